"""Pins of the oracle's lattice variants.

Union lattice (paper Sec. 3.3): the reduced state space is the set of the
m <= k*n distinct tokens among all heads' top_k, with the m x m sub-table of
Q; position t scores a token with head t's own distribution.  Anchored first
position: the transition from the previously emitted token into position 0
joins the path score.  Both are checked against exhaustive enumeration of
every path, written from the definition (full-vocabulary softmax, the
transition table itself), against exact ties on integer-valued lattices and
against the special cases they reduce to.
"""
import numpy as np
import pytest

from oracle import brute
from oracle.selection import select, top_k, union_inputs, union_states, viterbi
from paper_2410_13839_amd.workloads import EOS_ID, VOCAB, make_logq


@pytest.fixture(scope="module")
def logq_syn():
    return make_logq(kind="synthetic")


def _logits(rng, K, V=VOCAB, scale=0.64):
    return (rng.standard_normal((K, V)) * scale).astype(np.float32)


def _softmax64(x):
    x = np.asarray(x, np.float64)
    e = np.exp(x - x.max())
    return e / e.sum()


def test_union_states_are_the_sorted_union_of_every_heads_top_k():
    rng = np.random.default_rng(5)
    for K, k in [(1, 4), (3, 3), (4, 4), (8, 8)]:
        lg = _logits(rng, K)
        lg[1 % K] = lg[0]                      # overlapping heads
        U = union_states(lg, k, 10 ** 6, 0, EOS_ID)
        expect = set()
        for t in range(K):
            expect |= set(np.argsort(-lg[t].astype(np.float64), kind="stable")[:k].tolist())
        assert U.tolist() == sorted(expect)
        assert len(U) <= K * k


@pytest.mark.parametrize("K,k", [(1, 3), (2, 3), (3, 2), (3, 3)])
def test_union_viterbi_matches_exhaustive_product_form(logq_syn, K, k):
    """The best path over the union states maximises prod_t S_t(a_t) *
    prod_{t>=1} Q(a_{t-1}, a_t), S_t the head's full-vocabulary softmax."""
    rng = np.random.default_rng(300 + 10 * K + k)
    Q = np.exp(logq_syn.astype(np.float64))
    for trial in range(10):
        lg = _logits(rng, K)
        lat = select(lg, logq_syn, k, 10 ** 6, 0, EOS_ID, lattice="union")
        U = lat.cand[0]
        probs = np.stack([_softmax64(lg[t])[U] for t in range(K)])
        for t in range(K):   # e_t = log S_t + the head's log-sum-exp (a per-position constant)
            x = lg[t].astype(np.float64)
            lse = np.log(np.exp(x - x.max()).sum())
            assert np.allclose(lat.ehat[t], np.log(probs[t]) + lse, atol=1e-5)
        P, score = brute.path_scores_product(lat.cand, probs, Q)
        ours = score[np.all(P == lat.slots, axis=1)][0]
        assert ours >= score.max() * (1 - 1e-5)
        srt = np.sort(score)[::-1]
        if len(srt) == 1 or srt[0] > srt[1] * (1 + 1e-4):
            assert np.array_equal(P[np.argmax(score)], lat.slots)
        assert np.array_equal(lat.tokens, U[lat.slots])


def test_union_exact_ties_pick_lowest_states():
    """Integer-valued logits and transitions: exact ties everywhere, and the
    recursion must return the reverse-lexicographically smallest optimal path
    over the ascending-id state order."""
    rng = np.random.default_rng(11)
    for trial in range(30):
        K, k = 3, 2
        lg = rng.integers(-3, 3, size=(K, 64)).astype(np.float32)
        lq = rng.integers(-2, 1, size=(64, 64)).astype(np.float32)
        cand, ehat = union_inputs(lg, k, 10 ** 6, 0, 63)
        lat = viterbi(cand, ehat, lq)
        P, score = brute.path_scores_log(cand, ehat, lq)
        assert np.array_equal(lat.slots, brute.tie_rule_path(brute.best_paths(P, score)))


def test_union_optimum_is_at_least_the_own_top_k_optimum(logq_syn):
    """Every own-top_k path is also a union path with the same score."""
    rng = np.random.default_rng(17)
    for trial in range(20):
        K, k = 3, 3
        lg = _logits(rng, K)
        own = select(lg, logq_syn, k, 10 ** 6, 0, EOS_ID)
        uni = select(lg, logq_syn, k, 10 ** 6, 0, EOS_ID, lattice="union")
        assert float(uni.delta[-1].max()) >= float(own.delta[-1].max()) - 1e-5


def test_union_one_head_and_uniform_q_reduce_to_argmax():
    rng = np.random.default_rng(23)
    uni_q = make_logq(kind="uniform")
    for trial in range(10):
        lg = _logits(rng, 4)
        one = select(lg[:1], uni_q, 4, 10 ** 6, 0, EOS_ID, lattice="union")
        assert one.tokens.tolist() == [int(np.argmax(lg[0]))]
        lat = select(lg, uni_q, 4, 10 ** 6, 0, EOS_ID, lattice="union")
        assert lat.tokens.tolist() == [int(np.argmax(lg[t])) for t in range(4)]


def test_union_masked_eos_is_a_dead_state_for_early_heads():
    """EOS in the union (a late head ranks it) is -inf at positions whose
    generated index is below eos_min, so no path uses it there."""
    rng = np.random.default_rng(29)
    lg = _logits(rng, 3)
    lg[2, EOS_ID] = 10.0                        # head 2 ranks EOS first
    cand, ehat = union_inputs(lg, 2, gen=5, eos_min=7, eos_id=EOS_ID)
    j = int(np.where(cand[0] == EOS_ID)[0][0])
    assert np.isneginf(ehat[0, j]) and np.isneginf(ehat[1, j]) and np.isfinite(ehat[2, j])
    lat = viterbi(cand, ehat, make_logq(kind="uniform"))
    assert EOS_ID not in lat.tokens[:2].tolist()


@pytest.mark.parametrize("lattice", ["own", "union"])
def test_anchored_viterbi_matches_exhaustive(logq_syn, lattice):
    rng = np.random.default_rng(41)
    for trial in range(10):
        K, k = 3, 3
        lg = _logits(rng, K)
        prev = int(rng.integers(0, VOCAB - 1))
        lat = select(lg, logq_syn, k, 10 ** 6, 0, EOS_ID, lattice=lattice, anchor=prev)
        P, score = brute.path_scores_log(lat.cand, lat.ehat, logq_syn, anchor=prev)
        ours = score[np.all(P == lat.slots, axis=1)][0]
        assert abs(ours - score.max()) <= 1e-5


def test_anchor_direction_is_previous_to_first():
    """An asymmetric Q that favours prev -> b (but not b -> prev) must pull the
    first position from a to b when a leads b only slightly."""
    V = 16
    lq = np.full((V, V), np.log(1.0 / V), np.float32)
    prev, a, b = 3, 5, 9
    lq[prev, b] = np.log(0.9)
    lq[b, prev] = np.log(0.001)
    lg = np.full((1, V), -5.0, np.float32)
    lg[0, a], lg[0, b] = 1.0, 0.9
    free = select(lg, lq, 2, 10 ** 6, 0, V - 1)
    anch = select(lg, lq, 2, 10 ** 6, 0, V - 1, anchor=prev)
    assert free.tokens.tolist() == [a] and anch.tokens.tolist() == [b]
    lq2 = lq.copy()
    lq2[prev, b], lq2[b, prev] = lq[b, prev], lq[prev, b]     # transpose the bias
    assert select(lg, lq2, 2, 10 ** 6, 0, V - 1, anchor=prev).tokens.tolist() == [a]


def test_anchor_with_uniform_q_only_shifts_scores():
    rng = np.random.default_rng(43)
    uq = make_logq(kind="uniform")
    for lattice in ("own", "union"):
        lg = _logits(rng, 4)
        free = select(lg, uq, 3, 10 ** 6, 0, EOS_ID, lattice=lattice)
        anch = select(lg, uq, 3, 10 ** 6, 0, EOS_ID, lattice=lattice, anchor=7)
        assert np.array_equal(free.tokens, anch.tokens)
        assert np.allclose(anch.delta[0] - free.delta[0], uq[0, 0], atol=1e-6)
