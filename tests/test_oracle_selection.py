"""Pins of the oracle's selection (top_k, emission, Viterbi, accept).

Paper Sec. 3.3: the emitted n tokens are the path through each head's top_k
candidates that maximises prod_t Q(a_{t-1}, a_t) S_t(a_t).  The recursion is
checked against exhaustive enumeration of every path (in both the product and
the log form), exact ties on integer-valued lattices, and the special cases the
method reduces to (one head = greedy AR, Eq. 1; uniform Q = per-head argmax;
identical heads with a self-favouring Q = the greedy token repeated).
"""
import json
import os

import numpy as np
import pytest

from oracle import brute
from oracle.selection import (accept, emission, mask_eos, path_margin, select,
                              top_k, topk_boundary_gap, viterbi)
from paper_2410_13839_amd.workloads import EOS_ID, VOCAB, make_logq

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_lattice(rng, K, k, logq, V=VOCAB):
    logits = (rng.standard_normal((K, V)) * 0.64).astype(np.float32)
    cand = np.zeros((K, k), np.int32)
    ehat = np.zeros((K, k), np.float32)
    for t in range(K):
        ids, vals = top_k(logits[t], k)
        cand[t], ehat[t] = ids, emission(vals)
    return logits, cand, ehat


@pytest.fixture(scope="module")
def logq_syn():
    return make_logq(kind="synthetic")


@pytest.mark.parametrize("K,k", [(1, 1), (1, 5), (2, 3), (3, 4), (4, 4), (5, 3), (6, 2), (4, 6)])
def test_viterbi_matches_exhaustive_log_form(logq_syn, K, k):
    rng = np.random.default_rng(1000 + 10 * K + k)
    for trial in range(20):
        _, cand, ehat = _rand_lattice(rng, K, k, logq_syn)
        lat = viterbi(cand, ehat, logq_syn)
        P, score = brute.path_scores_log(cand, ehat, logq_syn)
        best = score.max()
        ours = score[np.all(P == lat.slots, axis=1)][0]
        assert abs(ours - best) <= 1e-5
        srt = np.sort(score)[::-1]
        if len(srt) == 1 or srt[0] - srt[1] > 1e-4:
            assert np.array_equal(P[np.argmax(score)], lat.slots)
        assert np.array_equal(lat.tokens, cand[np.arange(K), lat.slots])


@pytest.mark.parametrize("K,k", [(2, 3), (3, 3), (4, 4), (3, 5)])
def test_viterbi_matches_exhaustive_product_form(logq_syn, K, k):
    """The paper's own objective: product of Q(a_{t-1}, a_t) and the head's
    full-vocabulary softmax probability S_t(a_t)."""
    rng = np.random.default_rng(77 + K * k)
    Q = np.exp(logq_syn.astype(np.float64))
    for trial in range(20):
        logits, cand, ehat = _rand_lattice(rng, K, k, logq_syn)
        S_full = np.exp(logits.astype(np.float64) - logits.max(axis=1, keepdims=True))
        S_full /= S_full.sum(axis=1, keepdims=True)
        probs = np.take_along_axis(S_full, cand.astype(np.int64), axis=1)
        P, score = brute.path_scores_product(cand, probs, Q)
        lat = viterbi(cand, ehat, logq_syn)
        srt = np.sort(np.log(score))[::-1]
        if srt[0] - srt[1] > 1e-4:
            assert np.array_equal(P[np.argmax(score)], lat.slots)


@pytest.mark.parametrize("K,k", [(2, 2), (3, 3), (4, 3), (5, 2), (3, 4)])
def test_viterbi_exact_ties_pick_lowest_slots(K, k):
    """Integer lattices make exact ties common; the recursion must return the
    optimal path that is smallest when read from the last position back."""
    rng = np.random.default_rng(5 * K + k)
    V = 8
    for trial in range(200):
        logq = rng.integers(-2, 1, size=(V, V)).astype(np.float32)
        cand = np.stack([rng.permutation(V)[:k] for _ in range(K)]).astype(np.int32)
        ehat = rng.integers(-2, 1, size=(K, k)).astype(np.float32)
        lat = viterbi(cand, ehat, logq)
        P, score = brute.path_scores_log(cand, ehat, logq)
        opt = brute.best_paths(P, score)
        assert np.array_equal(lat.slots, brute.tie_rule_path(opt)), (trial, opt, lat.slots)


def test_viterbi_hand_worked_example():
    """A 3-position, 2-slot lattice whose best path was worked out by hand."""
    with open(os.path.join(GOLDEN, "viterbi_hand_example.json")) as f:
        ex = json.load(f)
    V = ex["vocab"]
    logq = np.full((V, V), -100.0, np.float32)
    for (a, b, v) in ex["logq_entries"]:
        logq[a, b] = v
    lat = viterbi(np.array(ex["cand"], np.int32), np.array(ex["ehat"], np.float32), logq)
    assert lat.delta.tolist() == ex["delta"]
    assert lat.psi[1:].tolist() == ex["psi"][1:]
    assert lat.slots.tolist() == ex["slots"]
    assert lat.tokens.tolist() == ex["tokens"]


def test_one_head_is_greedy_ar(logq_syn):
    """n = 1: Eq. 1's plain AR decoding, argmax with the lowest id on ties."""
    rng = np.random.default_rng(3)
    for trial in range(50):
        logits = (rng.standard_normal((1, VOCAB)) * 0.64).astype(np.float32)
        if trial % 5 == 0:  # plant an exact tie at the top
            j = int(np.argmax(logits[0]))
            logits[0, (j + 17) % (VOCAB - 1)] = logits[0, j]
        for k in (1, 3, 8):
            lat = select(logits, logq_syn, k, gen=0, eos_min=0, eos_id=EOS_ID)
            assert lat.tokens[0] == int(np.argmax(logits[0]))


def test_uniform_q_is_per_head_argmax():
    """With a uniform Q the transition factor is constant: the 'without
    Viterbi' baseline (each head's own argmax)."""
    logq = make_logq(kind="uniform")
    rng = np.random.default_rng(4)
    for trial in range(30):
        K, k = int(rng.integers(1, 9)), int(rng.integers(1, 9))
        logits = (rng.standard_normal((K, VOCAB)) * 0.64).astype(np.float32)
        lat = select(logits, logq, k, gen=0, eos_min=0, eos_id=EOS_ID)
        assert np.array_equal(lat.tokens, np.argmax(logits, axis=1))


@pytest.mark.parametrize("kind", ["uniform", "sticky"])
def test_identical_heads_accept_full_greedy_run(kind):
    logq = make_logq(kind=kind, alpha=0.5)
    rng = np.random.default_rng(11)
    for trial in range(20):
        K, k = int(rng.integers(1, 9)), int(rng.integers(1, 9))
        row = (rng.standard_normal(VOCAB) * 0.64).astype(np.float32)
        logits = np.tile(row, (K, 1))
        lat = select(logits, logq, k, gen=0, eos_min=VOCAB, eos_id=EOS_ID)
        g = int(np.argmax(np.where(np.arange(VOCAB) == EOS_ID, -np.inf, row)))
        assert lat.tokens.tolist() == [g] * K
        assert accept(lat.tokens, gen=0, max_new=1000, eos_id=EOS_ID) == (K, False)


def test_top_k_order_and_eos_mask():
    rng = np.random.default_rng(6)
    for trial in range(30):
        x = np.round(rng.standard_normal(VOCAB) * 4).astype(np.float32)  # many exact ties
        k = int(rng.integers(1, 33))
        ids, vals = top_k(x, k)
        ref = sorted(range(VOCAB), key=lambda i: (-float(x[i]), i))[:k]
        assert ids.tolist() == ref
        assert vals.tolist() == [float(x[i]) for i in ref]
    x = np.zeros(VOCAB, np.float32)
    x[EOS_ID] = 5.0
    assert top_k(mask_eos(x, 3, 4, EOS_ID), 1)[0][0] == 0          # masked: gen 3 < 4
    assert top_k(mask_eos(x, 4, 4, EOS_ID), 1)[0][0] == EOS_ID     # allowed from index 4


def test_emission_is_logsoftmax_up_to_a_constant():
    rng = np.random.default_rng(8)
    x = (rng.standard_normal(VOCAB) * 0.64).astype(np.float32)
    ids, vals = top_k(x, 8)
    e = emission(vals)
    assert e[0] == 0.0
    ls = x.astype(np.float64) - np.log(np.exp(x.astype(np.float64)).sum())
    np.testing.assert_allclose(e - (ls[ids] - ls[ids[0]]), 0, atol=1e-6)


def test_accept_rules():
    E = EOS_ID
    assert accept(np.array([5, 6, 7, 8]), gen=0, max_new=750, eos_id=E) == (4, False)
    assert accept(np.array([5, 6, 7, 8]), gen=748, max_new=750, eos_id=E) == (2, True)
    assert accept(np.array([5, E, 7, 8]), gen=10, max_new=750, eos_id=E) == (2, True)
    assert accept(np.array([E, 1, 2, 3]), gen=10, max_new=750, eos_id=E) == (1, True)
    assert accept(np.array([1, 2, 3, E]), gen=746, max_new=750, eos_id=E) == (4, True)
    assert accept(np.array([1, 2, E, 4]), gen=748, max_new=750, eos_id=E) == (2, True)  # EOS past the budget


def test_path_margin_matches_exhaustive(logq_syn):
    rng = np.random.default_rng(12)
    for trial in range(20):
        K, k = int(rng.integers(1, 5)), int(rng.integers(2, 5))
        _, cand, ehat = _rand_lattice(rng, K, k, logq_syn)
        _, score = brute.path_scores_log(cand, ehat, logq_syn)
        s = np.sort(score)[::-1]
        assert abs(path_margin(cand, ehat, logq_syn) - (s[0] - s[1])) < 1e-9


def test_topk_boundary_gap():
    x = np.array([3.0, 1.0, 2.0, 0.5], np.float32)
    assert topk_boundary_gap(x, 2) == pytest.approx(1.0)
    assert topk_boundary_gap(x, 3) == pytest.approx(0.5)
