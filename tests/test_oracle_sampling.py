"""Pins of the oracle's top_k sampling inside the lattice (Fig. 2 caption,
Sec. 3.3): the Philox generator against numpy's independent implementation
and the published zero known-answer block, exp32 against the float64
exponential, the forward weights and every backward draw against exhaustive
enumeration of the path distribution, the empirical path frequencies, and the
special cases the distribution reduces to (one head = top_k sampling with
temperature, a flat Q = independent per-head sampling, tau -> 0 = per-head
argmax)."""
import numpy as np
import pytest

from oracle import brute
from oracle.sampling import (draw, exp32, ffbs, philox4x64_10, select_sample, step_uniforms, uniform24)
from oracle.selection import select, union_inputs
from paper_2410_13839_amd.workloads import EOS_ID, VOCAB, make_logq

F32 = np.float32


@pytest.fixture(scope="module")
def logq_syn():
    return make_logq(kind="synthetic")


def _logits(rng, K, V=VOCAB, scale=0.64):
    return (rng.standard_normal((K, V)) * scale).astype(np.float32)


# ---------------------------------------------------------------- Philox


def test_philox_zero_block_known_answer():
    """Philox4x64-10 at counter 0, key 0 (the published known-answer block)."""
    assert philox4x64_10([0, 0, 0, 0], [0, 0]) == [
        0x16554D9ECA36314C, 0xDB20FE9D672D0FDC, 0xD7E772CEE186176B, 0x7E68B68AEC7BA23B]


def test_philox_matches_numpy():
    """numpy's Philox bit generator (a separate implementation of the same
    SC 2011 definition) increments its counter before each block, so its first
    block for counter c is ours at c + 1."""
    rng = np.random.default_rng(3)
    for _ in range(20):
        ctr = [int(x) for x in rng.integers(1, 2 ** 63, size=4, dtype=np.int64)]
        ctr[0] |= 1
        key = [int(x) for x in rng.integers(0, 2 ** 63, size=2, dtype=np.int64)]
        key[1] |= 1 << 63                       # high bits of the key too
        g = np.random.Philox(counter=np.array([ctr[0] - 1] + ctr[1:], np.uint64), key=np.array(key, np.uint64))
        assert [int(x) for x in g.random_raw(4)] == philox4x64_10(ctr, key)


def test_uniforms_are_24_bit_and_distinct():
    u = step_uniforms(seed=7, seq=2, gen=40, K=8)
    assert u.dtype == np.float32 and np.all((u >= 0) & (u < 1))
    assert np.all(u * F32(2 ** 24) == np.floor(u * F32(2 ** 24)))
    assert len(set(u.tolist())) == 8
    assert not np.array_equal(u, step_uniforms(7, 2, 41, 8))
    assert not np.array_equal(u, step_uniforms(7, 3, 40, 8))
    assert not np.array_equal(u, step_uniforms(8, 2, 40, 8))
    assert np.array_equal(u, step_uniforms(7, 2, 40, 8))
    assert np.array_equal(u[:4], step_uniforms(7, 2, 40, 4))
    assert uniform24(0) == 0 and uniform24((1 << 64) - 1) == F32(1 - 2 ** -24)


def test_uniforms_are_uniform():
    u = np.concatenate([step_uniforms(11, 0, g, 8) for g in range(500)]).astype(np.float64)
    hist = np.histogram(u, bins=10, range=(0, 1))[0]
    chi2 = ((hist - 400) ** 2 / 400).sum()
    assert chi2 < 30, chi2                      # 9 dof: p ~ 4e-4


# ---------------------------------------------------------------- exp32


def test_exp32_within_two_ulp_and_monotone():
    xs = np.linspace(-64, 0, 20001).astype(np.float32)
    ys = np.array([exp32(x) for x in xs])
    ref = np.exp(xs.astype(np.float64))
    ulp = np.spacing(ref.astype(np.float32)).astype(np.float64)
    assert (np.abs(ys - ref) / ulp).max() <= 2.0
    assert np.all(np.diff(ys) >= 0)


def test_exp32_special_values():
    assert exp32(0.0) == 1.0
    assert exp32(-np.inf) == 0.0
    assert exp32(np.float32(-64.0)) > 0 and exp32(np.float32(-64.0001)) == 0.0
    assert exp32(np.log(0.5)) == F32(0.5)


# ---------------------------------------------------------------- draws


def test_draw_edges():
    w = np.array([0, 0, 0.5, 0, 0.25], np.float32)
    assert draw(w, F32(0)) == 2                 # zero weights are never drawn
    assert draw(w, F32(1 - 2 ** -24)) == 4
    assert draw(w, F32(0.66)) == 2 and draw(w, F32(0.67)) == 4
    assert draw(np.zeros(4, np.float32), F32(0.3)) == 0


# ---------------------------------------------------------------- lattice distribution


def _lattice(rng, logq, K, k, lattice, gen=10 ** 6, eos_min=0):
    lg = _logits(rng, K)
    ref = select(lg, logq, k, gen, eos_min, EOS_ID, lattice=lattice)
    return ref.cand, ref.ehat


CASES = [("own", None, 3, 3), ("own", 17, 4, 3), ("union", None, 3, 2), ("union", 5, 2, 3), ("own", None, 5, 2)]


@pytest.mark.parametrize("lattice,anchor,K,k", CASES)
def test_forward_weights_are_prefix_marginals(logq_syn, lattice, anchor, K, k):
    """alpha_t, normalised, is the marginal of position t under the
    distribution of the first t + 1 positions."""
    rng = np.random.default_rng(100 + K * 10 + k)
    for tau in (1.0, 0.7):
        cand, ehat = _lattice(rng, logq_syn, K, k, lattice)
        sp = ffbs(cand, ehat, logq_syn, F32(1) / F32(tau), np.zeros(K, np.float32), anchor)
        for t in range(K):
            P, p = brute.path_weights(cand[:t + 1], ehat[:t + 1], logq_syn, tau, anchor)
            marg = np.bincount(P[:, t], weights=p, minlength=cand.shape[1])
            a = sp.alpha[t].astype(np.float64)
            assert 0.5 <= a.max() < 1.0
            assert np.allclose(a / a.sum(), marg, rtol=2e-5, atol=2e-7), (t, a / a.sum(), marg)


def _inverse_cdf(p, u):
    c = np.cumsum(p)
    j = int(np.searchsorted(c, u, side="right"))
    gap = np.min(np.abs(c[:-1] - u)) if len(c) > 1 else 1.0
    return min(j, len(p) - 1), gap


@pytest.mark.parametrize("lattice,anchor,K,k", CASES)
def test_backward_draws_follow_the_exact_conditionals(logq_syn, lattice, anchor, K, k):
    """Each draw is the inverse CDF of the exact conditional: the last position
    from its full-path marginal, position t from P(a_t | a_{t+1..K-1}), both
    summed from the enumerated path distribution in float64.  Draws whose
    uniform lies within 1e-5 of a CDF step are skipped (rounding decides them)."""
    rng = np.random.default_rng(200 + K * 10 + k)
    cand, ehat = _lattice(rng, logq_syn, K, k, lattice)
    tau = 0.9
    P, p = brute.path_weights(cand, ehat, logq_syn, tau, anchor)
    checked = 0
    for trial in range(150):
        u = rng.integers(0, 2 ** 24, size=K).astype(np.float32) * F32(2 ** -24)
        sp = ffbs(cand, ehat, logq_syn, F32(1) / F32(tau), u, anchor)
        m = cand.shape[1]
        expect = np.zeros(K, np.int64)
        near = False
        marg = np.bincount(P[:, K - 1], weights=p, minlength=m)
        expect[K - 1], gap = _inverse_cdf(marg / marg.sum(), float(u[0]))
        near |= gap < 1e-5
        for t in range(K - 2, -1, -1):
            sel = np.all(P[:, t + 1:] == expect[t + 1:], axis=1)
            cond = np.bincount(P[sel, t], weights=p[sel], minlength=m)
            expect[t], gap = _inverse_cdf(cond / cond.sum(), float(u[K - 1 - t]))
            near |= gap < 1e-5
        if near:
            continue
        checked += 1
        assert np.array_equal(sp.slots, expect), (trial, sp.slots, expect)
        assert np.array_equal(sp.tokens, cand[np.arange(K), sp.slots])
    assert checked >= 140


def test_path_frequencies_match_the_distribution(logq_syn):
    """Draws with the oracle's own uniform stream (one step per generated
    index) reproduce the path probabilities."""
    rng = np.random.default_rng(31)
    K, k, tau, N = 3, 3, 1.0, 3000
    cand, ehat = _lattice(rng, logq_syn, K, k, "own")
    P, p = brute.path_weights(cand, ehat, logq_syn, tau)
    counts = np.zeros(len(p))
    index = {tuple(r): i for i, r in enumerate(P.tolist())}
    for g in range(N):
        sp = ffbs(cand, ehat, logq_syn, F32(1), step_uniforms(5, 0, g, K))
        counts[index[tuple(sp.slots.tolist())]] += 1
    f = counts / N
    sd = np.sqrt(p * (1 - p) / N)
    assert np.all(np.abs(f - p) <= 5 * sd + 2e-3), np.abs(f - p) / (sd + 1e-12)


def test_one_head_is_top_k_sampling_with_temperature():
    rng = np.random.default_rng(37)
    for tau in (1.0, 0.5, 2.0):
        for trial in range(15):
            lg = _logits(rng, 1)
            sp = select_sample(lg, make_logq(kind="synthetic"), 5, 0, 0, EOS_ID, tau, seed=trial, seq=0)
            vals = np.sort(lg[0].astype(np.float64))[::-1][:5]
            p = np.exp((vals - vals[0]) / tau)
            j, gap = _inverse_cdf(p / p.sum(), float(sp.u[0]))
            if gap > 1e-5:
                assert int(sp.slots[0]) == j
            assert int(sp.tokens[0]) == int(sp.cand[0, sp.slots[0]])


def test_flat_q_makes_positions_independent():
    uq = make_logq(kind="uniform")
    rng = np.random.default_rng(41)
    for trial in range(40):
        lg = _logits(rng, 4)
        sp = select_sample(lg, uq, 4, 0, 0, EOS_ID, 0.8, seed=100 + trial, seq=1)
        for t in range(4):
            e = sp.ehat[t].astype(np.float64)
            p = np.exp(e / 0.8)
            j, gap = _inverse_cdf(p / p.sum(), float(sp.u[3 - t]))
            if gap > 1e-5:
                assert int(sp.slots[t]) == j, (trial, t)


def test_low_temperature_is_per_head_argmax(logq_syn):
    """tau = 1e-3: every emission weight but the top one is exactly 0, so the
    draw is the per-head argmax whatever Q and the uniforms are."""
    rng = np.random.default_rng(43)
    for trial in range(20):
        lg = _logits(rng, 4)
        for t in range(4):                       # keep the top logit 0.1 clear
            o = np.argsort(-lg[t].astype(np.float64))
            lg[t, o[0]] = lg[t, o[1]] + 0.1
        for lattice in ("own", "union"):
            sp = select_sample(lg, logq_syn, 4, 0, 0, EOS_ID, 1e-3, seed=trial, seq=0, lattice=lattice)
            assert sp.tokens.tolist() == [int(np.argmax(lg[t])) for t in range(4)]


def test_masked_eos_is_never_drawn():
    rng = np.random.default_rng(47)
    lg = _logits(rng, 3)
    lg[:, EOS_ID] = 5.0                          # every head ranks EOS first
    for g in range(30):
        sp = select_sample(lg, make_logq(kind="synthetic"), 3, gen=g, eos_min=10 ** 6, eos_id=EOS_ID,
                           temperature=1.0, seed=g, seq=0, lattice="union")
        assert EOS_ID not in sp.tokens.tolist()
    cand, ehat = union_inputs(lg, 3, 0, 0, EOS_ID)
    assert EOS_ID in cand[0].tolist()


def test_sampling_uses_the_selection_lattice(logq_syn):
    rng = np.random.default_rng(53)
    lg = _logits(rng, 4)
    for lattice in ("own", "union"):
        ref = select(lg, logq_syn, 3, 7, 9, EOS_ID, lattice=lattice)
        sp = select_sample(lg, logq_syn, 3, 7, 9, EOS_ID, 1.0, seed=1, seq=0, lattice=lattice)
        assert np.array_equal(sp.cand, ref.cand) and np.array_equal(sp.ehat, ref.ehat)
