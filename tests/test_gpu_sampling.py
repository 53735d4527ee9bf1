"""GPU parity of top_k sampling inside the lattice (Fig. 2 caption, Sec. 3.3).

The oracle's sampler applied to the GPU's own float32 logits, with the
sequence index, generated count, seed and temperature of the step, must give
the GPU's uniforms, lattice, rescaled forward weights, drawn slots and tokens
bit for bit: both sides follow the same float32 arithmetic (one rounding per
operation, flushed products, the same exp evaluation, Philox4x64-10)."""
import numpy as np
import pytest

from gpu_common import log, new_session
from oracle.sampling import select_sample
from oracle.selection import accept
from paper_2410_13839_amd.workloads import (EOS_ID, VOCAB, WORKLOADS, ModelShape, Workload, make_logq,
                                            make_prompts, make_weights)

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bits(x):
    return np.asarray(x, np.float32).view(np.uint32)


def _check_step(s, lg, logq, K, top_k, gen, live, lattice, anchors, tok, cnt, wl, tau, seed):
    from paper_2410_13839_amd.binding import MTP_LATTICE_UNION
    uni = lattice == MTP_LATTICE_UNION
    lat = s.union_lattice(K) if uni else s.lattice(K, top_k)
    u = s.uniforms(K)
    for b in range(lg.shape[0]):
        if not live[b]:
            assert cnt[b] == 0
            continue
        ref = select_sample(lg[b], logq, top_k, int(gen[b]), wl.eos_min, EOS_ID, tau, seed, b,
                            lattice="union" if uni else "own", anchor=anchors[b])
        ctx = f"seq {b} gen {gen[b]}"
        assert np.array_equal(_bits(u[b]), _bits(ref.u)), (ctx, u[b], ref.u)
        if uni:
            m = int(lat["m"][b])
            assert m == ref.cand.shape[1], ctx
            assert np.array_equal(lat["states"][b, :m], ref.cand[0]), ctx
            assert np.array_equal(_bits(lat["ehat"][b][:, :m]), _bits(ref.ehat)), ctx
            assert np.array_equal(_bits(lat["delta"][b][:, :m]), _bits(ref.alpha)), ctx
        else:
            assert np.array_equal(lat["cand"][b], ref.cand), ctx
            assert np.array_equal(_bits(lat["ehat"][b]), _bits(ref.ehat)), ctx
            assert np.array_equal(_bits(lat["delta"][b]), _bits(ref.alpha)), ctx
            assert np.all(lat["psi"][b] == -1), ctx
        assert np.array_equal(lat["slots"][b], ref.slots), (ctx, lat["slots"][b], ref.slots)
        n, _ = accept(ref.tokens, int(gen[b]), wl.max_new, EOS_ID)
        assert cnt[b] == n, (ctx, cnt[b], n)
        assert np.array_equal(tok[b][:n], ref.tokens[:n]), ctx


def _run(wl, w, logq, K, top_k, lattice, anchored, steps, tau, seed):
    from paper_2410_13839_amd.binding import MTP_SELECT_SAMPLE
    pr = make_prompts(wl)
    s = new_session(wl, w, logq)
    s.set_selection(lattice, anchored)
    s.set_sampling(MTP_SELECT_SAMPLE, tau, seed)
    s.prefill(pr.phon, pr.ac)
    anchors = [int(a[-1]) if (anchored and len(a)) else None for a in pr.ac]
    emitted = []
    for step in range(steps):
        st = s.seq_state()
        gen, live = st["gen"].copy(), st["done"] == 0
        if not live.any():
            break
        tok, cnt = s.step(K, top_k)
        lg = s.logits(K)
        _check_step(s, lg, logq, K, top_k, gen, live, lattice, anchors, tok, cnt, wl, tau, seed)
        for b in range(len(anchors)):
            if anchored and cnt[b] > 0:
                anchors[b] = int(tok[b][cnt[b] - 1])
        emitted.append(tok.copy())
    s.close()
    return emitted


def _ties_setup(K, top_k, seed):
    shape = ModelShape(n_layers=2, d_model=256, n_heads=4, d_ff=1024, k_heads=8, dtype="f32", max_pos=512)
    wl = Workload("ties", shape, K=K, top_k=top_k, batch=3, phon_len=(0, 4), ac_len=(5, 20), max_new=24,
                  eos_min=8)
    w = make_weights(shape, seed=21)
    rng = np.random.default_rng(seed)
    w["w_heads"][:] = 0.0
    w["b_heads"][:] = rng.integers(0, 3, size=w["b_heads"].shape).astype(np.float32)
    logq = rng.integers(-3, 1, size=(VOCAB, VOCAB)).astype(np.float32)
    return wl, w, logq


@pytest.mark.parametrize("K,top_k,tau", [(1, 1, 1.0), (1, 6, 1.0), (2, 3, 0.5), (4, 4, 1.0), (5, 7, 2.0),
                                         (8, 8, 0.7)])
def test_sampled_own_lattice_exact(K, top_k, tau):
    """Small-integer logits and log Q (ties everywhere, weights of many equal
    sizes), three sequences: every uniform, forward weight and draw exact."""
    wl, w, logq = _ties_setup(K, top_k, 700 + 10 * K + top_k)
    _run(wl, w, logq, K, top_k, 0, False, steps=3, tau=tau, seed=1234 + K)


@pytest.mark.parametrize("K,top_k,anchored", [(1, 5, False), (3, 4, False), (4, 4, True), (8, 8, False)])
def test_sampled_union_lattice_exact(K, top_k, anchored):
    wl, w, logq = _ties_setup(K, top_k, 800 + 10 * K + top_k)
    _run(wl, w, logq, K, top_k, 1, anchored, steps=3, tau=0.9, seed=(1 << 63) + K)


@pytest.mark.parametrize("lattice,anchored,tau", [(0, False, 1.0), (0, True, 0.7), (1, True, 1.3)])
def test_sampling_on_the_bf16_decoder(lattice, anchored, tau):
    """The 12-layer bf16 decoder with the synthetic Q, 40 sampled steps at
    K=4, top_k=4: every step exact against the oracle on the GPU's logits."""
    wl = WORKLOADS["valle_k4"]
    log(f"sampling lattice {lattice} anchored {anchored} tau {tau}: start")
    _run(wl, make_weights(wl.model), make_logq(), wl.K, wl.top_k, lattice, anchored, steps=40, tau=tau, seed=99)


def test_seed_reproducibility_and_mode_switches():
    """Same seed, same tokens; another seed, other tokens; switching between
    the best path and sampling, and changing the seed, take effect at the
    next step (the seed lives in device memory, not in a captured graph)."""
    from paper_2410_13839_amd.binding import MTP_SELECT_BEST, MTP_SELECT_SAMPLE
    from oracle.selection import select
    wl = WORKLOADS["valle_k4"]
    w, logq = make_weights(wl.model), make_logq()
    a = _run(wl, w, logq, 4, 4, 0, False, steps=6, tau=1.0, seed=5)
    b = _run(wl, w, logq, 4, 4, 0, False, steps=6, tau=1.0, seed=5)
    c = _run(wl, w, logq, 4, 4, 0, False, steps=6, tau=1.0, seed=6)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    assert not all(np.array_equal(x, y) for x, y in zip(a, c))

    pr = make_prompts(wl)
    s = new_session(wl, w, logq)
    s.prefill(pr.phon, pr.ac)
    plan = [(MTP_SELECT_BEST, 1.0, 0), (MTP_SELECT_SAMPLE, 1.0, 11), (MTP_SELECT_SAMPLE, 1.0, 12),
            (MTP_SELECT_SAMPLE, 0.6, 12), (MTP_SELECT_BEST, 1.0, 0), (MTP_SELECT_SAMPLE, 0.6, 12)]
    for mode, tau, seed in plan:
        s.set_sampling(mode, tau, seed)
        st = s.seq_state()
        gen, live = st["gen"].copy(), st["done"] == 0
        tok, cnt = s.step(4, 4)
        lg = s.logits(4)
        if mode == MTP_SELECT_SAMPLE:
            _check_step(s, lg, logq, 4, 4, gen, live, 0, [None] * len(gen), tok, cnt, wl, tau, seed)
        else:
            for bb in range(lg.shape[0]):
                ref = select(lg[bb], logq, 4, int(gen[bb]), wl.eos_min, EOS_ID)
                assert np.array_equal(tok[bb][:cnt[bb]], ref.tokens[:cnt[bb]])
    s.close()
