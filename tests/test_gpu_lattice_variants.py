"""GPU parity of the lattice variants of the selection (paper Sec. 3.3): the
union of all heads' top_k as every position's states, and the anchored first
position.  The oracle's selection applied to the GPU's own float32 logits must
give the GPU's lattice bit for bit (states, emissions, Viterbi scores,
back-pointers, chosen states) and its emitted tokens."""
import numpy as np
import pytest

from gpu_common import log, new_session
from oracle.selection import accept, select
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


def _check_step(s, lg, logq, K, top_k, gen, eos_min, live, lattice, anchors, tok, cnt, max_new):
    from paper_2410_13839_amd.binding import MTP_LATTICE_UNION
    uni = lattice == MTP_LATTICE_UNION
    lat = s.union_lattice(K) if uni else s.lattice(K, top_k)
    for b in range(lg.shape[0]):
        if not live[b]:
            assert cnt[b] == 0
            continue
        ref = select(lg[b], logq, top_k, int(gen[b]), eos_min, EOS_ID, lattice="union" if uni else "own",
                     anchor=anchors[b])
        ctx = f"seq {b}"
        if uni:
            m = int(lat["m"][b])
            assert m == ref.cand.shape[1], (ctx, m, ref.cand.shape)
            assert np.array_equal(lat["states"][b, :m], ref.cand[0]), ctx
            assert np.array_equal(_bits(lat["ehat"][b][:, :m]), _bits(ref.ehat)), ctx
            assert np.array_equal(_bits(lat["delta"][b][:, :m]), _bits(ref.delta)), ctx
            assert np.array_equal(lat["psi"][b][1:, :m], ref.psi[1:]), ctx
        else:
            assert np.array_equal(lat["cand"][b], ref.cand), ctx
            assert np.array_equal(_bits(lat["delta"][b]), _bits(ref.delta)), ctx
            assert np.array_equal(lat["psi"][b][1:], ref.psi[1:]), ctx
        assert np.array_equal(lat["slots"][b], ref.slots), ctx
        n, _ = accept(ref.tokens, int(gen[b]), max_new, EOS_ID)
        assert cnt[b] == n, (ctx, cnt[b], n)
        assert np.array_equal(tok[b][:n], ref.tokens[:n]), ctx


def _run(wl, w, logq, K, top_k, lattice, anchored, steps):
    pr = make_prompts(wl)
    s = new_session(wl, w, logq)
    s.set_selection(lattice, anchored)
    s.prefill(pr.phon, pr.ac)
    anchors = [int(a[-1]) if (anchored and len(a)) else None for a in pr.ac]
    for step in range(steps):
        st = s.seq_state()
        gen, live = st["gen"].copy(), st["done"] == 0
        if not live.any():
            break
        tok, cnt = s.step(K, top_k)
        lg = s.logits(K)
        _check_step(s, lg, logq, K, top_k, gen, wl.eos_min, live, lattice, anchors, tok, cnt, wl.max_new)
        for b in range(len(anchors)):
            if anchored and cnt[b] > 0:
                anchors[b] = int(tok[b][cnt[b] - 1])
    s.close()


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


@pytest.mark.parametrize("K,top_k", [(1, 1), (1, 6), (2, 3), (3, 5), (4, 4), (5, 2), (8, 8)])
def test_union_lattice_exact_with_planted_ties(K, top_k):
    """Small-integer logits and log Q: exact ties in the union, its ascending
    order, the emissions of tokens outside a head's own top_k, and the
    recursion's lowest-state tie rule."""
    from paper_2410_13839_amd.binding import MTP_LATTICE_UNION
    wl, w, logq = _ties_setup(K, top_k, 500 + 10 * K + top_k)
    _run(wl, w, logq, K, top_k, MTP_LATTICE_UNION, False, steps=3)


@pytest.mark.parametrize("lattice", [0, 1])
@pytest.mark.parametrize("K,top_k", [(1, 4), (3, 3), (4, 4)])
def test_anchored_selection_exact(lattice, K, top_k):
    """The first position carries the transition from the last emitted token
    (the acoustic prompt's last token at the first step)."""
    wl, w, logq = _ties_setup(K, top_k, 900 + 10 * K + top_k + lattice)
    _run(wl, w, logq, K, top_k, lattice, True, steps=4)


@pytest.mark.parametrize("lattice,anchored", [(1, False), (1, True), (0, True)])
def test_lattice_variants_on_the_bf16_decoder(lattice, anchored):
    """The 12-layer bf16 decoder with the synthetic Q, 40 steps at K=4,
    top_k=4: every step's lattice and tokens exact against the oracle on the
    GPU's logits."""
    wl = WORKLOADS["valle_k4"]
    log(f"lattice {lattice} anchored {anchored}: start")
    _run(wl, make_weights(wl.model), make_logq(), wl.K, wl.top_k, lattice, anchored, steps=40)


def test_union_needs_at_most_64_states():
    from paper_2410_13839_amd.binding import MTP_EINVAL, MTP_LATTICE_UNION, MTPError
    wl, w, logq = _ties_setup(8, 9, 7)
    pr = make_prompts(wl)
    s = new_session(wl, w, logq)
    s.set_selection(MTP_LATTICE_UNION, False)
    s.prefill(pr.phon, pr.ac)
    with pytest.raises(MTPError) as e:
        s.step(8, 9)
    assert e.value.code == MTP_EINVAL
    s.close()
