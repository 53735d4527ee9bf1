"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bars:
  * selection (top_k, emissions, Viterbi scores, back-pointers, slots, tokens,
    counts) is bit-exact given the same float32 logits;
  * logits within 1e-4 max-abs (fp32 model) / 3e-2 max-abs (bf16 model) of the
    float64 oracle on the same token history;
  * token trajectories agree wherever the oracle's own decision margin is
    outside the tie zone (twice the observed logit error).
"""
import math

import numpy as np
import pytest

from gpu_common import (OracleCheck, assert_selection_exact, log, new_session, oracle_logits_at)
from oracle.decoder import ARDecoder
from oracle.generate import Generator
from oracle.selection import mask_eos, path_margin, select, topk_boundary_gap
from paper_2410_13839_amd.workloads import (EOS_ID, VOCAB, WORKLOADS, ModelShape, Workload, make_logq,
                                            make_prompts, make_weights)

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _margin(logits, lat, logq, top_k, gen, eos_min):
    gaps = [topk_boundary_gap(mask_eos(logits[t], gen + t, eos_min, EOS_ID), top_k) for t in range(logits.shape[0])]
    gaps.append(path_margin(lat.cand, lat.ehat, logq))
    return min(gaps)


def run_teacher_forced(wl: Workload, K: int, top_k: int, steps_checked, tol: float, batch=None,
                       seqs_checked=None, emulate=False):
    """Run the GPU free; check selection every step and the oracle's logits
    (on the GPU's own history) at `steps_checked` for `seqs_checked`."""
    w = make_weights(wl.model)
    logq = make_logq()
    pr = make_prompts(wl, batch=batch)
    B = pr.batch
    s = new_session(wl, w, logq, batch=B)
    s.prefill(pr.phon, pr.ac)
    model = ARDecoder(wl.model, w, emulate_bf16=emulate)
    emitted = [[] for _ in range(B)]
    chk = OracleCheck()
    live = np.ones(B, bool)
    step = 0
    seqs_checked = list(range(B)) if seqs_checked is None else seqs_checked
    while live.any():
        st = s.seq_state()
        gen_before = st["gen"].copy()
        tok, cnt = s.step(K, top_k)
        lg = s.logits(K)
        lat = s.lattice(K, top_k)
        assert_selection_exact(lg, lat, logq, top_k, gen_before, wl.eos_min, EOS_ID, live)
        for b in range(B):
            if not live[b]:
                assert cnt[b] == 0
                continue
            ref_path = lat["cand"][b][np.arange(K), lat["slots"][b]]
            n_exp = min(K, wl.max_new - gen_before[b])
            eos_at = [p for p in range(n_exp) if ref_path[p] == EOS_ID]
            if eos_at:
                n_exp = eos_at[0] + 1
            assert cnt[b] == n_exp, (step, b, cnt[b], n_exp)
            assert np.array_equal(tok[b][:cnt[b]], ref_path[:cnt[b]])
            assert np.all(tok[b][cnt[b]:] == -1)
            if EOS_ID in ref_path[:cnt[b]]:
                assert gen_before[b] + list(ref_path).index(EOS_ID) >= wl.eos_min
            if step in steps_checked and b in seqs_checked:
                ref = oracle_logits_at(model, pr.phon[b], pr.ac[b], emitted[b], K)
                err = float(np.abs(ref - lg[b]).max())
                chk.max_err = max(chk.max_err, err)
                chk.checked += 1
                ref_lat = select(ref, logq, top_k, int(gen_before[b]), wl.eos_min, EOS_ID)
                m = _margin(ref, ref_lat, logq, top_k, int(gen_before[b]), wl.eos_min)
                same = np.array_equal(ref_lat.tokens[:cnt[b]], tok[b][:cnt[b]])
                if m <= 2 * tol:
                    chk.tie_zone += 1
                elif not same:
                    chk.mismatched += 1
                    chk.notes.append(f"step {step} seq {b}: margin {m:.3g}, err {err:.3g}")
                log(f"  [{wl.name}] step {step} seq {b}: logit err {err:.3g}, margin {m:.3g}, tokens agree {same}")
                assert err <= tol, (step, b, err)
            emitted[b].extend(int(x) for x in tok[b][:cnt[b]])
        st = s.seq_state()
        live = st["done"] == 0
        step += 1
    hist = s.tokens()
    for b in range(B):
        assert np.array_equal(hist[b][:len(emitted[b])], emitted[b])
    s.close()
    assert chk.mismatched == 0, chk.notes
    return step, emitted, chk


def test_tiny_fp32_follows_the_oracle_trajectory():
    """fp32 tiny model, 64 tokens at K=2, top_k=3, against the oracle's own
    free run (float64 trunk, float32 decisions): at every step the GPU's
    logits are within 1e-4 of the oracle's on the same history and its
    selection is bit-exact on its own logits.  Where the GPU's tokens differ
    from the oracle's, the oracle's decision margin must lie in the tie zone
    (1e-3); the GPU is then forced onto the oracle's tokens (teacher forcing)
    and the run continues on the oracle's trajectory.  The count of such
    steps is reported."""
    wl = WORKLOADS["tiny"]
    log("tiny: start")
    w = make_weights(wl.model)
    logq = make_logq()
    pr = make_prompts(wl)
    g = Generator(ARDecoder(wl.model, w), logq, wl.eos_min, wl.max_new)
    g.prefill(pr.phon[0], pr.ac[0])
    s = new_session(wl, w, logq)
    s.prefill(pr.phon, pr.ac)
    steps, forced, tie_zone, max_err = 0, 0, 0, 0.0
    while not g.done:
        gen = s.seq_state()["gen"].copy()
        assert gen[0] == g.gen
        rec = g.step(wl.K, wl.top_k)
        tok, cnt = s.step(wl.K, wl.top_k)
        lg = s.logits(wl.K)
        err = float(np.abs(rec.logits - lg[0]).max())
        max_err = max(max_err, err)
        assert err <= 1e-4, (steps, err)
        assert_selection_exact(lg, s.lattice(wl.K, wl.top_k), logq, wl.top_k, gen, wl.eos_min, EOS_ID,
                               np.ones(1, bool))
        margin = g.margins(rec, wl.top_k)
        tie_zone += margin <= 1e-3
        same = cnt[0] == rec.count and np.array_equal(tok[0][:cnt[0]], rec.emitted)
        if not same:
            assert margin <= 1e-3, (steps, margin, tok[0], rec.emitted)
            s.force(np.asarray(rec.emitted, np.int32)[None], [rec.count])
            forced += 1
        steps += 1
    st = s.seq_state()
    assert st["gen"][0] == wl.max_new and st["done"][0] == 1
    assert list(s.tokens()[0][:wl.max_new]) == g.run.tokens
    assert steps == math.ceil(wl.max_new / wl.K)
    s.close()
    log(f"tiny: {steps} steps on the oracle's trajectory, max logit err {max_err:.3g}, "
        f"tie-zone steps {tie_zone}, steps forced onto the oracle's tokens {forced}")


def test_force_tokens_teacher_forcing():
    """mtp_force_tokens (Sec. 3.1, Eq. 1: generation conditioned on a given
    history): forced tokens and counts replace the step's output, become the
    next step's pending chunk (the next logits match the oracle on the forced
    history), a forced EOS ends the sequence, and bad requests are refused
    with nothing changed."""
    from paper_2410_13839_amd.binding import MTP_EINVAL, MTPError
    shape = ModelShape(n_layers=2, d_model=256, n_heads=4, d_ff=1024, k_heads=4, dtype="f32", max_pos=512)
    wl = Workload("force", shape, K=4, top_k=3, batch=3, phon_len=(2, 6), ac_len=(5, 12), max_new=13,
                  eos_min=4)
    w = make_weights(shape, seed=41)
    logq = make_logq()
    pr = make_prompts(wl)
    model = ARDecoder(shape, w)
    s = new_session(wl, w, logq)
    s.prefill(pr.phon, pr.ac)
    rng = np.random.default_rng(5)
    hist = [[], [], []]
    K = wl.K
    # step 0: force sequence 0 to 4 tokens, 1 to 1 token, 2 to 3 tokens
    s.step(K, 3)
    want = rng.integers(0, 1024, size=(3, K)).astype(np.int32)
    counts = [4, 1, 3]
    before = (s.seq_state(), s.tokens().copy())
    for bad_tok, bad_cnt in ((want, [5, 1, 3]), (want, [0, 1, 3]), (np.where(want == want, 1025, want), counts),
                             (np.where(np.arange(K) == 0, EOS_ID, want), counts)):   # count > K, 0, id, early EOS
        with pytest.raises(MTPError) as e:
            s.force(bad_tok, bad_cnt)
        assert e.value.code == MTP_EINVAL
    after = (s.seq_state(), s.tokens())
    for k in before[0]:
        assert np.array_equal(before[0][k], after[0][k])
    assert np.array_equal(before[1], after[1])
    s.force(want, counts)
    for b in range(3):
        hist[b] += [int(x) for x in want[b][:counts[b]]]
    st = s.seq_state()
    assert list(st["gen"]) == counts and list(st["pend_len"]) == counts and list(st["done"]) == [0, 0, 0]
    # step 1 runs the forced chunks: logits against the oracle on the forced history
    tok, cnt = s.step(K, 3)
    lg = s.logits(K)
    for b in range(3):
        ref = oracle_logits_at(model, pr.phon[b], pr.ac[b], hist[b], K)
        assert np.abs(ref - lg[b]).max() <= 1e-4, b
    # force sequence 1 to end with EOS at generated index 4 (>= eos_min), the others their own tokens
    ft = tok.copy()
    fc = list(cnt)
    ft[1, :] = [7, 8, 9, 10]
    ft[1, 3] = EOS_ID
    fc[1] = 4
    s.force(ft, fc)
    for b in range(3):
        hist[b] += [int(x) for x in ft[b][:fc[b]]]
    st = s.seq_state()
    assert st["done"][1] == 1 and st["pend_len"][1] == 0 and st["gen"][1] == 5
    assert list(s.tokens()[1][:5]) == hist[1]
    # the ended sequence emits nothing and may only be forced to count 0
    tok, cnt = s.step(K, 3)
    assert cnt[1] == 0
    with pytest.raises(MTPError):
        s.force(tok, [cnt[0], 1, cnt[2]])
    lg = s.logits(K)
    for b in (0, 2):
        ref = oracle_logits_at(model, pr.phon[b], pr.ac[b], hist[b], K)
        assert np.abs(ref - lg[b]).max() <= 1e-4, b
    s.close()


@pytest.mark.parametrize("K,top_k", [(1, 1), (1, 4), (2, 3), (3, 5), (4, 4), (5, 2), (8, 8), (8, 32), (6, 17)])
def test_selection_exact_with_planted_ties(K, top_k):
    """Zero head weights and integer biases make the logits small integers,
    and an integer log Q makes Viterbi ties common: top_k must break ties by
    token id and the recursion by slot, bit-exactly like the oracle."""
    shape = ModelShape(n_layers=2, d_model=256, n_heads=4, d_ff=1024, k_heads=8, dtype="f32", max_pos=512)
    wl = Workload("ties", shape, K=K, top_k=top_k, batch=3, phon_len=(0, 4), ac_len=(5, 20), max_new=24,
                  eos_min=8)
    w = make_weights(shape, seed=21)
    rng = np.random.default_rng(K * 100 + top_k)
    w["w_heads"][:] = 0.0
    w["b_heads"][:] = rng.integers(0, 3, size=w["b_heads"].shape).astype(np.float32)
    logq = rng.integers(-3, 1, size=(VOCAB, VOCAB)).astype(np.float32)
    pr = make_prompts(wl)
    s = new_session(wl, w, logq)
    s.prefill(pr.phon, pr.ac)
    for step in range(3):
        gen = s.seq_state()["gen"].copy()
        live = s.seq_state()["done"] == 0
        tok, cnt = s.step(K, top_k)
        lg = s.logits(K)
        assert np.array_equal(lg[:, :, :], np.broadcast_to(w["b_heads"][:K], lg.shape))
        assert_selection_exact(lg, s.lattice(K, top_k), logq, top_k, gen, wl.eos_min, EOS_ID, live)
    s.close()


def test_one_head_is_greedy_on_gpu():
    wl = WORKLOADS["tiny"]
    w = make_weights(wl.model)
    pr = make_prompts(wl)
    s = new_session(wl, w, make_logq())
    s.prefill(pr.phon, pr.ac)
    for _ in range(6):
        gen = int(s.seq_state()["gen"][0])
        tok, cnt = s.step(1, 5)
        lg = s.logits(1)[0, 0].copy()
        if gen < wl.eos_min:
            lg[EOS_ID] = -np.inf
        assert cnt[0] == 1 and tok[0, 0] == int(np.argmax(lg))
    s.close()


def test_eager_and_graph_launch_agree():
    """The hipGraph replay and eager launches run the same kernels: identical
    tokens and bit-identical logits."""
    from paper_2410_13839_amd.binding import MTP_FLAG_NO_GRAPH
    wl = WORKLOADS["tiny"]
    w = make_weights(wl.model)
    pr = make_prompts(wl)
    out = []
    for flags in (0, MTP_FLAG_NO_GRAPH):
        s = new_session(wl, w, make_logq(), flags=flags)
        s.prefill(pr.phon, pr.ac)
        logs = []
        for _ in range(5):
            s.step(wl.K, wl.top_k)
            logs.append(s.logits(wl.K))
        out.append((s.tokens()[0][:10].copy(), np.stack(logs)))
        s.close()
    assert np.array_equal(out[0][0], out[1][0])
    assert np.array_equal(out[0][1].view(np.uint32), out[1][1].view(np.uint32))


def test_changing_K_between_steps():
    """Heads can be dropped per call (Fig. 1): a K=4 step followed by K=2 and
    K=3 steps matches the oracle on the same history."""
    shape = ModelShape(n_layers=2, d_model=256, n_heads=4, d_ff=1024, k_heads=4, dtype="f32", max_pos=512)
    wl = Workload("varK", shape, K=4, top_k=3, batch=2, phon_len=(3, 6), ac_len=(8, 12), max_new=40, eos_min=40)
    w = make_weights(shape, seed=31)
    logq = make_logq()
    pr = make_prompts(wl)
    s = new_session(wl, w, logq)
    s.prefill(pr.phon, pr.ac)
    model = ARDecoder(shape, w)
    emitted = [[], []]
    for K in (4, 2, 3, 1, 4):
        gen = s.seq_state()["gen"].copy()
        tok, cnt = s.step(K, 3)
        lg = s.logits(K)
        for b in range(2):
            ref = oracle_logits_at(model, pr.phon[b], pr.ac[b], emitted[b], K)
            assert np.abs(ref - lg[b]).max() <= 1e-4
            emitted[b].extend(int(x) for x in tok[b][:cnt[b]])
        assert_selection_exact(lg, s.lattice(K, 3), logq, 3, gen, wl.eos_min, EOS_ID, np.ones(2, bool))
    st = s.seq_state()
    assert list(st["gen"]) == [14, 14]
    s.close()


def test_bf16_changing_K_between_steps():
    """The same on a small bf16 decoder whose decode layers run the one-launch
    front and chained FFN (8 heads, three layers, one sequence at ~350 keys:
    two key splits): the pending chunk changes size every step (1 to 4 rows),
    so each step runs another plan over the same hand-off words and row sets;
    logits within 3e-2 of the oracle on the same history, selection exact."""
    shape = ModelShape(n_layers=3, d_model=512, n_heads=8, d_ff=1024, k_heads=4, dtype="bf16")
    wl = Workload("varK_bf16", shape, K=4, top_k=3, batch=1, phon_len=(20, 30), ac_len=(300, 330), max_new=40,
                  eos_min=40)
    w = make_weights(shape, seed=37)
    logq = make_logq()
    pr = make_prompts(wl)
    s = new_session(wl, w, logq)
    s.prefill(pr.phon, pr.ac)
    model = ARDecoder(shape, w)
    emitted = []
    max_err = 0.0
    for K in (4, 1, 2, 4, 3, 1, 4, 2):
        gen = s.seq_state()["gen"].copy()
        tok, cnt = s.step(K, 3)
        lg = s.logits(K)
        ref = oracle_logits_at(model, pr.phon[0], pr.ac[0], emitted, K)
        err = float(np.abs(ref - lg[0]).max())
        max_err = max(max_err, err)
        assert err <= 3e-2, (K, err)
        emitted.extend(int(x) for x in tok[0][:cnt[0]])
        assert_selection_exact(lg, s.lattice(K, 3), logq, 3, gen, wl.eos_min, EOS_ID, np.ones(1, bool))
    assert s.seq_state()["gen"][0] == 21
    s.close()
    log(f"bf16 changing K: max logit err {max_err:.3g}")


def test_valle_k4_bf16_batch1():
    """12-layer d1024 bf16 decoder, K=4, top_k=4, batch 1, up to 750 tokens
    with EOS allowed from index 600: selection exact at every step, logits
    within 3e-2 at sampled steps."""
    wl = WORKLOADS["valle_k4"]
    log("valle_k4: start")
    steps, emitted, chk = run_teacher_forced(wl, wl.K, wl.top_k, steps_checked={0, 1, 97, 160}, tol=3e-2)
    assert len(emitted[0]) >= wl.eos_min or emitted[0][-1] == EOS_ID
    log(f"valle_k4: {steps} steps, {len(emitted[0])} tokens, max logit err {chk.max_err:.3g}, tie-zone {chk.tie_zone}")


def test_valle_k8_bf16_batch1():
    """Eight heads (the paper's largest K), batch 1: 8 pending rows per step,
    the out-projection merging up to eight attention key splits."""
    wl = WORKLOADS["valle_k8"]
    log("valle_k8: start")
    steps, emitted, chk = run_teacher_forced(wl, wl.K, wl.top_k, steps_checked={0, 47, 93}, tol=3e-2)
    assert steps == math.ceil(wl.max_new / wl.K)
    log(f"valle_k8: {steps} steps, max logit err {chk.max_err:.3g}, tie-zone {chk.tie_zone}")


def test_valle_batch2_k8_sixteen_rows():
    """Two ragged sequences at K=8: 16 decode rows, the largest fused row
    count, with the out-projection merge at its narrowest split budget."""
    wl = WORKLOADS["valle_b32"]
    log("valle batch 2, K=8: start")
    steps, emitted, chk = run_teacher_forced(wl, 8, 8, steps_checked={0, 61}, tol=3e-2, batch=2)
    assert steps == math.ceil(wl.max_new / 8)
    log(f"valle batch 2: {steps} steps, max logit err {chk.max_err:.3g}, tie-zone {chk.tie_zone}")


# Small bf16 decoders for the fronts of a small-batch decode layer:
#  * chain (the default where it applies: heads a multiple of 8): one launch
#    whose attention workgroups wait for their head's QKV columns, with 256-
#    or 512-key splits (MTP_FRONT=256 / 512 force one);
#  * separate QKV and attention launches (MTP_FRONT=0);
#  * every one of them with FFN1 and FFN2 in one launch whose FFN2
#    workgroups wait for their K range (the default), and the chained front
#    or separate launches with two FFN launches (MTP_FFN_CHAIN=0);
#  * one launch for LN1, QKV and the attention over the cached keys with 8 or
#    16 workgroups per head (MTP_QKV_ATTN=8 / 16; the out-projection then
#    merges the chunk's own keys).
FRONT_CASES = {
    # 8 heads (grouped per XCD), 2 ragged sequences of 4 rows, contexts up to ~690 keys;
    # three layers, so the one-launch kinds' last layer takes the third flag / row set
    "d512_b2_k4": (ModelShape(n_layers=3, d_model=512, n_heads=8, d_ff=1024, k_heads=4, dtype="bf16"),
                   4, 3, 2, (5, 40), (200, 600)),
    # 4 heads, one sequence of 2 rows, ~2,100 keys (more than 8 splits of 256 keys: the
    # 8-workgroup front is not available and falls back to separate launches)
    "d256_b1_k2": (ModelShape(n_layers=2, d_model=256, n_heads=4, d_ff=512, k_heads=2, dtype="bf16"),
                   2, 4, 1, (30, 40), (1900, 2000)),
    # 16 heads, 8 sequences of one row each (K = 1: plain AR decoding)
    "d1024_b8_k1": (ModelShape(n_layers=2, d_model=1024, n_heads=16, d_ff=2048, k_heads=1, dtype="bf16"),
                    1, 2, 8, (3, 20), (10, 300)),
}


FRONT_ENV = {"separate": {"MTP_FRONT": "0"}, "chain": {}, "chain256": {"MTP_FRONT": "256"},
             "chain512": {"MTP_FRONT": "512"}, "8": {"MTP_QKV_ATTN": "8"}, "16": {"MTP_QKV_ATTN": "16"},
             "ffn2": {"MTP_FFN_CHAIN": "0"}, "unchained": {"MTP_FRONT": "0", "MTP_FFN_CHAIN": "0"}}


def set_front(monkeypatch, front):
    monkeypatch.delenv("MTP_FRONT", raising=False)
    monkeypatch.delenv("MTP_QKV_ATTN", raising=False)
    monkeypatch.delenv("MTP_FFN_CHAIN", raising=False)
    for k, v in FRONT_ENV[front].items():
        monkeypatch.setenv(k, v)


@pytest.mark.parametrize("front", sorted(FRONT_ENV))
@pytest.mark.parametrize("case", sorted(FRONT_CASES))
def test_decode_fronts_match_the_oracle(case, front, monkeypatch):
    """Every front of the small-batch decode layer: selection exact at every
    step, logits within 3e-2 of the float64 oracle at every third step for
    every sequence (Sec. 3.1 Eq. 1 on the GPU's own history)."""
    shape, K, top_k, B, phon, ac = FRONT_CASES[case]
    wl = Workload(f"front_{case}", shape, K=K, top_k=top_k, batch=B, phon_len=phon, ac_len=ac, max_new=48,
                  eos_min=48)
    set_front(monkeypatch, front)
    log(f"front {front}, {case}: start")
    steps, emitted, chk = run_teacher_forced(wl, K, top_k, steps_checked=set(range(0, 64, 3)), tol=3e-2)
    assert steps == math.ceil(wl.max_new / K)
    assert chk.checked >= B * (steps // 3)
    log(f"front {front}, {case}: {steps} steps, {chk.checked} oracle checks, max logit err {chk.max_err:.3g}, "
        f"tie-zone {chk.tie_zone}")


@pytest.mark.parametrize("front", ["chain", "16"])
def test_fused_front_eager_and_graph_agree(front, monkeypatch):
    """The one-launch fronts give bit-identical logits eagerly and replayed
    from a captured graph, step after step."""
    from paper_2410_13839_amd.binding import MTP_FLAG_NO_GRAPH
    shape, K, top_k, B, phon, ac = FRONT_CASES["d512_b2_k4"]
    wl = Workload("front_graph", shape, K=K, top_k=top_k, batch=B, phon_len=phon, ac_len=ac, max_new=48, eos_min=48)
    set_front(monkeypatch, front)
    w = make_weights(shape)
    pr = make_prompts(wl)
    out = []
    for flags in (0, MTP_FLAG_NO_GRAPH):
        s = new_session(wl, w, make_logq(), flags=flags)
        s.prefill(pr.phon, pr.ac)
        logs = []
        for _ in range(6):
            s.step(K, top_k)
            logs.append(s.logits(K))
        out.append((s.tokens()[:, :24].copy(), np.stack(logs)))
        s.close()
    assert np.array_equal(out[0][0], out[1][0])
    assert np.array_equal(out[0][1].view(np.uint32), out[1][1].view(np.uint32))


@pytest.mark.parametrize("front", ["chain", "separate"])
def test_front_wait_that_runs_out_is_reported(front, monkeypatch):
    """The one-launch front's and chained FFN's waits (with `separate`, the
    chained FFN's alone), set from the host to give up at once
    (MTP_FRONT_SPIN=0: every kernel still runs to its end), make the step
    return MTP_ETIMEOUT; the context then refuses to step until a new
    prefill, after which it runs separate launches and gives bit for bit the
    tokens and logits of a context that always did."""
    from paper_2410_13839_amd.binding import MTP_ESTATE, MTP_ETIMEOUT, MTPError
    shape, K, top_k, B, phon, ac = FRONT_CASES["d512_b2_k4"]
    wl = Workload("front_timeout", shape, K=K, top_k=top_k, batch=B, phon_len=phon, ac_len=ac, max_new=48,
                  eos_min=48)
    w = make_weights(shape)
    pr = make_prompts(wl)
    logq = make_logq()
    set_front(monkeypatch, front)
    monkeypatch.setenv("MTP_FRONT_SPIN", "0")
    s = new_session(wl, w, logq)
    monkeypatch.delenv("MTP_FRONT_SPIN")
    s.prefill(pr.phon, pr.ac)
    s.step(K, top_k)            # the first step after a prefill runs no trunk layer
    with pytest.raises(MTPError) as e:
        s.step(K, top_k)
    assert e.value.code == MTP_ETIMEOUT
    with pytest.raises(MTPError) as e:
        s.step(K, top_k)
    assert e.value.code == MTP_ESTATE
    runs = []
    for sess in (s, None):
        if sess is None:
            set_front(monkeypatch, "unchained")
            sess = new_session(wl, w, logq)
        sess.prefill(pr.phon, pr.ac)
        logs = []
        for _ in range(5):
            sess.step(K, top_k)
            logs.append(sess.logits(K))
        runs.append((sess.tokens()[:, :20].copy(), np.stack(logs)))
        sess.close()
    assert np.array_equal(runs[0][0], runs[1][0])
    assert np.array_equal(runs[0][1].view(np.uint32), runs[1][1].view(np.uint32))
    log("front timeout: reported, then separate launches match")


def test_valle_b32_batched():
    """32 ragged sequences, K=4 (128 decode rows through the tiled path):
    selection exact for every sequence at every step; logits and tokens of
    four sequences against the oracle at the first step and near the longest
    context (step 185: prompt + 740 keys)."""
    wl = WORKLOADS["valle_b32"]
    log("valle_b32: start")
    steps, emitted, chk = run_teacher_forced(wl, wl.K, wl.top_k, steps_checked={0, 185}, tol=3e-2,
                                             seqs_checked=[0, 9, 17, 31])
    assert steps == math.ceil(wl.max_new / wl.K)
    assert all(len(e) == wl.max_new for e in emitted)
    log(f"valle_b32: {steps} steps, max logit err {chk.max_err:.3g}, tie-zone {chk.tie_zone}")


@pytest.mark.timeout(1200)
def test_long_b8_batched():
    """24-layer d1536 decoder (24 heads of 64), batch 8, K=4, 3000 tokens
    each: 32 decode rows through the batched path over a paged cache that
    grows to 3650 keys per sequence; selection exact for every sequence at
    every step; logits and tokens of two sequences against the oracle at the
    first step and at step 700 (the chunk attends to 3450 keys)."""
    wl = WORKLOADS["long_b8"]
    log("long_b8: start")
    steps, emitted, chk = run_teacher_forced(wl, wl.K, wl.top_k, steps_checked={0, 700}, tol=3e-2,
                                             seqs_checked=[2, 6])
    assert steps == math.ceil(wl.max_new / wl.K)
    assert all(len(e) == wl.max_new for e in emitted)
    log(f"long_b8: {steps} steps, max logit err {chk.max_err:.3g}, tie-zone {chk.tie_zone}")


def test_replay_timing_then_prefill_again():
    """Kernel replay timing returns positive times for every class, forbids a
    decode step until the next prefill, and leaves no trace in the next
    generation (same tokens and logits as a fresh session)."""
    from paper_2410_13839_amd.binding import MTP_ESTATE, MTPError
    wl = WORKLOADS["valle_k4"]
    w = make_weights(wl.model)
    logq = make_logq()
    pr = make_prompts(wl)

    def run(s, n):
        s.prefill(pr.phon, pr.ac)
        lg = []
        for _ in range(n):
            s.step(wl.K, wl.top_k)
            lg.append(s.logits(wl.K))
        return s.tokens()[0][:n * wl.K].copy(), np.stack(lg)

    s = new_session(wl, w, logq)
    ref = run(s, 6)
    # the classes the step launched: the front is one launch (class 10) or
    # the QKV projection and the attention (3 and 4), the FFN one launch (11)
    # or two (1 and 2); the others raise MTP_ESTATE.  Replaying the one-launch
    # kinds also runs their hand-off state through many launches in a row,
    # which the next generation checks.
    replayed = []
    for kc in range(1, 12):
        for cold in (True, False):
            try:
                us = s.replay(kc, 3, cold)
            except MTPError as e:
                assert e.code == MTP_ESTATE, (kc, e)
                continue
            assert 0.5 < us < 1000.0, (kc, cold, us)
            replayed.append(kc)
    replayed = sorted(set(replayed))
    assert replayed in ([5, 6, 7, 10, 11], [3, 4, 5, 6, 7, 11], [1, 2, 5, 6, 7, 10], [1, 2, 3, 4, 5, 6, 7]), replayed
    with pytest.raises(MTPError) as e:
        s.step(wl.K, wl.top_k)
    assert e.value.code == MTP_ESTATE
    with pytest.raises(MTPError) as e:
        s.force(np.zeros((1, wl.K), np.int32), [wl.K])
    assert e.value.code == MTP_ESTATE
    again = run(s, 6)
    s.close()
    assert np.array_equal(ref[0], again[0])
    assert np.array_equal(ref[1].view(np.uint32), again[1].view(np.uint32))
