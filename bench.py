"""Decode throughput of the MTP + Viterbi path on one MI355X.

A step is one decode step of the whole hot path (trunk over the pending
chunk and the paged KV cache, final LN, K head projections, EOS mask +
top_k, Viterbi lattice, accept) for the whole batch.  Workload: the
12-layer d1024 bf16 VALL-E-shaped decoder, K=4 heads, top_k=4, batch 1,
prompt 100 phonemes + 225 acoustic tokens, up to 750 generated tokens (EOS
allowed from index 600).  Inputs are seeded synthetic (weights N(0, 0.02),
synthetic transition table, uniform prompt ids).

Prints one JSON line.  `value` is emitted codec tokens per second over the
timed decode steps (prefill excluded, inputs resident in HBM).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # three whole generations (187 full steps each) timed after one whole
    # generation of warm-up: the step time varies by a few percent between
    # generations
    ap.add_argument("--steps", type=int, default=561)
    ap.add_argument("--warmup", type=int, default=188)
    ap.add_argument("--workload", default="valle_k4")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true", help="skip the per-workload generation lines")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--copy-probe", action="store_true", help="also run a 256 MiB device copy (PMC calibration)")
    ap.add_argument("--replay-passes", type=int, default=20, help="passes of the per-class replay timing")
    ap.add_argument("--no-warm-replay", action="store_true", help="skip the cache-warm replay figures")
    ap.add_argument("--no-variants", action="store_true", help="skip the selection-variant figures")
    ap.add_argument("--no-qest", action="store_true", help="skip the transition-table estimation figures")
    ap.add_argument("--no-nar", action="store_true", help="skip the NAR module figures")
    ap.add_argument("--nar-only", action="store_true", help="only the NAR module figures (one JSON line of them)")
    ap.add_argument("--config-only", default=None,
                    help="only one workload's generation line (tiny, valle_k4, valle_k8, valle_b32, long_b8)")
    ap.add_argument("--batched-only", action="store_true",
                    help="only the batched decode kernel classes against their roofline ceilings")
    ap.add_argument("--batched-workloads", default="valle_b32,long_b8",
                    help="comma-separated workloads of --batched-only")
    ap.add_argument("--no-graph", action="store_true",
                    help="--batched-only: decode steps launched eagerly instead of replayed graphs")
    ap.add_argument("--peaks-only", action="store_true", help="only the copy and library-GEMM figures")
    ap.add_argument("--qest-only", action="store_true",
                    help="only the transition-table estimation figures (one JSON line of them)")
    return ap.parse_args()


def _steps_per_generation(wl):
    return -(-wl.max_new // wl.K)


def time_decode(sess, wl, prompts, steps, warmup, torch, top_k=None):
    """Warm up, then time exactly `steps` decode steps that each run the whole
    path.  The first step after a prefill has no pending chunk (it runs the
    heads and the selection on the prompt's last hidden state), so it is never
    timed; a generation's remaining steps 1 .. S-1 are.  Whole generations
    are timed while `steps` covers them; the rest (or all of a shorter run) is
    the window of consecutive steps centred on the middle of a generation, so
    its mean context, and with it the step time, is the generation's mean.
    Prefills are outside the timed intervals.  Returns (ms, tokens)."""
    top_k = wl.top_k if top_k is None else top_k
    per_gen = _steps_per_generation(wl)
    full = per_gen - 1                       # steps with a pending chunk per generation
    st = sess.stream
    # warmup (also instantiates the hipGraphs of the step)
    sess.prefill(prompts.phon, prompts.ac)
    for i in range(warmup):
        if i and i % per_gen == 0:
            sess.prefill(prompts.phon, prompts.ac)
        sess.step_async(wl.K, top_k)
    torch.cuda.synchronize()
    total_ms, tokens, done = 0.0, 0, 0
    while done < steps:
        n = min(full, steps - done)
        first = 1 + (full - n) // 2          # window start (step index within the generation)
        sess.prefill(prompts.phon, prompts.ac)
        for _ in range(first):
            sess.step_async(wl.K, top_k)
        torch.cuda.synchronize()
        gen0 = int(sess.seq_state()["gen"].sum())
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(n):
            sess.step_async(wl.K, top_k)
        e1.record(st)
        torch.cuda.synchronize()
        total_ms += e0.elapsed_time(e1)
        tokens += int(sess.seq_state()["gen"].sum()) - gen0
        done += n
    return total_ms, tokens


KCLASSES = {  # kernel class -> (name, launches per decode step as a function of layers)
    10: ("LN1 + QKV + decode attention, one launch (qkv_front_kernel)", lambda L: L),
    9: ("LN1 + QKV + attention over the cached keys (qkv_attn_kernel)", lambda L: L),
    4: ("attention (attn_dec_kernel)", lambda L: L),
    3: ("QKV projection (gemv_kernel<EpiQKVDec>)", lambda L: L),
    11: ("LN2 + FFN1 + FFN2, one launch (ffn_chain_kernel)", lambda L: L),
    1: ("FFN1 (gemv_kernel<EpiGeluB>)", lambda L: L),
    5: ("heads (gemv_kernel<EpiLogitsB>)", lambda L: 1),
    6: ("out-projection (gemv_kernel<EpiPart>, attention merge)", lambda L: L),
    2: ("FFN2 (gemv_kernel<EpiPart>)", lambda L: L),
}


def launch_bytes(wl, kclass, ctx):
    """Algorithmic HBM bytes of one launch of a kernel class at batch B, K
    pending rows per sequence, `ctx` cached tokens per sequence (bf16 weights
    and KV, fp32 residual stream).  Every tensor an ideal fused kernel must
    touch counts once: weights, biases, LayerNorm parameters, input and output
    rows; the residual rows are read and written by the LayerNorm consumer
    that completes them (QKV, FFN1), the projections before them (O-proj,
    FFN2) write one fp32 contribution per row.  Split-K partial sums beyond
    that one contribution are overhead, not algorithmic bytes."""
    m = wl.model
    d, f, V, B, K = m.d_model, m.d_ff, m.vocab, wl.batch, wl.K
    M = B * K
    if kclass == 4:   # K and V rows of every head of every key + queries + output
        return B * (ctx + K) * 2 * d * 2 + M * d * 4 + M * d * 2
    if kclass == 3:
        return 3 * d * d * 2 + 3 * d * 4 + M * d * 4 + 2 * d * 4 + M * d * 4 + 2 * M * d * 2
    if kclass in (9, 10):   # the QKV projection, the cached K and V rows of every head, the attention output
        return launch_bytes(wl, 3, ctx) + B * ctx * 2 * d * 2 + M * d * 2
    if kclass == 1:
        return f * d * 2 + f * 4 + 2 * M * d * 4 + 2 * d * 4 + M * f * 2
    if kclass == 5:
        return K * V * d * 2 + K * V * 4 + B * d * 4 + 2 * d * 4 + B * K * V * 4
    if kclass == 6:
        return d * d * 2 + M * d * 2 + M * d * 4
    if kclass == 2:
        return d * f * 2 + M * f * 2 + M * d * 4
    if kclass == 11:  # both FFN products; the GELU rows between them need not reach HBM
        return launch_bytes(wl, 1, ctx) + launch_bytes(wl, 2, ctx) - 2 * M * f * 2
    raise ValueError(kclass)


KCLASS_SOURCES = {  # kernel class -> the sources its kernels are built from
    4: ("attn_mfma.hip", "attn_dec.h", "common.h", "launch.h", "wave.h"),
    9: ("qkv_attn.hip", "ln_rows.h", "common.h", "launch.h", "wave.h"),
}
GEMV_SOURCES = ("gemv.hip", "attn_dec.h", "ln_rows.h", "common.h", "launch.h", "wave.h")


def kernel_source_digest(kclass):
    """Digest of the HIP sources of one kernel class: PMC traffic figures are
    valid only for the kernels they were taken on."""
    import hashlib
    h = hashlib.sha256()
    for name in KCLASS_SOURCES.get(kclass, GEMV_SOURCES):
        h.update(name.encode())
        with open(os.path.join(ROOT, "paper_2410_13839_amd", "csrc", name), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def pmc_traffic(workload, kclass):
    """HBM bytes per launch of kernel class `kclass` from the committed PMC
    summary (FETCH_SIZE and WRITE_SIZE in KiB per dispatch, scaled by the
    factors a copy of known size gives), or None when there is none for this
    workload and class or the kernels changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    digest = kernel_source_digest(kclass)
    with open(path) as fh:
        for line in fh:
            if not line.startswith("pmc:"):
                continue
            kv = dict(item.split("=", 1) for item in line[4:].split())
            if int(kv["class"]) != kclass or kv["source"] != digest:
                continue
            return int(round(float(kv["fetch_kib"]) * 1024 * float(kv["fetch_factor"])
                             + float(kv["write_kib"]) * 1024 * float(kv["write_factor"])))
    return None


def replay_kernels(sess, wl, prompts, steps, iters, torch, cold=True):
    """Per kernel class: average launch time (us) over `iters` replays of the
    class's launches in one decode step (one per layer), mid-generation after
    `steps` decode steps; with `cold`, the caches are evicted before each pass
    as the other layers' weights evict them in a real step."""
    sess.prefill(prompts.phon, prompts.ac)
    for i in range(steps):
        sess.step_async(wl.K, wl.top_k)
        if i % 25 == 24:
            torch.cuda.synchronize()
            print(f"[bench] replay set-up: step {i + 1}/{steps}", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    from paper_2410_13839_amd.binding import MTP_ESTATE, MTPError
    ctx = int(sess.seq_state()["ctx_len"].max())
    out = {}
    for kc in KCLASSES:
        try:
            out[kc] = sess.replay(kc, iters, cold)
        except MTPError as e:
            if e.code != MTP_ESTATE:
                raise
            continue              # not launched on this workload's path (fused front or separate launches)
        print(f"[bench] replay {'cold' if cold else 'warm'} class {kc}: {out[kc]:.3f} us", file=sys.stderr, flush=True)
    return out, ctx


def cpu_baseline(wl, weights, logq, prompts, budget_s):
    """The float64 oracle as it stands, on this host's cores: prefill, then
    decode steps until about `budget_s` seconds of decode have run."""
    from oracle.decoder import ARDecoder
    from oracle.generate import Generator
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    model = ARDecoder(wl.model, weights)
    g = Generator(model, logq, wl.eos_min, wl.max_new)
    t0 = time.perf_counter()
    g.prefill(prompts.phon[0], prompts.ac[0])
    t_pre = time.perf_counter() - t0
    t1 = time.perf_counter()
    steps = 0
    while not g.done and time.perf_counter() - t1 < budget_s:
        g.step(wl.K, wl.top_k)
        steps += 1
    dt = time.perf_counter() - t1
    toks = len(g.run.tokens)
    return {"value": toks / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{wl.name}: prefill of {len(prompts.phon[0]) + len(prompts.ac[0])} tokens "
                      f"({t_pre:.1f} s, excluded) then {steps} decode steps = {toks} tokens in {dt:.1f} s, "
                      f"float64 numpy on {threads} BLAS threads of {len(os.sched_getaffinity(0))} visible cores"}


def cpu_baseline_1thread(wl, weights, logq, prompts, budget_s):
    """The same oracle limited to one BLAS thread (threadpoolctl), on a
    bounded sample: prefill, then decode steps for about `budget_s` s."""
    try:
        from threadpoolctl import threadpool_limits
    except Exception:
        return None
    with threadpool_limits(limits=1):
        out = cpu_baseline(wl, weights, logq, prompts, budget_s)
    out["cores"] = 1
    out["sample"] = out["sample"].split(", float64")[0] + ", float64 numpy on 1 BLAS thread"
    return out


def trunk_params(m):
    """Parameters one token streams through the trunk (per layer: QKV, out,
    FFN1, FFN2 weights and biases, two LayerNorms)."""
    d, F = m.d_model, m.d_ff
    return m.n_layers * (4 * d * d + 2 * d * F + 3 * d + d + F + d + 4 * d)


def head_params(m, K):
    return K * m.vocab * (m.d_model + 1)


def step_bytes(wl, ctx, trunk=True):
    """Algorithmic HBM bytes of one decode step at batch-wide cached lengths
    `ctx` (one entry per sequence): every weight of the trunk, the final LN
    and the first K heads once (bf16 matrices, fp32 vectors counted as bf16
    is close enough at these sizes), the K and V rows of every cached key of
    every layer (4 d bytes per key per layer for a bf16 cache), the new
    chunk's K and V, and the logits written and read."""
    m = wl.model
    d, L, B, K = m.d_model, m.n_layers, wl.batch, wl.K
    wb = 2 if m.dtype == "bf16" else 4
    heads = wb * (head_params(m, K) + 2 * d) + 8 * B * K * m.vocab
    if not trunk:
        return heads
    kv_read = wb * 2 * L * d * float(np.sum(ctx))
    kv_write = wb * 2 * L * d * B * K
    return wb * trunk_params(m) + kv_read + kv_write + heads


def prefill_flops(wl, lens):
    """Trunk flops of a prefill over prompts of lengths `lens`: the GEMMs
    (2 flops per weight per row) and causal attention (2 products of
    len * (len + 1) / 2 key-query pairs x d per layer)."""
    m = wl.model
    rows = float(np.sum(lens))
    attn = sum(2.0 * 2.0 * (n * (n + 1) / 2.0) * m.d_model for n in lens) * m.n_layers
    return 2.0 * rows * (trunk_params(m) - m.n_layers * (m.d_ff + 9 * m.d_model)) + attn


def bench_config(torch, name, weights_cache, logq):
    """One workload end to end: a warm-up generation, then one timed prefill
    and one timed full generation (every decode step until all sequences
    finish), HIP events on the library stream.  Reports codec tokens/s, the
    step time, the whole step's algorithmic bytes against the HBM peak and
    the prefill's flops against the bf16 MFMA peak."""
    from paper_2410_13839_amd.binding import Session
    from paper_2410_13839_amd.workloads import WORKLOADS, make_prompts, make_weights
    wl = WORKLOADS[name]
    key = wl.model
    if key not in weights_cache:
        weights_cache.clear()
        weights_cache[key] = make_weights(wl.model)
    w = weights_cache[key]
    pr = make_prompts(wl)
    s = Session(wl.model, w, logq, max_batch=wl.batch, max_prompt=wl.max_prompt, max_new=wl.max_new,
                eos_min=wl.eos_min, topk_max=max(8, wl.top_k))
    per_gen = _steps_per_generation(wl)
    st = s.stream
    lens = [len(p) + len(a) for p, a in zip(pr.phon, pr.ac)]
    res = None
    for rep in range(2):
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev[0].record(st)
        s.prefill(pr.phon, pr.ac)
        ev[1].record(st)
        for _ in range(per_gen):
            s.step_async(wl.K, wl.top_k)
        ev[2].record(st)
        torch.cuda.synchronize()
        pre_ms, dec_ms = ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2])
        gen = s.seq_state()["gen"]
        res = (pre_ms, dec_ms, int(gen.sum()))
    s.close()
    del s
    torch.cuda.empty_cache()
    pre_ms, dec_ms, toks = res
    # the first step after the prefill runs the heads only; step i >= 1 runs
    # the K pending rows over the prompt and the K (i - 1) tokens before them
    tot_bytes = sum(step_bytes(wl, [n + wl.K * i for n in lens], trunk=i > 0) for i in range(per_gen))
    us_step = dec_ms * 1000.0 / per_gen
    fl = prefill_flops(wl, lens)
    out = {"workload": f"{wl.name}: {wl.description}", "batch": wl.batch, "K": wl.K, "top_k": wl.top_k,
           "dtype": wl.model.dtype, "steps": per_gen, "tokens": toks,
           "tokens_per_s": round(toks / (dec_ms * 1e-3), 1), "us_per_step": round(us_step, 2),
           "ms_per_token_per_seq": round(dec_ms / (toks / wl.batch), 5),
           "step_algorithmic_bytes_avg": int(tot_bytes / per_gen),
           "step_hbm_GB_s": round(tot_bytes / (dec_ms * 1e-3) / 1e9, 1),
           "step_hbm_frac": round(tot_bytes / (dec_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "prefill_rows": int(np.sum(lens)), "prefill_ms": round(pre_ms, 3),
           "end_to_end_ms": round(pre_ms + dec_ms, 3),
           "end_to_end_tokens_per_s": round(toks / ((pre_ms + dec_ms) * 1e-3), 1),
           "prefill_tflops": round(fl / (pre_ms * 1e-3) / 1e12, 1),
           "prefill_mfma_frac_bf16": round(fl / (pre_ms * 1e-3) / 2.5e15, 4) if wl.model.dtype == "bf16" else None}
    print(f"[bench] config {name}: {out}", file=sys.stderr, flush=True)
    return out


MFMA_PEAK_BF16 = 2.5e15


def batched_class_figures(wl, kclass, ctx_sum):
    """Algorithmic flops and HBM bytes of one launch of a batched decode
    kernel class (M = B K rows, bf16 weights / activations / KV, fp32
    residual stream and queries); every operand an ideal kernel must touch,
    once.  `ctx_sum`: cached keys summed over the batch."""
    m = wl.model
    d, F, B, K, V = m.d_model, m.d_ff, wl.batch, wl.K, m.vocab
    M = B * K
    if kclass == 3:   # LN1 rows -> q (fp32), K / V rows into the cache (bf16)
        return 2.0 * M * 3 * d * d, 3 * d * d * 2 + 3 * d * 4 + M * d * 2 + M * d * 4 + 2 * M * d * 2
    if kclass == 6:   # attention rows -> one fp32 contribution per row
        return 2.0 * M * d * d, d * d * 2 + M * d * 2 + M * d * 4
    if kclass == 1:   # LN2 rows -> GELU rows (bf16)
        return 2.0 * M * F * d, F * d * 2 + F * 4 + M * d * 2 + M * F * 2
    if kclass == 2:   # GELU rows -> one fp32 contribution per row
        return 2.0 * M * d * F, d * F * 2 + M * F * 2 + M * d * 4
    if kclass == 4:   # K pending queries per sequence over its cached keys
        keys = ctx_sum + B * K
        return 4.0 * K * keys * d, keys * 2 * d * 2 + M * d * 4 + M * d * 2
    if kclass == 8:   # residual + contribution + bias -> residual (fp32) and LN rows (bf16)
        return 8.0 * M * d, 3 * M * d * 4 + M * d * 2 + 3 * d * 4
    raise ValueError(kclass)


BATCHED_CLASSES = {3: "QKV (gemm_med_bf16<EpiQKV>)", 4: "attention (attn_dec_kernel)",
                   6: "out-projection (gemm_med_bf16<EpiPartial>)", 1: "FFN1 (gemm_med_bf16<EpiGelu>)",
                   2: "FFN2 (gemm_med_bf16<EpiPartial>)", 8: "residual + LayerNorm (resid_ln_kernel)"}


def bench_batched_kernels(torch, name, weights_cache, logq, passes, flags=0):
    """Per kernel class of a batched decode step (mid-generation): average
    launch time from cold replays (caches evicted before each pass), the
    achieved TFLOP/s and GB/s, and the fraction of the class's own roofline
    ceiling min(MFMA peak, AI x HBM peak)."""
    from paper_2410_13839_amd.binding import Session
    from paper_2410_13839_amd.workloads import WORKLOADS, make_prompts, make_weights
    wl = WORKLOADS[name]
    if wl.model not in weights_cache:
        weights_cache.clear()
        weights_cache[wl.model] = make_weights(wl.model)
    pr = make_prompts(wl)
    s = Session(wl.model, weights_cache[wl.model], logq, max_batch=wl.batch, max_prompt=wl.max_prompt,
                max_new=wl.max_new, eos_min=wl.eos_min, topk_max=max(8, wl.top_k), flags=flags)
    mid = _steps_per_generation(wl) // 2
    s.prefill(pr.phon, pr.ac)
    for _ in range(mid):
        s.step_async(wl.K, wl.top_k)
    torch.cuda.synchronize()
    ctx_sum = int(s.seq_state()["ctx_len"].sum())
    out = {}
    for kc, cname in BATCHED_CLASSES.items():
        us = s.replay(kc, passes, True)
        fl, nb = batched_class_figures(wl, kc, ctx_sum)
        ai = fl / nb
        ceil = min(MFMA_PEAK_BF16, ai * HBM_PEAK_GBS * 1e9)
        ach = fl / (us * 1e-6)
        out[cname] = {"avg_launch_us": round(us, 3), "flops": fl, "bytes": nb, "flop_per_byte": round(ai, 1),
                      "tflops": round(ach / 1e12, 1), "GB_s": round(nb / (us * 1e-6) / 1e9, 1),
                      "ceiling_tflops": round(ceil / 1e12, 1), "frac_of_ceiling": round(ach / ceil, 4),
                      "frac_of_mfma_peak": round(ach / MFMA_PEAK_BF16, 4)}
        print(f"[bench] {name} class {kc}: {out[cname]}", file=sys.stderr, flush=True)
    s.close()
    del s
    torch.cuda.empty_cache()
    return {"workload": f"{wl.name}: {wl.description}", "step": mid, "cached_keys_total": ctx_sum,
            "passes": passes, "classes": out}


def bench_peaks(torch):
    """What this GPU delivers to plain library work, next to the published
    peaks: a 1 GiB device-to-device copy (bytes read + written per second)
    and an 8192^3 bf16 matrix product through torch (hipBLASLt), fp32
    accumulation, bf16 output.  HIP events on torch's current stream."""
    st = torch.cuda.current_stream()
    a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 10
    e0.record(st)
    for _ in range(reps):
        b.copy_(a)
    e1.record(st)
    torch.cuda.synchronize()
    copy_gbs = 2.0 * a.numel() * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a, b
    n = 8192
    x = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    y = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    for _ in range(3):
        z = x @ y
    e0.record(st)
    for _ in range(reps):
        z = x @ y
    e1.record(st)
    torch.cuda.synchronize()
    gemm_tf = 2.0 * n ** 3 * reps / (e0.elapsed_time(e1) * 1e-3) / 1e12
    del x, y, z
    torch.cuda.empty_cache()
    out = {"copy_GB_s": round(copy_gbs, 1), "copy_frac_of_hbm_peak": round(copy_gbs / HBM_PEAK_GBS, 3),
           "bf16_gemm_8192_tflops": round(gemm_tf, 1), "bf16_gemm_frac_of_mfma_peak": round(gemm_tf * 1e12 / MFMA_PEAK_BF16, 3),
           "how": "torch copy_ of 1 GiB (read + write bytes) and torch.matmul bf16 8192^3 (hipBLASLt), HIP events"}
    print(f"[bench] achievable peaks: {out}", file=sys.stderr, flush=True)
    return out


def bench_qest(torch, reps, cpu):
    """Transition-table estimation over the LibriTTS-train-shaped corpus
    (354,780 utterances, ~105 M tokens): zero the counts, count bigrams with
    the end-of-utterance EOS pair, normalise to log Q (alpha = 1).  HIP events
    on the stream the kernels run on."""
    from paper_2410_13839_amd.binding import MTP_Q_COUNT_EOS, mtp_q_count, mtp_q_normalize, mtp_q_workspace_size
    from paper_2410_13839_amd.workloads import CORPORA, EOS_ID, VOCAB, make_corpus
    cp = make_corpus(CORPORA["libritts_train"])
    n_tok, n_seq, V = int(cp.tokens.size), int(cp.offsets.size - 1), VOCAB
    print(f"[bench] q estimation: {n_tok} tokens in {n_seq} utterances", file=sys.stderr, flush=True)
    t = torch.from_numpy(cp.tokens).cuda()
    o = torch.from_numpy(cp.offsets).cuda()
    counts = torch.empty((V, V), dtype=torch.int32, device="cuda")
    status = torch.empty(3, dtype=torch.int64, device="cuda")
    ws_bytes = mtp_q_workspace_size(n_tok, n_seq, V)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    logq = torch.empty((V, V), dtype=torch.float32, device="cuda")
    st = torch.cuda.current_stream()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(reps + 1)]
    for r in range(reps + 1):                       # pass 0 is a warm-up
        e = ev[r]
        e[0].record(st)
        counts.zero_()
        status.zero_()
        e[1].record(st)
        mtp_q_count(t.data_ptr(), n_tok, o.data_ptr(), n_seq, V, EOS_ID, MTP_Q_COUNT_EOS, counts.data_ptr(),
                    status.data_ptr(), ws.data_ptr(), ws_bytes, st.cuda_stream)
        e[2].record(st)
        mtp_q_normalize(counts.data_ptr(), V, 1.0, logq.data_ptr(), st.cuda_stream)
        e[3].record(st)
    torch.cuda.synchronize()
    tot = np.mean([ev[r][0].elapsed_time(ev[r][3]) for r in range(1, reps + 1)]) * 1e3
    cnt = np.mean([ev[r][1].elapsed_time(ev[r][2]) for r in range(1, reps + 1)]) * 1e3
    nrm = np.mean([ev[r][2].elapsed_time(ev[r][3]) for r in range(1, reps + 1)]) * 1e3
    assert status.cpu().tolist() == [0, 0, 0]
    count_bytes = n_tok * 4 + (n_seq + 1) * 8 + V * V * 4
    out = {"corpus": "libritts_train (synthetic Markov chain of Q)", "tokens": n_tok, "utterances": n_seq,
           "tokens_per_s": round(n_tok / (tot * 1e-6), 1), "us_total": round(tot, 2), "reps": reps,
           "count_kernel_us": round(cnt, 2), "count_algorithmic_bytes": count_bytes,
           "count_GB_s": round(count_bytes / (cnt * 1e-6) / 1e9, 1),
           "count_bigrams_per_s": round((n_tok) / (cnt * 1e-6), 1),
           "normalize_kernel_us": round(nrm, 2), "normalize_GB_s": round(2 * V * V * 4 / (nrm * 1e-6) / 1e9, 1),
           "paper_context": "paper: the LibriTTS transition table takes 3 minutes (hardware and implementation unstated)"}
    if cpu:
        from oracle.qestimate import bigram_counts, log_q
        n_s = 100000
        sl = cp.offsets[:n_s + 1]
        tk = cp.tokens[:int(sl[-1])]
        t0 = time.perf_counter()
        c, _, _ = bigram_counts(tk, sl, V, EOS_ID, True)
        log_q(c, 1.0)
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": round(tk.size / dt, 1), "unit": "tokens/s", "cores": 1, "kind": "oracle",
                               "sample": f"first {n_s} utterances ({tk.size} tokens), counts + log Q"}
    print(f"[bench] q estimation: {out}", file=sys.stderr, flush=True)
    del t, o, counts, status, logq, ws
    torch.cuda.empty_cache()
    return out


def nar_flops(wl, inp):
    """Algorithmic flops of one NAR forward (all stages): the GEMMs (QKV,
    out-projection, FFN, the stage head) and the attention products
    (2 * 2 * len^2 * d per layer and utterance, bidirectional)."""
    m = wl.model
    d, F, cb = m.d_model, m.d_ff, m.codebook
    lens = [len(p) + q.shape[1] + len(a) for p, q, a in zip(inp.phon, inp.prompt, inp.a1)]
    rows = sum(lens)
    per_layer = 2 * rows * (3 * d * d + d * d + 2 * d * F) + sum(4 * L * L * d for L in lens)
    return m.k_heads * (m.n_layers * per_layer + 2 * rows * d * cb)


def bench_nar(torch, reps, cpu):
    """NAR module (codec layers 2..8) on the VALL-E-shaped bf16 model: one
    utterance of 100 phonemes + 225 prompt + 750 target rows, and a ragged
    batch of 8.  HIP events around mtp_nar_run on the session's stream."""
    from paper_2410_13839_amd.binding import NarSession
    from paper_2410_13839_amd.workloads import NAR_WORKLOADS, make_nar_inputs, make_weights
    out = {}
    w = make_weights(NAR_WORKLOADS["nar_valle"].model)
    for name in ("nar_valle", "nar_valle_b8"):
        wl = NAR_WORKLOADS[name]
        inp = make_nar_inputs(wl)
        s = NarSession(wl.model, w, max_batch=wl.batch, max_seq=wl.max_seq)
        s.prepare(inp.phon, inp.prompt, inp.a1)
        s.run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s.stream)
        for _ in range(reps):
            s.run()
        e1.record(s.stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        fl = nar_flops(wl, inp)
        n_codes = wl.model.k_heads * sum(len(a) for a in inp.a1)
        out[name] = {"workload": wl.description, "ms_per_forward": round(ms, 3), "reps": reps,
                     "codes_per_s": round(n_codes / (ms * 1e-3), 1),
                     "tflops": round(fl / (ms * 1e-3) / 1e12, 1), "flops_per_forward": fl,
                     "mfma_frac_bf16": round(fl / (ms * 1e-3) / 2.5e15, 3)}
        print(f"[bench] {name}: {out[name]}", file=sys.stderr, flush=True)
        s.close()
        del s
        torch.cuda.empty_cache()
    if cpu:
        from oracle.nar import NARModel
        wl = NAR_WORKLOADS["nar_valle"]
        inp = make_nar_inputs(wl)
        m = NARModel(wl.model, w)
        teacher = np.vstack([inp.a1[0][None], np.zeros((wl.model.k_heads, len(inp.a1[0])), np.int64)])
        import os as _os
        t0 = time.perf_counter()
        m.forward(m.embed(2, inp.phon[0], inp.prompt[0], teacher))
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": round(len(inp.a1[0]) / dt, 1), "unit": "codes/s", "kind": "oracle",
                               "cores": _os.cpu_count(), "sample": "one stage (layer 2) of nar_valle, float64"}
    return out


def main():
    args = _parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the decode path runs on a single MI355X).", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2410_13839_amd.binding import Session
    from paper_2410_13839_amd.workloads import WORKLOADS, make_logq, make_prompts, make_weights

    if args.qest_only:
        print(json.dumps(bench_qest(torch, 5, not args.no_cpu_baseline)))
        return
    if args.nar_only:
        print(json.dumps(bench_nar(torch, 3, not args.no_cpu_baseline)))
        return
    if args.config_only:
        print(json.dumps(bench_config(torch, args.config_only, {}, make_logq())))
        return
    if args.batched_only:
        from paper_2410_13839_amd.binding import MTP_FLAG_NO_GRAPH
        wc, lq = {}, make_logq()
        fl = MTP_FLAG_NO_GRAPH if args.no_graph else 0
        print(json.dumps({n: bench_batched_kernels(torch, n, wc, lq, args.replay_passes, fl)
                          for n in args.batched_workloads.split(",")}))
        return
    if args.peaks_only:
        print(json.dumps(bench_peaks(torch)))
        return

    wl = WORKLOADS[args.workload]
    weights = make_weights(wl.model)
    logq = make_logq()
    prompts = make_prompts(wl)
    sess = Session(wl.model, weights, logq, max_batch=wl.batch, max_prompt=wl.max_prompt, max_new=wl.max_new,
                   eos_min=wl.eos_min, topk_max=max(8, wl.top_k))
    print(f"[bench] {wl.name}: warmup {args.warmup}, timing {args.steps} steps", file=sys.stderr, flush=True)
    ms, tokens = time_decode(sess, wl, prompts, args.steps, args.warmup, torch)
    tok_s = tokens / (ms / 1000.0)
    ms_step = ms / args.steps
    ms_token = ms / (tokens / wl.batch)
    print(f"[bench] {tokens} tokens in {ms:.2f} ms: {tok_s:.0f} tokens/s, {ms_step * 1000:.1f} us/step",
          file=sys.stderr, flush=True)

    # per-kernel launch times (back-to-back replays) and the dominant kernel
    mid = _steps_per_generation(wl) // 2
    passes = args.replay_passes
    times, ctx = replay_kernels(sess, wl, prompts, mid, passes, torch, cold=True)
    if args.no_warm_replay:
        warm = {kc: float("nan") for kc in times}
    else:
        warm, _ = replay_kernels(sess, wl, prompts, mid, passes, torch, cold=False)
    L = wl.model.n_layers
    kernels = {}
    for kc, us in times.items():
        name, per_step = KCLASSES[kc]
        nbytes = launch_bytes(wl, kc, ctx)
        kernels[name] = {"avg_launch_us": round(us, 3), "launches_per_step": per_step(L),
                         "bytes_per_launch": nbytes, "GB_s": round(nbytes / (us * 1e-6) / 1e9, 1),
                         "share_of_step": round(us * per_step(L) / (ms_step * 1000.0), 3),
                         "avg_launch_us_cache_warm": round(warm[kc], 3) if warm[kc] == warm[kc] else None}
    # dominant kernel class: the largest time per step (the rocprofv3
    # summary's top kernel); the classes within 5% of it, too close to rank
    # by one measurement, are listed beside it, and every class's fraction
    per_step = {kc: times[kc] * KCLASSES[kc][1](L) for kc in times}
    top = max(per_step.values())
    near = [kc for kc in per_step if per_step[kc] >= 0.95 * top]
    dom = max(per_step, key=lambda kc: per_step[kc])
    dname = KCLASSES[dom][0]
    dk = kernels[dname]
    roof = {"kernel": dname, "bound": "hbm", "achieved": dk["GB_s"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(dk["GB_s"] / HBM_PEAK_GBS, 4), "traffic": pmc_traffic(wl.name, dom),
            "bytes_per_launch": dk["bytes_per_launch"], "avg_launch_us": dk["avg_launch_us"],
            "measured": f"{passes} passes over the {KCLASSES[dom][1](L)} launches of one step at step {mid} "
                        f"(context {ctx} tokens), caches evicted before each pass, HIP events on the library stream",
            "selection": "largest time per step; near_dominant: the classes within 5% of it",
            "near_dominant": [KCLASSES[kc][0] for kc in near],
            "classes_frac": {KCLASSES[kc][0]: round(kernels[KCLASSES[kc][0]]["GB_s"] / HBM_PEAK_GBS, 4)
                             for kc in times}}
    print(f"[bench] dominant kernel {dname}: {dk}", file=sys.stderr, flush=True)

    # selection variants (Sec. 3.3): throughput of the whole step and the
    # selection kernel's own launch time (cold passes at step `mid`)
    from paper_2410_13839_amd.binding import MTP_KCLASS_SELECT, MTP_SELECT_BEST, MTP_SELECT_SAMPLE
    variants = []
    if not args.no_variants:
        for lat, anch, tk, smp, what in (
                (0, False, wl.top_k, False, "each head's own top_k (default)"),
                (1, False, wl.top_k, False, "union of all heads' top_k, m x m transitions"),
                (0, True, wl.top_k, False, "own top_k, first position anchored"),
                (1, True, wl.top_k, False, "union, first position anchored"),
                (0, False, 1, False, "top_k = 1: per-head argmax, no Viterbi"),
                (0, False, wl.top_k, True, "top_k sampling in the own lattice, temperature 1"),
                (1, False, wl.top_k, True, "top_k sampling in the union lattice, temperature 1")):
            sess.set_selection(lat, anch)
            sess.set_sampling(MTP_SELECT_SAMPLE if smp else MTP_SELECT_BEST, 1.0, 2024)
            n_full = _steps_per_generation(wl) - 1
            vms, vtok = time_decode(sess, wl, prompts, n_full, 5, torch, top_k=tk)
            sess.prefill(prompts.phon, prompts.ac)
            for _ in range(mid):
                sess.step_async(wl.K, tk)
            torch.cuda.synchronize()
            sel_us = sess.replay(MTP_KCLASS_SELECT, passes, True)
            v = {"lattice": "union" if lat else "own", "anchored": anch, "top_k": tk, "sampled": smp, "selection": what,
                 "tokens_per_s": round(vtok / (vms / 1000.0), 1), "us_per_step": round(vms * 1000.0 / n_full, 2),
                 "select_kernel_us": round(sel_us, 3)}
            variants.append(v)
            print(f"[bench] variant {v}", file=sys.stderr, flush=True)
        sess.set_selection(0, False)
        sess.set_sampling(MTP_SELECT_BEST)
    sess.close()
    del sess
    torch.cuda.empty_cache()

    configs = None
    if not args.no_secondary and args.workload == "valle_k4":
        configs = []
        wcache = {}
        for name in ("tiny", "valle_k4", "valle_k8", "valle_b32", "long_b8"):
            configs.append(bench_config(torch, name, wcache, logq))
        wcache.clear()

    batched = None
    if not args.no_secondary and args.workload == "valle_k4":
        batched = {}
        wcache = {}
        for name in ("valle_b32", "long_b8"):
            batched[name] = bench_batched_kernels(torch, name, wcache, logq, passes)
        wcache.clear()

    qest = None
    if not args.no_qest:
        qest = bench_qest(torch, 5, not args.no_cpu_baseline)
    peaks = None if args.no_secondary else bench_peaks(torch)
    nar = None
    if not args.no_nar:
        nar = bench_nar(torch, 3, not args.no_cpu_baseline)

    if args.copy_probe:
        a = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()

    cpu = None
    cpu1 = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, weights, logq, prompts, args.cpu_seconds)
        print(f"[bench] cpu oracle: {cpu['value']:.2f} tokens/s", file=sys.stderr, flush=True)
        # one-thread figures for the two batch-1 parity workloads (small samples)
        cpu1 = {}
        wt = WORKLOADS["tiny"]
        cpu1["tiny"] = cpu_baseline_1thread(wt, make_weights(wt.model), logq, make_prompts(wt), 3.0)
        cpu1[wl.name] = cpu_baseline_1thread(wl, weights, logq, prompts, 5.0)
        print(f"[bench] cpu oracle, one thread: {cpu1}", file=sys.stderr, flush=True)

    out = {
        "metric": "codec tokens/sec (and ms/token) at batch 1, K=4 heads, top_k=4",
        "value": round(tok_s, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4), "ms_per_token": round(ms_token, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.description}", "batch": wl.batch, "K": wl.K, "top_k": wl.top_k,
                   "layers": wl.model.n_layers, "d_model": wl.model.d_model, "prompt": "100 phon + 225 acoustic",
                   "max_new": wl.max_new, "parallelism": "single GPU"},
        "roofline": roof,
        "kernels": kernels,
        "cpu_baseline": cpu,
        "cpu_baseline_one_thread": cpu1,
        "selection_variants": variants,
        "configs": configs,
        "batched_decode_kernels": batched,
        "achievable_peaks": peaks,
        "q_estimation": qest,
        "nar": nar,
        "paper_context": "paper reports 20.5 -> 4.5 ms/token (x4.56, VALL-E, 8 heads) on unstated inference hardware",
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
