"""The C ABI library loads, exports every call include/mtp.h declares, and
rejects bad arguments before touching the GPU (no compute calls here)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mtp.h")


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|void|const char\s*\*)\s*(mtp_\w+)\s*\(", src, re.M)))


def test_library_exports_every_declared_call():
    from paper_2410_13839_amd import binding
    lib = ctypes.CDLL(binding.LIB_PATH)
    names = _declared()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(binding.EXPORTED) == names


def _cfg(**kw):
    from paper_2410_13839_amd import binding as b
    from paper_2410_13839_amd.workloads import WORKLOADS
    wl = WORKLOADS["valle_k4"]
    cfg = b.make_config(wl.model, 1, wl.max_prompt, wl.max_new, wl.eos_min)
    for k, v in kw.items():
        setattr(cfg, k, v)
    return cfg


@pytest.mark.parametrize("field,value", [("d_model", 1000), ("n_heads", 15), ("k_heads", 9), ("k_heads", 0),
                                         ("topk_max", 33), ("page_size", 12), ("page_size", 8), ("page_size", 32),
                                         ("page_size", 64), ("dtype", 7), ("vocab", 5000),
                                         ("max_new", 5000), ("eos_id", 1025), ("max_batch", 0)])
def test_query_sizes_rejects_bad_configs(field, value):
    from paper_2410_13839_amd import binding as b
    with pytest.raises(b.MTPError) as e:
        b.mtp_query_sizes(_cfg(**{field: value}))
    assert e.value.code == b.MTP_EINVAL


def test_weight_layout_is_aligned_and_disjoint():
    from paper_2410_13839_amd import binding as b
    cfg = _cfg()
    spans = []
    for t in range(b.MTP_T_COUNT):
        layers = range(cfg.n_layers) if b.MTP_T_LN1_G <= t <= b.MTP_T_B_2 else [0]
        for l in layers:
            off, n = b.mtp_weight_offset(cfg, t, l)
            assert off % 256 == 0
            elt = 2 if t in b._MATRICES else 4
            spans.append((off, off + n * elt))
    spans.sort()
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        assert a1 <= b0
    sz = b.mtp_query_sizes(cfg)
    assert spans[-1][1] <= sz.weights_bytes
    # 12 x (3d^2 + d^2 + 2 d f) + tables + 8 heads x V x d, bf16
    d, f, V = 1024, 4096, 1025
    mats = 12 * (4 * d * d + 2 * d * f) + (512 + V + 4096) * d + 8 * V * d
    assert mats * 2 <= sz.weights_bytes < mats * 2 + 4 * 1024 * 1024
    assert sz.logq_bytes == V * V * 4


def test_calls_validate_before_gpu_work():
    from paper_2410_13839_amd import binding as b
    cfg = _cfg()
    with pytest.raises(b.MTPError):
        b.mtp_create(cfg, b.mtp_buffers(256, 512, 1024, 100), 0)   # misaligned workspace
    ctx = b.mtp_create(cfg, b.mtp_buffers(256, 512, 1024, 2048), 0)
    try:
        with pytest.raises(b.MTPError) as e:
            b.mtp_decode_step(ctx, 1, 4, 4)
        assert e.value.code == b.MTP_ESTATE
        with pytest.raises(b.MTPError) as e:       # prompt too long
            b.mtp_prefill(ctx, [np.zeros(100, np.int32)], [np.zeros(cfg.max_prompt, np.int32)])
        assert e.value.code == b.MTP_EINVAL
        with pytest.raises(b.MTPError) as e:       # batch above max_batch
            b.mtp_prefill(ctx, [np.zeros(1, np.int32)] * 2, [np.zeros(3, np.int32)] * 2)
        assert e.value.code == b.MTP_EINVAL
        with pytest.raises(b.MTPError) as e:       # acoustic id 1024 (EOS) is not a prompt token
            b.mtp_prefill(ctx, [np.zeros(1, np.int32)], [np.full(3, 1024, np.int32)])
        assert e.value.code == b.MTP_EINVAL
        with pytest.raises(b.MTPError) as e:       # phoneme id out of range
            b.mtp_prefill(ctx, [np.full(2, 512, np.int32)], [np.zeros(3, np.int32)])
        assert e.value.code == b.MTP_EINVAL
        with pytest.raises(b.MTPError) as e:
            b.mtp_profile_replay(ctx, 99, 10)
        assert e.value.code == b.MTP_EINVAL
        with pytest.raises(b.MTPError) as e:       # nothing launched yet
            b.mtp_profile_replay(ctx, b.MTP_KCLASS_GEMM_FFN1, 10)
        assert e.value.code == b.MTP_ESTATE
        for buf, nbytes in ((4096, 0), (0, 4096), (4096, 1000), (4104, 4096), (4096, 512)):
            with pytest.raises(b.MTPError) as e:   # eviction buffer without size, unaligned or too small
                b.mtp_profile_replay(ctx, b.MTP_KCLASS_GEMM_FFN1, 10, buf, nbytes)
            assert e.value.code == b.MTP_EINVAL
        with pytest.raises(b.MTPError) as e:       # teacher forcing before any decode step
            b.mtp_force_tokens(ctx, np.zeros((1, 4), np.int32), [4])
        assert e.value.code == b.MTP_ESTATE
    finally:
        b.mtp_destroy(ctx)


def test_kv_pool_exhaustion_is_reported():
    from paper_2410_13839_amd import binding as b
    cfg = _cfg(num_pages=10)
    ctx = b.mtp_create(cfg, b.mtp_buffers(256, 512, 1024, 2048), 0)
    try:
        with pytest.raises(b.MTPError) as e:
            b.mtp_prefill(ctx, [np.zeros(10, np.int32)], [np.zeros(10, np.int32)])
        assert e.value.code == b.MTP_ENOMEM
    finally:
        b.mtp_destroy(ctx)


def test_strerror():
    from paper_2410_13839_amd import binding as b
    assert b.mtp_strerror(b.MTP_ENOMEM).startswith("KV")


def test_bf16_weight_fragment_order():
    """The binding's packer follows the fragment order mtp.h documents for bf16
    Linear weights: element (n, k) at ((n/16)(K/32) + k/32)*512 + ((k%32)/8)*128
    + (n%16)*8 + k%8, rows padded with zeros to a multiple of 16."""
    from paper_2410_13839_amd.binding import tile_bf16_matrix
    rng = np.random.default_rng(5)
    N, K = 37, 96
    w = rng.integers(1, 65535, size=(N, K), dtype=np.uint16)
    t = tile_bf16_matrix(w)
    assert t.size == 48 * K
    n, k = np.meshgrid(np.arange(N), np.arange(K), indexing="ij")
    idx = ((n // 16) * (K // 32) + k // 32) * 512 + ((k % 32) // 8) * 128 + (n % 16) * 8 + k % 8
    assert np.array_equal(t[idx], w)
    mask = np.ones(t.size, bool)
    mask[idx.reshape(-1)] = False
    assert np.all(t[mask] == 0)


def test_packed_weights_hold_every_tensor():
    """pack_weights places each tensor of a bf16 model at its offset: row-major
    tables and vectors as given, Linear weights in fragment order."""
    from paper_2410_13839_amd import binding as b
    from paper_2410_13839_amd.workloads import ModelShape, Workload, make_weights
    shape = ModelShape(n_layers=1, d_model=256, n_heads=4, d_ff=512, k_heads=2, dtype="bf16", max_pos=64)
    w = make_weights(shape, seed=3)
    cfg = b.make_config(shape, 1, 16, 16, 16)
    img = b.pack_weights(cfg, w)
    u16 = lambda a: (np.ascontiguousarray(a, np.float32).view(np.uint32) >> 16).astype(np.uint16)
    off, n = b.mtp_weight_offset(cfg, b.MTP_T_EMB_AC, 0)
    assert np.array_equal(img[off:off + 2 * n].view(np.uint16), u16(w["emb_ac"]).reshape(-1))
    off, n = b.mtp_weight_offset(cfg, b.MTP_T_W_1, 0)
    tiled = b.tile_bf16_matrix(u16(w["l0.w_1"]))
    assert np.array_equal(img[off:off + 2 * tiled.size].view(np.uint16), tiled)
    off, n = b.mtp_weight_offset(cfg, b.MTP_T_W_HEADS, 0)
    tiled = b.tile_bf16_matrix(u16(w["w_heads"]).reshape(-1, 256))
    assert tiled.size == (2 * 1025 + 15) // 16 * 16 * 256
    assert np.array_equal(img[off:off + 2 * tiled.size].view(np.uint16), tiled)
    off, n = b.mtp_weight_offset(cfg, b.MTP_T_B_1, 0)
    assert np.array_equal(img[off:off + 4 * n].view(np.float32), w["l0.b_1"])


def test_set_selection_validates():
    from paper_2410_13839_amd import binding as b
    cfg = _cfg()
    ctx = b.mtp_create(cfg, b.mtp_buffers(256, 512, 1024, 2048), 0)
    try:
        for lattice, anchored in ((2, 0), (-1, 0), (0, 2)):
            with pytest.raises(b.MTPError) as e:
                b.mtp_set_selection(ctx, lattice, anchored)
            assert e.value.code == b.MTP_EINVAL
        b.mtp_set_selection(ctx, b.MTP_LATTICE_UNION, True)
        with pytest.raises(b.MTPError) as e:       # no step yet
            b.mtp_get_union_lattice(ctx, 1, 4)
        assert e.value.code == b.MTP_ESTATE
    finally:
        b.mtp_destroy(ctx)


def test_set_sampling_validates():
    from paper_2410_13839_amd import binding as b
    cfg = _cfg()
    ctx = b.mtp_create(cfg, b.mtp_buffers(256, 512, 1024, 2048), 0)
    try:
        for mode, tau in ((2, 1.0), (-1, 1.0), (1, 0.0), (1, -1.0), (1, float("nan")), (1, float("inf")),
                          (1, 1e-45)):
            with pytest.raises(b.MTPError) as e:
                b.mtp_set_sampling(ctx, mode, tau, 1)
            assert e.value.code == b.MTP_EINVAL, (mode, tau)
        b.mtp_set_sampling(ctx, b.MTP_SELECT_SAMPLE, 0.7, (1 << 64) - 1)
        b.mtp_set_sampling(ctx, b.MTP_SELECT_BEST, 0.0, 0)      # temperature unused when not sampling
        with pytest.raises(b.MTPError) as e:                    # no step yet
            b.mtp_get_uniforms(ctx, 1, 4)
        assert e.value.code == b.MTP_ESTATE
    finally:
        b.mtp_destroy(ctx)


def test_q_estimation_validates_before_gpu_work():
    from paper_2410_13839_amd import binding as b
    need = b.mtp_q_workspace_size(10, 2, 1025)
    assert need >= 10 * 4 + 33 * (1 << 17)
    assert b.mtp_q_workspace_size(10 ** 8, 350000, 1025) > 4 * 10 ** 8
    ok = dict(tokens=256, n_tokens=10, offsets=512, n_seqs=2, vocab=1025, eos_id=1024, flags=0, counts=1024,
              status=2048, workspace=4096, ws_bytes=need, stream=0)
    for k, v in (("n_tokens", -1), ("n_tokens", 1 << 31), ("n_seqs", -1), ("vocab", 0), ("vocab", 8193),
                 ("eos_id", 1025), ("eos_id", -1), ("flags", 2), ("counts", 0), ("status", 0), ("offsets", 0),
                 ("tokens", 0), ("workspace", 0), ("tokens", 260), ("workspace", 4096 + 64)):
        with pytest.raises(b.MTPError) as e:
            b.mtp_q_count(**{**ok, k: v})
        assert e.value.code == b.MTP_EINVAL, (k, v)
    with pytest.raises(b.MTPError) as e:
        b.mtp_q_count(**{**ok, "ws_bytes": need - 1})
    assert e.value.code == b.MTP_ENOMEM
    b.mtp_q_count(**{**ok, "n_seqs": 0, "ws_bytes": b.mtp_q_workspace_size(10, 0, 1025)})   # nothing launched
    for k, v in (("alpha", -1.0), ("alpha", float("nan")), ("alpha", float("inf")), ("vocab", 0), ("counts", 0),
                 ("logq", 0)):
        args = dict(counts=256, vocab=1025, alpha=1.0, logq=512, stream=0)
        args[k] = v
        with pytest.raises(b.MTPError) as e:
            b.mtp_q_normalize(**args)
        assert e.value.code == b.MTP_EINVAL, (k, v)


def test_probe_library_exports():
    """The measurement-probe library is built beside libmtp.so and exports
    its entry points (no GPU call is made)."""
    import ctypes
    from paper_2410_13839_amd.probe import LIB_PATH
    lib = ctypes.CDLL(LIB_PATH)
    for name in ("mtp_probe_launch_floor", "mtp_probe_stream", "mtp_probe_flag_barrier", "mtp_probe_xcc_map",
                 "mtp_probe_handoff", "mtp_probe_bf16_round"):
        assert hasattr(lib, name), name
