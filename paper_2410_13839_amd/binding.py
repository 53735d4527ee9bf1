"""ctypes binding of libmtp (include/mtp.h): argument marshalling only.

Functions keep the C names.  PyTorch provides device memory (torch tensors'
data_ptr()) and the HIP stream; every step of the decode path runs in the
library's HIP kernels.  If libmtp.so is missing this module raises on import:
there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmtp.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() (hipcc, gfx950)")
_lib = ctypes.CDLL(LIB_PATH)

MTP_OK, MTP_EINVAL, MTP_ENOMEM, MTP_ESTATE, MTP_EHIP, MTP_ETIMEOUT = 0, -1, -2, -3, -4, -5
MTP_DTYPE_F32, MTP_DTYPE_BF16 = 0, 1
MTP_FLAG_NO_GRAPH, MTP_FLAG_NAR = 1, 2
(MTP_T_EMB_PHONE, MTP_T_EMB_AC, MTP_T_POS, MTP_T_LN1_G, MTP_T_LN1_B, MTP_T_W_QKV, MTP_T_B_QKV, MTP_T_W_O,
 MTP_T_B_O, MTP_T_LN2_G, MTP_T_LN2_B, MTP_T_W_1, MTP_T_B_1, MTP_T_W_2, MTP_T_B_2, MTP_T_LNF_G, MTP_T_LNF_B,
 MTP_T_W_HEADS, MTP_T_B_HEADS, MTP_T_STAGE, MTP_T_COUNT) = range(21)
(MTP_KCLASS_GEMM_FFN1, MTP_KCLASS_GEMM_FFN2, MTP_KCLASS_GEMM_QKV, MTP_KCLASS_ATTENTION, MTP_KCLASS_HEADS,
 MTP_KCLASS_GEMM_OPROJ, MTP_KCLASS_SELECT, MTP_KCLASS_RESID_LN, MTP_KCLASS_QKV_ATTN,
 MTP_KCLASS_QKV_FRONT, MTP_KCLASS_FFN_CHAIN) = 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11

EXPORTED = ["mtp_query_sizes", "mtp_weight_offset", "mtp_create", "mtp_prefill", "mtp_decode_step",
            "mtp_decode_step_async", "mtp_get_logits", "mtp_get_lattice", "mtp_force_tokens", "mtp_get_seq_state",
            "mtp_get_tokens",
            "mtp_profile_replay", "mtp_reset", "mtp_destroy", "mtp_last_error", "mtp_strerror",
            "mtp_set_selection", "mtp_get_union_lattice", "mtp_set_sampling", "mtp_get_uniforms",
            "mtp_q_workspace_size", "mtp_q_count", "mtp_q_count_noalloc", "mtp_q_normalize",
            "mtp_nar_prepare", "mtp_nar_run", "mtp_nar_get_codes", "mtp_nar_get_logits"]
MTP_Q_COUNT_EOS = 1
MTP_LATTICE_OWN, MTP_LATTICE_UNION = 0, 1
MTP_SELECT_BEST, MTP_SELECT_SAMPLE = 0, 1


class mtp_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "d_model", "n_heads", "d_ff", "vocab", "eos_id", "n_phone", "max_pos", "k_heads",
        "topk_max", "max_batch", "max_prompt", "max_new", "eos_min", "page_size", "num_pages", "dtype", "flags")]


class mtp_sizes(ctypes.Structure):
    _fields_ = [("weights_bytes", ctypes.c_uint64), ("logq_bytes", ctypes.c_uint64),
                ("kv_bytes", ctypes.c_uint64), ("workspace_bytes", ctypes.c_uint64)]


class mtp_buffers(ctypes.Structure):
    _fields_ = [("weights", ctypes.c_void_p), ("logq", ctypes.c_void_p),
                ("kv_pool", ctypes.c_void_p), ("workspace", ctypes.c_void_p)]


_P = ctypes.POINTER
_i32p = _P(ctypes.c_int32)
_f32p = _P(ctypes.c_float)
_ctx = ctypes.c_void_p

_lib.mtp_query_sizes.argtypes = [_P(mtp_config), _P(mtp_sizes)]
_lib.mtp_weight_offset.argtypes = [_P(mtp_config), ctypes.c_int, ctypes.c_int, _P(ctypes.c_uint64), _P(ctypes.c_uint64)]
_lib.mtp_create.argtypes = [_P(mtp_config), _P(mtp_buffers), ctypes.c_void_p, _P(_ctx)]
_lib.mtp_prefill.argtypes = [_ctx, ctypes.c_int, _i32p, _i32p, _i32p, _i32p]
_lib.mtp_decode_step.argtypes = [_ctx, ctypes.c_int, ctypes.c_int, _i32p, _i32p]
_lib.mtp_decode_step_async.argtypes = [_ctx, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
_lib.mtp_get_logits.argtypes = [_ctx, _f32p]
_lib.mtp_get_lattice.argtypes = [_ctx, _i32p, _f32p, _f32p, _i32p, _i32p]
_lib.mtp_force_tokens.argtypes = [_ctx, _i32p, _i32p]
_lib.mtp_set_selection.argtypes = [_ctx, ctypes.c_int, ctypes.c_int]
_lib.mtp_get_union_lattice.argtypes = [_ctx, _i32p, _i32p, _f32p, _f32p, _i32p, _i32p]
_lib.mtp_set_sampling.argtypes = [_ctx, ctypes.c_int, ctypes.c_float, ctypes.c_uint64]
_lib.mtp_get_uniforms.argtypes = [_ctx, _f32p]
_lib.mtp_q_workspace_size.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int, _P(ctypes.c_uint64)]
_lib.mtp_q_count.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                             ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                             ctypes.c_uint64, ctypes.c_void_p]
_lib.mtp_q_count_noalloc.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                     ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
MTP_Q_NOALLOC_SCRATCH_BYTES = 64 << 20
_lib.mtp_q_normalize.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p]
_lib.mtp_nar_prepare.argtypes = [_ctx, ctypes.c_int, _i32p, _i32p, _i32p, _i32p, _i32p, _i32p]
_lib.mtp_nar_run.argtypes = [_ctx]
_lib.mtp_nar_get_codes.argtypes = [_ctx, _i32p]
_lib.mtp_nar_get_logits.argtypes = [_ctx, ctypes.c_int, _f32p]
_lib.mtp_get_seq_state.argtypes = [_ctx, _i32p, _i32p, _i32p, _i32p]
_lib.mtp_get_tokens.argtypes = [_ctx, _i32p]
_lib.mtp_profile_replay.argtypes = [_ctx, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_uint64,
                                    _P(ctypes.c_double)]
_lib.mtp_reset.argtypes = [_ctx]
_lib.mtp_destroy.argtypes = [_ctx]
_lib.mtp_destroy.restype = None
_lib.mtp_last_error.argtypes = [_ctx]
_lib.mtp_last_error.restype = ctypes.c_char_p
_lib.mtp_strerror.argtypes = [ctypes.c_int]
_lib.mtp_strerror.restype = ctypes.c_char_p


class MTPError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{msg} (code {code})")
        self.code = code


def _check(rc: int, ctx=None, what: str = ""):
    if rc != MTP_OK:
        detail = _lib.mtp_last_error(ctx).decode() if ctx else _lib.mtp_strerror(rc).decode()
        raise MTPError(rc, f"{what}: {detail}")


def _i32(a) -> Tuple[np.ndarray, object]:
    arr = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return arr, arr.ctypes.data_as(_i32p)


# ------------------------------------------------------------- C-named calls
def mtp_query_sizes(cfg: mtp_config) -> mtp_sizes:
    out = mtp_sizes()
    _check(_lib.mtp_query_sizes(ctypes.byref(cfg), ctypes.byref(out)), None, "mtp_query_sizes")
    return out


def mtp_weight_offset(cfg: mtp_config, tensor: int, layer: int = 0) -> Tuple[int, int]:
    off, n = ctypes.c_uint64(), ctypes.c_uint64()
    _check(_lib.mtp_weight_offset(ctypes.byref(cfg), tensor, layer, ctypes.byref(off), ctypes.byref(n)),
           None, "mtp_weight_offset")
    return off.value, n.value


def mtp_create(cfg: mtp_config, bufs: mtp_buffers, stream: int):
    ctx = _ctx()
    _check(_lib.mtp_create(ctypes.byref(cfg), ctypes.byref(bufs), ctypes.c_void_p(stream), ctypes.byref(ctx)),
           None, "mtp_create")
    return ctx


def mtp_prefill(ctx, phon: Sequence[np.ndarray], ac: Sequence[np.ndarray]) -> None:
    B = len(ac)
    pl, plp = _i32([len(p) for p in phon])
    al, alp = _i32([len(a) for a in ac])
    pf, pfp = _i32(np.concatenate([np.asarray(p, np.int32) for p in phon]) if sum(pl) else np.zeros(1, np.int32))
    af, afp = _i32(np.concatenate([np.asarray(a, np.int32) for a in ac]))
    _check(_lib.mtp_prefill(ctx, B, pfp, plp, afp, alp), ctx, "mtp_prefill")


def mtp_nar_prepare(ctx, phon: Sequence[np.ndarray], prompt: Sequence[np.ndarray], a1: Sequence[np.ndarray]) -> None:
    """prompt[b]: [n_q, P_b] codes of every layer; a1[b]: [T_b] first-layer codes."""
    B = len(a1)
    pl, plp = _i32([len(p) for p in phon])
    ql, qlp = _i32([np.asarray(q).shape[1] for q in prompt])
    tl, tlp = _i32([len(a) for a in a1])
    cat = lambda xs: np.concatenate([np.asarray(x, np.int32).reshape(-1) for x in xs]) if xs else np.zeros(1, np.int32)
    pf, pfp = _i32(cat(phon) if sum(pl) else np.zeros(1, np.int32))
    qf, qfp = _i32(cat(prompt) if sum(ql) else np.zeros(1, np.int32))
    af, afp = _i32(cat(a1) if sum(tl) else np.zeros(1, np.int32))
    _check(_lib.mtp_nar_prepare(ctx, B, pfp, plp, qfp, qlp, afp, tlp), ctx, "mtp_nar_prepare")


def mtp_nar_run(ctx) -> None:
    _check(_lib.mtp_nar_run(ctx), ctx, "mtp_nar_run")


def mtp_nar_get_codes(ctx, k_heads: int, target_lens: Sequence[int]) -> List[np.ndarray]:
    """Per utterance [k_heads, T_b]: the codes of layers 2..k_heads+1."""
    out = np.zeros(max(1, k_heads * int(sum(target_lens))), np.int32)
    _check(_lib.mtp_nar_get_codes(ctx, out.ctypes.data_as(_i32p)), ctx, "mtp_nar_get_codes")
    res, o = [], 0
    for t in target_lens:
        res.append(out[o:o + k_heads * t].reshape(k_heads, t).copy())
        o += k_heads * t
    return res


def mtp_nar_get_logits(ctx, stage: int, n_target: int, codebook: int) -> np.ndarray:
    out = np.zeros((max(1, n_target), codebook), np.float32)
    _check(_lib.mtp_nar_get_logits(ctx, stage, out.ctypes.data_as(_f32p)), ctx, "mtp_nar_get_logits")
    return out[:n_target]


def mtp_decode_step(ctx, B: int, K: int, top_k: int) -> Tuple[np.ndarray, np.ndarray]:
    tok = np.zeros((B, K), np.int32)
    cnt = np.zeros(B, np.int32)
    _check(_lib.mtp_decode_step(ctx, K, top_k, tok.ctypes.data_as(_i32p), cnt.ctypes.data_as(_i32p)),
           ctx, "mtp_decode_step")
    return tok, cnt


def mtp_decode_step_async(ctx, K: int, top_k: int, d_tokens: int = 0, d_count: int = 0) -> None:
    _check(_lib.mtp_decode_step_async(ctx, K, top_k, ctypes.c_void_p(d_tokens or None),
                                      ctypes.c_void_p(d_count or None)), ctx, "mtp_decode_step_async")


def mtp_get_logits(ctx, B: int, K: int, V: int) -> np.ndarray:
    out = np.zeros((B, K, V), np.float32)
    _check(_lib.mtp_get_logits(ctx, out.ctypes.data_as(_f32p)), ctx, "mtp_get_logits")
    return out


def mtp_set_selection(ctx, lattice: int, anchored: bool) -> None:
    _check(_lib.mtp_set_selection(ctx, lattice, int(anchored)), ctx, "mtp_set_selection")


def mtp_set_sampling(ctx, mode: int, temperature: float = 1.0, seed: int = 0) -> None:
    _check(_lib.mtp_set_sampling(ctx, mode, temperature, seed & ((1 << 64) - 1)), ctx, "mtp_set_sampling")


def mtp_get_uniforms(ctx, B: int, K: int) -> np.ndarray:
    u = np.zeros((B, 8), np.float32)
    _check(_lib.mtp_get_uniforms(ctx, u.ctypes.data_as(_f32p)), ctx, "mtp_get_uniforms")
    return u[:, :K]


def mtp_get_union_lattice(ctx, B: int, K: int) -> Dict[str, np.ndarray]:
    m = np.zeros(B, np.int32)
    states = np.zeros((B, 64), np.int32)
    ehat = np.zeros((B, 8, 64), np.float32)
    delta = np.zeros((B, 8, 64), np.float32)
    psi = np.zeros((B, 8, 64), np.int32)
    slots = np.zeros((B, K), np.int32)
    _check(_lib.mtp_get_union_lattice(ctx, m.ctypes.data_as(_i32p), states.ctypes.data_as(_i32p),
                                      ehat.ctypes.data_as(_f32p), delta.ctypes.data_as(_f32p),
                                      psi.ctypes.data_as(_i32p), slots.ctypes.data_as(_i32p)),
           ctx, "mtp_get_union_lattice")
    return {"m": m, "states": states, "ehat": ehat[:, :K], "delta": delta[:, :K], "psi": psi[:, :K], "slots": slots}


def mtp_get_lattice(ctx, B: int, K: int, top_k: int) -> Dict[str, np.ndarray]:
    cand = np.zeros((B, K, top_k), np.int32)
    ehat = np.zeros((B, K, top_k), np.float32)
    delta = np.zeros((B, K, top_k), np.float32)
    psi = np.zeros((B, K, top_k), np.int32)
    slots = np.zeros((B, K), np.int32)
    _check(_lib.mtp_get_lattice(ctx, cand.ctypes.data_as(_i32p), ehat.ctypes.data_as(_f32p),
                                delta.ctypes.data_as(_f32p), psi.ctypes.data_as(_i32p),
                                slots.ctypes.data_as(_i32p)), ctx, "mtp_get_lattice")
    return dict(cand=cand, ehat=ehat, delta=delta, psi=psi, slots=slots)


def mtp_get_seq_state(ctx, B: int) -> Dict[str, np.ndarray]:
    a = [np.zeros(B, np.int32) for _ in range(4)]
    _check(_lib.mtp_get_seq_state(ctx, *[x.ctypes.data_as(_i32p) for x in a]), ctx, "mtp_get_seq_state")
    return dict(ctx_len=a[0], pend_len=a[1], gen=a[2], done=a[3])


def mtp_get_tokens(ctx, B: int, max_new: int) -> np.ndarray:
    out = np.zeros((B, max_new), np.int32)
    _check(_lib.mtp_get_tokens(ctx, out.ctypes.data_as(_i32p)), ctx, "mtp_get_tokens")
    return out


def mtp_profile_replay(ctx, kclass: int, iters: int, flush_buf: int = 0, flush_bytes: int = 0) -> float:
    """flush_buf: device pointer (integer) of the caller's eviction buffer, 0 for cache-warm passes."""
    us = ctypes.c_double()
    _check(_lib.mtp_profile_replay(ctx, kclass, iters, ctypes.c_void_p(flush_buf or None), flush_bytes,
                                   ctypes.byref(us)), ctx, "mtp_profile_replay")
    return us.value


def mtp_force_tokens(ctx, tokens: np.ndarray, count: Sequence[int]) -> None:
    """tokens: [B, K] of the last step (row b's first count[b] entries used)."""
    tk, tkp = _i32(tokens)
    cn, cnp = _i32(count)
    _check(_lib.mtp_force_tokens(ctx, tkp, cnp), ctx, "mtp_force_tokens")


def mtp_q_workspace_size(n_tokens: int, n_seqs: int, vocab: int) -> int:
    out = ctypes.c_uint64()
    _check(_lib.mtp_q_workspace_size(n_tokens, n_seqs, vocab, ctypes.byref(out)), None, "mtp_q_workspace_size")
    return out.value


def mtp_q_count(tokens: int, n_tokens: int, offsets: int, n_seqs: int, vocab: int, eos_id: int, flags: int,
                counts: int, status: int, workspace: int, ws_bytes: int, stream: int) -> None:
    """Device pointers as integers; see include/mtp.h."""
    _check(_lib.mtp_q_count(ctypes.c_void_p(tokens or None), n_tokens, ctypes.c_void_p(offsets or None), n_seqs,
                            vocab, eos_id, flags, ctypes.c_void_p(counts or None), ctypes.c_void_p(status or None),
                            ctypes.c_void_p(workspace or None), ws_bytes, ctypes.c_void_p(stream or None)),
           None, "mtp_q_count")


def mtp_q_count_noalloc(tokens: int, n_tokens: int, offsets: int, n_seqs: int, vocab: int, eos_id: int, flags: int,
                        counts: int, status: int, stream: int) -> None:
    """mtp_q_count on the library's fixed scratch (no workspace); device pointers as integers."""
    _check(_lib.mtp_q_count_noalloc(ctypes.c_void_p(tokens or None), n_tokens, ctypes.c_void_p(offsets or None),
                                    n_seqs, vocab, eos_id, flags, ctypes.c_void_p(counts or None),
                                    ctypes.c_void_p(status or None), ctypes.c_void_p(stream or None)),
           None, "mtp_q_count_noalloc")


def mtp_q_normalize(counts: int, vocab: int, alpha: float, logq: int, stream: int) -> None:
    _check(_lib.mtp_q_normalize(ctypes.c_void_p(counts or None), vocab, alpha, ctypes.c_void_p(logq or None),
                                ctypes.c_void_p(stream or None)), None, "mtp_q_normalize")


def estimate_logq(tokens, offsets, vocab: int, eos_id: int, count_eos: bool, alpha: float, stream=None):
    """Counts and log Q of a corpus held in device tensors (int32 tokens,
    int64 offsets [n_seqs + 1]).  Allocates the outputs with torch and runs
    mtp_q_count and mtp_q_normalize on `stream` (default: torch's current
    stream).  Returns (counts as int32 bits of the uint32 counts [V, V],
    log Q float32 [V, V], status int64 [3])."""
    import torch
    dev = tokens.device
    assert tokens.dtype == torch.int32 and offsets.dtype == torch.int64 and tokens.is_cuda and offsets.is_cuda
    st = stream if stream is not None else torch.cuda.current_stream(dev)
    counts = torch.empty((vocab, vocab), dtype=torch.int32, device=dev)
    logq = torch.empty((vocab, vocab), dtype=torch.float32, device=dev)
    status = torch.empty(3, dtype=torch.int64, device=dev)
    n_seqs = offsets.numel() - 1
    ws_bytes = mtp_q_workspace_size(tokens.numel(), n_seqs, vocab)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    with torch.cuda.stream(st):
        counts.zero_()
        status.zero_()
    mtp_q_count(tokens.data_ptr(), tokens.numel(), offsets.data_ptr(), n_seqs, vocab, eos_id,
                MTP_Q_COUNT_EOS if count_eos else 0, counts.data_ptr(), status.data_ptr(), ws.data_ptr(), ws_bytes,
                st.cuda_stream)
    mtp_q_normalize(counts.data_ptr(), vocab, alpha, logq.data_ptr(), st.cuda_stream)
    ws.record_stream(st)
    return counts, logq, status


def mtp_reset(ctx) -> None:
    _check(_lib.mtp_reset(ctx), ctx, "mtp_reset")


def mtp_destroy(ctx) -> None:
    _lib.mtp_destroy(ctx)


def mtp_last_error(ctx) -> str:
    return _lib.mtp_last_error(ctx).decode()


def mtp_strerror(code: int) -> str:
    return _lib.mtp_strerror(code).decode()


# --------------------------------------------------------------- convenience
def make_config(shape, max_batch: int, max_prompt: int, max_new: int, eos_min: int, topk_max: int = 32,
                page_size: int = 16, num_pages: int = 0, flags: int = 0) -> mtp_config:
    return mtp_config(
        n_layers=shape.n_layers, d_model=shape.d_model, n_heads=shape.n_heads, d_ff=shape.d_ff,
        vocab=shape.vocab, eos_id=shape.eos_id, n_phone=shape.n_phone, max_pos=shape.max_pos,
        k_heads=shape.k_heads, topk_max=topk_max, max_batch=max_batch, max_prompt=max_prompt,
        max_new=max_new, eos_min=eos_min, page_size=page_size, num_pages=num_pages,
        dtype=MTP_DTYPE_BF16 if shape.dtype == "bf16" else MTP_DTYPE_F32,
        flags=flags | (MTP_FLAG_NAR if getattr(shape, "nar", False) else 0))


_TENSOR_OF = {"emb_phone": MTP_T_EMB_PHONE, "emb_ac": MTP_T_EMB_AC, "emb_codes": MTP_T_EMB_AC, "pos": MTP_T_POS,
              "lnf_g": MTP_T_LNF_G, "lnf_b": MTP_T_LNF_B, "w_heads": MTP_T_W_HEADS, "b_heads": MTP_T_B_HEADS,
              "stage": MTP_T_STAGE}
_LAYER_TENSOR_OF = {"ln1_g": MTP_T_LN1_G, "ln1_b": MTP_T_LN1_B, "w_qkv": MTP_T_W_QKV, "b_qkv": MTP_T_B_QKV,
                    "w_o": MTP_T_W_O, "b_o": MTP_T_B_O, "ln2_g": MTP_T_LN2_G, "ln2_b": MTP_T_LN2_B,
                    "w_1": MTP_T_W_1, "b_1": MTP_T_B_1, "w_2": MTP_T_W_2, "b_2": MTP_T_B_2}
_MATRICES = {MTP_T_EMB_PHONE, MTP_T_EMB_AC, MTP_T_POS, MTP_T_W_QKV, MTP_T_W_O, MTP_T_W_1, MTP_T_W_2, MTP_T_W_HEADS}


_TILED = {MTP_T_W_QKV, MTP_T_W_O, MTP_T_W_1, MTP_T_W_2, MTP_T_W_HEADS}


def tile_bf16_matrix(w: np.ndarray) -> np.ndarray:
    """[N][K] matrix (any dtype) -> flat MFMA fragment order of mtp.h: rows
    padded to a multiple of 16, then per (16-row block, 32-column block) a
    fragment whose slot 16 g + r holds row r, columns 8 g .. 8 g + 7."""
    n, k = w.shape
    assert k % 32 == 0, k
    npad = (n + 15) // 16 * 16
    p = np.zeros((npad, k), w.dtype)
    p[:n] = w
    return np.ascontiguousarray(p.reshape(npad // 16, 16, k // 32, 4, 8).transpose(0, 2, 3, 1, 4)).reshape(-1)


def pack_weights(cfg: mtp_config, weights: Dict[str, np.ndarray]) -> np.ndarray:
    """Host image of the packed weights buffer (uint8) in the library's layout."""
    total = mtp_query_sizes(cfg).weights_bytes
    img = np.zeros(total, np.uint8)
    for name, arr in weights.items():
        if name.startswith("l") and "." in name:
            l, short = name.split(".", 1)
            t, layer = _LAYER_TENSOR_OF[short], int(l[1:])
        else:
            t, layer = _TENSOR_OF[name], 0
        off, n = mtp_weight_offset(cfg, t, layer)
        a = np.ascontiguousarray(arr, dtype=np.float32).reshape(-1)
        assert a.size == n, (name, a.size, n)
        if t in _MATRICES and cfg.dtype == MTP_DTYPE_BF16:
            raw = (a.view(np.uint32) >> 16).astype(np.uint16)
            assert np.array_equal((raw.astype(np.uint32) << 16).view(np.float32), a), f"{name} is not bf16-exact"
            if t in _TILED:
                k = cfg.d_ff if t == MTP_T_W_2 else cfg.d_model
                raw = tile_bf16_matrix(raw.reshape(-1, k))
            img[off:off + 2 * raw.size] = raw.view(np.uint8)
        else:
            img[off:off + 4 * n] = a.view(np.uint8)
    return img


class Session:
    """Owns the torch device buffers of one context and its stream."""

    def __init__(self, shape, weights: Dict[str, np.ndarray], logq: np.ndarray, max_batch: int,
                 max_prompt: int, max_new: int, eos_min: int, topk_max: int = 32, page_size: int = 16,
                 num_pages: int = 0, flags: int = 0, device: str = "cuda:0", stream=None):
        import torch
        self.torch = torch
        self.shape = shape
        self.cfg = make_config(shape, max_batch, max_prompt, max_new, eos_min, topk_max, page_size, num_pages, flags)
        sz = mtp_query_sizes(self.cfg)
        self.sizes = sz
        self.device = torch.device(device)
        self.weights_dev = torch.from_numpy(pack_weights(self.cfg, weights)).to(self.device)
        self.logq_dev = torch.from_numpy(np.ascontiguousarray(logq, dtype=np.float32)).to(self.device)
        self.kv = torch.empty(int(sz.kv_bytes), dtype=torch.uint8, device=self.device)
        self.ws = torch.empty(int(sz.workspace_bytes), dtype=torch.uint8, device=self.device)
        self.stream = stream if stream is not None else torch.cuda.Stream(device=self.device)
        torch.cuda.synchronize(self.device)
        bufs = mtp_buffers(self.weights_dev.data_ptr(), self.logq_dev.data_ptr(), self.kv.data_ptr(),
                           self.ws.data_ptr())
        self.ctx = mtp_create(self.cfg, bufs, self.stream.cuda_stream)
        self.B = 0

    def prefill(self, phon: Sequence[np.ndarray], ac: Sequence[np.ndarray]) -> None:
        mtp_prefill(self.ctx, phon, ac)
        self.B = len(ac)

    def step(self, K: int, top_k: int) -> Tuple[np.ndarray, np.ndarray]:
        return mtp_decode_step(self.ctx, self.B, K, top_k)

    def step_async(self, K: int, top_k: int) -> None:
        mtp_decode_step_async(self.ctx, K, top_k)

    def logits(self, K: int) -> np.ndarray:
        return mtp_get_logits(self.ctx, self.B, K, self.cfg.vocab)

    def lattice(self, K: int, top_k: int) -> Dict[str, np.ndarray]:
        return mtp_get_lattice(self.ctx, self.B, K, top_k)

    def force(self, tokens: np.ndarray, count: Sequence[int]) -> None:
        mtp_force_tokens(self.ctx, tokens, count)

    FLUSH_BYTES = 512 << 20

    def replay(self, kclass: int, iters: int, cold: bool = True) -> float:
        """Average launch time of one kernel class of the last step (us); cold
        passes read a 512 MiB buffer of this session first (evicting L2 and
        the last-level cache)."""
        if not cold:
            return mtp_profile_replay(self.ctx, kclass, iters)
        if getattr(self, "flush", None) is None:
            self.flush = self.torch.empty(self.FLUSH_BYTES, dtype=self.torch.uint8, device=self.device)
        return mtp_profile_replay(self.ctx, kclass, iters, self.flush.data_ptr(), self.FLUSH_BYTES)

    def set_selection(self, lattice: int = MTP_LATTICE_OWN, anchored: bool = False) -> None:
        mtp_set_selection(self.ctx, lattice, anchored)

    def union_lattice(self, K: int) -> Dict[str, np.ndarray]:
        return mtp_get_union_lattice(self.ctx, self.B, K)

    def set_sampling(self, mode: int, temperature: float = 1.0, seed: int = 0) -> None:
        mtp_set_sampling(self.ctx, mode, temperature, seed)

    def uniforms(self, K: int) -> np.ndarray:
        return mtp_get_uniforms(self.ctx, self.B, K)

    def seq_state(self) -> Dict[str, np.ndarray]:
        return mtp_get_seq_state(self.ctx, self.B)

    def tokens(self) -> np.ndarray:
        return mtp_get_tokens(self.ctx, self.B, self.cfg.max_new)

    def close(self) -> None:
        if getattr(self, "ctx", None):
            mtp_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class NarSession:
    """Device buffers, stream and context of one NAR module (MTP_FLAG_NAR)."""

    def __init__(self, shape, weights: Dict[str, np.ndarray], max_batch: int, max_seq: int, page_size: int = 16,
                 flags: int = 0, device: str = "cuda:0", stream=None):
        import torch
        assert shape.nar
        self.torch = torch
        self.shape = shape
        self.cfg = make_config(shape, max_batch, max_seq, 1, 1, 1, page_size, 0, flags)
        sz = mtp_query_sizes(self.cfg)
        self.sizes = sz
        self.device = torch.device(device)
        self.weights_dev = torch.from_numpy(pack_weights(self.cfg, weights)).to(self.device)
        self.kv = torch.empty(int(sz.kv_bytes), dtype=torch.uint8, device=self.device)
        self.ws = torch.empty(int(sz.workspace_bytes), dtype=torch.uint8, device=self.device)
        self.stream = stream if stream is not None else torch.cuda.Stream(device=self.device)
        torch.cuda.synchronize(self.device)
        bufs = mtp_buffers(self.weights_dev.data_ptr(), None, self.kv.data_ptr(), self.ws.data_ptr())
        self.ctx = mtp_create(self.cfg, bufs, self.stream.cuda_stream)
        self.tlens: List[int] = []

    def prepare(self, phon, prompt, a1) -> None:
        mtp_nar_prepare(self.ctx, phon, prompt, a1)
        self.tlens = [len(a) for a in a1]

    def run(self) -> None:
        mtp_nar_run(self.ctx)

    def codes(self) -> List[np.ndarray]:
        return mtp_nar_get_codes(self.ctx, self.cfg.k_heads, self.tlens)

    def logits(self, stage: int) -> np.ndarray:
        return mtp_nar_get_logits(self.ctx, stage, int(sum(self.tlens)), self.cfg.vocab - 1)

    def close(self) -> None:
        if getattr(self, "ctx", None):
            mtp_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
