"""Oracle AR decoder (theta_AR) with n next-token heads, in float64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Paper Sec. 3.1 / Eq. 1: a decoder-only Transformer is trained on one sequence
that concatenates the phoneme prompt p, the acoustic prompt (first-quantizer
codec tokens of the reference audio) and the generated tokens, with no
separator tokens.  Sec. 3.2: the trunk encodes the prefix into a latent z and
n distinct heads map the latent at the last position to the distributions of
the next n tokens.

The paper does not state the block internals.  The readings used here:
  * pre-LayerNorm blocks, LN epsilon 1e-5;
  * multi-head causal self-attention, head dimension 64, scale 1/sqrt(64);
  * FFN with exact (erf) GELU;
  * learned absolute position table, one running position index over the
    whole concatenated sequence; phoneme positions use the phoneme
    embedding table, every other position the codec-token table;
  * final LayerNorm, then head i is one Linear d_model -> vocab with bias.

Everything is computed in float64 from the given weights.  With
`emulate_bf16=True` the GEMM inputs and the cached keys/values are rounded to
bfloat16 at the points where a bf16 GPU kernel stores them; this is optional
and only narrows the comparison, it is not part of the method.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np
import torch
from scipy.special import erf

LN_EPS = 1e-5


def _bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even), returned as float64."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint32) << 16
    return r.view(np.float32).reshape(f.shape).astype(np.float64)


def layer_norm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float = LN_EPS) -> np.ndarray:
    """LayerNorm over the last axis with biased variance."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def gelu(x: np.ndarray) -> np.ndarray:
    """Exact GELU: x * Phi(x) with the normal CDF written through erf."""
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def softmax(x: np.ndarray, axis: int = -1) -> np.ndarray:
    m = np.max(x, axis=axis, keepdims=True)
    e = np.exp(x - m)
    return e / e.sum(axis=axis, keepdims=True)


@dataclass
class KVCache:
    """Append-only per-layer key/value rows of one sequence ([T, d_model] each)."""
    k: List[np.ndarray]
    v: List[np.ndarray]

    @property
    def length(self) -> int:
        return self.k[0].shape[0]


class ARDecoder:
    """theta_AR plus the n prediction heads, float64."""

    def __init__(self, shape, weights: Dict[str, np.ndarray], emulate_bf16: bool = False):
        self.shape = shape
        self.w = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
        self.emulate = emulate_bf16
        self.L = shape.n_layers
        self.d = shape.d_model
        self.H = shape.n_heads
        self.hd = self.d // self.H

    # -- rounding points of a bf16 kernel (identity unless emulating) --------
    def _r(self, x: np.ndarray) -> np.ndarray:
        return _bf16(x) if self.emulate else x

    def new_cache(self) -> KVCache:
        z = np.zeros((0, self.d))
        return KVCache([z.copy() for _ in range(self.L)], [z.copy() for _ in range(self.L)])

    def embed(self, ids: np.ndarray, positions: np.ndarray, phon_len: int) -> np.ndarray:
        """Token embedding plus position embedding.

        Positions below `phon_len` hold phoneme ids and use the phoneme table;
        the rest hold codec ids and use the codec table.
        """
        out = np.empty((len(ids), self.d))
        for r, (tok, pos) in enumerate(zip(ids, positions)):
            table = self.w["emb_phone"] if pos < phon_len else self.w["emb_ac"]
            out[r] = table[int(tok)] + self.w["pos"][int(pos)]
        return out

    def attention(self, q: np.ndarray, k_all: np.ndarray, v_all: np.ndarray, q_pos: np.ndarray,
                  rows_per_block: int = 256) -> np.ndarray:
        """Causal multi-head attention of the query rows over cached rows.

        q: [n, d]; k_all, v_all: [T, d] with row index = absolute position;
        query r at position q_pos[r] sees keys 0..q_pos[r].  Per head h the
        textbook form softmax(Q_h K_h^T / sqrt(64) + M) V_h, with M = -inf
        where the key's position exceeds the query's.  Query rows are taken
        `rows_per_block` at a time only to bound the size of the score
        matrix; each row's result does not depend on the blocking.  A few
        query rows (a decode chunk) are evaluated with numpy, many (a prompt
        or a full recompute) with float64 PyTorch CPU operations, which run
        the large score matrices multi-threaded; both evaluate the same
        formula in float64.
        """
        q_pos = np.asarray(q_pos, dtype=np.int64)
        if q.shape[0] <= 64:
            return self._attention_np(q, k_all, v_all, q_pos)
        return self._attention_torch(q, k_all, v_all, q_pos, rows_per_block)

    def _attention_np(self, q, k_all, v_all, q_pos):
        n = q.shape[0]
        out = np.zeros((n, self.d))
        scale = 1.0 / np.sqrt(self.hd)
        T = int(q_pos.max()) + 1
        visible = np.arange(T)[None, :] <= q_pos[:, None]
        for h in range(self.H):
            sl = slice(h * self.hd, (h + 1) * self.hd)
            s = np.where(visible, (q[:, sl] @ k_all[:T, sl].T) * scale, -np.inf)
            out[:, sl] = softmax(s, axis=-1) @ v_all[:T, sl]
        return out

    def _attention_torch(self, q, k_all, v_all, q_pos, rows_per_block):
        n = q.shape[0]
        out = torch.zeros((n, self.d), dtype=torch.float64)
        scale = 1.0 / np.sqrt(self.hd)
        qt = torch.from_numpy(np.ascontiguousarray(q, dtype=np.float64))
        kt = torch.from_numpy(np.ascontiguousarray(k_all, dtype=np.float64))
        vt = torch.from_numpy(np.ascontiguousarray(v_all, dtype=np.float64))
        qp = torch.as_tensor(q_pos)
        kp = torch.arange(kt.shape[0])
        for h in range(self.H):
            sl = slice(h * self.hd, (h + 1) * self.hd)
            k_h, v_h = kt[:, sl].contiguous(), vt[:, sl].contiguous()
            for r0 in range(0, n, rows_per_block):
                r1 = min(n, r0 + rows_per_block)
                T = int(qp[r0:r1].max()) + 1            # keys any row of the block can see
                s = (qt[r0:r1, sl] @ k_h[:T].T) * scale
                s = s.masked_fill(kp[None, :T] > qp[r0:r1, None], float("-inf"))
                out[r0:r1, sl] = torch.softmax(s, dim=-1) @ v_h[:T]
        return out.numpy()

    def forward(self, cache: KVCache, ids: np.ndarray, phon_len: int) -> np.ndarray:
        """Run the trunk over new tokens appended after the cached prefix.

        Returns the final residual-stream rows h [n, d] (before the final LN)
        and extends `cache` by n positions.
        """
        ids = np.asarray(ids)
        start = cache.length
        pos = np.arange(start, start + len(ids))
        h = self.embed(ids, pos, phon_len)
        for l in range(self.L):
            p = f"l{l}."
            u = self._r(layer_norm(h, self.w[p + "ln1_g"], self.w[p + "ln1_b"]))
            qkv = u @ self.w[p + "w_qkv"].T + self.w[p + "b_qkv"]
            q, k, v = qkv[:, :self.d], qkv[:, self.d:2 * self.d], qkv[:, 2 * self.d:]
            cache.k[l] = np.concatenate([cache.k[l], self._r(k)], axis=0)
            cache.v[l] = np.concatenate([cache.v[l], self._r(v)], axis=0)
            a = self._r(self.attention(q, cache.k[l], cache.v[l], pos))
            h = h + a @ self.w[p + "w_o"].T + self.w[p + "b_o"]
            u2 = self._r(layer_norm(h, self.w[p + "ln2_g"], self.w[p + "ln2_b"]))
            f = self._r(gelu(u2 @ self.w[p + "w_1"].T + self.w[p + "b_1"]))
            h = h + f @ self.w[p + "w_2"].T + self.w[p + "b_2"]
        return h

    def heads(self, h_last: np.ndarray, n: int) -> np.ndarray:
        """Logits of the first n heads on the last position's latent.

        z = LN_f(h_last); head i gives W_i z + b_i, the scores of token
        t+1+i (Sec. 3.2).  Returns float64 [n, vocab].
        """
        z = self._r(layer_norm(h_last, self.w["lnf_g"], self.w["lnf_b"]))
        W = self.w["w_heads"][:n]
        b = self.w["b_heads"][:n]
        return np.einsum("ivd,d->iv", W, z) + b
