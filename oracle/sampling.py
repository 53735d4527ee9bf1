"""Oracle of top_k sampling inside the lattice.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

The paper (Fig. 2 caption) keeps diversity by top_k sampling but gives no
procedure.  Reading taken here: instead of the single best path, the emitted
path is DRAWN from the distribution over the lattice's paths (each position's
own top_k, or the union of all heads' top_k, Sec. 3.3) in which a path has
weight

    prod_t exp(e_t(a_t) / tau) * prod_{t>=1} Q(a_{t-1}, a_t)
    [ * Q(a_prev, a_0) when the first position is anchored ],

e_t(c) = l_t[c] - max l_t the head's emission score (EOS masked to -inf while
its generated index is below eos_min) and tau the temperature.  With one head
this is ordinary top_k sampling at temperature tau; as tau -> 0 with a flat Q
it becomes the per-head argmax.  The draw is exact by forward filtering,
backward sampling:

  forward   alpha_0(j) = W_0(j) [* Q(a_prev, c_0j)],
            alpha_t(j) = W_t(j) * sum_i alpha_{t-1}(i) * Q(c_{t-1,i}, c_{t,j}),
            W_t(j) = exp(e_t(j) / tau), each alpha_t rescaled by a power of
            two so that its largest entry lies in [1/2, 1);
  backward  a_{K-1} ~ alpha_{K-1};  a_t ~ alpha_t(i) * Q(c_{t,i}, c_{t+1,a_{t+1}}).

A draw from weights w_0..w_{m-1} with a uniform u in [0, 1) takes the first j
whose running sum w_0 + .. + w_j exceeds u * (w_0 + .. + w_{m-1}).

Arithmetic, chosen so that any IEEE float32 implementation that follows it
reproduces every draw exactly: all of it is float32 with one rounding per
operation (no fused multiply-add), sums run in ascending state order, every
product is flushed to zero below 2^-100 (so no result depends on how
subnormals are handled), the rescaling is an exact power of two, and exp is
the float32 evaluation defined in `exp32`.

Uniforms: draw r of a step (r = 0 for the last position, r = K-1-t for
position t) of sequence b whose generated count before the step is g takes
64-bit word r % 4 of Philox4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC 2011) at counter (g, b, r // 4, 0)
with key (seed, 0); u = (word >> 40) * 2^-24.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

from .selection import emission, mask_eos, top_k, union_inputs

F32 = np.float32
_M64 = (1 << 64) - 1

# Philox4x64 round constants (SC 2011): the two multipliers and the Weyl
# increments of the key schedule (golden ratio and sqrt(3) - 1, 64-bit).
PHILOX_M = (0xD2E7470EE14C6C93, 0xCA5A826395121157)
PHILOX_W = (0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)

TINY = F32(2.0 ** -100)      # products below this are flushed to zero


def philox4x64_10(counter: Sequence[int], key: Sequence[int]) -> List[int]:
    """One Philox4x64 block, 10 rounds.  Each round multiplies words 0 and 2
    by the two multipliers (128-bit products split into hi and lo) and
    outputs (hi_1 ^ c_1 ^ k_0, lo_1, hi_0 ^ c_3 ^ k_1, lo_0); the key
    advances by the Weyl increments between rounds."""
    c = [int(x) & _M64 for x in counter]
    k0, k1 = int(key[0]) & _M64, int(key[1]) & _M64
    for _ in range(10):
        p0 = PHILOX_M[0] * c[0]
        p1 = PHILOX_M[1] * c[2]
        c = [(p1 >> 64) ^ c[1] ^ k0, p1 & _M64, (p0 >> 64) ^ c[3] ^ k1, p0 & _M64]
        k0 = (k0 + PHILOX_W[0]) & _M64
        k1 = (k1 + PHILOX_W[1]) & _M64
    return c


def uniform24(word: int) -> np.float32:
    """The top 24 bits of a 64-bit word as a float32 in [0, 1) (exact)."""
    return F32(int(word) >> 40) * F32(2.0 ** -24)


def step_uniforms(seed: int, seq: int, gen: int, K: int) -> np.ndarray:
    """The K uniforms of one step of sequence `seq` (draw order r = 0..K-1)."""
    out = np.zeros(K, dtype=np.float32)
    for r in range(K):
        out[r] = uniform24(philox4x64_10([gen, seq, r // 4, 0], [seed, 0])[r % 4])
    return out


# exp in float32: x = n ln2 + r with n = rint(x log2 e) and ln 2 split into a
# 16-significant-bit head (n * head exact for |n| < 128) and a tail, then the
# Taylor series of e^r to degree 7 by Horner (|r| <= ln2 / 2: truncation below
# 2^-27), then the exact scaling by 2^n.
_LN2 = math.log(2.0)
_LN2_HI = (np.array([_LN2], np.float32).view(np.uint32) & np.uint32(0xFFFFFF00)).view(np.float32)[0]
_LN2_LO = F32(_LN2 - float(_LN2_HI))
_LOG2E = F32(1.0 / _LN2)
_TAYLOR = [F32(1) / F32(math.factorial(n)) for n in range(8)]   # 1/n!, correctly rounded float32
EXP_MIN = F32(-64.0)          # exp32 returns 0 below this (e^-64 ~ 2^-92)


def exp32(x) -> np.float32:
    """e^x in float32 for x <= 0 by the evaluation above; 0 for x < -64 and
    for -inf."""
    x = F32(x)
    if not x >= EXP_MIN:
        return F32(0.0)
    n = np.rint(F32(x * _LOG2E))
    r = F32(F32(x - F32(n * _LN2_HI)) - F32(n * _LN2_LO))
    p = _TAYLOR[7]
    for c in _TAYLOR[6::-1]:
        p = F32(F32(p * r) + c)
    return F32(np.ldexp(p, int(n)))


def _flush(x: np.float32) -> np.float32:
    return x if x >= TINY else F32(0.0)


def _rescale(v: np.ndarray) -> np.ndarray:
    """Multiply by the power of two that puts max(v) in [1/2, 1) (exact), then flush."""
    mx = F32(np.max(v))
    if not mx > 0:
        return v
    e = int(np.frexp(mx)[1])
    return np.array([_flush(F32(np.ldexp(F32(x), -e))) for x in v], dtype=np.float32)


def draw(w: np.ndarray, u: np.float32) -> int:
    """Inverse-CDF draw: the first j whose running float32 sum exceeds
    u * total; if none does (u * total rounded up to the total), the last j
    of positive weight; slot 0 if every weight is 0."""
    total = F32(0.0)
    for x in w:
        total = F32(total + F32(x))
    thr = F32(F32(u) * total)
    run = F32(0.0)
    for j, x in enumerate(w):
        run = F32(run + F32(x))
        if run > thr:
            return j
    pos = [j for j, x in enumerate(w) if x > 0]
    return pos[-1] if pos else 0


@dataclass
class SampledPath:
    cand: np.ndarray     # int32 [K, m]  state tokens per position
    ehat: np.ndarray     # float32 [K, m] emission scores
    alpha: np.ndarray    # float32 [K, m] rescaled forward weights
    u: np.ndarray        # float32 [K]   uniforms in draw order
    slots: np.ndarray    # int32 [K]
    tokens: np.ndarray   # int32 [K]


def ffbs(cand: np.ndarray, ehat: np.ndarray, logq: np.ndarray, inv_tau: np.float32, u: np.ndarray,
         anchor: Optional[int] = None) -> SampledPath:
    """Forward filtering, backward sampling over K positions x m states
    (arithmetic as in the module docstring).  inv_tau = float32(1 / tau)."""
    cand = np.asarray(cand, dtype=np.int32)
    ehat = np.asarray(ehat, dtype=np.float32)
    inv_tau = F32(inv_tau)
    K, m = cand.shape

    def G(t, i, j):       # Q between slot i of position t and slot j of position t + 1
        return exp32(logq[cand[t, i], cand[t + 1, j]])

    W = np.array([[exp32(F32(ehat[t, j] * inv_tau)) for j in range(m)] for t in range(K)], dtype=np.float32)
    alpha = np.zeros((K, m), dtype=np.float32)
    a0 = W[0].copy()
    if anchor is not None:
        a0 = np.array([_flush(F32(W[0, j] * exp32(logq[anchor, cand[0, j]]))) for j in range(m)], dtype=np.float32)
    alpha[0] = _rescale(a0)
    for t in range(1, K):
        row = np.zeros(m, dtype=np.float32)
        for j in range(m):
            s = F32(0.0)
            for i in range(m):
                s = F32(s + _flush(F32(alpha[t - 1, i] * G(t - 1, i, j))))
            row[j] = _flush(F32(W[t, j] * s))
        alpha[t] = _rescale(row)
    u = np.asarray(u, dtype=np.float32)
    slots = np.zeros(K, dtype=np.int32)
    slots[K - 1] = draw(alpha[K - 1], u[0])
    for t in range(K - 2, -1, -1):
        w = np.array([_flush(F32(alpha[t, i] * G(t, i, slots[t + 1]))) for i in range(m)], dtype=np.float32)
        slots[t] = draw(w, u[K - 1 - t])
    tokens = np.array([cand[t, slots[t]] for t in range(K)], dtype=np.int32)
    return SampledPath(cand, ehat, alpha, u, slots, tokens)


def select_sample(logits: np.ndarray, logq: np.ndarray, k: int, gen: int, eos_min: int, eos_id: int,
                  temperature: float, seed: int, seq: int, lattice: str = "own",
                  anchor: Optional[int] = None) -> SampledPath:
    """One step's sampled selection from the float32 logits of K heads:
    the lattice of `oracle.selection.select` (own or union states, EOS mask,
    anchor), uniforms of (seed, seq, gen), inv_tau = float32(1) / float32(tau)."""
    logits = np.asarray(logits, dtype=np.float32)
    K = logits.shape[0]
    if lattice == "union":
        cand, ehat = union_inputs(logits, k, gen, eos_min, eos_id)
    else:
        cand = np.zeros((K, k), dtype=np.int32)
        ehat = np.zeros((K, k), dtype=np.float32)
        for t in range(K):
            ids, vals = top_k(mask_eos(logits[t], gen + t, eos_min, eos_id), k)
            cand[t] = ids
            ehat[t] = emission(vals)
    inv_tau = F32(1.0) / F32(temperature)
    return ffbs(cand, ehat, logq, inv_tau, step_uniforms(seed, seq, gen, K), anchor)
