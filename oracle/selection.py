"""Oracle selection: emission scores, per-head top_k, Viterbi, accept.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Paper Sec. 3.3: tokens follow a Markov chain with transition table Q, Q(i, j)
the probability that token a_i is immediately followed by a_j; head t gives
S_t(a), the probability of token a at time t.  Moving from a_i at t-1 to a_j
at t scores Q(a_i, a_j) * S_t(a_j), and the emitted sequence A* is the
best-scoring path.  Fig. 2 / Sec. 3.3: the search is restricted to each
head's top_k tokens, so every step uses small gathered sub-tables of Q
instead of the full |V| x |V| table.

Readings where the paper is silent (its Algorithm 1 body is not available):
  * max-product Viterbi in the log domain; the first position carries its
    emission only (no transition from the previously emitted token), so one
    head reduces to plain greedy AR decoding (Eq. 1);
  * states at position t are head t's own top_k tokens;
  * emission log S_t(c) is replaced by l_t[c] - max l_t.  The dropped
    log-sum-exp is the same for every path through position t, so the
    argmax path is unchanged, and the selection then needs only IEEE add,
    subtract and max, which the GPU reproduces bit for bit;
  * ties: top_k orders by (logit desc, token id asc); Viterbi keeps the
    lowest predecessor slot and the lowest final slot;
  * EOS (id 1024) is masked to -inf while its generated index is below
    `eos_min`; no verify/reject step exists, every selected token up to the
    budget and the first EOS is emitted.

All decisions are taken in float32 (numpy float32 scalars, never Python
floats), the precision the GPU kernels take them in.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np

F32 = np.float32


def mask_eos(logits: np.ndarray, gen_index: int, eos_min: int, eos_id: int) -> np.ndarray:
    """Copy of one head's float32 logits with EOS at -inf while gen_index < eos_min."""
    out = np.array(logits, dtype=np.float32, copy=True)
    if gen_index < eos_min:
        out[eos_id] = -np.inf
    return out


def top_k(logits: np.ndarray, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """The k largest logits of one head, ordered by (value desc, token id asc).

    Returns (token ids int32 [k], values float32 [k]).
    """
    logits = np.asarray(logits, dtype=np.float32)
    ids = np.arange(logits.shape[0])
    order = np.lexsort((ids, -logits.astype(np.float64)))[:k]
    return order.astype(np.int32), logits[order]


def emission(values: np.ndarray) -> np.ndarray:
    """e_hat(j) = l[c_j] - max l in float32; values are top_k-ordered so max = values[0]."""
    values = np.asarray(values, dtype=np.float32)
    top = values[0]
    return np.array([F32(v - top) for v in values], dtype=np.float32)


@dataclass
class Lattice:
    cand: np.ndarray    # int32 [K, k]  token id of slot j at position t
    ehat: np.ndarray    # float32 [K, k] emission score
    delta: np.ndarray   # float32 [K, k] best path score ending in (t, j)
    psi: np.ndarray     # int32 [K, k]  best predecessor slot (psi[0] = 0)
    slots: np.ndarray   # int32 [K]     chosen slot per position
    tokens: np.ndarray  # int32 [K]     chosen token per position


def viterbi(cand: np.ndarray, ehat: np.ndarray, logq: np.ndarray, anchor: Optional[int] = None) -> Lattice:
    """Max-product Viterbi over K positions x k candidate slots (log domain).

    delta_0(j) = e_0(j), or logQ(anchor, c_{0,j}) + e_0(j) when the first
    position is anchored to the previously emitted token `anchor`;
    delta_t(j) = max_i [delta_{t-1}(i) + logQ(c_{t-1,i}, c_{t,j})] + e_t(j),
    psi_t(j) = the maximising i (lowest on ties); the path ends in the lowest
    slot of maximal delta_{K-1} and is read back through psi.
    Every sum is a float32 add in exactly this association.
    """
    cand = np.asarray(cand, dtype=np.int32)
    ehat = np.asarray(ehat, dtype=np.float32)
    K, k = cand.shape
    delta = np.zeros((K, k), dtype=np.float32)
    psi = np.zeros((K, k), dtype=np.int32)
    for j in range(k):
        delta[0, j] = ehat[0, j] if anchor is None else F32(logq[anchor, cand[0, j]] + ehat[0, j])
    for t in range(1, K):
        for j in range(k):
            best = None
            arg = 0
            for i in range(k):
                s = F32(delta[t - 1, i] + logq[cand[t - 1, i], cand[t, j]])
                if best is None or s > best:
                    best, arg = s, i
            delta[t, j] = F32(best + ehat[t, j])
            psi[t, j] = arg
    last = 0
    for j in range(1, k):
        if delta[K - 1, j] > delta[K - 1, last]:
            last = j
    slots = np.zeros(K, dtype=np.int32)
    slots[K - 1] = last
    for t in range(K - 1, 0, -1):
        slots[t - 1] = psi[t, slots[t]]
    tokens = np.array([cand[t, slots[t]] for t in range(K)], dtype=np.int32)
    return Lattice(cand, ehat, delta, psi, slots, tokens)


def union_states(logits: np.ndarray, k: int, gen: int, eos_min: int, eos_id: int) -> np.ndarray:
    """The m <= K*k distinct tokens among the K heads' top_k (EOS-masked per
    head), in ascending token id: the reduced state space of Sec. 3.3, whose
    transition table is the m x m sub-table of Q."""
    logits = np.asarray(logits, dtype=np.float32)
    ids = [top_k(mask_eos(logits[t], gen + t, eos_min, eos_id), k)[0] for t in range(logits.shape[0])]
    return np.unique(np.concatenate(ids)).astype(np.int32)


def union_inputs(logits: np.ndarray, k: int, gen: int, eos_min: int, eos_id: int) -> Tuple[np.ndarray, np.ndarray]:
    """(cand, ehat) of the union lattice: every position has the same m states
    (union_states), and position t scores state c with head t's own
    distribution, e_t(c) = l_t[c] - max l_t (float32; -inf for a masked EOS)."""
    logits = np.asarray(logits, dtype=np.float32)
    K = logits.shape[0]
    U = union_states(logits, k, gen, eos_min, eos_id)
    cand = np.tile(U, (K, 1))
    ehat = np.zeros((K, U.size), dtype=np.float32)
    for t in range(K):
        lt = mask_eos(logits[t], gen + t, eos_min, eos_id)
        top = np.max(lt)
        ehat[t] = np.array([F32(lt[c] - top) for c in U], dtype=np.float32)
    return cand, ehat


def select(logits: np.ndarray, logq: np.ndarray, k: int, gen: int, eos_min: int, eos_id: int,
           lattice: str = "own", anchor: Optional[int] = None) -> Lattice:
    """One step's selection from the float32 logits of K heads ([K, V]).

    lattice="own": position t's states are head t's top_k (ordered by logit);
    lattice="union": every position's states are the union of all heads'
    top_k (ascending id), scored by head t at position t.  `anchor` (the last
    emitted token, or None) adds its transition into the first position.
    """
    logits = np.asarray(logits, dtype=np.float32)
    K = logits.shape[0]
    if lattice == "union":
        cand, ehat = union_inputs(logits, k, gen, eos_min, eos_id)
        return viterbi(cand, ehat, logq, anchor)
    cand = np.zeros((K, k), dtype=np.int32)
    ehat = np.zeros((K, k), dtype=np.float32)
    for t in range(K):
        ids, vals = top_k(mask_eos(logits[t], gen + t, eos_min, eos_id), k)
        cand[t] = ids
        ehat[t] = emission(vals)
    return viterbi(cand, ehat, logq, anchor)


def accept(tokens: np.ndarray, gen: int, max_new: int, eos_id: int) -> Tuple[int, bool]:
    """Number of selected tokens emitted this step and whether the sequence ends.

    count = min(K, max_new - gen); if EOS is at position p < count the step
    emits tokens 0..p (EOS included) and the sequence ends; it also ends when
    the budget is used up.
    """
    n = min(len(tokens), max_new - gen)
    done = False
    for p in range(n):
        if int(tokens[p]) == eos_id:
            n = p + 1
            done = True
            break
    if gen + n >= max_new:
        done = True
    return n, done


def topk_boundary_gap(logits: np.ndarray, k: int) -> float:
    """Gap between the k-th and (k+1)-th largest logit (float64); how far the
    candidate set is from changing."""
    s = np.sort(np.asarray(logits, dtype=np.float64))[::-1]
    s = s[np.isfinite(s)]
    return float(s[k - 1] - s[k]) if len(s) > k else float("inf")


def path_margin(cand: np.ndarray, ehat: np.ndarray, logq: np.ndarray) -> float:
    """Best minus second-best path score over all k^K slot paths (float64).

    Two-best list Viterbi: each state keeps its two best prefix scores.
    """
    cand = np.asarray(cand)
    e = np.asarray(ehat, dtype=np.float64)
    K, k = cand.shape
    if K == 1:
        s = np.sort(e[0])[::-1]
        return float(s[0] - s[1]) if k > 1 else float("inf")
    top = [[(e[0, j],) for j in range(k)]]
    for t in range(1, K):
        row = []
        for j in range(k):
            c = []
            for i in range(k):
                tr = float(logq[cand[t - 1, i], cand[t, j]])
                for s in top[t - 1][i]:
                    c.append(s + tr + e[t, j])
            c.sort(reverse=True)
            row.append(tuple(c[:2]))
        top.append(row)
    fin = sorted([s for st in top[K - 1] for s in st], reverse=True)
    return float(fin[0] - fin[1]) if len(fin) > 1 else float("inf")
