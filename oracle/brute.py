"""Exhaustive path search: the definition the Viterbi recursion must reproduce.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Paper Sec. 3.3: the emitted sequence is the path through the candidate
tokens that maximises the product over positions of Q(a_{t-1}, a_t) * S_t(a_t)
(no transition factor at the first position, see selection.py).  Here every
one of the k^K slot paths is scored directly, in float64, so a wrong index,
sign or dropped term in the recursion shows up as a different argmax.
"""
from __future__ import annotations

import itertools
from typing import List, Optional, Tuple

import numpy as np


def all_paths(K: int, k: int) -> np.ndarray:
    """Every slot path, [k^K, K] int64, in lexicographic order."""
    return np.array(list(itertools.product(range(k), repeat=K)), dtype=np.int64).reshape(-1, K)


def path_scores_log(cand: np.ndarray, ehat: np.ndarray, logq: np.ndarray,
                    anchor: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Log-domain score sum_t e_t(s_t) + sum_{t>=1} logQ(c_{t-1,s_{t-1}}, c_{t,s_t})
    (+ logQ(anchor, c_{0,s_0}) for an anchored first position), float64."""
    cand = np.asarray(cand)
    K, k = cand.shape
    P = all_paths(K, k)
    e = np.asarray(ehat, dtype=np.float64)
    lq = np.asarray(logq, dtype=np.float64)
    score = np.zeros(P.shape[0])
    if anchor is not None:
        score += lq[anchor, cand[0, P[:, 0]]]
    for t in range(K):
        score += e[t, P[:, t]]
        if t > 0:
            score += lq[cand[t - 1, P[:, t - 1]], cand[t, P[:, t]]]
    return P, score


def path_scores_product(cand: np.ndarray, probs: np.ndarray, q: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Probability-domain score prod_t S_t(c_t) * prod_{t>=1} Q(c_{t-1}, c_t) (float64).

    probs[t, j] = S_t of the token in slot j (the head's full-vocabulary
    softmax probability), q = the transition table itself.
    """
    cand = np.asarray(cand)
    K, k = cand.shape
    P = all_paths(K, k)
    S = np.asarray(probs, dtype=np.float64)
    Q = np.asarray(q, dtype=np.float64)
    score = np.ones(P.shape[0])
    for t in range(K):
        score *= S[t, P[:, t]]
        if t > 0:
            score *= Q[cand[t - 1, P[:, t - 1]], cand[t, P[:, t]]]
    return P, score


def best_paths(P: np.ndarray, score: np.ndarray) -> np.ndarray:
    """All slot paths attaining the maximal score exactly."""
    return P[score == score.max()]


def tie_rule_path(optimal: np.ndarray) -> np.ndarray:
    """Among optimal paths, the one with the smallest last slot, then the
    smallest second-to-last slot, and so on (lexicographic on the reversed
    path): what lowest-index tie-breaking in the recursion and backtrack yields."""
    rev = optimal[:, ::-1]
    order = np.lexsort(rev.T[::-1])
    return optimal[order[0]]


def path_weights(cand: np.ndarray, ehat: np.ndarray, logq: np.ndarray, tau: float,
                 anchor: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Normalised probability of every slot path under the sampling
    distribution prod_t exp(e_t / tau) * prod_{t>=1} Q(a_{t-1}, a_t)
    [* Q(anchor, a_0)], float64 with numpy's exp."""
    cand = np.asarray(cand)
    K, k = cand.shape
    P = all_paths(K, k)
    e = np.asarray(ehat, dtype=np.float64)
    lq = np.asarray(logq, dtype=np.float64)
    logw = np.zeros(P.shape[0])
    if anchor is not None:
        logw += lq[anchor, cand[0, P[:, 0]]]
    for t in range(K):
        logw += e[t, P[:, t]] / tau
        if t > 0:
            logw += lq[cand[t - 1, P[:, t - 1]], cand[t, P[:, t]]]
    w = np.exp(logw - logw.max())
    return P, w / w.sum()
