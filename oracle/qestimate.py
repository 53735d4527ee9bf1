"""Oracle of the transition-table estimation.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Sec. 3.3: Q(i, j) models how likely token a_i is immediately followed by
a_j, and Q is derived from the training data (Fig. 2 caption: computed for
LibriTTS in minutes).  The paper gives no estimator; reading taken here:

  counts   C[i][j] = the number of places where token i is immediately
           followed by token j inside one utterance (no pair spans two
           utterances); optionally the end of every non-empty utterance adds
           the pair (last token, EOS), so the EOS column carries the
           probability of stopping after a token;
  table    Q(i, j) = (C[i][j] + alpha) / (sum_j' C[i][j'] + alpha * V), the
           row-normalised counts with additive (Laplace) smoothing alpha >= 0,
           row = previous token; log Q rounded to float32.  A row with no
           counts and alpha = 0 is uniform.

Input checks: a pair with an id outside [0, V) is skipped and counted as a
bad pair; an utterance whose offsets are not 0 <= start <= end <= n_tokens is
skipped and counted as a bad sequence.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np


def bigram_pairs(tokens: np.ndarray, offsets: np.ndarray, eos_id: int, count_eos: bool):
    """Every (previous, next) pair of the corpus, utterance by utterance, and
    the number of utterances with bad offsets."""
    tokens = np.asarray(tokens, dtype=np.int64)
    offsets = np.asarray(offsets, dtype=np.int64)
    n = tokens.shape[0]
    xs, ys = [], []
    bad_seqs = 0
    for u in range(offsets.shape[0] - 1):
        s, e = int(offsets[u]), int(offsets[u + 1])
        if not (0 <= s <= e <= n):
            bad_seqs += 1
            continue
        xs.append(tokens[s:e - 1] if e > s else tokens[0:0])
        ys.append(tokens[s + 1:e])
        if count_eos and e > s:
            xs.append(tokens[e - 1:e])
            ys.append(np.array([eos_id], np.int64))
    x = np.concatenate(xs) if xs else np.zeros(0, np.int64)
    y = np.concatenate(ys) if ys else np.zeros(0, np.int64)
    return x, y, bad_seqs


def bigram_counts(tokens: np.ndarray, offsets: np.ndarray, vocab: int, eos_id: int,
                  count_eos: bool) -> Tuple[np.ndarray, int, int]:
    """C as uint32 [V][V] (row = previous token), the number of bad pairs and
    the number of bad utterances."""
    x, y, bad_seqs = bigram_pairs(tokens, offsets, eos_id, count_eos)
    ok = (x >= 0) & (x < vocab) & (y >= 0) & (y < vocab)
    key = x[ok] * vocab + y[ok]
    counts = np.bincount(key, minlength=vocab * vocab).astype(np.uint32).reshape(vocab, vocab)
    return counts, int((~ok).sum()), bad_seqs


def log_q(counts: np.ndarray, alpha: float) -> np.ndarray:
    """float32 log Q from uint32 counts: log(C + a) - log(row sum + a V) in
    float64, a = the float32 alpha; -log V for a row whose denominator is 0."""
    c = np.asarray(counts, dtype=np.float64)
    V = c.shape[1]
    a = float(np.float32(alpha))
    den = c.sum(axis=1, keepdims=True) + a * V
    with np.errstate(divide="ignore", invalid="ignore"):
        out = np.log(c + a) - np.log(den)
    empty = (den[:, 0] == 0)
    out[empty, :] = -np.log(float(V))
    return out.astype(np.float32)
