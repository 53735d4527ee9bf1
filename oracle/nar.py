"""Oracle NAR module (theta_NAR) for the codec layers 2..n_q, in float64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Paper Sec. 3.1 / Eq. 2: after the AR module has produced the first-layer
tokens a^1, a non-autoregressive LM predicts each further layer's whole token
sequence a^j (j = 2..8) in one pass, conditioned on the phonemes p, the
acoustic prompt (all its codec layers) and the already known layers a^{<j}.

The paper does not state the module's internals.  Readings used here:
  * the same pre-LN Transformer block as the AR module (decoder.py), but the
    self-attention is bidirectional: every position sees the whole
    sequence [p; prompt; target] of its utterance;
  * input of stage j at a position: the phoneme table for phoneme positions;
    for prompt positions the sum over all n_q layers of the layer's codebook
    table at the prompt's token; for target positions the sum over layers
    i < j of table i at a^i; plus the learned position (one running index)
    and a learned stage vector s_j added to every position;
  * output of stage j: final LayerNorm, then the stage's own Linear
    d_model -> codebook size with bias at the target positions; a^j is the
    argmax (lowest index on ties), i.e. greedy decoding.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .decoder import _bf16, gelu, layer_norm, softmax


class NARModel:
    """theta_NAR with one head and one stage vector per predicted layer."""

    def __init__(self, shape, weights: Dict[str, np.ndarray], emulate_bf16: bool = False):
        self.shape = shape
        self.w = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
        self.emulate = emulate_bf16
        self.L = shape.n_layers
        self.d = shape.d_model
        self.H = shape.n_heads
        self.hd = self.d // self.H
        self.n_stages = self.w["w_heads"].shape[0]          # predicted layers 2 .. n_stages + 1
        self.n_q = self.n_stages + 1

    def _r(self, x: np.ndarray) -> np.ndarray:
        return _bf16(x) if self.emulate else x

    def embed(self, j: int, phon: np.ndarray, prompt: np.ndarray, target: np.ndarray) -> np.ndarray:
        """Stage j input rows for [phon; prompt; target].

        prompt: [n_q, P] codes of every layer; target: [>= j-1, T] codes of
        layers 1..j-1 (rows beyond j-1 are ignored)."""
        phon = np.asarray(phon)
        prompt = np.asarray(prompt).reshape(self.n_q, -1)
        target = np.asarray(target)
        P, T = prompt.shape[1], target.shape[1]
        n = len(phon) + P + T
        E = self.w["emb_codes"]
        out = np.zeros((n, self.d))
        r = 0
        for tok in phon:
            out[r] = self.w["emb_phone"][int(tok)]
            r += 1
        for t in range(P):
            out[r] = sum(E[i][int(prompt[i, t])] for i in range(self.n_q))
            r += 1
        for t in range(T):
            out[r] = sum(E[i][int(target[i, t])] for i in range(j - 1))
            r += 1
        out += self.w["pos"][:n] + self.w["stage"][j - 2]
        return out

    def attention(self, q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
        """Bidirectional multi-head attention: every row sees every row."""
        out = np.zeros_like(q)
        scale = 1.0 / np.sqrt(self.hd)
        for h in range(self.H):
            sl = slice(h * self.hd, (h + 1) * self.hd)
            p = softmax((q[:, sl] @ k[:, sl].T) * scale, axis=-1)
            out[:, sl] = p @ v[:, sl]
        return out

    def forward(self, x: np.ndarray) -> np.ndarray:
        """The trunk over one utterance's rows; returns h before the final LN."""
        h = x
        for l in range(self.L):
            p = f"l{l}."
            u = self._r(layer_norm(h, self.w[p + "ln1_g"], self.w[p + "ln1_b"]))
            qkv = u @ self.w[p + "w_qkv"].T + self.w[p + "b_qkv"]
            q, k, v = qkv[:, :self.d], qkv[:, self.d:2 * self.d], qkv[:, 2 * self.d:]
            a = self._r(self.attention(q, self._r(k), self._r(v)))
            h = h + a @ self.w[p + "w_o"].T + self.w[p + "b_o"]
            u2 = self._r(layer_norm(h, self.w[p + "ln2_g"], self.w[p + "ln2_b"]))
            f = self._r(gelu(u2 @ self.w[p + "w_1"].T + self.w[p + "b_1"]))
            h = h + f @ self.w[p + "w_2"].T + self.w[p + "b_2"]
        return h

    def stage_logits(self, h_target: np.ndarray, j: int) -> np.ndarray:
        """Stage j's head on the final-LN target rows: [T, codebook]."""
        z = self._r(layer_norm(h_target, self.w["lnf_g"], self.w["lnf_b"]))
        return z @ self.w["w_heads"][j - 2].T + self.w["b_heads"][j - 2]

    def run(self, phon: Sequence[int], prompt: np.ndarray, a1: Sequence[int],
            teacher: Optional[np.ndarray] = None) -> Tuple[np.ndarray, List[np.ndarray]]:
        """All stages for one utterance.  Returns (codes [n_q, T] with layer 1
        = a1 and layers 2.. by argmax, the stage logits [T, codebook] each).
        With `teacher` ([n_q, T]), stage j reads layers 2..j-1 from it instead
        of its own argmax (to follow another implementation's choices)."""
        a1 = np.asarray(a1, dtype=np.int64)
        T = len(a1)
        codes = np.zeros((self.n_q, T), np.int64)
        codes[0] = a1
        logits = []
        n_pre = len(phon) + np.asarray(prompt).reshape(self.n_q, -1).shape[1]
        for j in range(2, self.n_q + 1):
            src = codes if teacher is None else np.vstack([codes[:1], np.asarray(teacher)[1:]])
            h = self.forward(self.embed(j, phon, prompt, src))
            lg = self.stage_logits(h[n_pre:], j)
            logits.append(lg)
            codes[j - 1] = np.argmax(lg, axis=1)
        return codes, logits
