"""Oracle AR loop with multi-token prediction and Viterbi selection.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Paper Fig. 1(b) and Sec. 3.2: each inference step encodes the prefix, the n
heads predict the next n tokens, the selected tokens are appended to the
input of the next step; the number of AR steps drops from L to about L/n.
Sec. 3.3 / Fig. 2: the n tokens come from the Viterbi selection over each
head's top_k candidates.

One sequence at a time (sequences are independent).  The trunk runs in
float64; logits are rounded to float32 and every decision is taken in
float32 (selection.py).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

from .decoder import ARDecoder
from .selection import Lattice, accept, path_margin, select, topk_boundary_gap


@dataclass
class StepRecord:
    gen_before: int
    logits: np.ndarray          # float32 [K, V] (unmasked)
    lattice: Lattice
    count: int
    done: bool
    emitted: np.ndarray         # int32 tokens actually emitted this step


@dataclass
class SequenceRun:
    tokens: List[int] = field(default_factory=list)
    steps: List[StepRecord] = field(default_factory=list)


class Generator:
    """Drives one sequence: prefill, then decode steps of K heads each."""

    def __init__(self, model: ARDecoder, logq: np.ndarray, eos_min: int, max_new: int):
        self.m = model
        self.logq = np.asarray(logq, dtype=np.float32)
        self.eos_min = eos_min
        self.max_new = max_new
        self.eos = model.shape.eos_id

    def prefill(self, phon: np.ndarray, ac: np.ndarray):
        self.cache = self.m.new_cache()
        self.phon_len = len(phon)
        ids = np.concatenate([np.asarray(phon, np.int64), np.asarray(ac, np.int64)])
        h = self.m.forward(self.cache, ids, self.phon_len)
        self.h_last = h[-1]
        self.pending: List[int] = []
        self.gen = 0
        self.done = False
        self.run = SequenceRun()

    def step(self, K: int, top_k: int, force: Optional[Sequence[int]] = None,
             force_count: Optional[int] = None) -> StepRecord:
        """One decode step.  With `force`, the emitted tokens/count are the
        caller's (teacher forcing) instead of the oracle's own selection."""
        assert not self.done
        if self.pending:
            h = self.m.forward(self.cache, np.asarray(self.pending, np.int64), self.phon_len)
            self.h_last = h[-1]
        logits = self.m.heads(self.h_last, K).astype(np.float32)
        lat = select(logits, self.logq, top_k, self.gen, self.eos_min, self.eos)
        n, done = accept(lat.tokens, self.gen, self.max_new, self.eos)
        emitted = lat.tokens[:n].copy()
        if force is not None:
            emitted = np.asarray(force, dtype=np.int32)[:force_count].copy()
            n = int(force_count)
            done = (n > 0 and int(emitted[-1]) == self.eos) or self.gen + n >= self.max_new
        rec = StepRecord(self.gen, logits, lat, n, done, emitted)
        self.run.steps.append(rec)
        self.run.tokens.extend(int(x) for x in emitted)
        self.gen += n
        self.done = done
        self.pending = [] if done else [int(x) for x in emitted]
        return rec

    def margins(self, rec: StepRecord, top_k: int) -> float:
        """Smallest decision gap of a step: top_k boundary of every head (with
        its EOS mask) and best-vs-second path score.  float64."""
        from .selection import mask_eos
        gaps = [topk_boundary_gap(mask_eos(rec.logits[t], rec.gen_before + t, self.eos_min, self.eos), top_k)
                for t in range(rec.logits.shape[0])]
        gaps.append(path_margin(rec.lattice.cand, rec.lattice.ehat, self.logq))
        return float(min(gaps))


def generate(model: ARDecoder, logq: np.ndarray, phon: np.ndarray, ac: np.ndarray,
             K: int, top_k: int, max_new: int, eos_min: int, max_steps: Optional[int] = None) -> SequenceRun:
    """Free-running generation of one sequence."""
    g = Generator(model, logq, eos_min, max_new)
    g.prefill(phon, ac)
    steps = 0
    while not g.done and (max_steps is None or steps < max_steps):
        g.step(K, top_k)
        steps += 1
    return g.run
