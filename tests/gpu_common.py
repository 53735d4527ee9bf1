"""Helpers shared by the GPU parity tests: build a HIP session and the oracle
on the same seeded inputs, and compare one decode step."""
from __future__ import annotations

import sys
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

from oracle.decoder import ARDecoder
from oracle.generate import Generator
from oracle.selection import select
from paper_2410_13839_amd.workloads import (Workload, make_logq, make_prompts, make_weights)


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def new_session(wl: Workload, weights, logq, batch: Optional[int] = None, flags: int = 0, topk_max: int = 32):
    from paper_2410_13839_amd.binding import Session
    B = wl.batch if batch is None else batch
    return Session(wl.model, weights, logq, max_batch=B, max_prompt=wl.max_prompt, max_new=wl.max_new,
                   eos_min=wl.eos_min, topk_max=topk_max, flags=flags)


def assert_selection_exact(gpu_logits: np.ndarray, lat: Dict[str, np.ndarray], logq: np.ndarray, top_k: int,
                           gen: np.ndarray, eos_min: int, eos_id: int, live: np.ndarray) -> None:
    """The oracle's selection applied to the GPU's own float32 logits must give
    the GPU's lattice bit for bit (candidates, emissions, Viterbi scores,
    back-pointers, slots)."""
    B, K, _ = gpu_logits.shape
    for b in range(B):
        if not live[b]:
            continue
        ref = select(gpu_logits[b], logq, top_k, int(gen[b]), eos_min, eos_id)
        ctx = f"seq {b}"
        assert np.array_equal(ref.cand, lat["cand"][b]), (ctx, ref.cand, lat["cand"][b])
        assert np.array_equal(ref.ehat.view(np.uint32), lat["ehat"][b].view(np.uint32)), ctx
        assert np.array_equal(ref.delta.view(np.uint32), lat["delta"][b].view(np.uint32)), (ctx, ref.delta, lat["delta"][b])
        assert np.array_equal(ref.psi[1:], lat["psi"][b][1:]), ctx
        assert np.array_equal(ref.slots, lat["slots"][b]), ctx


@dataclass
class OracleCheck:
    max_err: float = 0.0
    checked: int = 0
    tie_zone: int = 0
    mismatched: int = 0
    notes: List[str] = field(default_factory=list)


def oracle_logits_at(model: ARDecoder, phon: np.ndarray, ac: np.ndarray, emitted: List[int], K: int) -> np.ndarray:
    """Oracle head logits (float32 [K, V]) after the prompt and `emitted`."""
    ids = np.concatenate([np.asarray(phon, np.int64), np.asarray(ac, np.int64), np.asarray(emitted, np.int64)])
    h = model.forward(model.new_cache(), ids, len(phon))
    return model.heads(h[-1], K).astype(np.float32)
