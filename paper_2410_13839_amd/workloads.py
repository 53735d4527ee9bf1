"""Seeded synthetic workloads for the MTP + Viterbi decode path.

This module only *generates inputs*: model shapes, seeded weights, the
transition table Q and prompts.  It holds none of the method's arithmetic
(no forward pass, no scoring, no selection), so both the HIP path and the
CPU oracle can consume its arrays without sharing any computation.

Shapes follow a VALL-E style AR decoder: a decoder-only Transformer over the
concatenation [phonemes; acoustic prompt; generated codec tokens] (paper
Sec. 3.1, Eq. 1) with n parallel next-token heads on the last hidden state
(Sec. 3.2).  The codec vocabulary is 1024 first-quantizer codes plus EOS.

Seeding: every tensor is drawn from numpy's PCG64 seeded with
SeedSequence([seed, tensor_index]), N(0, 0.02) in float32.  For bf16 models
the float32 draw is rounded once to bf16 (round-to-nearest-even); both sides
use exactly those values.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

VOCAB = 1025          # 1024 first-quantizer codec codes + EOS
EOS_ID = 1024
N_PHONE = 512         # phoneme inventory (ids 0..511)
HEAD_DIM = 64
MAX_POS = 4096        # learned absolute position table length

DTYPE_F32 = "f32"
DTYPE_BF16 = "bf16"


@dataclass(frozen=True)
class ModelShape:
    """Decoder shape.  `k_heads` is the number of prediction heads loaded."""
    n_layers: int
    d_model: int
    n_heads: int
    d_ff: int
    k_heads: int
    dtype: str
    vocab: int = VOCAB
    eos_id: int = EOS_ID
    n_phone: int = N_PHONE
    max_pos: int = MAX_POS
    nar: bool = False    # NAR module: k_heads stages predict codec layers 2..k_heads+1

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    @property
    def codebook(self) -> int:
        """Codes per codec layer (the vocabulary without EOS)."""
        return self.vocab - 1


@dataclass(frozen=True)
class Workload:
    """One benchmark / parity configuration."""
    name: str
    model: ModelShape
    K: int                       # heads used per decode step (n in the paper)
    top_k: int                   # candidates kept per head
    batch: int
    phon_len: Tuple[int, int]    # inclusive range; (a, a) means fixed
    ac_len: Tuple[int, int]
    max_new: int                 # generation budget per sequence
    eos_min: int                 # EOS masked while generated index < eos_min
    description: str = ""

    @property
    def max_prompt(self) -> int:
        return self.phon_len[1] + self.ac_len[1]

    @property
    def max_seq(self) -> int:
        return self.max_prompt + self.max_new


_TINY = ModelShape(n_layers=2, d_model=256, n_heads=4, d_ff=1024, k_heads=2, dtype=DTYPE_F32)
_VALLE = ModelShape(n_layers=12, d_model=1024, n_heads=16, d_ff=4096, k_heads=8, dtype=DTYPE_BF16)
_LONG = ModelShape(n_layers=24, d_model=1536, n_heads=24, d_ff=6144, k_heads=4, dtype=DTYPE_BF16)

WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload(
        "tiny", _TINY, K=2, top_k=3, batch=1, phon_len=(0, 0), ac_len=(32, 32),
        max_new=64, eos_min=64,
        description="2L d256 H4 F1024 fp32, K=2 top_k=3, 32-token prompt, 64 tokens"),
    "valle_k4": Workload(
        "valle_k4", _VALLE, K=4, top_k=4, batch=1, phon_len=(100, 100), ac_len=(225, 225),
        max_new=750, eos_min=600,
        description="12L d1024 H16 F4096 bf16, K=4 top_k=4, batch 1, 100 phon + 225 acoustic, <=750 tokens, EOS from 600"),
    "valle_k8": Workload(
        "valle_k8", _VALLE, K=8, top_k=8, batch=1, phon_len=(100, 100), ac_len=(225, 225),
        max_new=750, eos_min=750,
        description="12L d1024 H16 F4096 bf16, K=8 top_k=8, batch 1, 750 tokens"),
    "valle_b32": Workload(
        "valle_b32", _VALLE, K=4, top_k=4, batch=32, phon_len=(50, 150), ac_len=(150, 300),
        max_new=750, eos_min=750,
        description="12L d1024 H16 F4096 bf16, K=4 top_k=4, batch 32 ragged prompts, 750 tokens each"),
    "long_b8": Workload(
        "long_b8", _LONG, K=4, top_k=4, batch=8, phon_len=(200, 200), ac_len=(450, 450),
        max_new=3000, eos_min=3000,
        description="24L d1536 H24 F6144 bf16, K=4 top_k=4, batch 8, 200 phon + 450 acoustic, 3000 tokens"),
}

WEIGHT_SEED = 0
Q_SEED = 1
PROMPT_SEED_BASE = 100


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return (rounded.astype(np.uint32) << 16).view(np.float32).reshape(x.shape)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) of float32 values that are already bf16-exact."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def weight_names(m: ModelShape) -> List[Tuple[str, Tuple[int, ...]]]:
    """Ordered (name, shape) list; the order fixes each tensor's seed index.

    NAR models (m.nar) have one codebook table per codec layer (emb_codes,
    [k_heads + 1, codebook, d]), one head per predicted layer (w_heads
    [k_heads, codebook, d]) and one stage vector per predicted layer (stage
    [k_heads, d]) instead of the AR's codec table and next-token heads."""
    d, f, v = m.d_model, m.d_ff, m.vocab
    out: List[Tuple[str, Tuple[int, ...]]] = [
        ("emb_phone", (m.n_phone, d)),
        ("emb_codes", (m.k_heads + 1, m.codebook, d)) if m.nar else ("emb_ac", (v, d)),
        ("pos", (m.max_pos, d)),
    ]
    for l in range(m.n_layers):
        out += [
            (f"l{l}.ln1_g", (d,)), (f"l{l}.ln1_b", (d,)),
            (f"l{l}.w_qkv", (3 * d, d)), (f"l{l}.b_qkv", (3 * d,)),
            (f"l{l}.w_o", (d, d)), (f"l{l}.b_o", (d,)),
            (f"l{l}.ln2_g", (d,)), (f"l{l}.ln2_b", (d,)),
            (f"l{l}.w_1", (f, d)), (f"l{l}.b_1", (f,)),
            (f"l{l}.w_2", (d, f)), (f"l{l}.b_2", (d,)),
        ]
    hv = m.codebook if m.nar else v
    out += [("lnf_g", (d,)), ("lnf_b", (d,)),
            ("w_heads", (m.k_heads, hv, d)), ("b_heads", (m.k_heads, hv))]
    if m.nar:
        out += [("stage", (m.k_heads, d))]
    return out


def make_weights(m: ModelShape, seed: int = WEIGHT_SEED) -> Dict[str, np.ndarray]:
    """Seeded float32 weights (bf16-exact values for bf16 models).

    Linear weights/biases, embeddings and the position table are N(0, 0.02).
    LayerNorm gains are 1 + N(0, 0.02) and shifts N(0, 0.02), so that a kernel
    that ignores either is caught by parity.
    """
    w: Dict[str, np.ndarray] = {}
    for idx, (name, shape) in enumerate(weight_names(m)):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, idx])))
        a = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(0.02)
        if name.endswith("_g"):
            a = a + np.float32(1.0)
        a = a.astype(np.float32)
        if m.dtype == DTYPE_BF16:
            a = bf16_round(a)
        w[name] = a
    return w


def make_logq(v: int = VOCAB, seed: int = Q_SEED, kind: str = "synthetic",
              alpha: float = 0.5, eos_id: Optional[int] = EOS_ID) -> np.ndarray:
    """log of a strictly positive row-stochastic transition table Q [v, v] (float32).

    Row = previous token, column = next token.  The LibriTTS-estimated table is
    not available, so values are invented:
      uniform   -- every entry 1/v;
      sticky    -- alpha * I + (1 - alpha) / v;
      synthetic -- heavy-tailed per-row draws (Gamma(0.3)) with a boosted
                   diagonal, since consecutive speech tokens are often similar;
                   the EOS column gets the row's mean mass.
    Built in float64, then log and rounded to float32.
    """
    if kind == "uniform":
        q = np.full((v, v), 1.0 / v)
    elif kind == "sticky":
        q = np.full((v, v), (1.0 - alpha) / v) + alpha * np.eye(v)
    elif kind == "synthetic":
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7])))
        raw = rng.gamma(0.3, size=(v, v)) + 1e-6
        diag = np.arange(v)
        raw[diag, diag] += 0.15 * raw.sum(axis=1)
        if eos_id is not None:
            raw[:, eos_id] = raw.mean(axis=1)
        q = raw / raw.sum(axis=1, keepdims=True)
    else:
        raise ValueError(f"unknown Q kind {kind!r}")
    return np.log(q).astype(np.float32)


@dataclass
class Prompts:
    phon: List[np.ndarray]   # per sequence int32 phoneme ids
    ac: List[np.ndarray]     # per sequence int32 acoustic-prompt codec ids

    @property
    def batch(self) -> int:
        return len(self.phon)


def make_prompts(wl: Workload, seed_base: int = PROMPT_SEED_BASE, batch: Optional[int] = None) -> Prompts:
    """Per-sequence prompts: sequence b uses seed seed_base + b.

    Lengths are uniform over the workload's inclusive ranges; phoneme ids are
    uniform over 0..511 and acoustic ids uniform over 0..1023.
    """
    B = wl.batch if batch is None else batch
    phon, ac = [], []
    for b in range(B):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed_base + b])))
        lp = int(rng.integers(wl.phon_len[0], wl.phon_len[1] + 1))
        la = int(rng.integers(wl.ac_len[0], wl.ac_len[1] + 1))
        phon.append(rng.integers(0, N_PHONE, size=lp).astype(np.int32))
        ac.append(rng.integers(0, VOCAB - 1, size=la).astype(np.int32))
    return Prompts(phon, ac)


def random_logits(rng: np.random.Generator, shape, scale: float = 0.64) -> np.ndarray:
    """iid N(0, scale^2) float32 logits, the spread of the VALL-E-shaped heads."""
    return (rng.standard_normal(size=shape) * scale).astype(np.float32)


# ---------------------------------------------------------------- token corpora
# Synthetic stand-ins for the codec-token streams a transition table is
# counted from (the paper derives Q from the LibriTTS training set).


@dataclass(frozen=True)
class CorpusSpec:
    """Token-stream corpus shape: `n_seqs` utterances whose lengths are
    Gamma(2)-distributed with mean `mean_len`, clipped to [min_len, max_len]."""
    name: str
    n_seqs: int
    mean_len: float
    min_len: int
    max_len: int
    seed: int


CORPORA: Dict[str, CorpusSpec] = {
    # LibriTTS train-clean-100 + train-clean-360 + train-other-500: 354,780
    # utterances, ~585 h, i.e. ~297 first-quantizer tokens per utterance at
    # SpeechTokenizer's 50 Hz frame rate (~105 M tokens in all)
    "libritts_train": CorpusSpec("libritts_train", 354780, 297.0, 13, 1750, seed=31),
    "small": CorpusSpec("small", 257, 37.0, 0, 160, seed=32),
}


@dataclass
class Corpus:
    tokens: np.ndarray    # int32 [n_tokens], utterances back to back
    offsets: np.ndarray   # int64 [n_seqs + 1], utterance u = tokens[offsets[u]:offsets[u+1]]


def _alias_tables(p: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Walker's alias tables (Vose's construction) for every row of a
    row-stochastic matrix: draw column c uniformly, keep it with probability
    keep[r, c], else take alias[r, c]."""
    R, n = p.shape
    keep = np.ones((R, n))
    alias = np.tile(np.arange(n, dtype=np.int32), (R, 1))
    for r in range(R):
        w = (p[r] * n).tolist()
        small = [i for i in range(n) if w[i] < 1.0]
        large = [i for i in range(n) if w[i] >= 1.0]
        kr, ar = keep[r], alias[r]
        while small and large:
            s_, l_ = small.pop(), large.pop()
            kr[s_] = w[s_]
            ar[s_] = l_
            w[l_] = (w[l_] + w[s_]) - 1.0
            (small if w[l_] < 1.0 else large).append(l_)
    return keep, alias


def make_corpus(spec: CorpusSpec, logq: Optional[np.ndarray] = None, chains: int = 65536,
                n_codes: int = EOS_ID) -> Corpus:
    """Codec-token utterances drawn from the Markov chain of Q (rows and
    columns of the first `n_codes` ids, renormalised; the synthetic table by
    default).  `chains` chains run side by side from uniform starting tokens;
    their concatenation is cut into the utterances."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([spec.seed, 5])))
    lens = np.clip(np.rint(rng.gamma(2.0, spec.mean_len / 2.0, size=spec.n_seqs)), spec.min_len, spec.max_len)
    lens = lens.astype(np.int64)
    offsets = np.zeros(spec.n_seqs + 1, np.int64)
    np.cumsum(lens, out=offsets[1:])
    total = int(offsets[-1])
    if logq is None:
        logq = make_logq()
    V = n_codes
    q = np.exp(logq[:V, :V].astype(np.float64))
    keep, alias = _alias_tables(q / q.sum(axis=1, keepdims=True))
    C = max(1, min(chains, total))
    steps = (total + C - 1) // C
    x = rng.integers(0, V, size=C)
    out = np.empty((steps, C), np.int32)
    for s in range(steps):
        out[s] = x
        c = rng.integers(0, V, size=C)
        x = np.where(rng.random(C) < keep[x, c], c, alias[x, c])
    tokens = np.ascontiguousarray(out.T).ravel()[:total].astype(np.int32)
    return Corpus(tokens, offsets)


# ---------------------------------------------------------------- NAR inputs
# The NAR module (Eq. 2) completes codec layers 2..8 of the utterance the AR
# module generated; its inputs are the phonemes, all 8 layers of the acoustic
# prompt and the generated first layer.


@dataclass(frozen=True)
class NarWorkload:
    name: str
    model: ModelShape
    batch: int
    phon_len: Tuple[int, int]      # inclusive ranges
    prompt_len: Tuple[int, int]
    target_len: Tuple[int, int]
    description: str = ""

    @property
    def max_seq(self) -> int:
        return self.phon_len[1] + self.prompt_len[1] + self.target_len[1]


_NAR_TINY = ModelShape(n_layers=2, d_model=256, n_heads=4, d_ff=1024, k_heads=7, dtype=DTYPE_F32, max_pos=512,
                       nar=True)
_NAR_VALLE = ModelShape(n_layers=12, d_model=1024, n_heads=16, d_ff=4096, k_heads=7, dtype=DTYPE_BF16, nar=True)

NAR_WORKLOADS: Dict[str, NarWorkload] = {
    "nar_tiny": NarWorkload("nar_tiny", _NAR_TINY, batch=3, phon_len=(0, 9), prompt_len=(6, 20),
                            target_len=(1, 40), description="2L d256 H4 F1024 fp32, 7 stages, batch 3 ragged"),
    "nar_valle": NarWorkload("nar_valle", _NAR_VALLE, batch=1, phon_len=(100, 100), prompt_len=(225, 225),
                             target_len=(750, 750),
                             description="12L d1024 H16 F4096 bf16, 7 stages, 100 phon + 225 prompt + 750 target"),
    "nar_valle_b8": NarWorkload("nar_valle_b8", _NAR_VALLE, batch=8, phon_len=(50, 150), prompt_len=(150, 300),
                                target_len=(300, 750),
                                description="12L d1024 H16 F4096 bf16, 7 stages, batch 8 ragged"),
}


@dataclass
class NarInputs:
    phon: List[np.ndarray]     # per utterance int32 phoneme ids
    prompt: List[np.ndarray]   # per utterance int32 [n_q, P] codes of every codec layer
    a1: List[np.ndarray]       # per utterance int32 [T] first-layer codes to complete


def make_nar_inputs(wl: NarWorkload, seed_base: int = 300) -> NarInputs:
    """Uniform ids: phonemes over 0..511, codes over 0..codebook-1; lengths
    uniform over the inclusive ranges; utterance b uses seed seed_base + b."""
    m = wl.model
    phon, prompt, a1 = [], [], []
    for b in range(wl.batch):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed_base + b])))
        lp = int(rng.integers(wl.phon_len[0], wl.phon_len[1] + 1))
        lq = int(rng.integers(wl.prompt_len[0], wl.prompt_len[1] + 1))
        lt = int(rng.integers(wl.target_len[0], wl.target_len[1] + 1))
        phon.append(rng.integers(0, m.n_phone, size=lp).astype(np.int32))
        prompt.append(rng.integers(0, m.codebook, size=(m.k_heads + 1, lq)).astype(np.int32))
        a1.append(rng.integers(0, m.codebook, size=lt).astype(np.int32))
    return NarInputs(phon, prompt, a1)
