"""Pins of the oracle's NAR module (Sec. 3.1, Eq. 2: codec layers 2..8 from
the phonemes, the whole acoustic prompt and the known layers a^{<j}).

The trunk and a stage head are checked against PyTorch's pre-LN
TransformerEncoderLayer (norm_first, exact GELU, no mask) in float64; the
conditioning against the structure Eq. 2 fixes: stage j reads layers 1..j-1
of the target and nothing above, and every layer of the prompt; attention is
bidirectional (a later target token changes earlier logits, and with the
position table removed the outputs are permutation-equivariant)."""
import numpy as np
import pytest
import torch

from oracle.nar import NARModel
from paper_2410_13839_amd.workloads import ModelShape, make_weights

SMALL = ModelShape(n_layers=2, d_model=128, n_heads=2, d_ff=256, k_heads=7, dtype="f32", max_pos=128, nar=True)


def _inputs(rng, lp=5, lq=9, lt=12):
    phon = rng.integers(0, SMALL.n_phone, size=lp)
    prompt = rng.integers(0, SMALL.codebook, size=(8, lq))
    target = rng.integers(0, SMALL.codebook, size=(8, lt))
    return phon, prompt, target


def _torch_stage(w, j, phon, prompt, target):
    """Stage j's target logits from torch.nn building blocks (float64)."""
    d = SMALL.d_model
    t64 = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    E = [torch.nn.Embedding.from_pretrained(t64(w["emb_codes"][i])) for i in range(8)]
    ph = torch.nn.Embedding.from_pretrained(t64(w["emb_phone"]))(torch.as_tensor(phon))
    pr = sum(E[i](torch.as_tensor(prompt[i])) for i in range(8))
    tg = sum(E[i](torch.as_tensor(target[i])) for i in range(j - 1))
    x = torch.cat([ph, pr, tg])
    n = x.shape[0]
    x = (x + t64(w["pos"][:n]) + t64(w["stage"][j - 2]))[None]
    with torch.no_grad():
        for l in range(SMALL.n_layers):
            p = f"l{l}."
            lay = torch.nn.TransformerEncoderLayer(d, SMALL.n_heads, SMALL.d_ff, dropout=0.0, activation="gelu",
                                                   batch_first=True, norm_first=True, dtype=torch.float64)
            for dst, src in ((lay.self_attn.in_proj_weight, "w_qkv"), (lay.self_attn.in_proj_bias, "b_qkv"),
                             (lay.self_attn.out_proj.weight, "w_o"), (lay.self_attn.out_proj.bias, "b_o"),
                             (lay.norm1.weight, "ln1_g"), (lay.norm1.bias, "ln1_b"),
                             (lay.norm2.weight, "ln2_g"), (lay.norm2.bias, "ln2_b"),
                             (lay.linear1.weight, "w_1"), (lay.linear1.bias, "b_1"),
                             (lay.linear2.weight, "w_2"), (lay.linear2.bias, "b_2")):
                dst.copy_(t64(w[p + src]))
            lay.eval()
            x = lay(x)
        z = torch.nn.functional.layer_norm(x[0, len(phon) + prompt.shape[1]:], (d,), t64(w["lnf_g"]),
                                           t64(w["lnf_b"]), eps=1e-5)
        return torch.nn.functional.linear(z, t64(w["w_heads"][j - 2]), t64(w["b_heads"][j - 2])).numpy()


@pytest.mark.parametrize("j", [2, 5, 8])
def test_stage_logits_match_torch_transformer(j):
    w = make_weights(SMALL, seed=4)
    rng = np.random.default_rng(j)
    phon, prompt, target = _inputs(rng)
    m = NARModel(SMALL, w)
    h = m.forward(m.embed(j, phon, prompt, target))
    ours = m.stage_logits(h[len(phon) + prompt.shape[1]:], j)
    ref = _torch_stage(w, j, phon, prompt, target)
    assert np.max(np.abs(ours - ref)) < 1e-10


def _stage(m, j, phon, prompt, target):
    h = m.forward(m.embed(j, phon, prompt, target))
    return m.stage_logits(h[len(phon) + prompt.shape[1]:], j)


def test_stage_reads_exactly_the_lower_layers():
    m = NARModel(SMALL, make_weights(SMALL, seed=5))
    rng = np.random.default_rng(1)
    phon, prompt, target = _inputs(rng)
    for j in range(2, 9):
        base = _stage(m, j, phon, prompt, target)
        upper = target.copy()
        upper[j - 1:] = rng.integers(0, SMALL.codebook, size=upper[j - 1:].shape)
        assert np.array_equal(_stage(m, j, phon, prompt, upper), base), j      # layers >= j unused
        lower = target.copy()
        lower[j - 2, 3] = (lower[j - 2, 3] + 1) % SMALL.codebook
        assert np.max(np.abs(_stage(m, j, phon, prompt, lower) - base)) > 1e-6, j   # layer j-1 used


def test_every_prompt_layer_conditions_every_stage():
    m = NARModel(SMALL, make_weights(SMALL, seed=6))
    rng = np.random.default_rng(2)
    phon, prompt, target = _inputs(rng)
    base = _stage(m, 2, phon, prompt, target)
    for i in range(8):
        p2 = prompt.copy()
        p2[i, 0] = (p2[i, 0] + 1) % SMALL.codebook
        assert np.max(np.abs(_stage(m, 2, phon, p2, target) - base)) > 1e-6, i


def test_attention_is_bidirectional():
    w = make_weights(SMALL, seed=7)
    m = NARModel(SMALL, w)
    rng = np.random.default_rng(3)
    phon, prompt, target = _inputs(rng)
    base = _stage(m, 3, phon, prompt, target)
    t2 = target.copy()
    t2[0, -1] = (t2[0, -1] + 1) % SMALL.codebook            # the last target position
    assert np.max(np.abs(_stage(m, 3, phon, prompt, t2)[0] - base[0])) > 1e-6
    # without positions the module is permutation-equivariant over the target
    w0 = dict(w)
    w0["pos"] = np.zeros_like(w["pos"])
    m0 = NARModel(SMALL, w0)
    perm = rng.permutation(target.shape[1])
    a = _stage(m0, 4, phon, prompt, target)
    b = _stage(m0, 4, phon, prompt, target[:, perm])
    assert np.allclose(b, a[perm], atol=1e-12)


def test_run_is_greedy_per_stage_and_teacher_forcing_is_consistent():
    m = NARModel(SMALL, make_weights(SMALL, seed=8))
    rng = np.random.default_rng(4)
    phon, prompt, target = _inputs(rng)
    codes, logits = m.run(phon, prompt, target[0])
    assert np.array_equal(codes[0], target[0])
    for j in range(2, 9):
        assert np.array_equal(codes[j - 1], np.argmax(logits[j - 2], axis=1))
        assert np.allclose(logits[j - 2], _stage(m, j, phon, prompt, codes))
    codes2, _ = m.run(phon, prompt, target[0], teacher=codes)
    assert np.array_equal(codes2, codes)
