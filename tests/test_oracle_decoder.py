"""Pins of the oracle's AR decoder and loop.

The trunk is checked against PyTorch's own pre-LN Transformer layer
(torch.nn.TransformerEncoderLayer with norm_first=True, exact GELU, causal
mask) loaded with the same weights, in float64 on the CPU: a library routine
that computes the same decoder-only block, written by someone else.  The KV
cache is checked against full recomputation, and the loop against the step
count the method implies (Sec. 3.2: about L/n AR steps for L tokens).
"""
import dataclasses
import math

import numpy as np
import pytest
import torch

from oracle.decoder import ARDecoder
from oracle.generate import Generator, generate
from oracle.selection import select
from paper_2410_13839_amd.workloads import (WORKLOADS, ModelShape, bf16_round,
                                            make_logq, make_prompts, make_weights)

SMALL = ModelShape(n_layers=2, d_model=128, n_heads=2, d_ff=512, k_heads=3, dtype="f32", max_pos=256)


def _torch_reference(shape, w, ids, phon_len, n_heads_out):
    """Same computation from torch.nn building blocks (float64, CPU)."""
    d, L = shape.d_model, shape.n_layers
    layers = []
    for l in range(L):
        p = f"l{l}."
        lay = torch.nn.TransformerEncoderLayer(d, shape.n_heads, shape.d_ff, dropout=0.0,
                                               activation="gelu", batch_first=True,
                                               norm_first=True, dtype=torch.float64)
        with torch.no_grad():
            lay.self_attn.in_proj_weight.copy_(torch.from_numpy(w[p + "w_qkv"].astype(np.float64)))
            lay.self_attn.in_proj_bias.copy_(torch.from_numpy(w[p + "b_qkv"].astype(np.float64)))
            lay.self_attn.out_proj.weight.copy_(torch.from_numpy(w[p + "w_o"].astype(np.float64)))
            lay.self_attn.out_proj.bias.copy_(torch.from_numpy(w[p + "b_o"].astype(np.float64)))
            lay.norm1.weight.copy_(torch.from_numpy(w[p + "ln1_g"].astype(np.float64)))
            lay.norm1.bias.copy_(torch.from_numpy(w[p + "ln1_b"].astype(np.float64)))
            lay.norm2.weight.copy_(torch.from_numpy(w[p + "ln2_g"].astype(np.float64)))
            lay.norm2.bias.copy_(torch.from_numpy(w[p + "ln2_b"].astype(np.float64)))
            lay.linear1.weight.copy_(torch.from_numpy(w[p + "w_1"].astype(np.float64)))
            lay.linear1.bias.copy_(torch.from_numpy(w[p + "b_1"].astype(np.float64)))
            lay.linear2.weight.copy_(torch.from_numpy(w[p + "w_2"].astype(np.float64)))
            lay.linear2.bias.copy_(torch.from_numpy(w[p + "b_2"].astype(np.float64)))
        lay.eval()
        layers.append(lay)
    T = len(ids)
    emb_p = torch.nn.Embedding.from_pretrained(torch.from_numpy(w["emb_phone"].astype(np.float64)))
    emb_a = torch.nn.Embedding.from_pretrained(torch.from_numpy(w["emb_ac"].astype(np.float64)))
    emb_pos = torch.nn.Embedding.from_pretrained(torch.from_numpy(w["pos"].astype(np.float64)))
    ids_t = torch.as_tensor(ids, dtype=torch.long)
    pos = torch.arange(T)
    x = torch.where((pos < phon_len)[:, None], emb_p(ids_t.clamp(max=shape.n_phone - 1)), emb_a(ids_t))
    x = (x + emb_pos(pos))[None]
    mask = torch.nn.Transformer.generate_square_subsequent_mask(T, dtype=torch.float64)
    with torch.no_grad():
        for lay in layers:
            x = lay(x, src_mask=mask, is_causal=True)
        z = torch.nn.functional.layer_norm(x[0, -1], (d,), torch.from_numpy(w["lnf_g"].astype(np.float64)),
                                           torch.from_numpy(w["lnf_b"].astype(np.float64)), eps=1e-5)
        heads = [torch.nn.functional.linear(z, torch.from_numpy(w["w_heads"][i].astype(np.float64)),
                                            torch.from_numpy(w["b_heads"][i].astype(np.float64)))
                 for i in range(n_heads_out)]
    return x[0].numpy(), torch.stack(heads).numpy()


@pytest.mark.parametrize("phon_len,T", [(0, 21), (7, 21), (5, 600)])
def test_trunk_and_heads_match_torch_transformer(phon_len, T):
    """T = 600 spans three of the oracle's 256-row attention blocks and a
    ragged last one."""
    shape = dataclasses.replace(SMALL, max_pos=1024)
    w = make_weights(shape, seed=3)
    rng = np.random.default_rng(0)
    ids = np.concatenate([rng.integers(0, 512, phon_len), rng.integers(0, 1024, T - phon_len)])
    m = ARDecoder(shape, w)
    cache = m.new_cache()
    h = m.forward(cache, ids, phon_len)
    logits = m.heads(h[-1], 3)
    h_ref, logits_ref = _torch_reference(shape, w, ids, phon_len, 3)
    np.testing.assert_allclose(h, h_ref, atol=1e-10, rtol=1e-10)
    np.testing.assert_allclose(logits, logits_ref, atol=1e-10, rtol=1e-10)


def test_kv_cache_chunks_equal_full_recompute():
    w = make_weights(SMALL, seed=4)
    m = ARDecoder(SMALL, w)
    rng = np.random.default_rng(1)
    ids = np.concatenate([rng.integers(0, 512, 5), rng.integers(0, 1024, 25)])
    full = m.forward(m.new_cache(), ids, 5)
    cache = m.new_cache()
    parts = [m.forward(cache, ids[a:b], 5) for a, b in [(0, 11), (11, 12), (12, 20), (20, 30)]]
    np.testing.assert_allclose(np.concatenate(parts), full, atol=1e-12)
    assert cache.length == 30


def test_bf16_emulation_changes_little():
    shape = ModelShape(n_layers=2, d_model=128, n_heads=2, d_ff=512, k_heads=2, dtype="bf16", max_pos=256)
    w = make_weights(shape, seed=5)
    for v in w.values():
        assert np.array_equal(v, bf16_round(v))
    ids = np.arange(17) * 13 % 1024
    a = ARDecoder(shape, w).heads(ARDecoder(shape, w).forward(ARDecoder(shape, w).new_cache(), ids, 0)[-1], 2)
    m = ARDecoder(shape, w, emulate_bf16=True)
    b = m.heads(m.forward(m.new_cache(), ids, 0)[-1], 2)
    assert 0 < np.abs(a - b).max() < 3e-2


def test_bf16_round_matches_torch():
    x = (np.random.default_rng(2).standard_normal(10000) * 3).astype(np.float32)
    x[:4] = [1.00390625, 1.01171875, -2.00390625, 0.0]  # exact halfway cases
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(bf16_round(x), ref)


@pytest.mark.parametrize("K", [1, 2, 3])
def test_step_count_is_ceil_tokens_over_heads(K):
    """Sec. 3.2: n heads emit n tokens per AR step, so G tokens take ceil(G/n) steps."""
    w = make_weights(SMALL, seed=6)
    m = ARDecoder(SMALL, w)
    logq = make_logq(kind="synthetic")
    G = 10
    run = generate(m, logq, np.array([1, 2, 3]), np.array([4, 5, 6, 7]), K=K, top_k=3, max_new=G, eos_min=G)
    assert len(run.steps) == math.ceil(G / K)
    assert len(run.tokens) == G
    assert [s.count for s in run.steps][:-1] == [K] * (len(run.steps) - 1)


def test_one_head_generation_is_greedy_ar():
    """With K = 1 the loop is plain AR decoding (Eq. 1): each token is the
    argmax of the one-step-ahead head given everything emitted so far."""
    w = make_weights(SMALL, seed=7)
    m = ARDecoder(SMALL, w)
    logq = make_logq(kind="synthetic")
    phon, ac = np.array([3, 9]), np.array([10, 20, 30])
    run = generate(m, logq, phon, ac, K=1, top_k=4, max_new=6, eos_min=6)
    seq = list(np.concatenate([phon, ac]))
    for tok in run.tokens:
        h = m.forward(m.new_cache(), np.array(seq), 2)
        lg = m.heads(h[-1], 1)[0].astype(np.float32)
        lg[1024] = -np.inf
        assert tok == int(np.argmax(lg))
        seq.append(tok)


def test_eos_ends_the_sequence_at_the_first_allowed_index():
    w = make_weights(SMALL, seed=8)
    w["b_heads"][:, 1024] = 50.0   # EOS dominates every head once allowed
    m = ARDecoder(SMALL, w)
    logq = make_logq(kind="synthetic")
    run = generate(m, logq, np.array([], np.int64), np.array([1, 2, 3]), K=3, top_k=3, max_new=40, eos_min=7)
    # generated indices 0..6 are non-EOS; index 7 (second position of the third step) is EOS
    assert len(run.tokens) == 8 and run.tokens[-1] == 1024
    assert 1024 not in run.tokens[:-1]
    assert [s.count for s in run.steps] == [3, 3, 2]


def test_teacher_forcing_follows_given_tokens():
    w = make_weights(SMALL, seed=9)
    m = ARDecoder(SMALL, w)
    logq = make_logq(kind="synthetic")
    g = Generator(m, logq, eos_min=100, max_new=100)
    g.prefill(np.array([1]), np.array([2, 3]))
    g.step(2, 3, force=[7, 8], force_count=2)
    rec = g.step(2, 3)
    m2 = ARDecoder(SMALL, w)
    h = m2.forward(m2.new_cache(), np.array([1, 2, 3, 7, 8]), 1)
    np.testing.assert_allclose(rec.logits, m2.heads(h[-1], 2).astype(np.float32), atol=0)


def test_workloads_shapes():
    wl = WORKLOADS["valle_b32"]
    pr = make_prompts(wl)
    assert pr.batch == 32
    assert all(50 <= len(p) <= 150 for p in pr.phon)
    assert all(150 <= len(a) <= 300 for a in pr.ac)
    assert all(p.max() < 512 for p in pr.phon) and all(a.max() < 1024 for a in pr.ac)
    pr2 = make_prompts(wl)
    assert all(np.array_equal(a, b) for a, b in zip(pr.ac, pr2.ac))


def test_attention_paths_agree():
    """The oracle evaluates the same causal attention formula with numpy for
    a few query rows and with PyTorch for many: on the same inputs (query
    rows at arbitrary positions, ragged blocks) both give the same rows."""
    m = ARDecoder(SMALL, make_weights(SMALL, seed=5))
    rng = np.random.default_rng(7)
    T = 300
    k = rng.standard_normal((T, SMALL.d_model))
    v = rng.standard_normal((T, SMALL.d_model))
    pos = np.sort(rng.choice(T, size=40, replace=False))
    q = rng.standard_normal((40, SMALL.d_model))
    a = m._attention_np(q, k, v, pos)
    b = m._attention_torch(q, k, v, pos, rows_per_block=16)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)
