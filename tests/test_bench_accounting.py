"""The algorithmic byte and flop counts the benchmark reports, pinned to
hand-computed figures for the 12-layer d1024 decoder (no GPU needed)."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2410_13839_amd.workloads import WORKLOADS  # noqa: E402


def test_parameter_counts():
    m = WORKLOADS["valle_k4"].model
    d, F, L, V = 1024, 4096, 12, 1025
    per_layer = 4 * d * d + 2 * d * F + (3 * d + d + F + d) + 4 * d
    assert bench.trunk_params(m) == L * per_layer
    assert bench.head_params(m, 4) == 4 * V * (d + 1)
    # 155.36 M parameters stream per step at K = 4
    assert abs((bench.trunk_params(m) + bench.head_params(m, 4)) / 1e6 - 155.357) < 1e-3


def test_step_bytes():
    wl = WORKLOADS["valle_k4"]
    m = wl.model
    ctx = [700]
    got = bench.step_bytes(wl, ctx)
    kv = 2 * 2 * m.n_layers * m.d_model * 700 + 2 * 2 * m.n_layers * m.d_model * wl.K
    weights = 2 * (bench.trunk_params(m) + bench.head_params(m, wl.K) + 2 * m.d_model)
    assert got == weights + kv + 8 * wl.K * m.vocab
    heads_only = bench.step_bytes(wl, ctx, trunk=False)
    assert heads_only == 2 * (bench.head_params(m, wl.K) + 2 * m.d_model) + 8 * wl.K * m.vocab


def test_prefill_flops():
    wl = WORKLOADS["valle_b32"]
    m = wl.model
    d, F, L = m.d_model, m.d_ff, m.n_layers
    lens = [3, 5]
    gemm = 2.0 * sum(lens) * L * (4 * d * d + 2 * d * F)
    attn = L * sum(4.0 * d * n * (n + 1) / 2 for n in lens)
    assert bench.prefill_flops(wl, lens) == pytest.approx(gemm + attn, rel=1e-12)
