"""Pins for the oracle's rounding helpers and operator definitions.

Each operator is checked against something other than its own formula: a
library routine (torch CPU in float64), brute-force loops, a closed form or
an invariant that a dropped term, wrong sign or swapped index would break.
"""
import math

import numpy as np
import pytest
import torch

from oracle import numerics
from oracle import execute as X


def test_bf16_rne_matches_torch_on_random_and_special_values():
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 1 << 32, size=1_000_000, dtype=np.uint64).astype(np.uint32)
    # ties: low 16 bits exactly 0x8000, with both parities of bit 16
    ties = (rng.integers(0, 1 << 16, size=20000, dtype=np.uint32) << 16) | 0x8000
    special = np.array([0, 0x80000000, 0x7F800000, 0xFF800000, 0x7F7FFFFF,
                        0x7F7F8000, 0x00000001, 0x00008000, 0x00018000,
                        0x807FFFFF, 0x3F808000, 0x3F818000], dtype=np.uint32)
    allbits = np.concatenate([bits, ties, special])
    f = allbits.view(np.float32)
    finite = ~np.isnan(f)
    ours = numerics.f32_to_bf16_bits(f[finite])
    ref = torch.from_numpy(f[finite].copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    nan = numerics.f32_to_bf16_bits(np.array([np.nan], np.float32))
    assert (nan[0] & 0x7FFF) > 0x7F80   # stays NaN


def test_round_bf16_goes_through_float32():
    # a float64 value just above a float32 tie that float32 RNE moves onto the
    # tie, then bf16 RNE rounds the tie to even: double rounding is intended
    v = 1.0 + 2.0 ** -8 + 2.0 ** -30
    assert numerics.round_bf16(np.array([v]))[0] == 1.0
    assert numerics.round_f32(np.array([1.0 + 2.0 ** -30]))[0] == 1.0


def test_matmul_matches_loops_with_batch_broadcast():
    rng = np.random.default_rng(1)
    a = rng.standard_normal((2, 3, 4, 5))
    b = rng.standard_normal((5, 6))
    got = X.op_matmul(a, b)
    ref = np.zeros((2, 3, 4, 6))
    for i in range(2):
        for j in range(3):
            for m in range(4):
                for n in range(6):
                    ref[i, j, m, n] = sum(a[i, j, m, k] * b[k, n] for k in range(5))
    assert np.allclose(got, ref, rtol=1e-13, atol=1e-13)
    b2 = rng.standard_normal((2, 3, 5, 7))
    got2 = X.op_matmul(a, b2)
    assert got2[1, 2, 3, 6] == pytest.approx(sum(a[1, 2, 3, k] * b2[1, 2, k, 6] for k in range(5)))


@pytest.mark.parametrize("causal", [0, 1])
def test_softmax_properties_and_torch(causal):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 3, 7, 7)) * 4
    y = X.op_softmax(x, 0.125, causal)
    assert np.allclose(y.sum(-1), 1.0, atol=1e-14)
    z = torch.from_numpy(x) * 0.125
    if causal:
        mask = torch.triu(torch.ones(7, 7, dtype=torch.bool), diagonal=1)
        z = z.masked_fill(mask, float("-inf"))
        assert np.all(y[..., mask.numpy()] == 0.0)
        assert y[0, 0, 0, 0] == 1.0
    ref = torch.softmax(z, dim=-1).numpy()
    assert np.allclose(y, ref, rtol=1e-14, atol=1e-16)
    # shift invariance along the reduced axis
    assert np.allclose(X.op_softmax(x + 3.0, 0.125, causal), y, atol=1e-14)


def test_layernorm_matches_torch_and_moments():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((3, 5, 16)) * 2 + 1
    gamma = rng.standard_normal(16)
    beta = rng.standard_normal(16)
    y = X.op_layernorm(x, gamma, beta, 1e-5)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (16,), torch.from_numpy(gamma),
                                         torch.from_numpy(beta), eps=1e-5).numpy()
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12)
    y1 = X.op_layernorm(x, np.ones(16), np.zeros(16), 1e-5)
    var = x.var(-1)
    assert np.allclose(y1.mean(-1), 0.0, atol=1e-13)
    assert np.allclose(y1.var(-1), var / (var + 1e-5), rtol=1e-12)


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((2, 6, 32))
    gamma = rng.standard_normal(32)
    y = X.op_rmsnorm(x, gamma, 1e-5)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (32,), torch.from_numpy(gamma),
                                       eps=1e-5).numpy()
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_gelu_silu_match_torch_and_math():
    x = np.linspace(-8, 8, 1001)
    g = X.op_gelu(x)
    assert np.allclose(g, torch.nn.functional.gelu(torch.from_numpy(x), approximate="none").numpy(),
                       rtol=1e-14, atol=1e-15)
    assert g[500] == 0.0
    assert X.op_gelu(np.array([1.0]))[0] == pytest.approx(0.5 * (1 + math.erf(1 / math.sqrt(2))), rel=1e-15)
    s = X.op_silu(x)
    assert np.allclose(s, torch.nn.functional.silu(torch.from_numpy(x)).numpy(), rtol=1e-14, atol=1e-15)


def test_rope_equals_complex_rotation_and_keeps_relative_positions():
    rng = np.random.default_rng(5)
    B, S, NH, D = 1, 9, 2, 8
    import synth_inputs
    cos, sin = synth_inputs.rope_tables(S, D, 10000.0)
    x = rng.standard_normal((B, S, NH, D))
    y = X.op_rope(x, cos.astype(np.float64), sin.astype(np.float64))
    # complex form: pair (i, i+D/2) is the number x_i + j x_{i+D/2}, multiplied
    # by exp(j * p * base^(-2i/D))
    h = D // 2
    theta = np.arange(S)[:, None] * np.power(10000.0, -2.0 * np.arange(h) / D)[None, :]
    z = (x[..., :h] + 1j * x[..., h:]) * np.exp(1j * theta)[None, :, None, :]
    ref = np.concatenate([z.real, z.imag], axis=-1)
    assert np.allclose(y, ref, atol=1e-6)        # tables are float32
    # position 0 is the identity; pair norms are preserved
    assert np.array_equal(y[:, 0], x[:, 0])
    n0 = x[..., :h] ** 2 + x[..., h:] ** 2
    n1 = y[..., :h] ** 2 + y[..., h:] ** 2
    assert np.allclose(n0, n1, rtol=1e-6)
    # dot products of rotated vectors depend only on the position difference
    q = np.broadcast_to(rng.standard_normal(D), (1, S, 1, D)).copy()
    k = np.broadcast_to(rng.standard_normal(D), (1, S, 1, D)).copy()
    qr = X.op_rope(q, cos.astype(np.float64), sin.astype(np.float64))
    kr = X.op_rope(k, cos.astype(np.float64), sin.astype(np.float64))
    d1 = qr[0, 5, 0] @ kr[0, 3, 0]
    d2 = qr[0, 4, 0] @ kr[0, 2, 0]
    assert d1 == pytest.approx(d2, rel=1e-5)
