"""Pins for the oracle's scalar building blocks (CPU only).

Each test checks an oracle function against something other than itself:
a library routine (torch CPU), a closed form, an invariant, or brute force.
"""
import math

import numpy as np
import pytest
import torch

from oracle import numerics as nx


# ------------------------------------------------------------ storage rounding

def test_round_bf16_matches_torch_on_float32_values():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(3.0),
        (rng.standard_normal(2000) * 1e30).astype(np.float32),
        (rng.standard_normal(2000) * 1e-36).astype(np.float32),   # bf16 subnormals
        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0, -0.0,
                  3.3895313892515355e38, 3.4e38, np.inf, -np.inf], dtype=np.float32),
    ])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = nx.round_bf16(x.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


def test_round_bf16_ties_to_even_and_nan():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to the even mantissa (1).
    assert nx.round_bf16(np.array([1.0 + 2 ** -8]))[0] == 1.0
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: ties to 1 + 2^-6.
    assert nx.round_bf16(np.array([1.0 + 3 * 2 ** -8]))[0] == 1.0 + 2 ** -6
    # just above a tie rounds up even from float64 (no double rounding)
    assert nx.round_bf16(np.array([1.0 + 2 ** -8 + 2 ** -40]))[0] == 1.0 + 2 ** -7
    assert np.isnan(nx.round_bf16(np.array([np.nan]))[0])


def test_round_f16_threshold_values():
    r = lambda v: nx.round_to(np.array([v]), "f16")[0]
    assert r(64504.0) == 64512.0          # the clamp value stores as 64512
    assert r(64495.9) == 64480.0
    assert r(64496.0) == 64512.0          # tie -> even mantissa (2016 * 32)
    assert r(65519.0) == 65504.0
    assert np.isinf(r(65520.0))


def test_round_f32_is_ieee():
    x = np.array([1.0 + 2 ** -30, math.pi, 1e-40])
    np.testing.assert_array_equal(nx.round_to(x, "f32"),
                                  x.astype(np.float32).astype(np.float64))


def test_decode_storage_roundtrip():
    v = nx.round_bf16(np.linspace(-3, 3, 101))
    np.testing.assert_array_equal(nx.decode(nx.to_storage(v, "bf16"), "bf16"), v)


# ------------------------------------------------------------ activations

def test_gelu_identities_and_library():
    x = np.linspace(-8, 8, 1001)
    g = nx.gelu(x)
    # Phi(x) + Phi(-x) = 1  =>  gelu(x) - gelu(-x) = x
    np.testing.assert_allclose(g - nx.gelu(-x), x, rtol=0, atol=1e-14)
    assert nx.gelu(np.array([0.0]))[0] == 0.0
    ref = torch.nn.functional.gelu(torch.from_numpy(x)).numpy()
    np.testing.assert_allclose(g, ref, rtol=1e-14, atol=1e-15)


def test_silu_identities_and_library():
    x = np.linspace(-30, 30, 1001)
    s = nx.silu(x)
    # sigmoid(x) + sigmoid(-x) = 1  =>  silu(x) - silu(-x) = x
    np.testing.assert_allclose(s - nx.silu(-x), x, rtol=0, atol=1e-13)
    ref = torch.nn.functional.silu(torch.from_numpy(x)).numpy()
    np.testing.assert_allclose(s, ref, rtol=1e-14, atol=1e-15)


# ------------------------------------------------------------ norms

def test_layer_norm_closed_form_and_library():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 96)) * 5 + 2
    y = nx.layer_norm(x, np.ones(96), np.zeros(96), 1e-5)
    np.testing.assert_allclose(y.mean(-1), 0, atol=1e-12)
    var = x.var(-1)
    np.testing.assert_allclose((y * y).mean(-1), var / (var + 1e-5), rtol=1e-12)
    g, b = rng.standard_normal(96), rng.standard_normal(96)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (96,), torch.from_numpy(g),
                                         torch.from_numpy(b), 1e-5).numpy()
    np.testing.assert_allclose(nx.layer_norm(x, g, b, 1e-5), ref, rtol=1e-12, atol=1e-12)


def test_rms_norm_closed_form():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 64)) * 3
    y = nx.rms_norm(x, np.ones(64), 0.0)
    np.testing.assert_allclose(np.sqrt((y * y).mean(-1)), 1.0, rtol=1e-13)
    # brute force on one row
    row = x[3]
    ms = sum(v * v for v in row) / len(row)
    np.testing.assert_allclose(y[3], row / math.sqrt(ms), rtol=1e-13)


# ------------------------------------------------------------ softmax

def test_masked_softmax_invariants():
    rng = np.random.default_rng(3)
    s = rng.standard_normal((4, 9, 9)) * 4
    allowed = rng.random((4, 9, 9)) < 0.6
    allowed[0, 2, :] = False                 # a fully masked row
    p = nx.masked_softmax(s, allowed)
    assert np.all(p[~allowed] == 0.0)
    rows = allowed.any(-1)
    np.testing.assert_allclose(p.sum(-1)[rows], 1.0, rtol=1e-14)
    assert np.all(p[0, 2] == 0.0)
    # equal scores over the allowed set -> uniform
    q = nx.masked_softmax(np.zeros((1, 5)), np.array([[1, 1, 0, 1, 0]], bool))
    np.testing.assert_allclose(q, [[1 / 3, 1 / 3, 0, 1 / 3, 0]], rtol=1e-15)
    # brute force on one row
    i = 1
    e = [math.exp(s[1, i, j]) if allowed[1, i, j] else 0.0 for j in range(9)]
    np.testing.assert_allclose(p[1, i], np.array(e) / sum(e), rtol=1e-13)


def test_masked_softmax_matches_torch_sdpa():
    rng = np.random.default_rng(4)
    q = rng.standard_normal((2, 3, 11, 8))
    k = rng.standard_normal((2, 3, 11, 8))
    v = rng.standard_normal((2, 3, 11, 8))
    allowed = np.tril(np.ones((11, 11), bool))[None, None] & (rng.random((2, 1, 1, 11)) < 0.8)
    allowed[..., 0] = True
    p = nx.masked_softmax(q @ k.transpose(0, 1, 3, 2) / math.sqrt(8), allowed)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v),
        attn_mask=torch.from_numpy(allowed)).numpy()
    np.testing.assert_allclose(p @ v, ref, rtol=1e-12, atol=1e-13)


# ------------------------------------------------------------ rotary

def test_rope_table_and_rotation_properties():
    hd, n = 16, 40
    cos, sin = nx.rope_table(n, hd, 10000.0)
    # position 0 is the identity
    assert np.all(cos[0] == 1.0) and np.all(sin[0] == 0.0)
    # frequencies: theta_0 = 1, theta_i decreasing
    np.testing.assert_allclose(np.arctan2(sin[1], cos[1])[0], 1.0, rtol=1e-7)
    rng = np.random.default_rng(5)
    q = rng.standard_normal((n, hd))
    k = rng.standard_normal((n, hd))
    rq = nx.apply_rope(q, cos, sin)
    # each (i, i + hd/2) pair keeps its norm
    h = hd // 2
    np.testing.assert_allclose(rq[:, :h] ** 2 + rq[:, h:] ** 2,
                               q[:, :h] ** 2 + q[:, h:] ** 2, rtol=1e-6)
    # <rot_m q, rot_n k> depends only on m - n (same q, k at every position)
    qq = np.repeat(q[:1], n, 0)
    kk = np.repeat(k[:1], n, 0)
    a = nx.apply_rope(qq, cos, sin)
    b = nx.apply_rope(kk, cos, sin)
    d1 = a[10] @ b[7]
    d2 = a[25] @ b[22]
    np.testing.assert_allclose(d1, d2, rtol=1e-5)
    # table of length n is a prefix of a longer table, bit for bit
    c2, s2 = nx.rope_table(2 * n, hd, 10000.0)
    np.testing.assert_array_equal(c2[:n], cos)
    np.testing.assert_array_equal(s2[:n], sin)
