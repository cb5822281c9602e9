"""Pins of the oracle's elementwise numerics to library routines, closed forms
and brute force (no device needed)."""
import math

import numpy as np
import pytest
import torch

from oracle import numerics as nm


# ------------------------------------------------------------------ bf16
def _bf16_neighbours(r):
    """The bf16 values just below and above r (r finite, bf16-valued)."""
    b = (np.asarray(r, np.float32).view(np.uint32) >> 16).astype(np.int64)
    sign = b & 0x8000
    mag = b & 0x7FFF
    up = np.where(sign == 0, b + 1, np.where(mag == 0, 0x0001, b - 1))
    dn = np.where(sign == 0, np.where(mag == 0, 0x8001, b - 1), b + 1)
    f = lambda x: ((x.astype(np.uint32) & 0xFFFF) << 16).view(np.float32).astype(np.float64)
    return f(dn), f(up)


def test_bf16_matches_torch_on_float32():
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 2**32, size=200000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    special = np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.3895314e38, 3.4e38,
                        1e-40, -1e-40, 9.2e-41, np.inf, -np.inf], np.float32)
    x = np.concatenate([x, special])
    ours = nm.bf16_round(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)


def test_bf16_nan_stays_nan():
    assert np.isnan(nm.bf16_round(np.array([np.nan]))[0])


def test_bf16_nearest_even_brute_force_float64():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))
    r = nm.bf16_round(x)
    dn, up = _bf16_neighbours(r)
    err = np.abs(x - r)
    assert np.all(err <= np.abs(x - dn))
    assert np.all(err <= np.abs(x - up))


def test_bf16_double_rounding_cases():
    one = 1.0
    tie = 1.0 + 2.0 ** -8             # exactly between 1 and 1+2^-7: even -> 1
    assert nm.bf16_round(np.array([tie]))[0] == one
    above = tie + 2.0 ** -40          # float32 rounds it onto the tie; the value is above it
    assert nm.bf16_round(np.array([above]))[0] == 1.0 + 2.0 ** -7
    tie_odd = 1.0 + 3 * 2.0 ** -8     # between 1+2^-7 (odd) and 1+2^-6: even -> up
    assert nm.bf16_round(np.array([tie_odd]))[0] == 1.0 + 2.0 ** -6
    below = tie_odd - 2.0 ** -40
    assert nm.bf16_round(np.array([below]))[0] == 1.0 + 2.0 ** -7
    assert nm.bf16_round(np.array([-above]))[0] == -(1.0 + 2.0 ** -7)


def test_bf16_overflow_and_bits_roundtrip():
    assert nm.bf16_round(np.array([3.4e38]))[0] == np.inf
    b = nm.bf16_bits(np.array([1.0, -2.0, 0.5]))
    np.testing.assert_array_equal(b, np.array([0x3F80, 0xC000, 0x3F00], np.uint16))
    np.testing.assert_array_equal(nm.from_bf16_bits(b), [1.0, -2.0, 0.5])


# ------------------------------------------------------------------ RMSNorm
def test_rmsnorm_constant_vector_closed_form():
    for c in (3.0, -0.25, 1e-3):
        x = np.full((1, 64), c)
        g = np.linspace(0.5, 2.0, 64)
        y = nm.rmsnorm(x, g, 1e-5)
        np.testing.assert_allclose(y[0], c / math.sqrt(c * c + 1e-5) * g, rtol=1e-14)


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 96)) * 3
    g = rng.standard_normal(96)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(nm.rmsnorm(x, g, 1e-5), ref, rtol=1e-13, atol=1e-15)


# ------------------------------------------------------------------ RoPE
def test_rope_worked_example():
    # d = 4, theta = 10000: inverse frequencies 1 and 1/100; pairs (0,2), (1,3)
    x = np.array([[[1.0, 2.0, 0.0, 0.0]]])
    y = nm.rope(x, np.array([1]), 10000.0)[0, 0]
    np.testing.assert_allclose(y, [math.cos(1), 2 * math.cos(0.01), math.sin(1), 2 * math.sin(0.01)], rtol=1e-15)


def test_rope_position_zero_is_identity_and_norm_preserved():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((6, 3, 128))
    np.testing.assert_array_equal(nm.rope(x, np.zeros(6, np.int64), 5e5), x)
    y = nm.rope(x, np.arange(6) * 777, 5e5)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)


def test_rope_is_complex_rotation():
    rng = np.random.default_rng(4)
    d = 64
    x = rng.standard_normal((4, 2, d))
    pos = np.array([0, 5, 300, 4095])
    y = nm.rope(x, pos, 500000.0)
    zc = x[..., : d // 2] + 1j * x[..., d // 2:]
    ang = pos[:, None, None] * 500000.0 ** (-np.arange(0, d, 2) / d)
    w = zc * np.exp(1j * ang)
    np.testing.assert_allclose(y[..., : d // 2], w.real, atol=1e-12)
    np.testing.assert_allclose(y[..., d // 2:], w.imag, atol=1e-12)


def test_rope_scores_depend_on_offset_only():
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, 1, 128))
    k = rng.standard_normal((1, 1, 128))
    s = []
    for shift in (0, 17, 1000):
        qq = nm.rope(q, np.array([40 + shift]), 5e5)
        kk = nm.rope(k, np.array([12 + shift]), 5e5)
        s.append(float(np.sum(qq * kk)))
    np.testing.assert_allclose(s, s[0], rtol=1e-10)


# ------------------------------------------------------------------ SiLU
def test_silu_closed_form_and_torch():
    assert nm.silu(np.array([0.0]))[0] == 0.0
    assert abs(nm.silu(np.array([1.0]))[0] - 1.0 / (1.0 + math.exp(-1.0))) < 1e-16
    z = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(nm.silu(z), torch.nn.functional.silu(torch.from_numpy(z)).numpy(),
                               rtol=1e-14, atol=1e-300)


# ------------------------------------------------------------------ attention
def test_attend_matches_torch_sdpa():
    rng = np.random.default_rng(6)
    for n in (1, 7, 129):
        q = rng.standard_normal(64)
        K = rng.standard_normal((n, 64))
        V = rng.standard_normal((n, 64))
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q)[None, None, None], torch.from_numpy(K)[None, None],
            torch.from_numpy(V)[None, None])[0, 0, 0].numpy()
        np.testing.assert_allclose(nm.attend(q, K, V), ref, rtol=1e-12, atol=1e-13)


def test_attend_special_cases():
    rng = np.random.default_rng(7)
    n, d = 37, 32
    K = rng.standard_normal((n, d)) * 4
    q = rng.standard_normal(d) * 4
    # V = 1: softmax rows sum to one
    np.testing.assert_allclose(nm.attend(q, K, np.ones((n, d))), np.ones(d), rtol=1e-14)
    # V = one-hot(position) exposes the probabilities
    P = nm.attend(q, K, np.eye(n))
    np.testing.assert_allclose(P, nm.attention_weights(q, K), rtol=1e-14)
    s = K @ q / math.sqrt(d)
    np.testing.assert_allclose(P, np.exp(s) / np.exp(s).sum(), rtol=1e-12)
    # q = 0: uniform attention, output = mean of V
    V = rng.standard_normal((n, d))
    np.testing.assert_allclose(nm.attend(np.zeros(d), K, V), V.mean(0), rtol=1e-13, atol=1e-15)
    # a single key returns its value
    np.testing.assert_allclose(nm.attend(q, K[:1], V[:1]), V[0], rtol=0, atol=0)


def test_attend_large_scores_stable():
    q = np.full(8, 100.0)
    K = np.stack([np.full(8, 100.0), np.full(8, -100.0)])
    V = np.array([[1.0] * 8, [2.0] * 8])
    np.testing.assert_allclose(nm.attend(q, K, V), np.ones(8))


# ------------------------------------------------------------------ argmax
def test_argmax_lowest_index_and_nan():
    z = np.array([[1.0, 3.0, 3.0, 2.0],
                  [np.nan, 0.5, np.nan, 0.5],
                  [np.nan, np.nan, np.nan, np.nan],
                  [-np.inf, -np.inf, -1.0, -1.0]])
    np.testing.assert_array_equal(nm.argmax_lowest(z), [1, 1, 0, 2])


def test_argmax_brute_force():
    rng = np.random.default_rng(8)
    z = rng.integers(-3, 4, size=(50, 40)).astype(np.float64)
    ids = nm.argmax_lowest(z)
    for r in range(50):
        m = max(z[r])
        assert ids[r] == min(j for j in range(40) if z[r, j] == m)
