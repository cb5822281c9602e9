"""Elementwise and per-row numerics of the decode step, float64.

Test infrastructure only (see the package docstring).

The paper serves Llama-3-family decoders (Section "Implementation") and does
not restate their layer definitions; the readings taken here are the
standard Llama ones:
  * RMSNorm: x / sqrt(mean(x^2) + eps) * g, eps = 1e-5.
  * Rotary positions, rotate-half pairing (i, i + d/2), inverse frequency
    theta^(-2i/d), positions counted from 0, no frequency rescaling.
  * SwiGLU MLP: silu(x Wg^T) * (x Wu^T), silu(z) = z / (1 + exp(-z)); the
    paper names this product in Algorithm 1 (RUN cohort step).
  * Attention scale 1/sqrt(head_dim); query head h reads KV head
    floor(h * n_kv / n_q).
  * Contract rounding points: tensors stored between kernels are bf16,
    rounded to nearest, ties to even.
"""
from __future__ import annotations

import numpy as np


# ------------------------------------------------------------------ bf16
def bf16_round(x) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (ties to even); returns float64.

    Goes through float32: the first rounding (to 24 bits) can only mislead
    the second (to 8 bits) when it lands exactly on a bf16 midpoint from a
    value that was not one; that case is resolved toward the original value.
    NaN stays NaN, overflow rounds to +-inf.
    """
    x = np.asarray(x, dtype=np.float64)
    x32 = x.astype(np.float32)
    u = x32.view(np.uint32).astype(np.uint64)
    low = u & 0xFFFF
    base = u & 0xFFFF0000
    up = (low > 0x8000) | ((low == 0x8000) & (((u >> 16) & 1) == 1))
    # double-rounding fix: an apparent tie that is not a tie in float64
    fake_tie = (low == 0x8000) & (x != x32.astype(np.float64))
    away = np.abs(x) > np.abs(x32.astype(np.float64))
    up = np.where(fake_tie, away, up)
    r = (base + np.where(up, 0x10000, 0)).astype(np.uint64)
    nan = np.isnan(x32)
    r = np.where(nan, np.uint64(0x7FC00000) | (u & 0x80000000), r)
    out = (r.astype(np.uint32)).view(np.float32).astype(np.float64)
    return out


def bf16_bits(x) -> np.ndarray:
    """bf16 bit patterns (uint16) of bf16_round(x)."""
    r = bf16_round(x).astype(np.float32)
    return (r.view(np.uint32) >> 16).astype(np.uint16)


def from_bf16_bits(bits) -> np.ndarray:
    """Exact float64 values of bf16 bit patterns."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


# ------------------------------------------------------------------ RMSNorm
def rmsnorm(x, g, eps: float, dt=np.float64) -> np.ndarray:
    """Row-wise x / sqrt(mean(x^2) + eps) * g over the last axis, in dtype dt
    (float64 by default; float32 for the contract-mode variant)."""
    x = np.asarray(x, dtype=dt)
    ms = np.mean(x * x, axis=-1, keepdims=True, dtype=dt)
    return x / np.sqrt(ms + dt(eps)) * np.asarray(g, dtype=dt)


# ------------------------------------------------------------------ rotary
def rope_inv_freq(head_dim: int, theta: float) -> np.ndarray:
    i = np.arange(head_dim // 2, dtype=np.float64)
    return theta ** (-2.0 * i / head_dim)


def rope(x, pos, theta: float, dt=np.float64) -> np.ndarray:
    """Rotate-half rotary embedding.

    x   : [..., n_heads, head_dim]
    pos : int array broadcastable to x's leading axes (one position per row)
    Pair (j, j + d/2) turns by the angle pos * theta^(-2j/d).  The angles and
    their cosines and sines are taken in float64; the rotation runs in dtype
    dt (with float32 the factors are first rounded to float32).
    """
    x = np.asarray(x, dtype=dt)
    d = x.shape[-1]
    half = d // 2
    ang = np.asarray(pos, dtype=np.float64)[..., None, None] * rope_inv_freq(d, theta)
    c, s = np.cos(ang).astype(dt), np.sin(ang).astype(dt)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


# ------------------------------------------------------------------ MLP
def silu(z, dt=np.float64) -> np.ndarray:
    z = np.asarray(z, dtype=dt)
    with np.errstate(over="ignore"):
        return z / (dt(1.0) + np.exp(-z))


# ------------------------------------------------------------------ attention
def attend(q, K, V, dt=np.float64) -> np.ndarray:
    """One query head over n keys: softmax(q.K^T / sqrt(d)) V.

    q [d], K [n, d], V [n, d] -> [d]  (max-subtracted softmax, in dtype dt).
    """
    q = np.asarray(q, dtype=dt)
    d = q.shape[-1]
    s = (np.asarray(K, dtype=dt) @ q) / dt(np.sqrt(d))
    p = np.exp(s - np.max(s))
    p /= np.sum(p, dtype=dt)
    return p @ np.asarray(V, dtype=dt)


def attention_weights(q, K) -> np.ndarray:
    """The softmax row of attend(), exposed for invariant tests."""
    q = np.asarray(q, dtype=np.float64)
    s = (np.asarray(K, dtype=np.float64) @ q) / np.sqrt(q.shape[-1])
    p = np.exp(s - np.max(s))
    return p / np.sum(p)


# ------------------------------------------------------------------ greedy
def argmax_lowest(z) -> np.ndarray:
    """Per row, the lowest index attaining the maximum; NaN never wins.

    An all-NaN row returns index 0.
    """
    z = np.asarray(z, dtype=np.float64)
    zz = np.where(np.isnan(z), -np.inf, z)
    out = np.argmax(zz, axis=-1)  # numpy returns the first maximal index
    return out.astype(np.int32)
