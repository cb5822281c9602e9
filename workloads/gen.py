"""Seeded, counter-based synthetic input generators.

This module holds no arithmetic of the decode step itself.  It only turns
(seed, tensor key, element index) into input values, so that the device
side (torch on the GPU) and the CPU oracle can each materialise exactly the
same bf16 tensors, or any slice of them, without shipping gigabytes between
them.

Definition of one generated element
-----------------------------------
* ``key``   : a 32-bit tensor key, ``key_of(seed, *labels)``.
* ``i``     : the element's flat index in the tensor (row-major), < 2**48.
* ``h``     : ``mix32(((i mod 2**32) * 0x9E3779B1 mod 2**32) XOR k_hi)`` where
              ``k_hi = mix32(key XOR mix32((i >> 32) + 0x85EBCA6B))``.
* value     : ``TABLE_sigma[h >> 16]``, a bf16 bit pattern.

``mix32`` is the "lowbias32" integer finaliser published by C. Wellons
(hash-prospector): x ^= x>>16; x *= 0x7feb352d; x ^= x>>15; x *= 0x846ca68b;
x ^= x>>16 (all mod 2**32).  ``TABLE_sigma[j]`` is the bf16 (round to
nearest even, through float32) of ``sigma * Phi^-1((j + 0.5) / 65536)``: a
65536-level quantised normal distribution N(0, sigma^2), truncated at about
4.3 sigma.  Integer-valued tables (``TABLE_INT``) are used by tests that need
exact fp32 sums.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

M32 = 0xFFFFFFFF
_C_LO = 0x9E3779B1
_C_HI = 0x85EBCA6B
_C1 = 0x7FEB352D
_C2 = 0x846CA68B
TABLE_BITS = 16
TABLE_SIZE = 1 << TABLE_BITS


def mix32_int(x: int) -> int:
    """lowbias32 on a Python int (scalar path, used for key derivation)."""
    x &= M32
    x ^= x >> 16
    x = (x * _C1) & M32
    x ^= x >> 15
    x = (x * _C2) & M32
    x ^= x >> 16
    return x


def key_of(seed: int, *labels) -> int:
    """32-bit tensor key from a seed and a tuple of ints/strings."""
    k = mix32_int(seed ^ 0x5BD1E995)
    for lab in labels:
        if isinstance(lab, str):
            v = 0
            for ch in lab.encode():
                v = mix32_int(v ^ ch) + 1
        else:
            v = int(lab)
        # 64-bit labels are folded in two halves
        k = mix32_int(k ^ mix32_int(v & M32))
        k = mix32_int(k ^ mix32_int((v >> 32) + 0x27D4EB2F))
    return k


# ---------------------------------------------------------------- tables
_TABLES: dict = {}


def _f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def normal_table(sigma: float) -> np.ndarray:
    """bf16 bit patterns of the 65536 quantiles of N(0, sigma^2)."""
    key = ("normal", float(sigma))
    t = _TABLES.get(key)
    if t is None:
        from scipy.special import ndtri
        p = (np.arange(TABLE_SIZE, dtype=np.float64) + 0.5) / TABLE_SIZE
        t = _f32_to_bf16_bits((sigma * ndtri(p)).astype(np.float32))
        t.setflags(write=False)
        _TABLES[key] = t
    return t


def int_table(lo: int, hi: int) -> np.ndarray:
    """bf16 bit patterns of small integers lo..hi spread evenly over 65536 slots."""
    key = ("int", lo, hi)
    t = _TABLES.get(key)
    if t is None:
        n = hi - lo + 1
        vals = lo + (np.arange(TABLE_SIZE) * n) // TABLE_SIZE
        t = _f32_to_bf16_bits(vals.astype(np.float32))
        t.setflags(write=False)
        _TABLES[key] = t
    return t


def table_for(dist) -> np.ndarray:
    """dist: ('normal', sigma) or ('int', lo, hi)."""
    if dist[0] == "normal":
        return normal_table(dist[1])
    if dist[0] == "int":
        return int_table(dist[1], dist[2])
    raise ValueError(dist)


# ---------------------------------------------------------------- numpy path
def _mix32_np(x: np.ndarray) -> np.ndarray:
    x = x ^ (x >> np.uint32(16))
    x = x * np.uint32(_C1)
    x = x ^ (x >> np.uint32(15))
    x = x * np.uint32(_C2)
    x = x ^ (x >> np.uint32(16))
    return x


def hash_np(key: int, start: int, n: int) -> np.ndarray:
    """uint32 hashes of element indices start..start+n-1 (n small enough for RAM)."""
    out = np.empty(n, np.uint32)
    i = start
    pos = 0
    while pos < n:
        hi = i >> 32
        lo0 = i & M32
        take = min(n - pos, (1 << 32) - lo0)
        k_hi = np.uint32(mix32_int(key ^ mix32_int(hi + _C_HI)))
        lo = np.arange(lo0, lo0 + take, dtype=np.uint64).astype(np.uint32)
        with np.errstate(over="ignore"):
            out[pos:pos + take] = _mix32_np((lo * np.uint32(_C_LO)) ^ k_hi)
        pos += take
        i += take
    return out


_CHUNK = 1 << 20


def _threads() -> int:
    n = len(os.sched_getaffinity(0))
    return max(1, min(16, n))


_POOL = None


def _pool() -> ThreadPoolExecutor:
    """One worker pool for the process (starting threads per call is slow)."""
    global _POOL
    if _POOL is None:
        _POOL = ThreadPoolExecutor(_threads())
    return _POOL


def bf16_bits_np(key: int, n: int, dist=("normal", 0.02), start: int = 0) -> np.ndarray:
    """n generated bf16 bit patterns (uint16) for elements start..start+n-1."""
    table = table_for(dist)
    out = np.empty(n, np.uint16)

    def work(c0):
        c1 = min(n, c0 + _CHUNK)
        h = hash_np(key, start + c0, c1 - c0)
        np.take(table, (h >> np.uint32(16)), out=out[c0:c1])

    starts = range(0, n, _CHUNK)
    if n > 4 * _CHUNK:
        list(_pool().map(work, starts))
    else:
        for c0 in starts:
            work(c0)
    return out


def bf16_values_np(key: int, n: int, dist=("normal", 0.02), start: int = 0, dtype=np.float64) -> np.ndarray:
    """The same elements as bf16_bits_np, widened exactly to float64 (or float32),
    chunk by chunk on the thread pool."""
    table = table_for(dist)
    vals = (table.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(dtype)
    out = np.empty(n, dtype)

    def work(c0):
        c1 = min(n, c0 + _CHUNK)
        h = hash_np(key, start + c0, c1 - c0)
        np.take(vals, (h >> np.uint32(16)), out=out[c0:c1])

    starts = range(0, n, _CHUNK)
    if n > 4 * _CHUNK:
        list(_pool().map(work, starts))
    else:
        for c0 in starts:
            work(c0)
    return out


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float64."""
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


# ---------------------------------------------------------------- torch path
def _mix32_t(x):
    import torch  # noqa: F401
    x = x ^ (x >> 16)
    x = _mul32_t(x, _C1)
    x = x ^ (x >> 15)
    x = _mul32_t(x, _C2)
    x = x ^ (x >> 16)
    return x


def _mul32_t(x, c: int):
    """(x * c) mod 2**32 for int64 tensors holding values in [0, 2**32) without overflow."""
    lo = (x & 0xFFFF) * c                 # < 2**48
    hi = ((x >> 16) * c) & 0xFFFF         # only the low 16 bits survive the << 16
    return (lo + (hi << 16)) & M32


def bf16_tensor(key: int, shape, dist=("normal", 0.02), device="cuda", start: int = 0):
    """torch.bfloat16 tensor of the given shape with the same values as bf16_bits_np."""
    import torch
    n = 1
    for s in shape:
        n *= int(s)
    table = torch.from_numpy(table_for(dist).view(np.int16).copy()).to(device)
    out = torch.empty(n, dtype=torch.int16, device=device)
    chunk = 1 << 26
    for c0 in range(0, n, chunk):
        c1 = min(n, c0 + chunk)
        i0 = start + c0
        # split at 2**32 boundaries of the element index
        p = c0
        i = i0
        while p < c1:
            hi = i >> 32
            lo0 = i & M32
            take = min(c1 - p, (1 << 32) - lo0)
            k_hi = mix32_int(key ^ mix32_int(hi + _C_HI))
            lo = torch.arange(lo0, lo0 + take, dtype=torch.int64, device=device)
            h = _mix32_t(_mul32_t(lo, _C_LO) ^ k_hi)
            out[p:p + take] = table[h >> 16]
            p += take
            i += take
    return out.view(torch.bfloat16).view(*shape)
