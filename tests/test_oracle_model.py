"""Pins of the oracle's whole pass.

The main pin is a textbook full-sequence forward written with torch's own
building blocks (rms_norm, scaled_dot_product_attention with a causal mask
and grouped KV heads, silu), recomputing every position from scratch with
no cache.  The oracle instead runs a cached prefill then decode steps over
a paged, permuted block table.  Agreement pins the cache writes, the
position bookkeeping, the rotary convention, the GQA head map, the
rounding points and the residual/MLP wiring at once.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import numerics as nm
from oracle.kvcache import BlockAllocator, PagedKV, build_batch
from oracle.model import GeneratedWeights, forward
from workloads.configs import ModelCfg

PIN = ModelCfg("pin-2L", n_layers=2, hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=16, ffn=96,
               vocab=97, rope_theta=10000.0, weight_sigma=0.25)


def bf16r_indep(t: torch.Tensor) -> torch.Tensor:
    """Exact float64 -> bf16 rounding written independently: scale by the ulp, round half to even."""
    x = t.numpy()
    out = np.zeros_like(x)
    nz = x != 0
    e = np.floor(np.log2(np.abs(x[nz])))
    ulp = np.exp2(e - 7)
    out[nz] = np.round(x[nz] / ulp) * ulp
    return torch.from_numpy(out)


def rope_t(x, pos, theta):
    """Rotary embedding as a complex rotation of (x_j, x_{j+d/2})."""
    d = x.shape[-1]
    z = torch.complex(x[..., : d // 2], x[..., d // 2:])
    ang = pos[:, None, None].double() * theta ** (-torch.arange(0, d, 2, dtype=torch.float64) / d)
    w = z * torch.polar(torch.ones_like(ang), ang)
    return torch.cat([w.real, w.imag], dim=-1)


def textbook_forward(m, W, tokens):
    """Full causal forward over a whole token sequence; returns per-layer (k, v) and last-row z."""
    T = len(tokens)
    g = lambda n, l=-1: torch.from_numpy(W.get(n, l))
    x = torch.from_numpy(W.rows("embed", tokens))
    pos = torch.arange(T)
    kvs = []
    for l in range(m.n_layers):
        h = bf16r_indep(F.rms_norm(x, (m.hidden,), g("attn_norm", l), eps=m.rms_eps))
        q = (h @ g("wq", l).T).view(T, m.n_q_heads, m.head_dim)
        k = (h @ g("wk", l).T).view(T, m.n_kv_heads, m.head_dim)
        v = (h @ g("wv", l).T).view(T, m.n_kv_heads, m.head_dim)
        q = bf16r_indep(rope_t(q, pos, m.rope_theta))
        k = bf16r_indep(rope_t(k, pos, m.rope_theta))
        v = bf16r_indep(v)
        kvs.append((k.numpy(), v.numpy()))
        o = F.scaled_dot_product_attention(q.transpose(0, 1)[None], k.transpose(0, 1)[None],
                                           v.transpose(0, 1)[None], is_causal=True, enable_gqa=True)
        o = bf16r_indep(o[0].transpose(0, 1).reshape(T, -1))
        x = x + o @ g("wo", l).T
        h2 = bf16r_indep(F.rms_norm(x, (m.hidden,), g("mlp_norm", l), eps=m.rms_eps))
        a = bf16r_indep(F.silu(h2 @ g("w_gate", l).T) * (h2 @ g("w_up", l).T))
        x = x + a @ g("w_down", l).T
    hf = bf16r_indep(F.rms_norm(x[-1:], (m.hidden,), g("final_norm"), eps=m.rms_eps))
    z = hf @ torch.from_numpy(W.get("lm_head")).T
    return kvs, z[0].numpy()


def run_oracle_sequence(m, W, tokens, prefill_len, table_perm, n_blocks=16):
    """Cached prefill of the first prefill_len tokens, then one decode step per remaining token."""
    a = BlockAllocator(n_blocks, 16)
    a.seq_create(0)
    nb = (len(tokens) + 15) // 16
    a.seq_set_blocks(0, table_perm[:nb], 0)
    kv = PagedKV(m.n_layers, n_blocks, m.n_kv_heads, m.head_dim)
    a.reserve(0, prefill_len)
    b = build_batch(a, [0], [prefill_len])
    outs = [forward(m, W, kv, b, tokens[:prefill_len], [prefill_len - 1])]
    for t in range(prefill_len, len(tokens)):
        a.reserve(0, 1)
        b = build_batch(a, [0], [1])
        outs.append(forward(m, W, kv, b, tokens[t:t + 1], [0]))
    return a, kv, outs


@pytest.mark.parametrize("perm_seed", [0, 1])
def test_oracle_matches_textbook_forward(perm_seed):
    m = PIN
    # random norm gains, so a dropped, swapped or misplaced gain changes the result
    g = np.random.default_rng(30 + perm_seed)
    gains = {(n, l): g.uniform(0.5, 1.5, m.hidden) for n in ("attn_norm", "mlp_norm") for l in range(m.n_layers)}
    gains[("final_norm", -1)] = g.uniform(0.5, 1.5, m.hidden)
    W = GeneratedWeights(m, seed=11, overrides=gains, cache=True)
    rng = np.random.default_rng(3)
    tokens = rng.integers(0, m.vocab, size=37)
    perm = list(np.random.default_rng(perm_seed).permutation(16))
    a, kv, outs = run_oracle_sequence(m, W, tokens, 33, perm)
    # logits after the prefill and after each decode step
    for i, T in enumerate(range(33, 38)):
        kvs, z_ref = textbook_forward(m, W, tokens[:T])
        z = outs[i]["z"][0]
        np.testing.assert_allclose(z, z_ref, rtol=0, atol=1e-9)
        assert outs[i]["ids"][0] == int(np.argmax(z_ref))
    # the cache holds every layer's own K, V for every position (Invariant 1)
    slots = [a.slot(0, p) for p in range(37)]
    for l in range(m.n_layers):
        K, V = kv.read(l, slots)
        np.testing.assert_allclose(K, kvs[l][0], rtol=0, atol=1e-12)
        np.testing.assert_allclose(V, kvs[l][1], rtol=0, atol=1e-12)


def test_block_permutation_is_bit_invariant():
    m = PIN
    W = GeneratedWeights(m, seed=5, cache=True)
    tokens = np.random.default_rng(9).integers(0, m.vocab, size=40)
    _, _, o1 = run_oracle_sequence(m, W, tokens, 38, list(range(16)))
    _, _, o2 = run_oracle_sequence(m, W, tokens, 38, list(np.random.default_rng(4).permutation(16)))
    for x, y in zip(o1, o2):
        np.testing.assert_array_equal(x["z"], y["z"])


def test_batch_independence():
    m = PIN
    W = GeneratedWeights(m, seed=6, cache=True)
    rng = np.random.default_rng(10)
    ctx = [20, 33, 5]
    kv = PagedKV(m.n_layers, 16, m.n_kv_heads, m.head_dim)
    a = BlockAllocator(16, 16)
    for s, c in enumerate(ctx):
        a.seq_create(s)
        a.reserve(s, c)
        for l in range(m.n_layers):
            slots = [a.slot(s, p) for p in range(c)]
            kv.write(l, slots, rng.standard_normal((c, 2, 16)), rng.standard_normal((c, 2, 16)))
    for s in range(3):
        a.reserve(s, 1)
    tok = rng.integers(0, m.vocab, size=3)
    kv_copy = PagedKV(m.n_layers, 16, m.n_kv_heads, m.head_dim)
    kv_copy.K[:] = kv.K
    kv_copy.V[:] = kv.V
    full = forward(m, W, kv, build_batch(a, [0, 1, 2], [1, 1, 1]), tok, [0, 1, 2])
    one = forward(m, W, kv_copy, build_batch(a, [1], [1]), tok[1:2], [0])
    np.testing.assert_allclose(full["z"][1], one["z"][0], rtol=0, atol=1e-12)


def test_zero_mixing_reduces_to_norm_of_embedding():
    """Wo = Wd = 0 leaves x = E[t], so z = R(RMSNorm(E[t])) Wlm^T."""
    m = PIN
    over = {}
    for l in range(m.n_layers):
        over[("wo", l)] = np.zeros((m.hidden, m.q_dim))
        over[("w_down", l)] = np.zeros((m.hidden, m.ffn))
    W = GeneratedWeights(m, seed=2, overrides=over, cache=True)
    tokens = np.array([3, 50, 96])
    kv = PagedKV(m.n_layers, 4, m.n_kv_heads, m.head_dim)
    a = BlockAllocator(4, 16)
    for s in range(3):
        a.seq_create(s)
        a.reserve(s, 1)
    out = forward(m, W, kv, build_batch(a, [0, 1, 2], [1, 1, 1]), tokens, [0, 1, 2])
    E = torch.from_numpy(W.rows("embed", tokens))
    hf = bf16r_indep(F.rms_norm(E, (m.hidden,), eps=m.rms_eps))
    z_ref = (hf @ torch.from_numpy(W.get("lm_head")).T).numpy()
    np.testing.assert_allclose(out["z"], z_ref, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(out["logits"], nm.bf16_round(out["z"]))


def test_first_token_attends_to_itself_only():
    """With no cached context the attention output is the new row's own v."""
    m = ModelCfg("pin-1L", 1, 32, 2, 2, 16, 64, 31, rope_theta=10000.0, weight_sigma=0.3)
    H = m.hidden
    over = {("wo", 0): np.eye(H), ("w_down", 0): np.zeros((H, m.ffn))}
    W = GeneratedWeights(m, seed=8, overrides=over)
    kv = PagedKV(1, 2, 2, 16)
    a = BlockAllocator(2, 16)
    a.seq_create(0)
    a.reserve(0, 1)
    tok = np.array([7])
    out = forward(m, W, kv, build_batch(a, [0], [1]), tok, [0], want_hidden=True)
    x0 = W.rows("embed", tok)
    h = nm.bf16_round(nm.rmsnorm(x0, np.ones(H), m.rms_eps))
    v = nm.bf16_round(h @ W.get("wv", 0).T)
    # q heads 0,1 map to kv heads 0,1; o = v, then x = x0 + o (Wo = I)
    np.testing.assert_allclose(out["x"], x0 + v, rtol=0, atol=1e-12)


def test_layer_range_composes_to_the_whole_pass():
    """Running layers [0, k) then [k, L) from the first part's residual is the whole pass."""
    m = PIN
    W = GeneratedWeights(m, seed=21, cache=True)
    tokens = np.random.default_rng(22).integers(0, m.vocab, size=20)
    perm = list(range(16))
    a = BlockAllocator(16, 16)
    a.seq_create(0)
    a.seq_set_blocks(0, perm[:2], 0)
    a.reserve(0, 20)
    b = build_batch(a, [0], [20])
    kv1 = PagedKV(m.n_layers, 16, m.n_kv_heads, m.head_dim)
    kv2 = PagedKV(m.n_layers, 16, m.n_kv_heads, m.head_dim)
    full = forward(m, W, kv1, b, tokens, [19], want_hidden=True)
    part = forward(m, W, kv2, b, tokens, None, layers=[0])
    rest = forward(m, W, kv2, b, tokens, [19], x0=part["x"], layers=[1], want_hidden=True)
    np.testing.assert_array_equal(full["x"], rest["x"])
    np.testing.assert_array_equal(full["z"], rest["z"])
    np.testing.assert_array_equal(kv1.K, kv2.K)


# ---------------------------------------------------------------- float32 contract mode
def _int_pass(m, variant, dtype, rows=5, seed=0):
    from intcase import fresh_workload, int_overrides
    from helpers import oracle_state
    w = fresh_workload(m, rows, seed=seed)
    W = GeneratedWeights(m, w.seed, overrides=int_overrides(m, variant, seed=seed))
    a, batch, sub, r, kv, idx = oracle_state(w)
    out = forward(m, W, kv, sub, w.tokens[r], np.arange(rows), want_hidden=True, dtype=dtype)
    K, V = kv.read(0, sub["slot"])
    return out, K, V


@pytest.mark.parametrize("variant", ["qkv", "o", "mlp"])
def test_f32_contract_mode_equals_float64_on_exact_inputs(variant):
    """On inputs whose every sum is an exact integer (tests/intcase.py) the
    float32 contract mode and the float64 definition must agree bit for bit:
    any formula the float32 path states differently shows up here."""
    m = PIN
    o64, K64, V64 = _int_pass(m, variant, "f64")
    o32, K32, V32 = _int_pass(m, variant, "f32")
    np.testing.assert_array_equal(K32, K64)
    np.testing.assert_array_equal(V32, V64)
    np.testing.assert_array_equal(o32["x"], o64["x"])
    assert np.all(K64 == np.round(K64)) and np.all(V64 == np.round(V64))
    if variant == "qkv":
        np.testing.assert_array_equal(o32["z"], o64["z"])
        np.testing.assert_array_equal(o32["ids"], o64["ids"])
        assert np.all(o64["z"] == np.round(o64["z"]))
    else:
        assert np.all(o64["x"] == np.round(o64["x"]))
        assert np.abs(o64["x"] - np.round(o64["x"])).max() == 0 and np.abs(o64["x"]).max() > 2


def test_f32_contract_mode_runs_in_float32_and_stays_close():
    """On generic inputs the float32 mode differs from the float64 one (it is
    not silently the same computation), holds float32 values only, and stays
    close on a 2-layer model (a bf16 rounding flip moves some logits by a few
    hundredths; the mean moves by much less)."""
    m = PIN
    W = GeneratedWeights(m, seed=41, cache=True)
    tokens = np.random.default_rng(42).integers(0, m.vocab, size=30)
    res = {}
    for dt in ("f64", "f32"):
        a = BlockAllocator(16, 16)
        a.seq_create(0)
        a.seq_set_blocks(0, list(range(2)), 0)
        a.reserve(0, 30)
        b = build_batch(a, [0], [30])
        kv = PagedKV(m.n_layers, 16, m.n_kv_heads, m.head_dim)
        res[dt] = forward(m, W, kv, b, tokens, np.arange(30), want_hidden=True, dtype=dt)
    x32, z32 = res["f32"]["x"], res["f32"]["z"]
    np.testing.assert_array_equal(x32, x32.astype(np.float32).astype(np.float64))
    np.testing.assert_array_equal(z32, z32.astype(np.float32).astype(np.float64))
    assert not np.array_equal(res["f64"]["x"], x32)
    d = np.abs(z32 - res["f64"]["z"])
    assert d.max() <= 0.1 and d.mean() <= 5e-3, (d.max(), d.mean())
