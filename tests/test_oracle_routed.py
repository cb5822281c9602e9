"""Pins of the oracle's routed mode (Algorithm 1; Section 3.1; appendices
"Route-Guided Cohort Execution at the Kernel Level" and "A Minimal Skipper
Plugin").

The main pin is a textbook full-sequence forward written with torch's own
building blocks in which a routed layer is a mask, not a cohort: every row
runs attention, MLP and projector, a Project-Only row's attention output is
replaced by zero, and the residual takes w * MLP where the row runs and
(1 - w) * projector where it projects.  The oracle instead gathers the two
cohorts through Algorithm 1's maps, skips the Project-Only rows' attention
and scatters the weighted results back, over a cached prefill and decode
steps on a permuted block table.  Agreement pins the maps, the masking of
the attention, the KV writes of Project-Only rows (later tokens attend to
them), the weights and the projector wiring.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle.kvcache import BlockAllocator, PagedKV, build_batch
from oracle.model import GeneratedWeights, forward, route_maps
from workloads import routes
from workloads.configs import ModelCfg

from test_oracle_model import bf16r_indep, rope_t

# 3 layers, the last 2 routed, projector width 32
PINR = ModelCfg("pinr-3L", n_layers=3, hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=16, ffn=96,
                vocab=97, rope_theta=10000.0, weight_sigma=0.25, routed_layers=2, proj_ffn=32)


def textbook_routed(m, W, tokens, run, w):
    """Full causal forward; run/w [n_routed][T] per token.  Returns per-layer (k, v) and z of every row."""
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
        o = o[0].transpose(0, 1).reshape(T, -1)
        lr = l - m.first_routed
        if lr >= 0:
            keep = torch.from_numpy(run[lr].astype(np.float64))[:, None]
            o = o * keep
        o = bf16r_indep(o)
        x = x + o @ g("wo", l).T
        h2 = bf16r_indep(F.rms_norm(x, (m.hidden,), g("mlp_norm", l), eps=m.rms_eps))
        mlp = bf16r_indep(F.silu(h2 @ g("w_gate", l).T) * (h2 @ g("w_up", l).T)) @ g("w_down", l).T
        if lr >= 0:
            prj = bf16r_indep(F.silu(h2 @ g("p_gate", l).T) * (h2 @ g("p_up", l).T)) @ g("p_down", l).T
            rr = torch.from_numpy(run[lr])[:, None]
            ww = torch.from_numpy(w[lr].astype(np.float64))[:, None]
            x = x + torch.where(rr, ww * mlp, (1 - ww) * prj)
        else:
            x = x + mlp
    hf = bf16r_indep(F.rms_norm(x, (m.hidden,), g("final_norm"), eps=m.rms_eps))
    z = hf @ torch.from_numpy(W.get("lm_head")).T
    return kvs, z.numpy()


def oracle_routed_sequence(m, W, tokens, prefill_len, perm, run, w, n_blocks=16):
    """Cached prefill then decode steps, each pass given its rows' slice of the tape."""
    a = BlockAllocator(n_blocks, 16)
    a.seq_create(0)
    a.seq_set_blocks(0, perm[:(len(tokens) + 15) // 16], 0)
    kv = PagedKV(m.n_layers, n_blocks, m.n_kv_heads, m.head_dim)
    a.reserve(0, prefill_len)
    b = build_batch(a, [0], [prefill_len])
    sl = slice(0, prefill_len)
    outs = [forward(m, W, kv, b, tokens[sl], [prefill_len - 1], route=(run[:, sl], w[:, sl]))]
    for t in range(prefill_len, len(tokens)):
        a.reserve(0, 1)
        b = build_batch(a, [0], [1])
        outs.append(forward(m, W, kv, b, tokens[t:t + 1], [0], route=(run[:, t:t + 1], w[:, t:t + 1])))
    return a, kv, outs


@pytest.mark.parametrize("policy", ["router", "random", "static_half", "all_po"])
def test_routed_oracle_matches_textbook_masking(policy):
    m = PINR
    T, P = 37, 33
    W = GeneratedWeights(m, seed=51, cache=True)
    tokens = np.random.default_rng(52).integers(0, m.vocab, size=T)
    if policy == "router":
        run, w = routes.router_weights(53, m.n_routed, T)
    elif policy == "random":
        run, w = routes.random_skip(54, m.n_routed, np.zeros(T, np.int64), np.arange(T), 1.0, 0.5)
    elif policy == "static_half":
        run, w = routes.static_depth(m.n_routed, T, 0.5)
    else:
        run, w = routes.static_depth(m.n_routed, T, 1.0)
    assert run.any() or policy == "all_po"
    perm = list(np.random.default_rng(55).permutation(16))
    a, kv, outs = oracle_routed_sequence(m, W, tokens, P, perm, run, w)
    kvs, z_ref = textbook_routed(m, W, tokens, run, w.astype(np.float64))
    for i, t in enumerate(range(P - 1, T)):
        np.testing.assert_allclose(outs[i]["z"][0], z_ref[t], rtol=0, atol=1e-9)
    slots = [a.slot(0, p) for p in range(T)]
    for l in range(m.n_layers):  # Project-Only rows wrote their K, V too (Invariant 1)
        K, V = kv.read(l, slots)
        np.testing.assert_allclose(K, kvs[l][0], rtol=0, atol=1e-12)
        np.testing.assert_allclose(V, kvs[l][1], rtol=0, atol=1e-12)


def _decode_batch(m, ctx, seed):
    rng = np.random.default_rng(seed)
    n_blocks = sum((c + 16) // 16 for c in ctx) + 4
    a = BlockAllocator(n_blocks, 16)
    kv = PagedKV(m.n_layers, n_blocks, m.n_kv_heads, m.head_dim)
    for s, c in enumerate(ctx):
        a.seq_create(s)
        a.reserve(s, c)
        for l in range(m.n_layers):
            sl = [a.slot(s, p) for p in range(c)]
            kv.write(l, sl, rng.standard_normal((c, m.n_kv_heads, m.head_dim)),
                     rng.standard_normal((c, m.n_kv_heads, m.head_dim)))
    for s in range(len(ctx)):
        a.reserve(s, 1)
    b = build_batch(a, list(range(len(ctx))), [1] * len(ctx))
    return a, b, kv, rng.integers(0, m.vocab, size=len(ctx))


def _copy_kv(kv):
    import copy
    return copy.deepcopy(kv)


def test_all_run_with_unit_weight_is_dense_bit_for_bit():
    m = PINR
    W = GeneratedWeights(m, seed=61, cache=True)
    a, b, kv, tok = _decode_batch(m, [5, 40, 17, 0], 62)
    kv2 = _copy_kv(kv)
    dense = forward(m, W, kv, b, tok, np.arange(4), want_hidden=True)
    routed = forward(m, W, kv2, b, tok, np.arange(4), want_hidden=True, route=routes.all_run(m.n_routed, 4))
    np.testing.assert_array_equal(dense["x"], routed["x"])
    np.testing.assert_array_equal(dense["z"], routed["z"])
    np.testing.assert_array_equal(kv.K, kv2.K)
    np.testing.assert_array_equal(kv.V, kv2.V)
    # StaticDepth at ratio 0 runs every routed layer
    kv3 = _copy_kv(kv)
    sd0 = forward(m, W, kv3, b, tok, np.arange(4), route=routes.static_depth(m.n_routed, 4, 0.0))
    np.testing.assert_array_equal(dense["z"], sd0["z"])


def test_project_only_with_zero_projector_leaves_the_residual():
    """All rows Project-Only at the last layer with a zero projector: the
    attention emits zero and the projector adds zero, so the residual leaving
    the layer is the residual entering it -- but the layer's K, V are written."""
    m = PINR
    L = m.n_layers
    over = {("p_down", L - 1): np.zeros((m.hidden, m.proj_dim))}
    W = GeneratedWeights(m, seed=63, overrides=over, cache=True)
    a, b, kv, tok = _decode_batch(m, [9, 30, 1], 64)
    run = np.ones((m.n_routed, 3), bool)
    run[-1] = False
    wts = np.where(run, 1.0, 0.0).astype(np.float32)
    kv_a = _copy_kv(kv)
    before = forward(m, W, kv_a, b, tok, None, layers=range(L - 1), route=(run, wts))
    kv_b = _copy_kv(kv_a)
    after = forward(m, W, kv_b, b, tok, None, x0=before["x"], layers=[L - 1], route=(run, wts))
    np.testing.assert_array_equal(after["x"], before["x"])
    # the K, V written at the last layer are those of its own projections
    kv_c = _copy_kv(kv_a)
    forward(m, W, kv_c, b, tok, None, x0=before["x"], layers=[L - 1])  # dense: same K, V
    np.testing.assert_array_equal(kv_b.K[L - 1], kv_c.K[L - 1])
    np.testing.assert_array_equal(kv_b.V[L - 1], kv_c.V[L - 1])
    assert not np.array_equal(kv_b.K[L - 1], kv_a.K[L - 1])


def test_route_maps_partition_the_rows():
    rng = np.random.default_rng(70)
    for n in [0, 1, 2, 17, 130]:
        mask = rng.random(n) < 0.4
        run, proj, n_r, n_p = route_maps(mask)
        assert n_r + n_p == n
        assert sorted(np.concatenate([run, proj]).tolist()) == list(range(n))
        assert all(mask[i] for i in run) and not any(mask[i] for i in proj)
        assert list(run) == sorted(run) and list(proj) == sorted(proj)


def test_policies():
    run, w = routes.static_depth(16, 5, 0.5)
    assert run[:8].all() and not run[8:].any() and (w == run).all()
    assert routes.static_depth(16, 5, 1.0)[0].sum() == 0
    assert routes.static_depth(16, 5, 0.0)[0].all()
    run, w = routes.random_skip(1, 16, np.arange(400) // 4, np.arange(400) % 4, 0.5, 0.5)
    share = 1 - run.mean()
    assert abs(share - 0.25) < 0.05, share
    run2, _ = routes.random_skip(1, 16, np.arange(400) // 4, np.arange(400) % 4, 0.5, 0.5)
    assert (run == run2).all()
    run, w = routes.router_weights(3, 4, 100)
    assert (run == (w > 0.5)).all()
