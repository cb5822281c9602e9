"""Routed mode on the device (Algorithm 1) against the oracle, through the C ABI.

  * maps: the device's run[] / proj[] / inv[] / counts of every routed layer
    equal the oracle's route_maps bit for bit (n_r + n_p = rows);
  * all rows RUN with w = 1: bit-identical to the dense pass (logits, ids,
    residual and every layer's K,V);
  * router weights, random skip, static depth and all Project-Only tapes:
    logits end to end against the oracle's routed pass (compare_logits), and
    every row's K,V at the first routed layer -- Project-Only rows included
    (Invariant 1) -- within one bf16 ulp;
  * row counts that take every launch shape of the count-bounded projections
    (1, 20, 70 and 130 rows: one row tile of 1, 2 and 8 row groups, and a
    row-tiled pass), cohorts of zero rows (whose launches read no weights);
  * routed prefill (a chunk of prompt rows beside decode rows);
  * full size: the 3B workload (14 of 28 layers routed, random skip s = 0.5)
    and the 8B workload (16 of 32), head on every row and end to end.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle.model import GeneratedWeights, forward, route_maps  # noqa: E402
from workloads import routes  # noqa: E402
from workloads.configs import ModelCfg, decode_workload, mixed_workload, prefix_groups_workload, workload  # noqa: E402

from helpers import assert_bf16_close, e2e_compare, oracle_state  # noqa: E402

pytestmark = pytest.mark.gpu

# 3 layers, the last 2 routed, projector width 128
MIDR = ModelCfg("midr-3L", n_layers=3, hidden=512, n_q_heads=8, n_kv_heads=2, head_dim=128, ffn=1536,
                vocab=2048, rope_theta=500000.0, routed_layers=2, proj_ffn=128)


def _tape(policy, m, w, seed=0):
    R = w.n_rows
    if policy == "all_run":
        return routes.all_run(m.n_routed, R)
    if policy == "router":
        return routes.router_weights(seed, m.n_routed, R)
    if policy == "random":
        req = np.repeat(np.arange(w.n_seqs), [s.q_len for s in w.seqs])
        pos = np.concatenate([np.arange(s.ctx, s.ctx + s.q_len) for s in w.seqs])
        return routes.random_skip(seed, m.n_routed, req, pos, 0.5, 1.0)
    if policy == "static_half":
        return routes.static_depth(m.n_routed, R, 0.5)
    if policy == "all_po":
        return routes.static_depth(m.n_routed, R, 1.0)
    raise ValueError(policy)


def _first_routed_kv(d, w, tape, subset):
    """K,V the first routed layer wrote for the subset's rows -- Project-Only
    rows included (Invariant 1) -- against the oracle applied to that layer
    alone from the device's own input residual: within one bf16 ulp."""
    m = w.model
    d.set_layers(m.first_routed)
    d.step_routed()
    x_in = d.residual()
    d.set_layers(0)
    d.step_routed()
    a, batch, sub, rows, kv, idx = oracle_state(w, subset)
    W = GeneratedWeights(m, w.seed)
    tape_sub = (np.asarray(tape[0])[:, rows], np.asarray(tape[1])[:, rows])
    forward(m, W, kv, sub, w.tokens[rows], None, x0=x_in[rows], layers=[m.first_routed], route=tape_sub)
    K, V = d.read_kv(m.first_routed, sub["slot"])
    Ko, Vo = kv.read(m.first_routed, sub["slot"])
    assert_bf16_close(K, Ko, "K first routed layer")
    assert_bf16_close(V, Vo, "V first routed layer")


def _device(w, **kw):
    from paper_2609_37062_amd.runner import DeviceRun
    print(f"[gpu] {w.name} rows={w.n_rows} routed", flush=True)
    kw.setdefault("poison_pool", True)
    return DeviceRun(w, routed=True, **kw)


@pytest.mark.parametrize("rows", [1, 20, 70, 130])
def test_all_run_unit_weight_is_the_dense_pass(rows):
    m = MIDR
    ctx = np.random.default_rng(rows).integers(0, 400, size=rows)
    w = decode_workload(m, ctx, seed=rows, name=f"routed-allrun-{rows}")
    d = _device(w)
    slots = d.eng.batch_host()["slot"]
    d.step()
    lg0, ids0 = d.results()
    x0 = d.residual()
    kv0 = [d.read_kv(l, slots) for l in range(m.n_layers)]
    d.set_route(*_tape("all_run", m, w))
    d.step_routed()
    lg1, ids1 = d.results()
    np.testing.assert_array_equal(lg0, lg1)
    np.testing.assert_array_equal(ids0, ids1)
    np.testing.assert_array_equal(x0, d.residual())
    for l in range(m.n_layers):
        K, V = d.read_kv(l, slots)
        np.testing.assert_array_equal(K, kv0[l][0])
        np.testing.assert_array_equal(V, kv0[l][1])
    run, proj, inv, cnt = d.route_maps()
    assert (cnt[:, 0] == rows).all() and (cnt[:, 1] == 0).all()
    d.release()


@pytest.mark.parametrize("rows", [1, 20, 70, 130])
@pytest.mark.parametrize("policy", ["router", "random", "static_half", "all_po"])
def test_routed_decode_matches_oracle(policy, rows):
    m = MIDR
    ctx = np.random.default_rng(10 + rows).integers(0, 400, size=rows)
    w = decode_workload(m, ctx, seed=10 + rows, name=f"routed-{policy}-{rows}")
    tape = _tape(policy, m, w, seed=rows)
    d = _device(w)
    d.set_route(*tape)
    d.step_routed()
    lg, ids = d.results()
    # the maps, bit for bit
    run, proj, inv, cnt = d.route_maps()
    for lr in range(m.n_routed):
        r_or, p_or, n_r, n_p = route_maps(tape[0][lr])
        assert (cnt[lr, 0], cnt[lr, 1]) == (n_r, n_p) and n_r + n_p == rows
        np.testing.assert_array_equal(run[lr, :n_r], r_or)
        np.testing.assert_array_equal(proj[lr, :n_p], p_or)
        np.testing.assert_array_equal(inv[lr, r_or], np.arange(n_r))
        np.testing.assert_array_equal(inv[lr, p_or], np.arange(n_p))
    subset = None if rows <= 20 else list(range(0, rows, max(1, rows // 12)))
    st, *_ = e2e_compare(w, lg, ids, subset, route=tape)
    print(f"[gpu] routed {policy} rows={rows}: {st} cohorts {cnt.tolist()}", flush=True)
    _first_routed_kv(d, w, tape, subset)
    # a replay is bit-identical
    d.step_routed()
    lg2, ids2 = d.results()
    np.testing.assert_array_equal(lg, lg2)
    np.testing.assert_array_equal(ids, ids2)
    d.release()


def test_routed_decode_with_shared_prefixes():
    """Shared-prefix groups in a routed pass (Project-Only members read no KV
    of their own and emit zero; the prefix partials of RUN members are folded
    in): end to end against the oracle, and a second pass bit-identical."""
    m = MIDR
    suf = np.random.default_rng(61).integers(1, 50, size=26)
    w = prefix_groups_workload(m, [(160, 20), (64, 3)], suf, seed=61, name="routed-groups")
    req = np.arange(w.n_seqs)
    pos = np.array([s.ctx for s in w.seqs])
    tape = routes.random_skip(5, m.n_routed, req, pos, 1.0, 0.5)
    d = _device(w)
    d.eng.set_tuning(0, 8)
    d.set_route(*tape)
    d.step_routed()
    lg, ids = d.results()
    st, *_ = e2e_compare(w, lg, ids, [0, 3, 19, 20, 22, 23, 25], route=tape)
    print(f"[gpu] routed groups: {st}", flush=True)
    d.step_routed()
    lg2, ids2 = d.results()
    np.testing.assert_array_equal(lg, lg2)
    np.testing.assert_array_equal(ids, ids2)
    d.release()


@pytest.mark.parametrize("policy", ["router", "all_po"])
def test_routed_prefill_matches_oracle(policy):
    m = MIDR
    ctx = np.random.default_rng(40).integers(10, 200, size=5)
    w = mixed_workload(m, n_pre=2, plen=45, ctx=ctx, seed=41, name=f"routed-prefill-{policy}")
    tape = _tape(policy, m, w, seed=42)
    d = _device(w)
    d.set_route(*tape)
    d.step_routed()
    lg, ids = d.results()
    st, *_ = e2e_compare(w, lg, ids, route=tape)
    print(f"[gpu] routed prefill {policy}: {st}", flush=True)
    _first_routed_kv(d, w, tape, None)
    d.release()


def test_routed_decode_graph_replay():
    """A routed decode pass (random skip, 70 rows; cohort counts read on the
    device by the count-bounded launches) captured in a graph: every replay,
    with eager passes between, reproduces the eager pass bit for bit."""
    from test_gpu_parity import _graph_replays_match
    m = MIDR
    ctx = np.random.default_rng(81).integers(0, 400, size=70)
    w = decode_workload(m, ctx, seed=81, name="routed-graph")
    tape = _tape("random", m, w, seed=82)
    d = _device(w)
    d.set_route(*tape)
    lg, ids = _graph_replays_match(d, d.step_routed)
    st, *_ = e2e_compare(w, lg, ids, list(range(0, 70, 7)), route=tape)
    print(f"[gpu] routed graph: {st}", flush=True)
    d.release()


@pytest.mark.parametrize("row_tile", [0, 7, 11])
def test_routed_prefill_row_tiled(row_tile):
    """Routed prefill of 405 rows (two 200-row prompts beside 5 decoding
    sequences): the cohort-bounded projections of a row-tiled pass at the
    default tile heights and with 7 and 11 row groups per tile (tuning key
    10; a tile starting at or past its cohort's count exits), end to end
    against the oracle and the first routed layer's K,V within one ulp."""
    m = MIDR
    ctx = np.random.default_rng(43).integers(10, 200, size=5)
    w = mixed_workload(m, n_pre=2, plen=200, ctx=ctx, seed=44, name=f"routed-prefill-rt{row_tile}")
    tape = _tape("random", m, w, seed=45)
    d = _device(w)
    d.eng.set_tuning(10, row_tile)
    d.set_route(*tape)
    d.step_routed()
    lg, ids = d.results()
    st, *_ = e2e_compare(w, lg, ids, route=tape)
    print(f"[gpu] routed prefill rows={w.n_rows} row_tile={row_tile}: {st}", flush=True)
    _first_routed_kv(d, w, tape, [0, 1, 2, 6])
    d.release()


@pytest.mark.parametrize("cfg,subset", [(2, [0, 15]), (5, [0, 77])])
def test_routed_full_size(cfg, subset):
    """Random skip (r = 1, d = 0.5: half the routed decisions project) over
    the routed half of the 3B / 8B models: the oracle's head on the device's
    final residual for every row within 2e-2, and end to end on sampled
    sequences."""
    from test_gpu_fullsize import head_all_rows
    w = workload(cfg)
    m = w.model
    req = np.arange(w.n_seqs)
    pos = np.array([s.ctx for s in w.seqs])
    tape = routes.random_skip(7, m.n_routed, req, pos, 1.0, 0.5)
    d = _device(w)
    d.set_route(*tape)
    d.step_routed()
    lg, ids = d.results()
    x_all = d.residual()
    W = GeneratedWeights(m, w.seed)
    head = head_all_rows(w, W, x_all, lg, ids)
    print(f"[gpu] routed {w.name} head: {head}", flush=True)
    st, *_ = e2e_compare(w, lg, ids, subset, route=tape)
    print(f"[gpu] routed {w.name} e2e: {st}; skip share {1 - tape[0].mean():.3f}", flush=True)
    d.release()
