"""Model shapes off the beaten path, end to end against the oracle: hidden
sizes that are not multiples of 256 (K steps not a multiple of the 8 K-split
waves, ragged activation chunks), query widths different from the hidden
size, GQA groups of 1, 3, 5 and 16, head dims 64 and 128, vocabularies of a
few 64-column tiles; decode passes at every launch-shape row class (1-16,
17-32, 33-64, 65-128, row-tiled) and a mixed prefill + decode pass.  Every
row writes its own K,V at every layer (Invariant 1), checked layer-local.
The model is the decoder of section 3 ("Design and Implementation")."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from workloads.configs import ModelCfg, decode_workload, mixed_workload  # noqa: E402

from helpers import assert_kv_layer_local, e2e_compare  # noqa: E402

pytestmark = pytest.mark.gpu

SHAPES = {
    # GQA 3, head_dim 64, query width = hidden = 192 (6 K steps)
    "h192-g3-d64": ModelCfg("h192-g3", n_layers=2, hidden=192, n_q_heads=3, n_kv_heads=1, head_dim=64, ffn=320,
                            vocab=192, rope_theta=10000.0),
    # GQA 16 (a full MFMA column tile of query heads), query width 1024 != hidden 320
    "h320-g16-d64": ModelCfg("h320-g16", n_layers=2, hidden=320, n_q_heads=16, n_kv_heads=1, head_dim=64, ffn=576,
                             vocab=320, rope_theta=10000.0),
    # multi-head (group 1), head_dim 128, query width 256 < hidden 448
    "h448-g1-d128": ModelCfg("h448-g1", n_layers=2, hidden=448, n_q_heads=2, n_kv_heads=2, head_dim=128, ffn=704,
                             vocab=448, rope_theta=500000.0),
    # GQA 5, query width 1280 > hidden 256, ffn 1088 (17 tiles of 64)
    "h256-g5-d128": ModelCfg("h256-g5", n_layers=2, hidden=256, n_q_heads=10, n_kv_heads=2, head_dim=128, ffn=1088,
                             vocab=832, rope_theta=500000.0),
}


def _run(w):
    from paper_2609_37062_amd.runner import DeviceRun
    print(f"[gpu] {w.name} seqs={w.n_seqs} rows={w.n_rows}", flush=True)
    d = DeviceRun(w, poison_pool=True)
    d.step()
    lg, ids = d.results()
    return d, lg, ids


@pytest.mark.parametrize("shape", list(SHAPES))
@pytest.mark.parametrize("B", [1, 7, 17, 40, 70, 130])
def test_odd_shape_decode(shape, B):
    m = SHAPES[shape]
    ctx = np.random.default_rng(B).integers(0, 180, size=B)
    w = decode_workload(m, ctx, seed=B + 11, name=f"{shape}-decode-b{B}")
    d, lg, ids = _run(w)
    sub = None if B <= 20 else list(range(0, B, max(1, B // 10)))
    st, *_ = e2e_compare(w, lg, ids, sub)
    assert_kv_layer_local(d, w, seq_subset=sub)
    d.release()
    print(st)


@pytest.mark.parametrize("shape", list(SHAPES))
def test_odd_shape_mixed_pass(shape):
    m = SHAPES[shape]
    ctx = np.random.default_rng(5).integers(1, 150, size=6)
    w = mixed_workload(m, n_pre=2, plen=37, ctx=ctx, seed=9, name=f"{shape}-mixed")
    d, lg, ids = _run(w)
    st, *_ = e2e_compare(w, lg, ids)
    assert_kv_layer_local(d, w)
    d.release()
    print(st)


@pytest.mark.parametrize("shape", list(SHAPES))
def test_odd_shape_shared_prefix(shape):
    """20 sequences sharing a 160-token prefix (read once per group): with
    groups of 3, 5 or 16 query heads a row's heads straddle the 16-column
    MFMA tiles and the 64-column prefix work items."""
    m = SHAPES[shape]
    ctx = 160 + np.random.default_rng(3).integers(3, 40, size=20)
    w = decode_workload(m, ctx, seed=21, shared=160, name=f"{shape}-shared")
    d, lg, ids = _run(w)
    pfx, ng = d.eng.batch_prefix_info()
    assert ng == 1 and (np.asarray(pfx) == 10).all(), (ng, pfx)  # one group, 10 prefix blocks per row
    st, *_ = e2e_compare(w, lg, ids)
    d.release()
    print(st)


@pytest.mark.parametrize("shape", list(SHAPES))
@pytest.mark.parametrize("rows", [20, 130])
def test_odd_shape_routed(shape, rows):
    """The last layer routed (random skip, half Project-Only) with a projector
    of width 128: cohort maps, count-bounded projections and the weighted
    scatter on these shapes, end to end against the oracle's routed pass."""
    from dataclasses import replace

    from paper_2609_37062_amd.runner import DeviceRun
    from workloads import routes

    m = replace(SHAPES[shape], routed_layers=1, proj_ffn=128)
    ctx = np.random.default_rng(rows).integers(0, 180, size=rows)
    w = decode_workload(m, ctx, seed=rows + 2, name=f"{shape}-routed-{rows}")
    req = np.arange(rows)
    pos = np.array([s.ctx for s in w.seqs])
    tape = routes.random_skip(rows, m.n_routed, req, pos, 1.0, 0.5)
    print(f"[gpu] {w.name} rows={rows} routed", flush=True)
    d = DeviceRun(w, routed=True, poison_pool=True)
    d.set_route(*tape)
    d.step_routed()
    lg, ids = d.results()
    sub = None if rows <= 20 else list(range(0, rows, 13))
    st, *_ = e2e_compare(w, lg, ids, sub, route=tape)
    d.release()
    print(st)


# positions up to the largest the library takes (max_pos 16384)
LONG = ModelCfg("long-2L", n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=512, vocab=512,
                rope_theta=500000.0, max_pos=16384)


@pytest.mark.parametrize("bps", [0, 8, 512])
def test_long_contexts(bps):
    """Decode rows at positions up to 16,383 (the last rotary position),
    with the default split, 8-block splits (up to 128 split partials per
    row and KV head, merged in order) and 512-block splits."""
    from paper_2609_37062_amd.runner import DeviceRun
    ctx = np.array([16383, 12000, 9001, 5000, 1, 8192])
    w = decode_workload(LONG, ctx, seed=41, name=f"long-bps{bps}")
    print(f"[gpu] {w.name} bps={bps}", flush=True)
    d = DeviceRun(w, poison_pool=True)
    d.eng.set_tuning(0, bps)
    d.step()
    lg, ids = d.results()
    st, *_ = e2e_compare(w, lg, ids)
    assert_kv_layer_local(d, w)
    d.release()
    print(st)


@pytest.mark.parametrize("prefill_kernel", [1, 0])
def test_long_context_prefill_chunk(prefill_kernel):
    """Prefill chunks continuing long cached sequences: 40 rows after 9,000
    tokens (past the 8,192 positions a causal prefill work item stages, so
    the pass takes one decode work item per row) and 30 rows after 3,000,
    beside two decode rows."""
    from paper_2609_37062_amd.runner import DeviceRun
    from workloads.configs import SeqSpec, Workload
    rng = np.random.default_rng(43)
    specs = [(9000, 40), (3000, 30), (12000, 1), (700, 1)]
    n_pool = sum((c + q + 15) // 16 for c, q in specs) + 8
    perm = [int(b) for b in rng.permutation(n_pool)]
    seqs, pos = [], 0
    for i, (ctx, q) in enumerate(specs):
        nb = (ctx + 15) // 16
        seqs.append(SeqSpec(ctx, q, perm[pos:pos + nb], [(0, ctx, i)]))
        pos += nb
    tokens = rng.integers(0, LONG.vocab, size=sum(q for _, q in specs)).astype(np.int32)
    w = Workload(0, f"long-chunk-{prefill_kernel}", LONG, seqs, n_pool, tokens, 7)
    print(f"[gpu] {w.name}", flush=True)
    d = DeviceRun(w, poison_pool=True)
    d.eng.set_tuning(6, prefill_kernel)
    d.step()
    lg, ids = d.results()
    st, *_ = e2e_compare(w, lg, ids)
    assert_kv_layer_local(d, w)
    d.release()
    print(st)


def test_large_prefill_chunk():
    """A 4,100-row pass: four 1,024-token prompts prefilled in one chunk
    (33 row tiles of 128, causal items of 128 / G rows) beside four decode
    rows; logits of the 8 last rows against the oracle, K,V of a subset of
    the sequences layer-local."""
    m = SHAPES["h256-g5-d128"]
    ctx = np.array([5, 300, 1000, 77])
    w = mixed_workload(m, n_pre=4, plen=1024, ctx=ctx, seed=31, name="large-prefill")
    assert w.n_rows == 4100
    d, lg, ids = _run(w)
    st, *_ = e2e_compare(w, lg, ids)
    assert_kv_layer_local(d, w, seq_subset=[0, 3, 5])
    d.release()
    print(st)
