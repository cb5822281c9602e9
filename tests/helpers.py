"""Test helpers: run the oracle on (a subset of) a workload and compare results."""
from __future__ import annotations

import numpy as np

from oracle import numerics as nm
from oracle.kvcache import BlockAllocator, PagedKV, build_batch, select_seqs
from oracle.model import GeneratedWeights, forward
from workloads.setup import apply_recipe, kv_fill_ranges, kv_values_np

# logits tolerance against the oracle's float64 z (the logits tolerance of the decode step); the
# magnitude from which a bf16 output cannot meet it (half-ulp 1/32); the
# factor on the oracle's own float32-vs-float64 spread that bounds a row end
# to end where that spread exceeds the bar (see compare_logits)
LOGIT_TOL = 2e-2
BF16_EXACT_LIMIT = 8.0
SPREAD_K = 3.0


def bf16_half_ulp(z):
    """Half a bf16 ulp at |z| (the largest rounding error of a bf16 output)."""
    a = np.maximum(np.abs(np.asarray(z, np.float64)), 2.0 ** -126)
    return np.exp2(np.floor(np.log2(a)) - 8)


def logit_bound(z, tol):
    """Allowed |bf16 logit - z| per element: tol where a bf16 output can meet it
    (|z| < 8), else the bf16 half-ulp at z plus the same allowance for
    summation order (tol - 2^-6)."""
    z = np.asarray(z, np.float64)
    tol = np.broadcast_to(np.asarray(tol, np.float64), z.shape)
    return np.where(np.abs(z) < BF16_EXACT_LIMIT, tol, bf16_half_ulp(z) + (tol - 2.0 ** -6))


def assert_bf16_close(gpu, ref, what):
    """Elementwise: equal, or one bf16 ulp apart (summation order may move a
    rounding).  Values far below the tensor's RMS come out of cancellations
    (a rotary pair whose terms nearly cancel), where an fp32 sum differs from
    the float64 one by more ulps of the small result: there the floor is
    1e-3 of the RMS."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    mag = np.maximum(np.abs(ref), 2.0 ** -126)
    ulp = np.exp2(np.floor(np.log2(mag)) - 7)
    floor = 1e-3 * np.sqrt(np.mean(ref ** 2))
    bad = np.abs(gpu - ref) > np.maximum(ulp * 1.0001, floor)
    exact = float(np.mean(gpu == ref))
    assert not bad.any(), f"{what}: {int(bad.sum())} elements beyond 1 ulp"
    assert exact > 0.9, f"{what}: only {exact:.3f} exact"
    return exact


def oracle_state(w, seq_subset=None):
    """Allocator + batch for the whole workload, KV store holding the subset's blocks."""
    m = w.model
    a = BlockAllocator(w.n_pool_blocks, 16)
    apply_recipe(a, w)
    batch = build_batch(a, list(range(w.n_seqs)), [s.q_len for s in w.seqs])
    idx = list(range(w.n_seqs)) if seq_subset is None else list(seq_subset)
    sub, rows = select_seqs(batch, idx)
    blocks = sorted({b for i in idx for b in a.table(i)})
    kv = PagedKV(m.n_layers, w.n_pool_blocks, m.n_kv_heads, m.head_dim, blocks=blocks)
    for (i, p0, n, cid) in kv_fill_ranges(w, idx):
        t = np.asarray(a.table(i), np.int64)
        p = np.arange(p0, p0 + n)
        slots = t[p // 16] * 16 + p % 16
        for l in range(m.n_layers):
            K = nm.from_bf16_bits(kv_values_np(w, l, 0, p0, n, cid))
            V = nm.from_bf16_bits(kv_values_np(w, l, 1, p0, n, cid))
            kv.write(l, slots, K, V)
    return a, batch, sub, rows, kv, idx


def assert_kv_layer_local(d, w, seq_subset=None, step=None):
    """Every layer's new K,V for the subset's rows (Invariant 1: each row writes
    its own slot at every layer) within one bf16 ulp of the oracle applied to
    that layer alone, from the device's own input residual of the layer (end to
    end, an earlier layer's bf16 rounding flips would move later layers' K,V by
    more than an ulp).  `step` runs the device pass (default d.step); the
    engine is left with the full pass run last."""
    m = w.model
    step = step or d.step
    a, batch, sub, rows, kv, idx = oracle_state(w, seq_subset)
    xs = {}
    for l in range(1, m.n_layers):
        d.set_layers(l)
        step()
        xs[l] = d.residual()[rows]
    d.set_layers(0)
    step()
    W = GeneratedWeights(m, w.seed)
    tok = w.tokens[rows]
    for l in range(m.n_layers):
        forward(m, W, kv, sub, tok, None, x0=xs.get(l), layers=[l])
        K, V = d.read_kv(l, sub["slot"])
        Ko, Vo = kv.read(l, sub["slot"])
        assert_bf16_close(K, Ko, f"K layer {l}")
        assert_bf16_close(V, Vo, f"V layer {l}")


def oracle_run(w, seq_subset=None, overrides=None, dist=None, dtype="f64", route=None):
    """Oracle pass over the listed sequences.  Returns (out, kv, sub_batch, idx, device_rows).

    dtype "f32" runs the oracle's contract-mode variant (float32 arithmetic,
    same rounding points) instead of the float64 definition.  route: a
    routed pass's tape (run, w) over all rows of the workload.

    device_rows[j] is the row of the device's logits output that holds the
    j-th returned oracle row.
    """
    m = w.model
    a, batch, sub, rows, kv, idx = oracle_state(w, seq_subset)
    W = GeneratedWeights(m, w.seed, overrides=overrides, dist=dist)
    decode = all(s.q_len == 1 for s in w.seqs)
    if decode:
        lrows = np.arange(len(idx))
        dev_rows = np.asarray(idx)
    else:
        # logits for the last row of each sequence marked for logits
        lrows, dev_rows = [], []
        out_pos = {}
        k = 0
        for i, s in enumerate(w.seqs):
            if s.logits:
                out_pos[i] = k
                k += 1
        for j, i in enumerate(idx):
            if w.seqs[i].logits:
                lrows.append(int(sub["cu_q"][j + 1]) - 1)
                dev_rows.append(out_pos[i])
        lrows, dev_rows = np.asarray(lrows), np.asarray(dev_rows)
    rt = None if route is None else (np.asarray(route[0])[:, rows], np.asarray(route[1])[:, rows])
    out = forward(m, W, kv, sub, w.tokens[rows], lrows, dtype=dtype, route=rt)
    return out, kv, sub, idx, dev_rows


def compare_logits(gpu_logits, gpu_ids, z, tol=LOGIT_TOL, z32=None, k=SPREAD_K):
    """Check bf16 device logits and greedy ids against the oracle's float64 z.

    The bound is `tol` (the logits tolerance of the decode step), or, given the oracle's float32
    contract-mode z32 of the same rows, max(tol, k * spread) with spread =
    max |z32 - z| over the rows compared: a correct float32 implementation
    drifts from the float64 definition by about that much, and no less.  One
    bf16 rounding flip anywhere in the pass is amplified by every later
    normalisation (a flip in one query element of a 2-layer model moved 566
    final-norm outputs and the logits by 0.014), and whether a given row
    flips is chance: a row where the float32 run had none may have one on the
    device.  So the spread is taken over the workload's rows, not row by row.
    Elementwise the bound is logit_bound(z, bound).  Greedy ids: a row whose
    top-2 gap in z exceeds twice the bound must agree exactly; otherwise the
    device id must be within twice the bound of the maximum (several ids are
    correct).  With z32, the mean error over the rows must also stay within
    k times the mean error of bf16(z32).
    Returns a stats dict; asserts all of it.
    """
    z = np.asarray(z, np.float64)
    gpu_logits = np.asarray(gpu_logits, np.float64)
    rows = len(z)
    row_tol = np.full(rows, float(tol))
    if z32 is not None:
        z32 = np.asarray(z32, np.float64)
        spread = np.abs(z32 - z).max(axis=1)
        row_tol = np.maximum(row_tol, k * spread.max())
    bound = logit_bound(z, row_tol[:, None])
    err = np.abs(gpu_logits - z)
    ratio = err / bound
    ref_ids = nm.argmax_lowest(z)
    srt = np.sort(z, axis=1)
    gap = srt[:, -1] - srt[:, -2] if z.shape[1] > 1 else np.full(rows, np.inf)
    gate = 2.0 * row_tol
    decided = gap > gate
    strict = gpu_ids == ref_ids
    chosen = z[np.arange(rows), gpu_ids]
    gated = chosen >= z.max(axis=1) - gate
    stats = {"max_err": float(err[np.abs(z) < BF16_EXACT_LIMIT].max()) if (np.abs(z) < BF16_EXACT_LIMIT).any()
             else 0.0, "max_err_over_bound": float(ratio.max()), "n_large": int((np.abs(z) >= BF16_EXACT_LIMIT).sum()),
             "rows": rows, "strict_agree": int(strict.sum()), "decided_rows": int(decided.sum()),
             "gated_agree": int(gated.sum()), "row_bound_max": float(row_tol.max())}
    if z32 is not None:
        mean_gpu = err.mean(axis=1)
        mean_32 = np.abs(nm.bf16_round(z32) - z).mean(axis=1)
        stats["spread_max"] = float(spread.max())
        stats["spread_mean"] = float(mean_32.mean())
        stats["mean_err"] = float(mean_gpu.mean())
        assert mean_gpu.mean() <= max(k * mean_32.mean(), tol / 4), (stats, mean_gpu, mean_32)
    assert ratio.max() <= 1.0, stats
    assert strict[decided].all(), stats
    assert gated.all(), stats
    return stats


def e2e_compare(w, gpu_logits, gpu_ids, seq_subset=None, overrides=None, dist=None, route=None):
    """End-to-end check of device logits against the oracle run from the token
    ids, with row bounds from the oracle's own float32 spread (compare_logits).
    Returns (stats, float64 oracle output, kv, sub_batch, idx, device rows)."""
    out, kv, sub, idx, dev_rows = oracle_run(w, seq_subset, overrides=overrides, dist=dist, route=route)
    print(f"[e2e] {w.name}: float64 oracle done", flush=True)
    out32, *_ = oracle_run(w, seq_subset, overrides=overrides, dist=dist, dtype="f32", route=route)
    st = compare_logits(gpu_logits[dev_rows], gpu_ids[dev_rows], out["z"], z32=out32["z"])
    return st, out, kv, sub, idx, dev_rows
