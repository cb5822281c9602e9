"""Test helpers: run the oracle on (a subset of) a workload and compare results."""
from __future__ import annotations

import numpy as np

from oracle import numerics as nm
from oracle.kvcache import BlockAllocator, PagedKV, build_batch, select_seqs
from oracle.model import GeneratedWeights, forward
from workloads.setup import apply_recipe, kv_fill_ranges, kv_values_np

# logits tolerance against the oracle's float64 z (the spec bar), and
# the magnitude above which a bf16 output cannot meet it (half-ulp 1/32)
LOGIT_TOL = 2e-2
BF16_EXACT_LIMIT = 8.0


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


def oracle_run(w, seq_subset=None, overrides=None, dist=None):
    """Oracle pass over the listed sequences.  Returns (out, kv, sub_batch, idx, device_rows).

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
    out = forward(m, W, kv, sub, w.tokens[rows], lrows)
    return out, kv, sub, idx, dev_rows


def compare_logits(gpu_logits, gpu_ids, z, tol=LOGIT_TOL):
    """Check bf16 device logits against oracle z.  Returns a stats dict; asserts the bar."""
    z = np.asarray(z, np.float64)
    small = np.abs(z) < BF16_EXACT_LIMIT
    err = np.abs(gpu_logits - z)
    max_err = float(err[small].max()) if small.any() else 0.0
    ref_ids = nm.argmax_lowest(z)
    strict = gpu_ids == ref_ids
    zmax = z.max(axis=1)
    chosen = z[np.arange(len(z)), gpu_ids]
    gated = chosen >= zmax - 2 * tol
    stats = {"max_err": max_err, "n_large": int((~small).sum()), "strict_agree": int(strict.sum()),
             "gated_agree": int(gated.sum()), "rows": len(z)}
    assert max_err <= tol, stats
    assert gated.all(), stats
    return stats
