"""Turning a workload recipe into allocator calls and KV fill ranges.

Used identically for the library's allocator and for the oracle's model of
it.  Holds no arithmetic of the decode step.
"""
from __future__ import annotations

import numpy as np

from . import gen
from .configs import Workload, kv_content_key


def apply_recipe(alloc, w: Workload):
    """Create every sequence, install its block table, reserve its new rows.

    ``alloc`` offers seq_create(seq), seq_set_blocks(seq, blocks, ctx) and
    reserve(seq, n) -> slots.  Returns the per-sequence new-row slots.
    """
    for i, _ in enumerate(w.seqs):
        alloc.seq_create(i)
    for i, s in enumerate(w.seqs):
        if s.blocks or s.ctx:
            alloc.seq_set_blocks(i, s.blocks, s.ctx)
    slots = []
    for i, s in enumerate(w.seqs):
        slots.append(np.asarray(alloc.reserve(i, s.q_len), np.int64))
    return slots


def kv_fill_ranges(w: Workload, seq_subset=None):
    """Cached (pre-pass) positions to fill, as (seq, first_pos, n_pos, content_id).

    A shared prefix appears once, under the first listed sequence that holds it.
    """
    out = []
    seen = set()
    idx = range(len(w.seqs)) if seq_subset is None else seq_subset
    for i in idx:
        s = w.seqs[i]
        for (p0, n, cid) in s.content:
            if n <= 0:
                continue
            if cid < 0:
                if cid in seen:
                    continue
                seen.add(cid)
            out.append((i, p0, n, cid))
    return out


def kv_values_np(w: Workload, layer: int, kind: int, p0: int, n: int, cid: int):
    """Generated bf16 bits [n][n_kv_heads][head_dim] of one content range."""
    m = w.model
    per = m.n_kv_heads * m.head_dim
    key = kv_content_key(w.seed, m, cid, layer, kind)
    bits = gen.bf16_bits_np(key, n * per, ("normal", m.kv_sigma), start=p0 * per)
    return bits.reshape(n, m.n_kv_heads, m.head_dim)


def kv_values_torch(w: Workload, layer: int, kind: int, p0: int, n: int, cid: int, device="cuda"):
    m = w.model
    per = m.n_kv_heads * m.head_dim
    key = kv_content_key(w.seed, m, cid, layer, kind)
    return gen.bf16_tensor(key, (n, m.n_kv_heads, m.head_dim), ("normal", m.kv_sigma),
                           device=device, start=p0 * per)


def subset(w: Workload, seq_idx):
    """A workload holding only the listed sequences (same tables and content)."""
    import copy
    w2 = copy.copy(w)
    w2.seqs = [w.seqs[i] for i in seq_idx]
    rows = []
    r = 0
    starts = []
    for s in w.seqs:
        starts.append(r)
        r += s.q_len
    for i in seq_idx:
        rows.extend(range(starts[i], starts[i] + w.seqs[i].q_len))
    w2.tokens = w.tokens[np.asarray(rows, np.int64)] if rows else w.tokens[:0]
    return w2
