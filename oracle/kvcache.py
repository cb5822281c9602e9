"""Paged KV cache model: block allocator, slots and a paged store.

Test infrastructure only (see the package docstring).

The serving engine keeps each layer's keys and values in a paged cache
whose page mappings are rebuilt whenever the row set changes (paper,
"Invariants for Correct Mixed-Depth Execution", Invariant 2), and every
layer writes its own KV for every cached token (Invariant 1).  This module
states the bookkeeping the decode step relies on:

* A pool of ``n_blocks`` blocks of ``block`` tokens.  Blocks carry
  reference counts; a block referenced by several sequences is a shared
  (prefix) block and may not be written.
* Position p of a sequence lives at slot ``table[p // block] * block + p % block``.
* Reserving n new positions takes the lowest-numbered free block whenever a
  position starts a block the table does not yet hold.
* Every operation is all-or-nothing: on error the state is unchanged.

Error names mirror the library's status codes.
"""
from __future__ import annotations

import numpy as np


class AllocError(Exception):
    def __init__(self, code: str, msg: str = ""):
        super().__init__(f"{code}: {msg}")
        self.code = code


class BlockAllocator:
    """Plain model of the block allocator (dict/list based, O(n) everywhere)."""

    def __init__(self, n_blocks: int, block: int = 16):
        if n_blocks <= 0 or block <= 0:
            raise AllocError("ARG", "empty pool")
        self.n_blocks = n_blocks
        self.block = block
        self.ref = [0] * n_blocks
        self.seqs: dict[int, dict] = {}

    # -- queries
    def free_blocks(self):
        return [b for b in range(self.n_blocks) if self.ref[b] == 0]

    def table(self, seq):
        return list(self.seqs[seq]["blocks"])

    def length(self, seq):
        return self.seqs[seq]["len"]

    def slot(self, seq, pos):
        s = self.seqs[seq]
        if not 0 <= pos < len(s["blocks"]) * self.block:
            raise AllocError("RANGE", f"position {pos} outside table")
        return s["blocks"][pos // self.block] * self.block + pos % self.block

    # -- operations
    def seq_create(self, seq):
        if seq in self.seqs:
            raise AllocError("STATE", f"sequence {seq} exists")
        self.seqs[seq] = {"blocks": [], "len": 0}

    def seq_release(self, seq):
        if seq not in self.seqs:
            raise AllocError("STATE", f"unknown sequence {seq}")
        for b in self.seqs[seq]["blocks"]:
            self.ref[b] -= 1
        del self.seqs[seq]

    def seq_set_blocks(self, seq, blocks, ctx_len):
        if seq not in self.seqs:
            raise AllocError("STATE", f"unknown sequence {seq}")
        s = self.seqs[seq]
        if s["blocks"] or s["len"]:
            raise AllocError("STATE", "sequence already holds blocks")
        blocks = [int(b) for b in blocks]
        if ctx_len < 0 or len(blocks) * self.block < ctx_len:
            raise AllocError("ARG", "table shorter than context")
        for b in blocks:
            if not 0 <= b < self.n_blocks:
                raise AllocError("RANGE", f"block {b}")
        if len(set(blocks)) != len(blocks):
            raise AllocError("ARG", "block listed twice")
        for b in blocks:
            self.ref[b] += 1
        s["blocks"] = blocks
        s["len"] = int(ctx_len)

    def seq_share_prefix(self, dst, src, n_tokens):
        if dst not in self.seqs or src not in self.seqs:
            raise AllocError("STATE", "unknown sequence")
        d, s = self.seqs[dst], self.seqs[src]
        if d["blocks"] or d["len"]:
            raise AllocError("STATE", "destination not empty")
        if n_tokens < 0 or n_tokens % self.block or n_tokens > s["len"]:
            raise AllocError("ARG", "prefix must be block aligned and resident")
        nb = n_tokens // self.block
        d["blocks"] = list(s["blocks"][:nb])
        for b in d["blocks"]:
            self.ref[b] += 1
        d["len"] = n_tokens

    def reserve(self, seq, n_new):
        """Append n_new positions; returns their slots.  All or nothing."""
        if seq not in self.seqs:
            raise AllocError("STATE", f"unknown sequence {seq}")
        if n_new < 0:
            raise AllocError("ARG", "negative count")
        s = self.seqs[seq]
        L = s["len"]
        blocks = list(s["blocks"])
        free = self.free_blocks()
        taken = []
        slots = []
        for p in range(L, L + n_new):
            bi = p // self.block
            if bi >= len(blocks):
                if not free:
                    raise AllocError("NOMEM", "pool exhausted")
                b = free.pop(0)
                taken.append(b)
                blocks.append(b)
            b = blocks[bi]
            if self.ref[b] > 1:
                raise AllocError("SHARED_WRITE", f"block {b} is shared")
            slots.append(b * self.block + p % self.block)
        for b in taken:
            self.ref[b] += 1
        s["blocks"] = blocks
        s["len"] = L + n_new
        return np.asarray(slots, np.int64)


def build_batch(alloc: BlockAllocator, seqs, q_lens):
    """Per-pass metadata (Invariant 2: rebuilt from the current row set).

    Returns a dict with, for n sequences and R = sum(q_lens) rows:
      block_table [n][max_blocks] int32 (unused entries -1)
      kv_len      [n]   resident tokens including the pass's new rows
      cu_q        [n+1] row offsets
      row_seq     [R]   sequence index of each row
      pos         [R]   position of each row
      slot        [R]   cache slot each row writes
    """
    n = len(seqs)
    if len(q_lens) != n:
        raise AllocError("ARG", "length mismatch")
    if n == 0:
        raise AllocError("ARG", "empty batch")
    if len(set(seqs)) != n:
        raise AllocError("ARG", "sequence listed twice in one pass")
    kv_len = []
    for s, q in zip(seqs, q_lens):
        if s not in alloc.seqs:
            raise AllocError("STATE", f"unknown sequence {s}")
        L = alloc.length(s)
        if q < 1 or q > L:
            raise AllocError("ARG", "rows of a sequence must be 1..resident length")
        kv_len.append(L)
    max_blocks = max([len(alloc.table(s)) for s in seqs] + [1])
    table = -np.ones((n, max_blocks), np.int32)
    for i, s in enumerate(seqs):
        t = alloc.table(s)
        table[i, :len(t)] = t
    cu = np.zeros(n + 1, np.int32)
    cu[1:] = np.cumsum(q_lens)
    row_seq, pos, slot = [], [], []
    for i, (s, q) in enumerate(zip(seqs, q_lens)):
        for p in range(kv_len[i] - q, kv_len[i]):
            row_seq.append(i)
            pos.append(p)
            slot.append(alloc.slot(s, p))
    return {
        "block_table": table,
        "kv_len": np.asarray(kv_len, np.int32),
        "cu_q": cu,
        "row_seq": np.asarray(row_seq, np.int32),
        "pos": np.asarray(pos, np.int32),
        "slot": np.asarray(slot, np.int64),
    }


class PagedKV:
    """Paged K/V store indexed by (layer, slot), holding bf16-valued float64.

    ``blocks`` (optional) lists the only physical blocks that will be touched;
    the store then keeps just those (for full-size pools sampled by a few
    sequences).  Touching any other block raises.
    """

    def __init__(self, n_layers, n_blocks, n_kv_heads, head_dim, block=16, blocks=None):
        self.L, self.nb, self.hk, self.d, self.block = n_layers, n_blocks, n_kv_heads, head_dim, block
        self.remap = np.arange(n_blocks, dtype=np.int64)
        n_store = n_blocks
        if blocks is not None:
            blocks = np.unique(np.asarray(blocks, np.int64))
            self.remap = -np.ones(n_blocks, np.int64)
            self.remap[blocks] = np.arange(len(blocks))
            n_store = len(blocks)
        self.K = np.zeros((n_layers, n_store * block, n_kv_heads, head_dim))
        self.V = np.zeros_like(self.K)

    def _rows(self, slots):
        slots = np.asarray(slots, np.int64)
        if np.any(slots < 0) or np.any(slots >= self.nb * self.block):
            raise IndexError("slot outside pool")
        b = self.remap[slots // self.block]
        if np.any(b < 0):
            raise IndexError("block not held by this store")
        return b * self.block + slots % self.block

    def write(self, layer, slots, k, v):
        """k, v: [n, n_kv_heads, head_dim] at the given slots."""
        r = self._rows(slots)
        self.K[layer, r] = k
        self.V[layer, r] = v

    def read(self, layer, slots):
        r = self._rows(slots)
        return self.K[layer, r], self.V[layer, r]


def select_seqs(batch, idx):
    """The metadata of a sub-batch made of the listed sequences (same tables and slots)."""
    idx = [int(i) for i in idx]
    cu = batch["cu_q"]
    rows = np.concatenate([np.arange(cu[i], cu[i + 1]) for i in idx]) if idx else np.zeros(0, np.int64)
    q = [int(cu[i + 1] - cu[i]) for i in idx]
    cu2 = np.zeros(len(idx) + 1, np.int32)
    cu2[1:] = np.cumsum(q)
    row_seq = np.repeat(np.arange(len(idx), dtype=np.int32), q)
    return {
        "block_table": batch["block_table"][idx],
        "kv_len": batch["kv_len"][idx],
        "cu_q": cu2,
        "row_seq": row_seq,
        "pos": batch["pos"][rows],
        "slot": batch["slot"][rows],
    }, rows
