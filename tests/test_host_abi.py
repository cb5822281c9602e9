"""The C-ABI library on the CPU: it loads, exports every declared entry point,
and its host allocator / batch builder agree bit-exactly with the oracle's
model of them (no device calls)."""
import os
import re

import numpy as np
import pytest

from oracle.kvcache import AllocError, BlockAllocator, build_batch
from workloads.configs import M3B, M8B, TINY, workload
from workloads.setup import apply_recipe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
vsk = pytest.importorskip("paper_2609_37062_amd.vsk")


def _lib():
    try:
        return vsk.lib()
    except ImportError as e:
        pytest.fail(f"library not built: {e}")


def test_every_declared_symbol_is_exported():
    _lib()
    header = open(os.path.join(ROOT, "include", "vsk.h")).read()
    declared = set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(vsk_\w+)\s*\(", header, re.M))
    assert len(declared) >= 30
    import ctypes
    L = ctypes.CDLL(vsk.LIB_PATH)
    for name in declared:
        assert hasattr(L, name), name
    bound = {n for n, _, _ in vsk.SIGNATURES}
    assert declared == bound, declared ^ bound


def test_status_strings_and_bad_config():
    L = _lib()
    assert L.vsk_status_str(0) == b"ok"
    assert L.vsk_status_str(-2) == b"KV pool exhausted"
    bad = vsk.model_cfg(TINY)
    bad.head_dim = 96
    import ctypes
    h = ctypes.c_void_p()
    assert L.vsk_create(ctypes.byref(bad), ctypes.byref(h)) == -1
    assert vsk.packed_weight_bytes(M3B) > 7e9
    # kv pool bytes: L x 2 x blocks x Hkv x 16 x d x 2
    assert vsk.kv_pool_bytes(M8B, 10) == 32 * 2 * 10 * 8 * 16 * 128 * 2


def _slots_of(eng_or_alloc, w):
    return [np.asarray(s, np.int64) for s in apply_recipe(eng_or_alloc, w)]


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_allocator_and_batch_match_oracle_model(cid):
    w = workload(cid)
    e = vsk.Engine(w.model)
    e.kv_init(None, w.n_pool_blocks)
    a = BlockAllocator(w.n_pool_blocks, 16)
    s_lib = _slots_of(e, w)
    s_ref = _slots_of(a, w)
    for x, y in zip(s_lib, s_ref):
        np.testing.assert_array_equal(x, y)
    flat = np.concatenate(s_lib)
    assert len(np.unique(flat)) == len(flat), "two rows write one slot"
    q = [s.q_len for s in w.seqs]
    e.batch_build(list(range(w.n_seqs)), q)
    got = e.batch_host()
    ref = build_batch(a, list(range(w.n_seqs)), q)
    for k in ("block_table", "kv_len", "cu_q", "row_seq", "pos", "slot"):
        np.testing.assert_array_equal(got[k], ref[k].astype(np.int32), err_msg=k)
    for i in range(w.n_seqs):
        ln, table = e.seq_info(i)
        assert ln == a.length(i) and table == a.table(i)
    assert e.free_blocks() == len(a.free_blocks())
    e.close()


def test_random_allocator_sequences_match_model():
    rng = np.random.default_rng(0)
    for trial in range(20):
        n = int(rng.integers(4, 40))
        e = vsk.Engine(TINY)
        e.kv_init(None, n)
        a = BlockAllocator(n, 16)
        live = []
        for step in range(60):
            op = rng.integers(0, 5)
            args = None
            try:
                if op == 0 or not live:
                    sid = int(rng.integers(0, 30))
                    args = ("seq_create", sid)
                elif op == 1:
                    args = ("reserve", int(rng.choice(live)), int(rng.integers(0, 40)))
                elif op == 2:
                    args = ("seq_release", int(rng.choice(live)))
                elif op == 3:
                    src = int(rng.choice(live))
                    args = ("seq_share_prefix", int(rng.integers(0, 30)), src, 16 * int(rng.integers(0, 3)))
                else:
                    k = int(rng.integers(0, 3))
                    args = ("seq_set_blocks", int(rng.integers(0, 30)),
                            [int(b) for b in rng.integers(-1, n + 1, size=k)], int(rng.integers(0, 16 * k + 1)))
                r_ref = err_ref = None
                try:
                    r_ref = getattr(a, args[0])(*args[1:])
                except AllocError as ex:
                    err_ref = ex.code
                r_lib = err_lib = None
                try:
                    r_lib = getattr(e, args[0])(*args[1:])
                except vsk.VskError as ex:
                    err_lib = ex.code
                assert err_ref == err_lib, (args, err_ref, err_lib)
                if args[0] == "reserve" and err_ref is None:
                    np.testing.assert_array_equal(r_ref, r_lib)
                live = sorted(a.seqs.keys())
                assert e.free_blocks() == len(a.free_blocks())
            finally:
                pass
        for s in live:
            assert e.seq_info(s) == (a.length(s), a.table(s))
        e.close()


def test_errors_leave_state_unchanged():
    e = vsk.Engine(TINY)
    e.kv_init(None, 3)
    e.seq_create(1)
    e.reserve(1, 20)
    before = (e.seq_info(1), e.free_blocks())
    with pytest.raises(vsk.VskError) as ex:
        e.reserve(1, 40)
    assert ex.value.code == "NOMEM"
    assert (e.seq_info(1), e.free_blocks()) == before
    with pytest.raises(vsk.VskError) as ex:
        e.batch_build([1, 1], [1, 1])
    assert ex.value.code == "ARG"
    with pytest.raises(vsk.VskError) as ex:
        e.batch_build([7], [1])
    assert ex.value.code == "STATE"
    # an empty pass, and rows outside 1..resident length of the sequence
    for seqs, q in (([], []), ([1], [0]), ([1], [21])):
        with pytest.raises(vsk.VskError) as ex:
            e.batch_build(seqs, q)
        assert ex.value.code == "ARG", (seqs, q)
    assert (e.seq_info(1), e.free_blocks()) == before
    e.close()


def _prefix_groups_model(tables, kv_lens, min_blocks=4):
    """Brute force of the grouping rule: sequences grouped by first block; a
    group's prefix is the longest run of leading blocks that every member
    holds, each wholly before every member's current token."""
    n = len(tables)
    out = np.zeros(n, np.int32)
    groups = 0
    full = [(kv_lens[i] - 1) // 16 for i in range(n)]
    firsts = {}
    for i in range(n):
        if full[i] >= min_blocks:
            firsts.setdefault(tables[i][0], []).append(i)
    for m in firsts.values():
        if len(m) < 2:
            continue
        lim = min(full[i] for i in m)
        p = 0
        while p < lim and all(tables[i][p] == tables[m[0]][p] for i in m):
            p += 1
        if p >= min_blocks:
            groups += 1
            out[m] = p
    return out, groups


@pytest.mark.parametrize("cid", [2, 3, 5])
def test_shared_prefix_groups_of_workloads(cid):
    w = workload(cid)
    e = vsk.Engine(w.model)
    e.kv_init(None, w.n_pool_blocks)
    apply_recipe(e, w)
    e.batch_build(list(range(w.n_seqs)), [1] * w.n_seqs)
    got, ng = e.batch_prefix_info()
    b = e.batch_host()
    tables = [list(b["block_table"][i][: (b["kv_len"][i] + 15) // 16]) for i in range(w.n_seqs)]
    ref, ng_ref = _prefix_groups_model(tables, b["kv_len"])
    np.testing.assert_array_equal(got, ref)
    assert ng == ng_ref
    if cid == 3:
        assert ng == 1 and np.all(got == 1536 // 16)  # the whole 96-block shared prefix
    else:
        assert ng == 0
    e.close()


def test_shared_prefix_groups_random():
    """Random trees of shared prefixes (fork, extend, fork again) against the
    brute-force rule; rows of a mixed (prefill) pass are never grouped."""
    rng = np.random.default_rng(7)
    for trial in range(30):
        e = vsk.Engine(TINY)
        e.kv_init(None, 400)
        n_root = int(rng.integers(1, 4))
        seqs = []
        sid = 0
        for r in range(n_root):
            e.seq_create(sid)
            e.reserve(sid, int(rng.integers(1, 200)))
            seqs.append(sid)
            sid += 1
        for k in range(int(rng.integers(0, 10))):
            src = int(rng.choice(seqs))
            ln, _ = e.seq_info(src)
            share = 16 * int(rng.integers(0, ln // 16 + 1))
            e.seq_create(sid)
            e.seq_share_prefix(sid, src, share)
            e.reserve(sid, int(rng.integers(1, 100)))
            seqs.append(sid)
            sid += 1
        order = list(rng.permutation(seqs))
        e.batch_build(order, [1] * len(order))
        got, ng = e.batch_prefix_info()
        b = e.batch_host()
        tables = [list(b["block_table"][i][: (b["kv_len"][i] + 15) // 16]) for i in range(len(order))]
        ref, ng_ref = _prefix_groups_model(tables, b["kv_len"])
        np.testing.assert_array_equal(got, ref)
        assert ng == ng_ref
        e.batch_build(order, [2] + [1] * (len(order) - 1))
        got, ng = e.batch_prefix_info()
        assert ng == 0 and not got.any()
        e.close()
