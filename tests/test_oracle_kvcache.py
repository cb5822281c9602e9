"""Pins of the oracle's allocator and paging model (brute force, invariants)."""
import numpy as np
import pytest

from oracle.kvcache import AllocError, BlockAllocator, PagedKV, build_batch, select_seqs


def snapshot(a):
    return (list(a.ref), {k: (list(v["blocks"]), v["len"]) for k, v in a.seqs.items()})


def test_reserve_takes_lowest_free_block_and_slots():
    a = BlockAllocator(8, 4)
    a.seq_create(7)
    a.seq_set_blocks(7, [5, 2], 6)           # positions 0..5 in blocks 5, 2
    slots = a.reserve(7, 5)                  # positions 6..10
    # 6,7 -> block 2 offsets 2,3; 8..10 -> lowest free block 0
    assert list(slots) == [2 * 4 + 2, 2 * 4 + 3, 0, 1, 2]
    assert a.table(7) == [5, 2, 0]
    a.seq_create(8)
    s2 = a.reserve(8, 1)
    assert list(s2) == [1 * 4]               # next lowest free is 1


def test_slots_brute_force_random():
    rng = np.random.default_rng(0)
    a = BlockAllocator(64, 16)
    perm = rng.permutation(64)
    pos = 0
    lens = {}
    for s in range(5):
        n = int(rng.integers(1, 80))
        nb = (n + 15) // 16
        a.seq_create(s)
        a.seq_set_blocks(s, perm[pos:pos + nb], n)
        lens[s] = n
        pos += nb
    all_slots = set()
    for s in range(5):
        for p in range(lens[s]):
            sl = a.slot(s, p)
            assert sl == a.table(s)[p // 16] * 16 + p % 16
            assert sl not in all_slots
            all_slots.add(sl)


def test_errors_are_transactional():
    a = BlockAllocator(3, 4)
    a.seq_create(0)
    a.seq_set_blocks(0, [1], 4)
    before = snapshot(a)
    with pytest.raises(AllocError) as e:
        a.reserve(0, 9)                      # needs 3 more blocks, only 2 free
    assert e.value.code == "NOMEM"
    assert snapshot(a) == before
    with pytest.raises(AllocError) as e:
        a.seq_set_blocks(0, [2], 1)
    assert e.value.code == "STATE"
    a.seq_create(1)
    with pytest.raises(AllocError) as e:
        a.seq_set_blocks(1, [3], 1)
    assert e.value.code == "RANGE"
    with pytest.raises(AllocError) as e:
        a.seq_set_blocks(1, [0], 5)
    assert e.value.code == "ARG"
    with pytest.raises(AllocError) as e:
        a.seq_release(9)
    assert e.value.code == "STATE"
    with pytest.raises(AllocError) as e:
        a.seq_create(0)
    assert e.value.code == "STATE"


def test_shared_prefix_refcount_and_shared_write():
    a = BlockAllocator(10, 4)
    a.seq_create(0)
    a.seq_set_blocks(0, [3, 4, 5], 10)
    a.seq_create(1)
    a.seq_share_prefix(1, 0, 8)
    assert a.table(1) == [3, 4] and a.length(1) == 8
    assert a.ref[3] == 2 and a.ref[5] == 1
    s = a.reserve(1, 1)                      # position 8 starts a new block: lowest free 0
    assert list(s) == [0]
    # a writer into a shared block is refused, state unchanged
    a.seq_create(2)
    a.seq_share_prefix(2, 0, 4)
    a2 = BlockAllocator(10, 4)
    a2.seq_create(0)
    a2.seq_set_blocks(0, [3, 4], 6)
    a2.seq_create(1)
    a2.seq_set_blocks(1, [3, 4], 6)          # same blocks: both references shared
    before = snapshot(a2)
    with pytest.raises(AllocError) as e:
        a2.reserve(1, 1)
    assert e.value.code == "SHARED_WRITE"
    assert snapshot(a2) == before
    with pytest.raises(AllocError) as e:
        a.seq_share_prefix(2, 0, 4)          # destination not empty
    assert e.value.code == "STATE"
    with pytest.raises(AllocError):
        a.seq_create(3)
        a.seq_share_prefix(3, 0, 6)          # not block aligned


def test_release_returns_blocks():
    a = BlockAllocator(4, 4)
    a.seq_create(0)
    a.reserve(0, 9)
    assert a.free_blocks() == [3]
    a.seq_release(0)
    assert a.free_blocks() == [0, 1, 2, 3]


def test_build_batch_brute_force():
    a = BlockAllocator(32, 16)
    a.seq_create(0)
    a.seq_set_blocks(0, [9, 4], 20)
    a.seq_create(1)
    a.reserve(0, 1)
    a.reserve(1, 3)
    b = build_batch(a, [0, 1], [1, 3])
    assert list(b["kv_len"]) == [21, 3]
    assert list(b["cu_q"]) == [0, 1, 4]
    assert list(b["pos"]) == [20, 0, 1, 2]
    assert list(b["row_seq"]) == [0, 1, 1, 1]
    assert list(b["slot"]) == [4 * 16 + 4, 0, 1, 2]
    assert b["block_table"].tolist() == [[9, 4], [0, -1]]
    sub, rows = select_seqs(b, [1])
    assert list(rows) == [1, 2, 3] and list(sub["cu_q"]) == [0, 3]
    with pytest.raises(AllocError):
        build_batch(a, [0], [22])


def test_paged_store_subset_equals_dense():
    rng = np.random.default_rng(1)
    dense = PagedKV(2, 8, 2, 4, block=4)
    part = PagedKV(2, 8, 2, 4, block=4, blocks=[1, 6])
    slots = np.array([4, 5, 27, 24])
    k = rng.standard_normal((4, 2, 4))
    v = rng.standard_normal((4, 2, 4))
    for st in (dense, part):
        st.write(1, slots, k, v)
    for st in (dense, part):
        K, V = st.read(1, slots[::-1])
        np.testing.assert_array_equal(K, k[::-1])
        np.testing.assert_array_equal(V, v[::-1])
    with pytest.raises(IndexError):
        part.read(0, [0])
