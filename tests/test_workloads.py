"""The seeded input generators and workload recipes (no device needed)."""
import json
import os

import numpy as np
import torch

from workloads import gen
from workloads.configs import M3B, M8B, TINY, workload
from workloads.setup import apply_recipe, kv_fill_ranges
from oracle.kvcache import BlockAllocator

HERE = os.path.dirname(__file__)


def test_numpy_and_torch_generators_agree_bitwise():
    key = gen.key_of(123, "w", "x", 3)
    for start in (0, 12345, (1 << 32) - 1000):
        a = gen.bf16_bits_np(key, 5000, ("normal", 0.02), start=start)
        t = gen.bf16_tensor(key, (5000,), ("normal", 0.02), device="cpu", start=start)
        np.testing.assert_array_equal(a, t.view(torch.int16).numpy().view(np.uint16))


def test_generator_slices_are_consistent_and_threaded_equal():
    key = gen.key_of(7, "kv")
    whole = gen.bf16_bits_np(key, 6 << 20)           # threaded path
    part = gen.bf16_bits_np(key, 1000, start=(3 << 20) + 17)
    np.testing.assert_array_equal(whole[(3 << 20) + 17:(3 << 20) + 1017], part)


def test_normal_table_statistics():
    vals = gen.bf16_to_f64(gen.bf16_bits_np(gen.key_of(1), 1 << 20, ("normal", 0.02)))
    assert abs(vals.mean()) < 1e-4
    assert abs(vals.std() - 0.02) < 2e-4
    t = gen.bf16_to_f64(gen.normal_table(1.0))
    assert np.all(np.diff(t) >= 0) and t[0] < -4 and t[-1] > 4


def test_int_table():
    v = gen.bf16_to_f64(gen.int_table(-2, 2))
    assert set(np.unique(v)) == {-2.0, -1.0, 0.0, 1.0, 2.0}


def test_kv_sizing_matches_paper_figures():
    g = json.load(open(os.path.join(HERE, "golden", "kv_sizing.json")))
    assert M8B.kv_bytes_per_token_layer == g["kv_bytes_per_token_layer"]
    assert M8B.kv_bytes_per_token_layer * M8B.n_layers == g["kv_bytes_per_token"]
    assert g["tokens"] * g["kv_bytes_per_token"] == g["megabytes_for_tokens"] * 2 ** 20


def test_recipes_shapes():
    w1 = workload(1)
    assert w1.n_seqs == 4 and all(32 <= s.ctx <= 128 for s in w1.seqs)
    w2 = workload(2)
    assert w2.n_seqs == 16 and all(512 <= s.ctx <= 1024 for s in w2.seqs)
    w3 = workload(3)
    assert w3.n_seqs == 64
    shared = 1 - w3.unique_resident_tokens() / w3.resident_tokens()
    assert 0.88 < shared < 0.95          # about 90% of KV blocks shared
    w4 = workload(4)
    assert w4.n_rows == 4 * 512 + 32 and len(w4.logit_rows()) == 36
    w5 = workload(5)
    ctx = np.array([s.ctx for s in w5.seqs])
    assert ctx.min() >= 16 and ctx.max() <= 4096 and 400 < np.median(ctx) < 900


def test_recipe_allocation_is_valid():
    for cid in (1, 3, 4):
        w = workload(cid)
        a = BlockAllocator(w.n_pool_blocks, 16)
        slots = apply_recipe(a, w)
        flat = np.concatenate(slots)
        assert len(np.unique(flat)) == len(flat)
        for i, s in enumerate(w.seqs):
            assert a.length(i) == s.ctx + s.q_len
    # prefill requests of the mixed workload take the lowest free blocks
    w = workload(4)
    a = BlockAllocator(w.n_pool_blocks, 16)
    apply_recipe(a, w)
    held = set()
    for i in range(4, w.n_seqs):
        held |= set(a.table(i))
    free_sorted = sorted(set(range(w.n_pool_blocks)) - held)
    assert a.table(0) == free_sorted[:32]


def test_fill_ranges_share_prefix_once():
    w = workload(3)
    r = kv_fill_ranges(w)
    assert sum(1 for x in r if x[3] == -1) == 1
