"""Greedy generation over consecutive decode passes, through the C ABI.

Every pass reserves one more position per sequence in the host allocator,
rebuilds and uploads the batch metadata (Invariant 2: the block tables,
lengths, positions and slots of the current row set, rebuilt per pass) and
runs the decode step on the greedy ids the previous pass left on the device
(next_ids of one pass is the ids input of the next, no host round trip);
once per-operation kernels, once the persistent step kernel (whose grid
synchronisation epochs then advance over passes of changing batches).
Sequences cross block boundaries on the way, so the allocator hands out new
blocks (lowest free id) between the passes.

The oracle follows the same path: its allocator reserves the same slots
(checked each pass), its KV store keeps every pass's K,V (each row writes
its own-layer K,V: Invariant 1, read back by the next passes), and each pass
runs on the ids the device consumed.  Every pass's logits are held to the
logits bar (widened per row only where the oracle's own float32
contract-mode run, with a store of its own, drifts further), and the
device's ids to the oracle's argmax on decided rows (compare_logits).  Greedy decoding is the paper's (section 4, experimental
setup)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import numerics as nm  # noqa: E402
from oracle.kvcache import BlockAllocator, PagedKV, build_batch, select_seqs  # noqa: E402
from oracle.model import GeneratedWeights, forward  # noqa: E402
from workloads.configs import ModelCfg, decode_workload  # noqa: E402
from workloads.setup import apply_recipe, kv_fill_ranges, kv_values_np  # noqa: E402

from helpers import compare_logits  # noqa: E402

pytestmark = pytest.mark.gpu

MODELS = {
    "gqa4-d128": ModelCfg("gen-g4", n_layers=2, hidden=512, n_q_heads=8, n_kv_heads=2, head_dim=128, ffn=1536,
                          vocab=2048, rope_theta=500000.0),
    "gqa3-d64": ModelCfg("gen-g3", n_layers=3, hidden=384, n_q_heads=6, n_kv_heads=2, head_dim=64, ffn=1024,
                         vocab=1024, rope_theta=10000.0),
    # inside the persistent kernel's shape rule (every projection K a
    # multiple of 256 with at least 2,048)
    "persistent": ModelCfg("gen-p", n_layers=2, hidden=2048, n_q_heads=16, n_kv_heads=4, head_dim=128, ffn=2048,
                           vocab=4096, rope_theta=500000.0),
}


def _oracle_store(w):
    """Allocator with the workload's tables and a KV store of the whole pool
    holding its cached K,V (new blocks are handed out while generating)."""
    m = w.model
    a = BlockAllocator(w.n_pool_blocks, 16)
    apply_recipe(a, w)
    kv = PagedKV(m.n_layers, w.n_pool_blocks, m.n_kv_heads, m.head_dim)
    for (i, p0, n, cid) in kv_fill_ranges(w, list(range(w.n_seqs))):
        t = np.asarray(a.table(i), np.int64)
        p = np.arange(p0, p0 + n)
        slots = t[p // 16] * 16 + p % 16
        for l in range(m.n_layers):
            K = nm.from_bf16_bits(kv_values_np(w, l, 0, p0, n, cid))
            V = nm.from_bf16_bits(kv_values_np(w, l, 1, p0, n, cid))
            kv.write(l, slots, K, V)
    return a, kv


@pytest.mark.parametrize("model", list(MODELS))
def test_greedy_generation_matches_oracle(model):
    from paper_2609_37062_amd.runner import DeviceRun
    m = MODELS[model]
    T, B = 16, 12
    # cached lengths around block boundaries: most sequences take a new block
    # within the 16 passes, some at the first one
    ctx = np.array([15, 16, 31, 1, 47, 100, 63, 8, 129, 200, 12, 255])
    assert len(ctx) == B
    w = decode_workload(m, ctx, seed=17, name=f"gen-{model}")
    print(f"[gpu] {w.name} rows={B} passes={T}", flush=True)
    d = DeviceRun(w, max_kv_len=int(ctx.max()) + T + 1, poison_pool=True)
    if model == "persistent":
        d.eng.set_tuning(2, 2)  # every pass one launch of the persistent step kernel
    sp = d.sp
    seqs, ones = list(range(B)), [1] * B
    meta_t = torch.empty(4 * d.meta_bytes + 4096, dtype=torch.uint8, device=d.device)
    meta = meta_t.data_ptr() + ((-meta_t.data_ptr()) % 256)
    ids = [d.ids.clone(), torch.empty_like(d.ids)]
    a, kv = _oracle_store(w)
    kv32 = _oracle_store(w)[1]  # the float32 contract-mode oracle's own store
    W = GeneratedWeights(m, w.seed)
    new_blocks = 0
    for t in range(T):
        if t > 0:
            for q in seqs:
                d.eng.reserve(q, 1)
                new_blocks += int(a.length(q) % 16 == 0)
                a.reserve(q, 1)
            d.eng.batch_build(seqs, ones)
            d.eng.batch_upload(meta, meta_t.numel() - 256, sp)
        d.eng.decode_step(ids[t % 2].data_ptr(), d.logits.data_ptr(), ids[(t + 1) % 2].data_ptr(), d.ws,
                          d.ws_bytes, sp)
        torch.cuda.synchronize()
        lg = d.logits.view(torch.bfloat16).float().cpu().numpy().astype(np.float64)
        tok_in = ids[t % 2].cpu().numpy()
        nxt = ids[(t + 1) % 2].cpu().numpy()
        # the oracle's pass on the same rows, slots and input ids
        batch = build_batch(a, seqs, ones)
        np.testing.assert_array_equal(d.eng.batch_host()["slot"], batch["slot"])
        sub, rows = select_seqs(batch, seqs)
        out = forward(m, W, kv, sub, tok_in[rows], np.arange(B))
        out32 = forward(m, W, kv32, sub, tok_in[rows], np.arange(B), dtype="f32")
        st = compare_logits(lg, nxt, out["z"], z32=out32["z"])
        print(f"[gen] pass {t}: {st}", flush=True)
        if model == "persistent":
            d.eng.device_status(sp)
            assert d.eng.exec_counters()[5] == 1, "the persistent kernel did not run"
    assert new_blocks >= B - 1, new_blocks  # all sequences but one took a new block
    d.release()


def test_prefill_then_generate():
    """Three fresh prompts of 37 tokens prefilled in one chunk (the causal
    multi-row kernel; logits of each prompt's last row), then 12 decode
    passes generating from the prefill's greedy ids, against the oracle
    following the same path."""
    from paper_2609_37062_amd.runner import DeviceRun
    from workloads.configs import mixed_workload
    m = MODELS["gqa4-d128"]
    T, plen = 12, 37
    w = mixed_workload(m, n_pre=3, plen=plen, ctx=np.zeros(0, np.int64), seed=23, name="gen-prefill")
    B = w.n_seqs
    print(f"[gpu] {w.name} rows={w.n_rows} then {T} decode passes", flush=True)
    d = DeviceRun(w, max_kv_len=plen + T + 1, poison_pool=True)
    sp = d.sp
    seqs, ones = list(range(B)), [1] * B
    meta_t = torch.empty(4 * d.meta_bytes + 4096, dtype=torch.uint8, device=d.device)
    meta = meta_t.data_ptr() + ((-meta_t.data_ptr()) % 256)
    a, kv = _oracle_store(w)
    kv32 = _oracle_store(w)[1]
    W = GeneratedWeights(m, w.seed)
    # the prefill pass
    d.step()
    lg, nxt = d.results()
    batch = build_batch(a, seqs, [s.q_len for s in w.seqs])
    sub, rows = select_seqs(batch, seqs)
    last = np.asarray(sub["cu_q"][1:]) - 1
    out = forward(m, W, kv, sub, w.tokens[rows], last)
    out32 = forward(m, W, kv32, sub, w.tokens[rows], last, dtype="f32")
    st = compare_logits(lg, nxt, out["z"], z32=out32["z"])
    print(f"[gen] prefill: {st}", flush=True)
    ids = [torch.from_numpy(nxt.astype(np.int32)).to(d.device), torch.empty(B, dtype=torch.int32, device=d.device)]
    logits = torch.empty((B, m.vocab), dtype=torch.int16, device=d.device)
    for t in range(T):
        for q in seqs:
            d.eng.reserve(q, 1)
            a.reserve(q, 1)
        d.eng.batch_build(seqs, ones)
        d.eng.batch_upload(meta, meta_t.numel() - 256, sp)
        d.eng.decode_step(ids[t % 2].data_ptr(), logits.data_ptr(), ids[(t + 1) % 2].data_ptr(), d.ws, d.ws_bytes,
                          sp)
        torch.cuda.synchronize()
        lg = logits.view(torch.bfloat16).float().cpu().numpy().astype(np.float64)
        tok_in = ids[t % 2].cpu().numpy()
        nxt = ids[(t + 1) % 2].cpu().numpy()
        batch = build_batch(a, seqs, ones)
        np.testing.assert_array_equal(d.eng.batch_host()["slot"], batch["slot"])
        sub, rows = select_seqs(batch, seqs)
        out = forward(m, W, kv, sub, tok_in[rows], np.arange(B))
        out32 = forward(m, W, kv32, sub, tok_in[rows], np.arange(B), dtype="f32")
        st = compare_logits(lg, nxt, out["z"], z32=out32["z"])
        print(f"[gen] pass {t}: {st}", flush=True)
    d.release()
