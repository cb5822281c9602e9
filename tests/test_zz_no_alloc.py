"""vsk_decode_step_scratch (the entry point that allocates nothing) against
vsk_decode_step on the same batches: bit-identical logits, greedy ids and
KV writes, on two calls in a row, the second with a smaller batch; and a
batch too large for the fixed scratch array is refused before any launch."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from workloads.configs import ModelCfg, decode_workload  # noqa: E402

pytestmark = pytest.mark.gpu

MID = ModelCfg("mid-2L", n_layers=2, hidden=512, n_q_heads=8, n_kv_heads=2, head_dim=128, ffn=1536,
               vocab=2048, rope_theta=500000.0)


def _both(w):
    """Logits, ids and new K,V from the workspace entry point and from the scratch one."""
    from paper_2609_37062_amd.runner import DeviceRun
    print(f"[gpu] scratch vs workspace: {w.name} rows={w.n_rows}", flush=True)
    d = DeviceRun(w, poison_pool=True)
    slots = d.eng.batch_host()["slot"]
    d.step()
    lg_ws, ids_ws = d.results()
    kv_ws = [d.read_kv(l, slots) for l in range(w.model.n_layers)]
    d.logits.fill_(0)
    d.next_ids.fill_(-1)
    d.eng.decode_step_scratch(d.ids.data_ptr(), d.logits.data_ptr(), d.next_ids.data_ptr(), d.sp)
    lg_s, ids_s = d.results()
    kv_s = [d.read_kv(l, slots) for l in range(w.model.n_layers)]
    d.release()
    return (lg_ws, ids_ws, kv_ws), (lg_s, ids_s, kv_s)


def _same(a, b):
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    for (k1, v1), (k2, v2) in zip(a[2], b[2]):
        np.testing.assert_array_equal(k1, k2)
        np.testing.assert_array_equal(v1, v2)


def test_scratch_entry_point_matches_workspace_entry_point():
    rng = np.random.default_rng(5)
    big = decode_workload(MID, rng.integers(100, 1500, size=40), seed=5, name="scratch-b40")
    small = decode_workload(MID, rng.integers(0, 300, size=9), seed=6, name="scratch-b9")
    for w in (big, small):  # the second call is smaller: stale bytes of the first stay in the array
        ws, sc = _both(w)
        _same(ws, sc)


def test_scratch_entry_point_refuses_a_batch_beyond_its_array():
    from paper_2609_37062_amd import vsk
    from paper_2609_37062_amd.runner import DeviceRun
    ctx = np.full(256, 6000)
    w = decode_workload(MID, ctx, seed=7, name="scratch-too-big")
    d = DeviceRun(w)
    need = d.eng.workspace_bytes(w.n_rows, w.n_seqs, int(ctx.max()) + 1)
    assert need > vsk.SCRATCH_BYTES, need
    with pytest.raises(vsk.VskError) as e:
        d.eng.decode_step_scratch(d.ids.data_ptr(), d.logits.data_ptr(), d.next_ids.data_ptr(), d.sp)
    assert e.value.code == "ARG"
    d.release()
