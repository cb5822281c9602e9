"""Device pins that need no tolerance: bit-exact cases and invariants of the
pass, all through the C ABI.

  * small-integer inputs (tests/intcase.py): every projection sum is an exact
    integer, so the device must reproduce the oracle bit for bit whatever its
    tiling -- K,V written by the QKV epilogue, the residual after the O and
    the MLP projections, bf16 logits and greedy ids (with ties) -- at row
    counts that take every launch shape of the projections;
  * V = 1 at every key: softmax weights sum to one, so every attention
    output is exactly bf16 1.0 (seen through Wo = I as a residual of 2.0);
  * V = one-hot(position): the attention output is the softmax row P itself;
  * a first token (no cached context) attends only to itself: o = v exactly;
  * Wq = 0: uniform attention, each output the mean of its head's values;
  * no stray KV writes: after a pass every pool block other than those
    holding the pass's new slots is byte-identical, and so is every other
    token of those blocks (Invariant 1 writes exactly the rows' own slots);
  * vsk_argmax_sample: bit-exact against the oracle's lowest-index argmax on
    bf16 and fp32 logits with planted ties, NaN, all-NaN and all -inf rows,
    +inf, signed zeros, at vocabulary 128256 and odd sizes; its flag marks
    exactly the all-NaN rows.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import numerics as nm  # noqa: E402
from oracle.model import GeneratedWeights, forward  # noqa: E402
from workloads.configs import TINY, ModelCfg, decode_workload, mixed_workload  # noqa: E402

from helpers import oracle_state  # noqa: E402
from intcase import fresh_workload, int_overrides  # noqa: E402

pytestmark = pytest.mark.gpu

MID = ModelCfg("mid-2L", n_layers=2, hidden=512, n_q_heads=8, n_kv_heads=2, head_dim=128, ffn=1536,
               vocab=2048, rope_theta=500000.0)


def _device(w, **kw):
    from paper_2609_37062_amd.runner import DeviceRun
    print(f"[gpu] {w.name} rows={w.n_rows} {sorted(k for k in kw)}", flush=True)
    kw.setdefault("poison_pool", True)
    return DeviceRun(w, **kw)


def _bf16_dev(a, device):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).to(device).view(torch.int16)


def _write_kv(d, layer, slots, K, V):
    s = torch.from_numpy(np.ascontiguousarray(slots, np.int32)).to(d.device)
    Kd, Vd = _bf16_dev(K, d.device), _bf16_dev(V, d.device)
    d.eng.kv_write(layer, s.data_ptr(), len(slots), Kd.data_ptr(), Vd.data_ptr(), d.sp)
    torch.cuda.synchronize(d.device)


def _cached_slots(d, w):
    out = []
    for i, s in enumerate(w.seqs):
        if s.ctx:
            out.append(d.seq_slots(i, 0, s.ctx))
    return np.concatenate(out) if out else np.zeros(0, np.int32)


# ---------------------------------------------------------------- small-integer inputs
@pytest.mark.parametrize("model,rows", [(TINY, 4), (MID, 1), (MID, 20), (MID, 70), (MID, 130)])
@pytest.mark.parametrize("variant", ["qkv", "o", "mlp"])
def test_integer_inputs_bit_exact(variant, model, rows):
    w = fresh_workload(model, rows, seed=rows, name=f"int-{variant}-{model.name}-r{rows}")
    over = int_overrides(model, variant, seed=rows)
    d = _device(w, overrides=over)
    d.step()
    lg, ids = d.results()
    x_dev = d.residual()
    a, batch, sub, r, kv, idx = oracle_state(w)
    W = GeneratedWeights(model, w.seed, overrides=over)
    out = forward(model, W, kv, sub, w.tokens[r], np.arange(rows), want_hidden=True)
    K, V = d.read_kv(0, sub["slot"])
    Ko, Vo = kv.read(0, sub["slot"])
    np.testing.assert_array_equal(K, Ko)
    np.testing.assert_array_equal(V, Vo)
    if variant == "qkv":
        for l in range(1, model.n_layers):  # every layer sees the embedding row
            K, V = d.read_kv(l, sub["slot"])
            Ko, Vo = kv.read(l, sub["slot"])
            np.testing.assert_array_equal(K, Ko)
            np.testing.assert_array_equal(V, Vo)
        np.testing.assert_array_equal(lg, out["logits"])
        np.testing.assert_array_equal(ids, out["ids"])
        ties = int(sum((out["z"][i] == out["z"][i].max()).sum() > 1 for i in range(rows)))
        print(f"[gpu] integer logits bit-exact; rows with tied maxima: {ties}/{rows}", flush=True)
    else:
        np.testing.assert_array_equal(x_dev, out["x"])
        assert np.abs(out["x"]).max() > 2
    d.release()


@pytest.mark.parametrize("rows", [200, 520])
@pytest.mark.parametrize("variant", ["qkv", "o", "mlp"])
def test_integer_inputs_bit_exact_row_tiled(variant, rows):
    """Passes of more than 128 rows (several 128-row tiles, the last one
    ragged) through every epilogue (QKV, RESID, SWIGLU, LOGITS), bit for bit
    against the oracle."""
    m = MID
    w = fresh_workload(m, rows, seed=rows, name=f"int-rowtiled-{variant}-r{rows}")
    over = int_overrides(m, variant, seed=rows)
    d = _device(w, overrides=over)
    d.step()
    lg, ids = d.results()
    x_dev = d.residual()
    a, batch, sub, r, kv, idx = oracle_state(w)
    W = GeneratedWeights(m, w.seed, overrides=over)
    out = forward(m, W, kv, sub, w.tokens[r], np.arange(rows), want_hidden=True)
    for l in range(m.n_layers if variant == "qkv" else 1):
        K, V = d.read_kv(l, sub["slot"])
        Ko, Vo = kv.read(l, sub["slot"])
        np.testing.assert_array_equal(K, Ko)
        np.testing.assert_array_equal(V, Vo)
    if variant == "qkv":
        np.testing.assert_array_equal(lg, out["logits"])
        np.testing.assert_array_equal(ids, out["ids"])
    else:
        np.testing.assert_array_equal(x_dev, out["x"])
    d.release()


# ---------------------------------------------------------------- attention invariants
def _probe_overrides(m, v_row):
    """Embedding rows of ones (the normed input is exactly 1), Wv making every
    new v the unit vector e_{v_row} (v_row None: all ones), Wo = I, Wd = 0."""
    H = m.hidden
    assert H == m.q_dim
    wv = np.zeros((m.kv_dim, H))
    if v_row is None:
        wv[:, 0] = 1.0
    else:
        for g in range(m.n_kv_heads):
            wv[g * m.head_dim + v_row, 0] = 1.0
    return {("embed", -1): np.ones((m.vocab, H)), ("wv", 0): wv, ("wo", 0): np.eye(H),
            ("w_down", 0): np.zeros((H, m.ffn))}


def test_v_ones_gives_exact_unit_outputs():
    m = TINY
    ctx = np.random.default_rng(1).integers(1, 300, size=12)
    w = decode_workload(m, ctx, seed=1, name="v-ones")
    d = _device(w, overrides=_probe_overrides(m, None))
    slots = _cached_slots(d, w)
    K, _ = d.read_kv(0, slots)
    _write_kv(d, 0, slots, K, np.ones_like(K))
    for bps in (0, 8):  # one split per row, then up to 3 merged splits
        d.eng.set_tuning(0, bps)
        d.step()
        x = d.residual()
        # x = 1 (embedding) + o Wo^T with Wo = I; o = 1 exactly
        assert np.all(x == 2.0), (bps, np.unique(x))
    d.release()


def test_one_hot_v_exposes_the_softmax_row():
    m = TINY
    n = 40  # every row at position 40 attends keys 0..40 (41 <= head_dim)
    w = decode_workload(m, np.full(9, n), seed=2, name="v-onehot")
    over = _probe_overrides(m, n)
    d = _device(w, overrides=over)
    slots = _cached_slots(d, w)
    K, _ = d.read_kv(0, slots)
    onehot = np.zeros_like(K)
    for j in range(len(slots)):
        onehot[j, :, j % n] = 1.0  # token at position p holds e_p in every KV head
    _write_kv(d, 0, slots, K, onehot)
    d.step()
    o_dev = d.residual() - 1.0  # x = 1 + o, exact in fp32 for o >= 2^-16
    # the oracle's softmax rows with the same keys
    a, batch, sub, r, kv, idx = oracle_state(w)
    kv.write(0, slots, K, onehot)
    W = GeneratedWeights(m, w.seed, overrides=over)
    o_or = forward(m, W, kv, sub, w.tokens[r], None)["x"] - 1.0
    o_dev = o_dev.reshape(len(r), m.n_q_heads, m.head_dim)
    o_or = o_or.reshape(len(r), m.n_q_heads, m.head_dim)
    assert np.all(o_dev[:, :, n + 1:] == 0)
    sums = o_dev[:, :, :n + 1].sum(axis=-1)
    assert np.abs(sums - 1.0).max() <= 2.0 ** -7, sums
    big = o_or >= 2.0 ** -16
    ulp = np.exp2(np.floor(np.log2(np.maximum(o_or, 2.0 ** -126))) - 7)
    diff = np.abs(o_dev - o_or)
    assert np.all(diff[big] <= ulp[big]), diff.max()  # one bf16 ulp at most
    assert np.all(diff[~big] <= 2.0 ** -16)
    assert np.mean(diff == 0) > 0.9, np.mean(diff == 0)
    d.release()


def test_zero_queries_average_v():
    """Wq = 0: every score is 0, the softmax is uniform, and each head's
    output is the mean of its KV head's values over keys 0..p (cached ones
    and the row's own new v); with Wo = I and unit embeddings the residual is
    1 + o.  Against the oracle within one bf16 ulp (the mean's float32 sum
    may round either way), with one split per row and with merged splits."""
    m = TINY
    ctx = np.random.default_rng(4).integers(1, 300, size=10)
    w = decode_workload(m, ctx, seed=4, name="q-zero")
    over = {("embed", -1): np.ones((m.vocab, m.hidden)), ("wq", 0): np.zeros((m.q_dim, m.hidden)),
            ("wo", 0): np.eye(m.hidden), ("w_down", 0): np.zeros((m.hidden, m.ffn))}
    d = _device(w, overrides=over)
    a, batch, sub, r, kv, idx = oracle_state(w)
    W = GeneratedWeights(m, w.seed, overrides=over)
    o_or = forward(m, W, kv, sub, w.tokens[r], None)["x"] - 1.0
    mag = np.maximum(np.abs(o_or), 2.0 ** -126)
    ulp = np.exp2(np.floor(np.log2(mag)) - 7)
    for bps in (0, 8):
        d.eng.set_tuning(0, bps)
        d.step()
        o_dev = d.residual() - 1.0
        diff = np.abs(o_dev - o_or)
        assert np.all(diff <= np.maximum(ulp * 1.0001, 2.0 ** -16)), (bps, diff.max())
        assert np.mean(diff == 0) > 0.9, np.mean(diff == 0)
    d.release()


def test_first_token_attends_to_itself_only():
    m = TINY
    w = fresh_workload(m, 6, seed=3, name="ctx0")
    over = {("wo", 0): np.eye(m.hidden), ("w_down", 0): np.zeros((m.hidden, m.ffn))}
    d = _device(w, overrides=over)
    d.step()
    x = d.residual()
    slots = d.eng.batch_host()["slot"]
    _, V = d.read_kv(0, slots)
    E = GeneratedWeights(m, w.seed).rows("embed", w.tokens)
    want = (E.astype(np.float32) + V.reshape(len(slots), -1).astype(np.float32)).astype(np.float64)
    np.testing.assert_array_equal(x, want)
    d.release()


# ---------------------------------------------------------------- no stray KV writes
def _pool_blocks(d, m):
    """Pool as [layer][K/V][block][elements of one block, all KV heads]."""
    per = m.n_kv_heads * 16 * m.head_dim
    return d.pool.view(m.n_layers, 2, d.n_blocks, per)


@pytest.mark.parametrize("kind", ["decode", "shared", "mixed"])
def test_pass_writes_only_its_own_slots(kind):
    m = MID
    rng = np.random.default_rng(40)
    if kind == "decode":
        w = decode_workload(m, rng.integers(0, 300, size=24), seed=40, name="sentinel-decode")
    elif kind == "shared":
        w = decode_workload(m, 128 + rng.integers(1, 60, size=10), seed=41, shared=128, name="sentinel-shared")
    else:
        w = mixed_workload(m, n_pre=2, plen=37, ctx=rng.integers(5, 200, size=6), seed=42, name="sentinel-mixed")
    d = _device(w)
    before = _pool_blocks(d, m).clone()
    slots = d.eng.batch_host()["slot"].astype(np.int64)
    others = []  # every other token of a block holding a new slot
    new_blocks = set(int(s) // 16 for s in slots)
    sset = set(int(s) for s in slots)
    for b in sorted(new_blocks):
        others += [b * 16 + t for t in range(16) if b * 16 + t not in sset]
    kv_before = [d.read_kv(l, np.asarray(others)) for l in range(m.n_layers)] if others else None
    d.step()
    torch.cuda.synchronize()
    after = _pool_blocks(d, m)
    changed = (after != before).any(dim=-1).cpu().numpy()  # [layer][kind][block]
    for l in range(m.n_layers):
        for k in range(2):
            blocks = set(np.nonzero(changed[l, k])[0].tolist())
            assert blocks <= new_blocks, (l, k, sorted(blocks - new_blocks)[:10])
            assert blocks == new_blocks, (l, k, "a new slot was not written")
    if others:
        for l in range(m.n_layers):
            Kb, Vb = kv_before[l]
            Ka, Va = d.read_kv(l, np.asarray(others))
            # poisoned (NaN) slots stay NaN, written ones keep their bytes
            np.testing.assert_array_equal(np.isnan(Ka), np.isnan(Kb))
            np.testing.assert_array_equal(np.nan_to_num(Ka), np.nan_to_num(Kb))
            np.testing.assert_array_equal(np.nan_to_num(Va), np.nan_to_num(Vb))
    d.release()


# ---------------------------------------------------------------- argmax_sample
def _argmax_rows(vocab, rng):
    rows = []
    rows.append(rng.standard_normal(vocab))                  # generic
    r = rng.standard_normal(vocab)
    r[[vocab // 3, vocab // 2, vocab - 1]] = 9.0             # tie: lowest index wins
    rows.append(r)
    r = rng.standard_normal(vocab)
    r[:: max(1, vocab // 7)] = np.nan                         # NaN never wins
    r[vocab // 2] = 7.5
    rows.append(r)
    rows.append(np.full(vocab, np.nan))                      # all NaN -> 0
    rows.append(np.full(vocab, -np.inf))                     # all -inf -> 0
    r = rng.standard_normal(vocab)
    r[[vocab - 1, vocab // 4]] = np.inf                       # +inf: lowest of them
    rows.append(r)
    r = np.zeros(vocab)
    r[::2] = -0.0                                            # signed zeros compare equal
    r[0] = -0.0
    rows.append(r)
    r = rng.standard_normal(vocab)
    r[-1] = 50.0                                             # maximum at the last index
    rows.append(r)
    r = np.full(vocab, -np.inf)
    r[vocab // 2:] = np.nan
    r[min(vocab - 1, 3)] = -1e30                             # one finite value among -inf/NaN
    rows.append(r)
    return np.stack(rows)


@pytest.mark.parametrize("vocab", [128256, 1001, 7, 1])
@pytest.mark.parametrize("dtype", [0, 1])
def test_argmax_sample_is_bit_exact(dtype, vocab):
    from paper_2609_37062_amd import vsk
    rng = np.random.default_rng(vocab + 7 * dtype)
    z = _argmax_rows(vocab, rng)
    if dtype == 0:
        t = torch.from_numpy(z.astype(np.float32)).to(torch.bfloat16)
        zin = t.float().numpy().astype(np.float64)
        t = t.view(torch.int16).cuda()
    else:
        t = torch.from_numpy(z.astype(np.float32)).cuda()
        zin = z.astype(np.float32).astype(np.float64)
    ids = torch.full((len(z),), -7, dtype=torch.int32, device="cuda")
    flags = torch.full((len(z),), -7, dtype=torch.int32, device="cuda")
    print(f"[gpu] argmax_sample dtype={dtype} vocab={vocab} rows={len(z)}", flush=True)
    vsk.argmax_sample(t.data_ptr(), dtype, len(z), vocab, ids.data_ptr(), torch.cuda.current_stream().cuda_stream,
                      flags.data_ptr())
    torch.cuda.synchronize()
    got = ids.cpu().numpy()
    want = nm.argmax_lowest(zin)
    np.testing.assert_array_equal(got, want)
    assert got[3] == 0 and got[4] == 0
    # the flag marks exactly the rows with no value that is not NaN
    np.testing.assert_array_equal(flags.cpu().numpy(), np.isnan(zin).all(axis=1).astype(np.int32))
    # without the flag buffer the ids are the same
    ids2 = torch.full((len(z),), -7, dtype=torch.int32, device="cuda")
    vsk.argmax_sample(t.data_ptr(), dtype, len(z), vocab, ids2.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ids2.cpu().numpy(), got)


def test_argmax_sample_rejects_bad_arguments():
    from paper_2609_37062_amd import vsk
    t = torch.zeros((2, 8), dtype=torch.float32, device="cuda")
    ids = torch.zeros(2, dtype=torch.int32, device="cuda")
    for args in [(t.data_ptr(), 2, 2, 8), (t.data_ptr(), 1, 0, 8), (t.data_ptr(), 1, 2, 0), (0, 1, 2, 8)]:
        with pytest.raises(vsk.VskError):
            vsk.argmax_sample(*args, ids.data_ptr())
