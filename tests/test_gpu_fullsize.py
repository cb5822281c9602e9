"""Device parity at the full workload sizes, in the launch configuration the
benchmark times, on sampled sequences.

Sequences of a pass are independent, so the oracle recomputes a few sampled
sequences of the full batch while the device runs the whole batch.

Checks per workload:
  * head (the spec bar): the oracle's final RMSNorm + lm_head applied
    to the device's own final residual stream must give the device's bf16
    logits within 2e-2, with the same greedy id up to near-ties;
  * layer-local: at the first, middle and last layer the oracle applies that
    one layer to the device's residual stream before it; the layer's new K,V
    must agree within one bf16 ulp and the residual after it within
    LAYER_TOL of its RMS.  Inside one layer a 1e-4-level difference in the
    attention output already moves bf16 roundings of the MLP input, whose
    large update then carries them (measured 5e-3 on the 3B first layer);
  * sub-path isolation (3B and 8B): with the layer's down projection zeroed
    the layer is attention + O projection only, with its O projection zeroed
    it is the MLP only; each must match within PATH_TOL;
  * end to end: the device logits against the oracle run from the token ids
    alone; ids must agree up to near-ties and the logits within E2E_BOUND.
    Over 28-32 layers the bf16 rounding points amplify summation-order
    differences: the oracle itself moves by up to 0.06 on these workloads
    when only its matrix products switch from float64 to float32 (measured
    on the 3B batch-16 workload), so the end-to-end bound is set at 4x that.
"""
import time

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle.model import GeneratedWeights, forward  # noqa: E402
from workloads.configs import workload  # noqa: E402

from helpers import LOGIT_TOL, compare_logits, oracle_run, oracle_state  # noqa: E402

pytestmark = pytest.mark.gpu

LAYER_TOL = 2e-2   # max |x_dev - x_oracle| / rms(x_oracle) after one full layer
PATH_TOL = 2e-3    # the same after one isolated sub-path (attention or MLP)
E2E_BOUND = 0.25   # end-to-end logits bound (see module docstring)


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


def _check(w, subset, tuning=()):
    """Layer-local, head and end-to-end checks of one workload; `tuning`:
    (key, value) pairs set on the device engine first."""
    from paper_2609_37062_amd.runner import DeviceRun
    t0 = time.time()
    m = w.model
    L = m.n_layers
    print(f"[gpu] {w.name}: seqs={w.n_seqs} rows={w.n_rows} sample={subset} tuning={list(tuning)}", flush=True)
    d = DeviceRun(w, poison_pool=True)
    for k, v in tuning:
        d.eng.set_tuning(k, v)
    a, batch, sub, rows, kv, idx = oracle_state(w, subset)
    ks = sorted({1, L // 2, L})
    need = sorted({k for k in ks} | {k - 1 for k in ks if k > 1})
    xs = {}
    for k in need:
        d.set_layers(k)
        d.step()
        xs[k] = d.residual()[rows]
    d.set_layers(0)
    d.step()
    lg, ids = d.results()
    knew = {}
    for k in ks:
        knew[k] = d.read_kv(k - 1, sub["slot"])
    t1 = time.time()
    W = GeneratedWeights(m, w.seed)
    stats = {}
    # ---- layer-local
    tok = w.tokens[rows]
    for k in ks:
        x0 = None if k == 1 else xs[k - 1]
        o = forward(m, W, kv, sub, tok, None, x0=x0, layers=[k - 1])
        err = np.abs(xs[k] - o["x"]).max() / np.sqrt(np.mean(o["x"] ** 2))
        stats[f"layer{k}_rel_err"] = float(err)
        Ko, Vo = kv.read(k - 1, sub["slot"])
        assert_bf16_close(knew[k][0], Ko, f"K layer {k - 1}")
        assert_bf16_close(knew[k][1], Vo, f"V layer {k - 1}")
        assert err <= LAYER_TOL, (k, err)
    # ---- head on the device's final residual (the 2e-2 bar)
    _, _, _, _, dev_rows = oracle_run_rows(w, idx)
    lrows = logit_rows_local(w, idx, sub)
    oh = forward(m, W, kv, sub, tok, lrows, x0=xs[L], layers=[])
    stats["head"] = compare_logits(lg[dev_rows], ids[dev_rows], oh["z"], tol=LOGIT_TOL)
    t2 = time.time()
    # ---- end to end from token ids
    out, *_ = oracle_run(w, subset)
    st = compare_logits(lg[dev_rows], ids[dev_rows], out["z"], tol=E2E_BOUND)
    stats["e2e"] = st
    print(f"[gpu] {w.name}: {stats} device {t1 - t0:.1f}s oracle {time.time() - t1:.1f}s", flush=True)
    d.release()
    return stats


def logit_rows_local(w, idx, sub):
    """Rows of the sub-batch that return logits."""
    if all(s.q_len == 1 for s in w.seqs):
        return np.arange(len(idx))
    return np.asarray([int(sub["cu_q"][j + 1]) - 1 for j, i in enumerate(idx) if w.seqs[i].logits])


def oracle_run_rows(w, idx):
    """Device output rows of the sampled sequences (same mapping as oracle_run)."""
    if all(s.q_len == 1 for s in w.seqs):
        return None, None, None, None, np.asarray(idx)
    out_pos, k = {}, 0
    for i, s in enumerate(w.seqs):
        if s.logits:
            out_pos[i] = k
            k += 1
    return None, None, None, None, np.asarray([out_pos[i] for i in idx if w.seqs[i].logits])


def _isolated_paths(w, subset):
    """First layer with W_down = 0 (attention + O only), then with W_o = 0 (MLP only)."""
    from paper_2609_37062_amd.runner import DeviceRun
    m = w.model
    out = {}
    for name, over in [("attention", {("w_down", 0): np.zeros((m.hidden, m.ffn), np.float32)}),
                       ("mlp", {("wo", 0): np.zeros((m.hidden, m.q_dim), np.float32)})]:
        d = DeviceRun(w, overrides=over)
        d.set_layers(1)
        d.step()
        x = d.residual()
        d.release()
        del d
        torch.cuda.empty_cache()
        a, batch, sub, rows, kv, idx = oracle_state(w, subset)
        W = GeneratedWeights(m, w.seed, overrides={k: v.astype(np.float64) for k, v in over.items()})
        o = forward(m, W, kv, sub, w.tokens[rows], None, layers=[0])
        err = float(np.abs(x[rows] - o["x"]).max() / np.sqrt(np.mean(o["x"] ** 2)))
        out[name] = err
        assert err <= PATH_TOL, (name, err)
    print(f"[gpu] {w.name} isolated sub-paths: {out}", flush=True)
    return out


def test_config2_3b_decode_b16():
    _check(workload(2), [0, 15])


def test_config2_isolated_paths():
    _isolated_paths(workload(2), [0, 5])


def test_config5_isolated_paths():
    _isolated_paths(workload(5), [0, 77])


def test_config3_3b_shared_prefix_b64():
    _check(workload(3), [0, 63])


def test_config4_3b_mixed_prefill_decode():
    # one 512-token prefill request and two decoding sequences
    _check(workload(4), [1, 4, 35])


def test_config5_8b_decode_b128():
    w = workload(5)
    ctx = np.array([s.ctx for s in w.seqs])
    _check(w, sorted({0, int(np.argmax(ctx))}))
