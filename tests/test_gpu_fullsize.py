"""Device parity at the full workload sizes, in the launch configuration the
benchmark times.

Sequences of a pass are independent, so the oracle recomputes a few sampled
sequences of the full batch end to end while the device runs the whole batch.

Checks per workload:
  * head, on every row that returns logits (the logits tolerance of the decode step): the
    oracle's final RMSNorm + lm_head applied to the device's own final
    residual stream must give the device's bf16 logits within 2e-2
    (logit_bound), and the device's greedy ids must equal the oracle's on
    every row whose top-2 gap exceeds 0.04 (the rest: within 0.04 of the
    maximum);
  * layer-local: at the first, middle and last layer the oracle applies that
    one layer to the device's residual stream before it; the layer's new K,V
    must agree within one bf16 ulp and the residual after it within
    LAYER_TOL of its RMS.  Inside one layer a 1e-4-level difference in the
    attention output already moves bf16 roundings of the MLP input, whose
    large update then carries them (measured 5e-3 on the 3B first layer);
  * sub-path isolation (3B and 8B): with the layer's down projection zeroed
    the layer is attention + O projection only, with its O projection zeroed
    it is the MLP only; each must match within PATH_TOL;
  * end to end from token ids on the sampled sequences: each row is held to
    max(2e-2, 3 x the oracle's own float32-vs-float64 spread on that row)
    (helpers.compare_logits).  Over 28-32 layers every row's bf16 rounding
    points flip under summation-order noise and each later normalisation
    amplifies the flips, so the float32 contract-mode oracle itself sits
    0.06-0.08 from the float64 one on these workloads.
"""
import time

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle.kvcache import PagedKV  # noqa: E402
from oracle.model import GeneratedWeights, forward  # noqa: E402
from workloads.configs import workload  # noqa: E402

from helpers import LOGIT_TOL, assert_bf16_close, compare_logits, e2e_compare, oracle_state  # noqa: E402

pytestmark = pytest.mark.gpu

LAYER_TOL = 2e-2   # max |x_dev - x_oracle| / rms(x_oracle) after one full layer
PATH_TOL = 2e-3    # the same after one isolated sub-path (attention or MLP)


def head_all_rows(w, W, x_final, lg, ids):
    """The 2e-2 bar on every logit row: the oracle's final norm + lm_head on
    the device's own final residual (x_final: all rows of the pass)."""
    m = w.model
    decode = all(s.q_len == 1 for s in w.seqs)
    lrows = np.arange(w.n_rows) if decode else w.logit_rows().astype(np.int64)
    dummy = PagedKV(m.n_layers, 1, m.n_kv_heads, m.head_dim)
    oh = forward(m, W, dummy, {"pos": None, "slot": None, "cu_q": None, "kv_len": None, "block_table": None},
                 np.zeros(len(lrows), np.int64), np.arange(len(lrows)), x0=x_final[lrows], layers=[])
    return compare_logits(lg[:len(lrows)], ids[:len(lrows)], oh["z"], tol=LOGIT_TOL)


def _check(w, subset, tuning=()):
    """Layer-local, head (all rows) and end-to-end checks of one workload;
    `tuning`: (key, value) pairs set on the device engine first."""
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
    x_all = None
    for k in need:
        d.set_layers(k)
        d.step()
        xa = d.residual()
        xs[k] = xa[rows]
        if k == L:
            x_all = xa
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
    print(f"[gpu] {w.name}: layer-local done {time.time() - t0:.1f}s", flush=True)
    # ---- head on the device's final residual, every logit row (the 2e-2 bar)
    stats["head"] = head_all_rows(w, W, x_all, lg, ids)
    print(f"[gpu] {w.name}: head {stats['head']}", flush=True)
    t2 = time.time()
    # ---- end to end from token ids on the sampled sequences
    stats["e2e"], *_ = e2e_compare(w, lg, ids, subset)
    print(f"[gpu] {w.name}: {stats} device {t1 - t0:.1f}s head {t2 - t1:.1f}s e2e {time.time() - t2:.1f}s",
          flush=True)
    d.release()
    return stats


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


def test_config2_persistent_step():
    """The persistent decode-step kernel (one launch per pass, tuning key 2 =
    2; the pass fails rather than fall back when it is not eligible) at the
    3B batch-16 workload: the same layer-local, head and end-to-end checks."""
    _check(workload(2), [0, 15], tuning=((2, 2),))


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
