"""Exact greedy-token agreement over more than 10,000 rows.

The device's greedy id (lowest index of the maximum fp32 logit) against the
oracle's on every row of 40 decode passes of 256 rows: the 1-layer tiny
model and a 2-layer GQA model, each over 20 seeds (weights, contexts, block
tables and tokens all drawn from the seed).

Several ids are correct on a near-tie.  Per pass the oracle's own float32
contract-mode run gives the bound of compare_logits (max(2e-2, 3 x its
largest float32-vs-float64 logit spread)); a row whose top-2 gap exceeds
twice that bound is decided and must agree exactly, and every other
disagreement must be within twice the bound of the maximum.  The raw exact
agreement is reported beside the float32 oracle's own raw agreement with the
float64 one and must reach 99.9%.  On the 2-layer model one bf16 rounding
flip moves logits by ~0.01, so raw agreement there is set by the near-tie
rate and by how often the implementation flips a rounding.  The device's
attention carries its softmax probabilities into P V as three bf16 terms
(about 24 significant bits, as a float32 run has); with two terms (about 16
bits) its attention outputs flipped more roundings and raw agreement was
10206/10240 = 99.67% against the float32 oracle's 99.92%; with three it is
10233/10240 = 99.93% (every decided row exact).  The full-size workloads add
their head rows in test_gpu_fullsize.py.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import numerics as nm  # noqa: E402
from workloads.configs import ModelCfg, decode_workload, workload  # noqa: E402

from helpers import LOGIT_TOL, SPREAD_K, oracle_run  # noqa: E402

pytestmark = pytest.mark.gpu

MID = ModelCfg("mid-2L", n_layers=2, hidden=512, n_q_heads=8, n_kv_heads=2, head_dim=128, ffn=1536,
               vocab=2048, rope_theta=500000.0)
SEEDS = range(20)
ROWS = 256


def _agreement(make):
    from paper_2609_37062_amd.runner import DeviceRun
    tot = {"rows": 0, "gpu": 0, "f32": 0, "decided": 0, "decided_agree": 0}
    for s in SEEDS:
        w = make(s)
        d = DeviceRun(w)
        d.step()
        lg, ids = d.results()
        d.release()
        out, *_, dev_rows = oracle_run(w)
        out32, *_ = oracle_run(w, dtype="f32")
        z, z32 = out["z"], out32["z"]
        got = ids[dev_rows]
        ref = nm.argmax_lowest(z)
        bound = max(LOGIT_TOL, SPREAD_K * float(np.abs(z32 - z).max()))
        srt = np.sort(z, axis=1)
        decided = srt[:, -1] - srt[:, -2] > 2 * bound
        ok = got == ref
        chosen = z[np.arange(len(z)), got]
        assert np.all(ok[decided]), (s, np.nonzero(decided & ~ok)[0])
        assert np.all(chosen >= z.max(axis=1) - 2 * bound), (s, np.nonzero(~ok)[0])
        tot["rows"] += len(z)
        tot["gpu"] += int(ok.sum())
        tot["f32"] += int((nm.argmax_lowest(z32) == ref).sum())
        tot["decided"] += int(decided.sum())
        tot["decided_agree"] += int(ok[decided].sum())
    return tot


def test_greedy_agreement_over_10k_rows():
    tiny = _agreement(lambda s: workload(1, seed=s, batch=ROWS))
    mid = _agreement(lambda s: decode_workload(MID, np.random.default_rng(1000 + s).integers(0, 600, size=ROWS),
                                               seed=s, name=f"mid-agree-{s}"))
    n = tiny["rows"] + mid["rows"]
    gpu = tiny["gpu"] + mid["gpu"]
    f32 = tiny["f32"] + mid["f32"]
    dec = tiny["decided"] + mid["decided"]
    print(f"[gpu] greedy agreement: tiny {tiny}, mid {mid}; device {gpu}/{n} = {gpu / n:.5f}, "
          f"float32 oracle {f32}/{n} = {f32 / n:.5f}, decided rows {dec}/{n} all exact", flush=True)
    assert n >= 10_000
    assert dec == tiny["decided_agree"] + mid["decided_agree"]
    assert tiny["gpu"] / tiny["rows"] >= 0.999
    assert gpu / n >= 0.999
