"""Route tapes: per routed layer and row, RUN or Project-Only and a weight.

Input generators for routed mode (no arithmetic of the pass).  A tape is
(run [n_routed][rows] bool, w [n_routed][rows] float32): a RUN row adds
w times its MLP output to the residual, a Project-Only row adds (1 - w) times
its projector output and reads no KV at that layer.  The policies follow the
paper's examples:

  * static_depth(ratio): the last floor(n_routed * ratio) routed layers
    project every valid row, the others run it (the static-depth plugin of
    the appendix "A Minimal Skipper Plugin"); binary weights (w = 1 for RUN,
    0 for Project-Only, so the chosen branch gets weight 1).
  * random_skip(r, d): a request skips with probability r (a seeded hash of
    the request), and a skipping request's token projects at each routed
    layer with probability d (a seeded hash of request, token position and
    layer), so the expected skip share is s = r * d (the RandomSkip grid of
    the roofline appendix); binary weights.
  * router_weights: a weight per (layer, row) uniform in [0, 1] standing in
    for a trained router's output, RUN when w > 0.5 (the released router's
    rule, appendix "Route-Guided Cohort Execution at the Kernel Level").
"""
from __future__ import annotations

import numpy as np

from . import gen


def _unit(key, idx):
    """Uniform [0, 1) from the counter-based hash of element indices idx."""
    h = np.array([gen.hash_np(key, int(i), 1)[0] for i in np.asarray(idx).ravel()], np.uint64)
    return (h.astype(np.float64) / 2.0 ** 32).reshape(np.shape(idx))


def static_depth(n_routed, rows, ratio):
    if not 0.0 <= ratio <= 1.0:
        raise ValueError("ratio must be in [0, 1]")
    take = int(n_routed * ratio)
    run = np.ones((n_routed, rows), bool)
    run[n_routed - take:, :] = False
    return run, run.astype(np.float32)


def random_skip(seed, n_routed, req_ids, positions, r, d):
    """req_ids, positions: per row (the request and the token position of the row)."""
    req_ids = np.asarray(req_ids, np.int64)
    positions = np.asarray(positions, np.int64)
    k_req = gen.key_of(seed, "randomskip-request")
    skipping = _unit(k_req, req_ids) < r
    run = np.ones((n_routed, len(req_ids)), bool)
    for l in range(n_routed):
        k = gen.key_of(seed, "randomskip-token", l)
        u = _unit(k, req_ids * 1_000_003 + positions)
        run[l] = ~(skipping & (u < d))
    return run, run.astype(np.float32)


def router_weights(seed, n_routed, rows):
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 77])))
    w = rng.random((n_routed, rows)).astype(np.float32)
    return w > 0.5, w


def all_run(n_routed, rows):
    return np.ones((n_routed, rows), bool), np.ones((n_routed, rows), np.float32)
