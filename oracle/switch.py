"""The mode switch: when routed execution pays, and who gets it.

Test infrastructure only (see the package docstring).

Written from Section 3.3 ("Profitability-Aware Mode Switching") and the
appendix "The Switching Thresholds from the Roofline":

* Decode below the ridge point streams the weights whatever the rows do, so
  a Project-Only row saves only its attention read of the layer's KV:
  b bytes per resident token per routed layer.  With a share s of the
  decisions projecting over L_r routed layers, a step holding V resident
  tokens skips s * L_r * b * V bytes, worth that over BW seconds, against the
  routed mode's fixed cost tau per step.  tau was measured over 16 routed
  layers and is reused per routed layer (scaled by L_r / 16), so
      V* = (tau * L_r / 16) * BW / (s * L_r * b).
* Thresholds of the hysteresis band: exit at V*, enter at 1.25 V*.  The
  printed thresholds are multiples of 10k tokens; reading: each is rounded to
  the nearest 10k (this reproduces every printed pair).
* Switching state: on once V reaches the enter threshold, off once V falls
  to the exit threshold, unchanged in between.  A request that starts
  decoding takes the current state; the off-to-on crossing promotes the
  requests already decoding densely; a routed request never goes back.
* Prefill: routed when the admitted batch holds at least 1,536 prompt tokens
  and the estimated Project-Only share exceeds 0.35.

Parity: pinned by the values the paper prints (tests/test_oracle_switch.py).
"""
from __future__ import annotations

import math


def v_star(tau_s, bw_bytes_per_s, skip, routed_layers, kv_bytes, tau_layers=16):
    """The crossover resident-token count V* (float)."""
    tau_eff = tau_s * routed_layers / tau_layers
    return tau_eff * bw_bytes_per_s / (skip * routed_layers * kv_bytes)


def round_tokens(v, unit=10000):
    """Nearest multiple of ``unit`` (halves round up); unit 0: nearest integer."""
    if unit <= 0:
        return int(math.floor(v + 0.5))
    return int(math.floor(v / unit + 0.5)) * int(unit)


def thresholds(tau_s, bw_bytes_per_s, skip, routed_layers, kv_bytes, tau_layers=16, enter_factor=1.25,
               unit=10000):
    """(V*, exit, enter)."""
    vs = v_star(tau_s, bw_bytes_per_s, skip, routed_layers, kv_bytes, tau_layers)
    return vs, round_tokens(vs, unit), round_tokens(enter_factor * vs, unit)


def switch_state(routing, resident, exit_tokens, enter_tokens):
    """Next switching state and whether this observation promotes running dense decodes."""
    if resident >= enter_tokens:
        nxt = 1
    elif resident <= exit_tokens:
        nxt = 0
    else:
        nxt = routing
    return nxt, int(routing == 0 and nxt == 1)


def decode_mode(mode_in, routing, promote):
    """mode_in: None (starts decoding now), 0 dense, 1 routed."""
    if mode_in is None:
        return routing
    if mode_in == 1:
        return 1
    return 1 if promote else 0


def prefill_routed(prompt_tokens, po_share, floor_tokens=1536, share_min=0.35):
    return int(prompt_tokens >= floor_tokens and po_share > share_min)


def simulate(trace, exit_tokens, enter_tokens):
    """Replay a serving trace through the switch.

    trace: list of steps; each step is (resident tokens V, ids of requests that
    start decoding at this step, ids that finish).  Returns the per-step
    switching state and the mode of every request at the end of each step.
    """
    routing = 0
    modes = {}
    out = []
    for V, starts, finishes in trace:
        routing, promote = switch_state(routing, V, exit_tokens, enter_tokens)
        for r in list(modes):
            modes[r] = decode_mode(modes[r], routing, promote)
        for r in starts:
            modes[r] = decode_mode(None, routing, promote)
        for r in finishes:
            modes.pop(r, None)
        out.append((routing, dict(modes)))
    return out
