// Profitability-aware mode switching: host pure functions of the C ABI.
//
// Routed mode (a per-layer RUN / Project-Only choice per row) carries a fixed
// cost per step; in decode below the ridge point the weights stream anyway,
// so what a Project-Only row saves is its attention read of that layer's KV.
// The paper's decode rule (Section 3.3 and appendix "The Switching
// Thresholds from the Roofline") therefore compares the fixed cost tau with
// the bytes skipped per step, s * L_r * b * V over the bandwidth, and routes
// when the resident KV tokens V exceed V* = tau * BW / (s * L_r * b).  tau
// is measured once over a reference number of routed layers and scales with
// the routed layers of the model at hand, so L_r cancels.  The served
// thresholds are a hysteresis band: exit at V*, enter at 1.25 V*, both
// rounded to 10k tokens (the rounding is read off the printed thresholds).
// Decode mode is set when a request starts decoding and may be promoted once
// from dense to routed when V crosses the enter threshold; it never reverts.
// Prefill routes a batch with at least a floor of prompt tokens whose
// estimated Project-Only share exceeds a threshold (Section 3.3, Prefill).
#include <cmath>

#include "../../include/vsk.h"

namespace {

bool finite_pos(double v) { return std::isfinite(v) && v > 0.0; }

int64_t round_to(double v, double unit) {
  if (!(unit > 0.0)) return static_cast<int64_t>(std::floor(v + 0.5));
  return static_cast<int64_t>(std::floor(v / unit + 0.5)) * static_cast<int64_t>(unit);
}

}  // namespace

extern "C" {

int vsk_switch_thresholds(const vsk_switch_params* p, vsk_switch_band* out) {
  if (!p || !out) return VSK_E_ARG;
  if (!finite_pos(p->tau_s) || p->tau_layers < 1 || !finite_pos(p->bw_bytes_per_s) || !finite_pos(p->skip) ||
      p->skip > 1.0 || p->routed_layers < 1 || !finite_pos(p->kv_bytes_per_token_layer) ||
      !(p->enter_factor >= 1.0) || !std::isfinite(p->enter_factor) || !(p->round_tokens >= 0.0))
    return VSK_E_ARG;
  // tau scales with the routed layers: tau_eff = tau * L_r / tau_layers
  const double tau_eff = p->tau_s * static_cast<double>(p->routed_layers) / static_cast<double>(p->tau_layers);
  const double saved_per_token = p->skip * static_cast<double>(p->routed_layers) * p->kv_bytes_per_token_layer;
  out->v_star = tau_eff * p->bw_bytes_per_s / saved_per_token;
  out->exit_tokens = round_to(out->v_star, p->round_tokens);
  out->enter_tokens = round_to(p->enter_factor * out->v_star, p->round_tokens);
  return VSK_OK;
}

int vsk_switch_step(const vsk_switch_band* t, int32_t routing_in, int64_t resident_tokens, int32_t* routing_out,
                    int32_t* promote) {
  if (!t || !routing_out || resident_tokens < 0 || (routing_in != 0 && routing_in != 1)) return VSK_E_ARG;
  if (t->exit_tokens > t->enter_tokens) return VSK_E_ARG;
  int32_t r = routing_in;
  if (resident_tokens >= t->enter_tokens) r = 1;
  else if (resident_tokens <= t->exit_tokens) r = 0;
  *routing_out = r;
  if (promote) *promote = (routing_in == 0 && r == 1) ? 1 : 0;
  return VSK_OK;
}

int vsk_switch_decode_mode(int32_t mode_in, int32_t routing, int32_t promote, int32_t* mode_out) {
  if (!mode_out || mode_in < -1 || mode_in > 1 || (routing != 0 && routing != 1) || (promote != 0 && promote != 1))
    return VSK_E_ARG;
  if (mode_in < 0) *mode_out = routing;          // starts decoding now: the current state
  else if (mode_in == 1) *mode_out = 1;          // routed never reverts
  else *mode_out = promote ? 1 : 0;              // dense: promoted once by a crossing
  return VSK_OK;
}

int vsk_switch_prefill(int64_t prompt_tokens, double po_share, int64_t floor_tokens, double share_min,
                       int32_t* routed) {
  if (!routed || prompt_tokens < 0 || floor_tokens < 0 || !std::isfinite(po_share) || po_share < 0.0 ||
      po_share > 1.0 || !std::isfinite(share_min))
    return VSK_E_ARG;
  *routed = (prompt_tokens >= floor_tokens && po_share > share_min) ? 1 : 0;
  return VSK_OK;
}

}  // extern "C"
