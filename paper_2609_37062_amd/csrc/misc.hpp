// Small-kernel launchers (see k_misc.hip).
#pragma once

#include "internal.hpp"

namespace vsk {

hipError_t launch_embed(const uint16_t* E, const int32_t* ids, int R, int H, int V, float* x, double* ssq,
                        hipStream_t s);
hipError_t launch_gather_rows(const float* x_in, int R_in, const int32_t* rows, int Ro, int H, float* x_out,
                              double* ssq_out, hipStream_t s);
// Where a normalised row goes in a routed layer: mask non-null puts row r at
// its cohort position inv[r], in the RUN buffer (the norm's own output) when
// mask[r] != 0 and in `po` otherwise.  A null mask keeps row r at row r.
struct CohortOut {
  const uint8_t* mask = nullptr;
  const int32_t* inv = nullptr;
  uint16_t* po = nullptr;
};
hipError_t launch_resid_norm(float* x, const float* y, int splits, int R, int H, const uint16_t* g, float eps,
                             uint16_t* hg, int Rg, hipStream_t s, CohortOut rc = {});
hipError_t launch_rmsnorm_frags(const float* x, const uint16_t* g, const double* ssq, int parts, int R, int H,
                                float eps, uint16_t* hg, int Rg, hipStream_t s, CohortOut rc = {});
// Routed layers (see k_misc.hip): Algorithm 1's maps of n_layers tapes of R
// rows ([n_layers][R] each, cnt [n_layers][2]), and the weighted scatter of
// the two cohorts' down-projection products into the residual (+ next norm).
hipError_t launch_route_maps(const uint8_t* tape, int n_layers, int R, int32_t* run, int32_t* proj, int32_t* inv,
                             int32_t* cnt, hipStream_t s);
hipError_t launch_route_reduce_norm(float* x, const float* y_run, int s_run, const float* y_po, int s_po,
                                    const uint8_t* mask, const int32_t* inv, const float* wts, int R, int H,
                                    const uint16_t* g, float eps, uint16_t* hg, int Rg, hipStream_t s);
hipError_t launch_argmax_partials(const float* pv, const int* pi, int n_groups, int R, int32_t* ids,
                                  hipStream_t s);
hipError_t launch_pack(const uint16_t* s0, const uint16_t* s1, const uint16_t* s2, int n0, int n1, int N, int K,
                       int perm_kind, int head_dim, int n_rope_rows, uint16_t* dst, hipStream_t s);
hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* out, int wgs, hipStream_t s);
hipError_t launch_kv_move(bool write, uint16_t* pool, int layer, int n_blocks, int Hkv, int hd,
                          const int32_t* slots, int n, uint16_t* k, uint16_t* v, hipStream_t s);

}  // namespace vsk
