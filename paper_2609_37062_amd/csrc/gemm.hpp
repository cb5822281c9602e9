// Projection kernel interface (see k_gemm.hip).
#pragma once

#include "internal.hpp"

namespace vsk {

enum { EPI_RESID = 0, EPI_QKV = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3 };

struct GemmArgs {
  const uint32_t __attribute__((ext_vector_type(4)))* W;  // packed tiles
  const uint32_t __attribute__((ext_vector_type(4)))* X;  // activation frags
  int Kt;       // K / 32
  int N;        // output columns
  int R;        // valid rows
  int Rg;       // 16-row groups of the X frag buffer
  float* x;          // RESID: fp32 residual [R][N], x += y
  double* ssq_out;   // RESID: partial sums of x^2 of the updated rows [R][n_groups]
  uint16_t* out;  // QKV: q [R][Nq]; SWIGLU: frags (out_Rg); LOGITS: logits [R][N]
  int out_Rg;
  uint16_t* pool;  // QKV: KV pool
  int layer, n_blocks, Hkv, hd, Nq, Nkv;
  const int32_t* slot;
  const int32_t* pos;
  const float2* rope;  // [max_pos][hd/2] (cos, sin)
  float* am_val;       // LOGITS: [n_groups][R]
  int* am_idx;
  float* ypart;  // RESID with K split over workgroups: y[split][R][N] instead of x += y
  const int* count;  // nullable: rows of this launch read on the device (<= R; a cohort's size)
  int xcd_remap;     // row-tiled passes: row tiles of one N group on one XCD at the same time
};

struct GemmPlan {
  int mg = 1;        // 16-row groups per tile
  int m_tiles = 1;   // tiles along the rows
  int n_groups = 1;  // workgroups along N (also the number of x^2 partials a RESID emits)
  int nt = 1;        // N tiles per wave
  int wn = 1;        // waves side by side along N
  int ksplit = 1;    // RESID: workgroups along K, their products added by k_resid_norm
  bool xl = false;   // X chunks staged in LDS by a loader wave, shared by the compute waves
};

constexpr int kMaxResidSplits = 8;
constexpr int kResidTargetWgs = 0;  // default split-K target of the residual projections (0: no split)
constexpr int kQkvTargetWgs = 192;  // default split-K target of QKV at 4..8 row groups
constexpr int kRowTiledSplitBelow = 128;  // row-tiled residual projections split K at or below these workgroups
constexpr int kRowTiledTarget = 256;      // into as many splits as stay within this many workgroups
constexpr int kComputeUnits = 256;        // MI355X: 8 XCDs x 32 compute units

// shape: launch shape for 4 or 8 row groups (0 default; see k_gemm.hip)
// resid_target: workgroups a residual projection's K split aims for (-1: no
// split; 0: the layout's default -- 192 or 384 with X in LDS, 192 for the
// two-tile layout of the down projection at <= 16 rows, else
// kResidTargetWgs)
// row_tile: 16-row groups per tile of a row-tiled projection other than the
// lm_head (0: chosen from the launch rounds; 6, 7, 8 or 11: that height)
GemmPlan plan_gemm(int N, int K, int R, int epi, int shape = 0, int resid_target = 0, int row_tile = 0);
hipError_t launch_gemm(GemmArgs a, const GemmPlan& p, int epi, hipStream_t s, LaunchEvents ev = {});
// QKV with K split: add the `splits` products in a.ypart and apply the QKV
// epilogue (a as for the QKV projection, with N = Nq + 2 Nkv).
hipError_t launch_qkv_reduce(const GemmArgs& a, int splits, hipStream_t s);

}  // namespace vsk
