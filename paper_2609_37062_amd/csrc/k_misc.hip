// Small kernels of the pass: embedding gather, logit-row gather, greedy
// argmax, weight repacking, KV scatter/gather, workspace clearing.
#include <climits>
#include <cmath>

#include "dev.hpp"
#include "misc.hpp"

namespace vsk {

// ---------------------------------------------------------------- embedding
// x[r][:] = float(E[ids[r]][:]) (fp32 residual), plus what the first QKV
// projection consumes: frags of bf16(x * g) and per-16-column partial sums
// of x^2 (one per row: ssq[r]).  Token ids outside [0, V) give a zero row.
__global__ __launch_bounds__(256) void k_embed(const uint16_t* __restrict__ E, const int32_t* __restrict__ ids,
                                               int H, int V, float* __restrict__ x, double* __restrict__ ssq) {
  __shared__ double s_ss[4];
  const int r = blockIdx.x;
  const int id = ids[r];
  const bool valid = id >= 0 && id < V;
  const size_t base = valid ? static_cast<size_t>(id) * H : 0;
  double ss = 0.0;
  for (int c = threadIdx.x * 8; c < H; c += blockDim.x * 8) {
    u32x4 v = valid ? *reinterpret_cast<const u32x4*>(E + base + c) : u32x4{0u, 0u, 0u, 0u};
    float e[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      e[2 * k] = bf2f(v[k] & 0xffffu);
      e[2 * k + 1] = bf2f(v[k] >> 16);
    }
    float4* dst = reinterpret_cast<float4*>(x + static_cast<size_t>(r) * H + c);
    dst[0] = make_float4(e[0], e[1], e[2], e[3]);
    dst[1] = make_float4(e[4], e[5], e[6], e[7]);
#pragma unroll
    for (int k = 0; k < 8; ++k) ss += static_cast<double>(e[k]) * e[k];
  }
  // whole-row sum of x^2 in a fixed order: one partial per row
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
  if ((threadIdx.x & 63) == 0) s_ss[threadIdx.x >> 6] = ss;
  __syncthreads();
  if (threadIdx.x == 0) ssq[r] = (s_ss[0] + s_ss[1]) + (s_ss[2] + s_ss[3]);
}

hipError_t launch_embed(const uint16_t* E, const int32_t* ids, int R, int H, int V, float* x, double* ssq,
                        hipStream_t s) {
  hipLaunchKernelGGL(k_embed, dim3(R), dim3(256), 0, s, E, ids, H, V, x, ssq);
  return hipGetLastError();
}

// ---------------------------------------------------------------- row gather
// Compact the residual rows that return logits (a prefill pass asks for a
// few rows out of many) with each row's sum of x^2 (one partial per row, in
// a fixed order).  Indices outside [0, R_in) give a zero row.
__global__ __launch_bounds__(256) void k_gather_rows(const float* __restrict__ x_in, int R_in,
                                                     const int32_t* __restrict__ rows, int H,
                                                     float* __restrict__ x_out, double* __restrict__ ssq_out) {
  __shared__ double s_ss[4];
  const int i = blockIdx.x;
  const int src = rows[i];
  const bool valid = src >= 0 && src < R_in;
  double ss = 0.0;
  for (int c = threadIdx.x * 4; c < H; c += blockDim.x * 4) {
    const float4 v = valid ? *reinterpret_cast<const float4*>(x_in + static_cast<size_t>(src) * H + c)
                           : make_float4(0.f, 0.f, 0.f, 0.f);
    *reinterpret_cast<float4*>(x_out + static_cast<size_t>(i) * H + c) = v;
    ss += static_cast<double>(v.x) * v.x + static_cast<double>(v.y) * v.y + static_cast<double>(v.z) * v.z +
          static_cast<double>(v.w) * v.w;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
  if ((threadIdx.x & 63) == 0) s_ss[threadIdx.x >> 6] = ss;
  __syncthreads();
  if (threadIdx.x == 0) ssq_out[i] = (s_ss[0] + s_ss[1]) + (s_ss[2] + s_ss[3]);
}

hipError_t launch_gather_rows(const float* x_in, int R_in, const int32_t* rows, int Ro, int H, float* x_out,
                              double* ssq_out, hipStream_t s) {
  hipLaunchKernelGGL(k_gather_rows, dim3(Ro), dim3(256), 0, s, x_in, R_in, rows, H, x_out, ssq_out);
  return hipGetLastError();
}

// ---------------------------------------------------------------- RMSNorm
// h = bf16(x * g / sqrt(mean(x^2) + eps)), written as frags for the
// projection that follows (the rounding point of the norm's output).  The
// residual projection that produced x also wrote per-workgroup partial sums
// of x^2; every workgroup of a row adds them in the same fixed order, so all
// of them hold the same r, and the row is normalised in one pass over x.
// One wave per 512 elements of a row: each lane writes 8 (one 16-byte frag
// piece); the product is taken in double and rounded once.
// Routed layer (rc.mask non-null): the row is written at its position in
// its cohort, into hg for a RUN row and rc.po for a Project-Only row -- the
// cohort gather of Algorithm 1 folded into the producer of the operand.
__global__ __launch_bounds__(64) void k_rmsnorm_frags(const float* __restrict__ x, const uint16_t* __restrict__ g,
                                                      const double* __restrict__ ssq, int parts, int R, int H,
                                                      float eps, uint16_t* __restrict__ hg, int Rg, CohortOut rc) {
  const int r = blockIdx.y;
  const int c = blockIdx.x * 512 + threadIdx.x * 8;
  const bool on = c < H;
  const float* xr = x + static_cast<size_t>(r) * H;
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
  u32x4 gv = u32x4{0u, 0u, 0u, 0u};
  if (on) {
    a = *reinterpret_cast<const float4*>(xr + c);
    b = *reinterpret_cast<const float4*>(xr + c + 4);
    gv = *reinterpret_cast<const u32x4*>(g + c);
  }
  // partials p = lane, lane + 64, ... added in that order; four are loaded
  // before the first is added, so their latencies overlap
  double s = 0.0;
  for (int p0 = threadIdx.x; p0 < parts; p0 += 256) {
    double v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = p0 + 64 * q < parts ? ssq[static_cast<size_t>(r) * parts + p0 + 64 * q] : 0.0;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (p0 + 64 * q < parts) s += v[q];
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
  const double rr = 1.0 / sqrt(s / static_cast<double>(H) + static_cast<double>(eps));
  if (!on) return;
  const float e[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  u32x4 o;
#pragma unroll
  for (int k = 0; k < 4; ++k)
    o[k] = d2bf(static_cast<double>(e[2 * k]) * bf2f(gv[k] & 0xffffu) * rr) |
           (d2bf(static_cast<double>(e[2 * k + 1]) * bf2f(gv[k] >> 16) * rr) << 16);
  int ro = r;
  uint16_t* dst = hg;
  if (rc.mask != nullptr) {
    ro = rc.inv[r];
    if (rc.mask[r] == 0) dst = rc.po;
  }
  *reinterpret_cast<u32x4*>(dst + frag_index(ro, c, Rg)) = o;
}

// ---------------------------------------------------------------- residual sum + RMSNorm
// A residual projection whose K was split over workgroups leaves one fp32
// partial product per split (y[split][row][col]).  One workgroup per row,
// one thread per 8 columns, adds them to the residual in split order,
// x += ((y0 + y1) + y2) + ..., stores x, and (gain non-null) normalises the
// row into bf16 frags of x * g / sqrt(mean(x^2) + eps) -- the sum of squares
// in double, added in a fixed order, the product in double and rounded once.
// Every load of a thread (x, all splits, g) is issued before the first add,
// so the row costs one memory round trip, not one per split.
// NS > 0: exactly NS splits (compile-time: every load unconditional); NS = 0:
// `splits` of them, at most kResidNormMaxSplits.
constexpr int kResidNormMaxSplits = 8;
template <int NS>
__global__ __launch_bounds__(1024) void k_resid_norm(float* __restrict__ x, const float* __restrict__ y, int splits,
                                                     int R, int H, const uint16_t* __restrict__ g, float eps,
                                                     uint16_t* __restrict__ hg, int Rg, CohortOut rc) {
  if constexpr (NS > 0) splits = NS;
  constexpr int kMax = NS > 0 ? NS : kResidNormMaxSplits;
  __shared__ double s_ss[16];
  const int r = blockIdx.x;
  const int c = threadIdx.x * 8;
  const bool on = c < H;
  float* xr = x + static_cast<size_t>(r) * H + c;
  float e[8];
  u32x4 gv = u32x4{0u, 0u, 0u, 0u};
  double ss = 0.0;
  if (on) {
    float4 a = *reinterpret_cast<const float4*>(xr);
    float4 b = *reinterpret_cast<const float4*>(xr + 4);
    float4 ya[kMax], yb[kMax];
#pragma unroll
    for (int sp = 0; sp < kMax; ++sp) {
      if (NS > 0 || sp < splits) {
        const float* yr = y + (static_cast<size_t>(sp) * R + r) * H + c;
        ya[sp] = *reinterpret_cast<const float4*>(yr);
        yb[sp] = *reinterpret_cast<const float4*>(yr + 4);
      }
    }
    if (g != nullptr) gv = *reinterpret_cast<const u32x4*>(g + c);
    float4 sa = ya[0], sb = yb[0];
#pragma unroll
    for (int sp = 1; sp < kMax; ++sp) {
      if (NS > 0 || sp < splits) {
        sa.x += ya[sp].x; sa.y += ya[sp].y; sa.z += ya[sp].z; sa.w += ya[sp].w;
        sb.x += yb[sp].x; sb.y += yb[sp].y; sb.z += yb[sp].z; sb.w += yb[sp].w;
      }
    }
    a.x += sa.x; a.y += sa.y; a.z += sa.z; a.w += sa.w;
    b.x += sb.x; b.y += sb.y; b.z += sb.z; b.w += sb.w;
    *reinterpret_cast<float4*>(xr) = a;
    *reinterpret_cast<float4*>(xr + 4) = b;
    e[0] = a.x; e[1] = a.y; e[2] = a.z; e[3] = a.w;
    e[4] = b.x; e[5] = b.y; e[6] = b.z; e[7] = b.w;
#pragma unroll
    for (int q = 0; q < 8; ++q) ss += static_cast<double>(e[q]) * e[q];
  }
  if (g == nullptr) return;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
  if ((threadIdx.x & 63) == 0) s_ss[threadIdx.x >> 6] = ss;
  __syncthreads();
  double tot = 0.0;
  for (int w = 0; w < static_cast<int>(blockDim.x >> 6); ++w) tot += s_ss[w];
  const double rr = 1.0 / sqrt(tot / static_cast<double>(H) + static_cast<double>(eps));
  if (!on) return;
  u32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    o[q] = d2bf(static_cast<double>(e[2 * q]) * bf2f(gv[q] & 0xffffu) * rr) |
           (d2bf(static_cast<double>(e[2 * q + 1]) * bf2f(gv[q] >> 16) * rr) << 16);
  int ro = r;
  uint16_t* dst = hg;
  if (rc.mask != nullptr) {  // routed layer: the row's place in its cohort
    ro = rc.inv[r];
    if (rc.mask[r] == 0) dst = rc.po;
  }
  *reinterpret_cast<u32x4*>(dst + frag_index(ro, c, Rg)) = o;
}

hipError_t launch_resid_norm(float* x, const float* y, int splits, int R, int H, const uint16_t* g, float eps,
                             uint16_t* hg, int Rg, hipStream_t s, CohortOut rc) {
  if (H % 8 != 0 || H > 8192 || splits < 1 || splits > kResidNormMaxSplits) return hipErrorInvalidValue;
  const int threads = (H / 8 + 63) / 64 * 64;
  switch (splits) {
    case 2: hipLaunchKernelGGL(k_resid_norm<2>, dim3(R), dim3(threads), 0, s, x, y, splits, R, H, g, eps, hg, Rg, rc); break;
    case 4: hipLaunchKernelGGL(k_resid_norm<4>, dim3(R), dim3(threads), 0, s, x, y, splits, R, H, g, eps, hg, Rg, rc); break;
    case 8: hipLaunchKernelGGL(k_resid_norm<8>, dim3(R), dim3(threads), 0, s, x, y, splits, R, H, g, eps, hg, Rg, rc); break;
    default: hipLaunchKernelGGL(k_resid_norm<0>, dim3(R), dim3(threads), 0, s, x, y, splits, R, H, g, eps, hg, Rg, rc);
  }
  return hipGetLastError();
}

hipError_t launch_rmsnorm_frags(const float* x, const uint16_t* g, const double* ssq, int parts, int R, int H,
                                float eps, uint16_t* hg, int Rg, hipStream_t s, CohortOut rc) {
  hipLaunchKernelGGL(k_rmsnorm_frags, dim3((H + 511) / 512, R), dim3(64), 0, s, x, g, ssq, parts, R, H, eps, hg, Rg,
                     rc);
  return hipGetLastError();
}

// ---------------------------------------------------------------- routed layers
// Algorithm 1's maps, rebuilt on the device from the route tape for every
// pass (Invariant 2): for each routed layer (one workgroup each), run[] and
// proj[] list the batch rows of the RUN and Project-Only cohorts in row
// order, inv[r] is row r's position in its own cohort, and cnt = (n_r, n_p).
// A block-wide exclusive scan of the RUN flags over chunks of blockDim rows.
__global__ __launch_bounds__(1024) void k_route_maps(const uint8_t* __restrict__ tape, int R,
                                                     int32_t* __restrict__ run, int32_t* __restrict__ proj,
                                                     int32_t* __restrict__ inv, int32_t* __restrict__ cnt) {
  __shared__ int s_w[16];
  __shared__ int s_base;
  const int l = blockIdx.x;
  const uint8_t* t = tape + static_cast<size_t>(l) * R;
  run += static_cast<size_t>(l) * R;
  proj += static_cast<size_t>(l) * R;
  inv += static_cast<size_t>(l) * R;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  if (threadIdx.x == 0) s_base = 0;
  __syncthreads();
  for (int r0 = 0; r0 < R; r0 += blockDim.x) {
    const int r = r0 + threadIdx.x;
    const bool valid = r < R;
    const bool is_run = valid && t[r] != 0;
    const uint64_t bal = __ballot(is_run);
    const int below = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) s_w[w] = __popcll(bal);
    __syncthreads();
    int before = s_base;
    for (int i = 0; i < w; ++i) before += s_w[i];
    int chunk = 0;
    for (int i = 0; i < nw; ++i) chunk += s_w[i];
    const int n_run_before = before + below;  // RUN rows before r
    if (valid) {
      if (is_run) {
        run[n_run_before] = r;
        inv[r] = n_run_before;
      } else {
        const int p = r - n_run_before;  // Project-Only rows before r
        proj[p] = r;
        inv[r] = p;
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) s_base += chunk;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    cnt[2 * l] = s_base;
    cnt[2 * l + 1] = R - s_base;
  }
}

hipError_t launch_route_maps(const uint8_t* tape, int n_layers, int R, int32_t* run, int32_t* proj, int32_t* inv,
                             int32_t* cnt, hipStream_t s) {
  if (n_layers <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_route_maps, dim3(n_layers), dim3(1024), 0, s, tape, R, run, proj, inv, cnt);
  return hipGetLastError();
}

// The end of a routed layer's MLP: one workgroup per batch row r adds its
// cohort's down-projection product (the splits of that cohort's launch, in
// split order, at row inv[r] of the cohort) to the residual with weight w[r]
// for a RUN row and 1 - w[r] for a Project-Only one -- the weighted scatter
// of Algorithm 1 -- and (gain non-null) normalises the row into bf16 frags
// for the next layer as k_resid_norm does.  With every row RUN and w = 1 the
// residual is the one k_resid_norm computes from the same products.
__global__ __launch_bounds__(1024) void k_route_reduce_norm(float* __restrict__ x, const float* __restrict__ y_run,
                                                            int s_run, const float* __restrict__ y_po, int s_po,
                                                            const uint8_t* __restrict__ mask,
                                                            const int32_t* __restrict__ inv,
                                                            const float* __restrict__ wts, int R, int H,
                                                            const uint16_t* __restrict__ g, float eps,
                                                            uint16_t* __restrict__ hg, int Rg) {
  __shared__ double s_ss[16];
  const int r = blockIdx.x;
  const int c = threadIdx.x * 8;
  const bool on = c < H;
  const bool is_run = mask[r] != 0;
  const float* y = is_run ? y_run : y_po;
  const int splits = is_run ? s_run : s_po;
  const int m = inv[r];
  const float wt = is_run ? wts[r] : 1.f - wts[r];
  float* xr = x + static_cast<size_t>(r) * H + c;
  float e[8];
  u32x4 gv = u32x4{0u, 0u, 0u, 0u};
  double ss = 0.0;
  if (on) {
    float4 a = *reinterpret_cast<const float4*>(xr);
    float4 b = *reinterpret_cast<const float4*>(xr + 4);
    float4 ya[kResidNormMaxSplits], yb[kResidNormMaxSplits];
#pragma unroll
    for (int sp = 0; sp < kResidNormMaxSplits; ++sp) {
      if (sp < splits) {
        const float* yr = y + (static_cast<size_t>(sp) * R + m) * H + c;
        ya[sp] = *reinterpret_cast<const float4*>(yr);
        yb[sp] = *reinterpret_cast<const float4*>(yr + 4);
      }
    }
    if (g != nullptr) gv = *reinterpret_cast<const u32x4*>(g + c);
    float4 sa = ya[0], sb = yb[0];
#pragma unroll
    for (int sp = 1; sp < kResidNormMaxSplits; ++sp) {
      if (sp < splits) {
        sa.x += ya[sp].x; sa.y += ya[sp].y; sa.z += ya[sp].z; sa.w += ya[sp].w;
        sb.x += yb[sp].x; sb.y += yb[sp].y; sb.z += yb[sp].z; sb.w += yb[sp].w;
      }
    }
    a.x += wt * sa.x; a.y += wt * sa.y; a.z += wt * sa.z; a.w += wt * sa.w;
    b.x += wt * sb.x; b.y += wt * sb.y; b.z += wt * sb.z; b.w += wt * sb.w;
    *reinterpret_cast<float4*>(xr) = a;
    *reinterpret_cast<float4*>(xr + 4) = b;
    e[0] = a.x; e[1] = a.y; e[2] = a.z; e[3] = a.w;
    e[4] = b.x; e[5] = b.y; e[6] = b.z; e[7] = b.w;
#pragma unroll
    for (int q = 0; q < 8; ++q) ss += static_cast<double>(e[q]) * e[q];
  }
  if (g == nullptr) return;
#pragma unroll
  for (int mm = 32; mm >= 1; mm >>= 1) ss += __shfl_xor(ss, mm, 64);
  if ((threadIdx.x & 63) == 0) s_ss[threadIdx.x >> 6] = ss;
  __syncthreads();
  double tot = 0.0;
  for (int w = 0; w < static_cast<int>(blockDim.x >> 6); ++w) tot += s_ss[w];
  const double rr = 1.0 / sqrt(tot / static_cast<double>(H) + static_cast<double>(eps));
  if (!on) return;
  u32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    o[q] = d2bf(static_cast<double>(e[2 * q]) * bf2f(gv[q] & 0xffffu) * rr) |
           (d2bf(static_cast<double>(e[2 * q + 1]) * bf2f(gv[q] >> 16) * rr) << 16);
  *reinterpret_cast<u32x4*>(hg + frag_index(r, c, Rg)) = o;
}

hipError_t launch_route_reduce_norm(float* x, const float* y_run, int s_run, const float* y_po, int s_po,
                                    const uint8_t* mask, const int32_t* inv, const float* wts, int R, int H,
                                    const uint16_t* g, float eps, uint16_t* hg, int Rg, hipStream_t s) {
  if (H % 8 != 0 || H > 8192 || s_run < 1 || s_run > kResidNormMaxSplits || s_po < 1 ||
      s_po > kResidNormMaxSplits)
    return hipErrorInvalidValue;
  const int threads = (H / 8 + 63) / 64 * 64;
  hipLaunchKernelGGL(k_route_reduce_norm, dim3(R), dim3(threads), 0, s, x, y_run, s_run, y_po, s_po, mask, inv, wts,
                     R, H, g, eps, hg, Rg);
  return hipGetLastError();
}

// ---------------------------------------------------------------- argmax
__device__ inline void block_am_reduce(float& bv, int& bi) {
  __shared__ float s_v[16];
  __shared__ int s_i[16];
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float v2 = shfl_xor(bv, m);
    const int i2 = shfl_xor(bi, m);
    am_merge(bv, bi, v2, i2);
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    s_v[w] = bv;
    s_i[w] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < (int)(blockDim.x >> 6); ++i) am_merge(bv, bi, s_v[i], s_i[i]);
  }
}

// ids[r] from the per-workgroup partials of the lm_head epilogue ([G][R]).
__global__ __launch_bounds__(256) void k_argmax_partials(const float* __restrict__ pv, const int* __restrict__ pi,
                                                         int n_groups, int R, int32_t* __restrict__ ids) {
  const int r = blockIdx.x;
  float bv = -INFINITY;
  int bi = INT_MAX;
  // eight partials per lane are loaded before any is merged (the merge is a
  // total order on (value, -index), so its order does not matter)
  constexpr int kU = 8;
  for (int g0 = threadIdx.x; g0 < n_groups; g0 += kU * blockDim.x) {
    float v[kU];
    int i[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int g = g0 + u * blockDim.x;
      v[u] = g < n_groups ? pv[static_cast<size_t>(g) * R + r] : -INFINITY;
      i[u] = g < n_groups ? pi[static_cast<size_t>(g) * R + r] : INT_MAX;
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) am_merge(bv, bi, v[u], i[u]);
  }
  block_am_reduce(bv, bi);
  if (threadIdx.x == 0) ids[r] = (bi == INT_MAX) ? 0 : bi;
}

hipError_t launch_argmax_partials(const float* pv, const int* pi, int n_groups, int R, int32_t* ids,
                                  hipStream_t s) {
  hipLaunchKernelGGL(k_argmax_partials, dim3(R), dim3(256), 0, s, pv, pi, n_groups, R, ids);
  return hipGetLastError();
}

template <int DT>
__global__ __launch_bounds__(1024) void k_argmax_logits(const void* __restrict__ logits, int vocab,
                                                        int32_t* __restrict__ ids, int32_t* __restrict__ no_value) {
  const int r = blockIdx.x;
  float bv = -INFINITY;
  int bi = INT_MAX;
  for (int j = threadIdx.x; j < vocab; j += blockDim.x) {
    float v;
    if constexpr (DT == 0)
      v = bf2f(reinterpret_cast<const uint16_t*>(logits)[static_cast<size_t>(r) * vocab + j]);
    else
      v = reinterpret_cast<const float*>(logits)[static_cast<size_t>(r) * vocab + j];
    if (!(v != v)) am_merge(bv, bi, v, j);
  }
  block_am_reduce(bv, bi);
  if (threadIdx.x == 0) {
    ids[r] = (bi == INT_MAX) ? 0 : bi;
    if (no_value != nullptr) no_value[r] = bi == INT_MAX ? 1 : 0;  // every value NaN
  }
}

hipError_t launch_argmax_logits(const void* logits, int dtype, int rows, int vocab, int32_t* ids, int32_t* no_value,
                                hipStream_t s) {
  if (dtype == 0)
    hipLaunchKernelGGL(k_argmax_logits<0>, dim3(rows), dim3(1024), 0, s, logits, vocab, ids, no_value);
  else
    hipLaunchKernelGGL(k_argmax_logits<1>, dim3(rows), dim3(1024), 0, s, logits, vocab, ids, no_value);
  return hipGetLastError();
}

// ---------------------------------------------------------------- weight packing
// dst tile order (see internal.hpp).  Logical source rows come from up to
// three matrices stacked vertically (n0, n1, n2 rows); perm_kind selects the
// packed->logical row map: 0 identity, 1 rotary pairing in the first
// n_rope_rows rows (per head of head_dim), 2 gate/up interleave (n0 = n1 = F).
__device__ inline int packed_to_logical(int p, int perm_kind, int head_dim, int n_rope_rows, int F) {
  if (perm_kind == 1 && p < n_rope_rows) {
    const int ph = p % head_dim;
    const int dim = (ph & 1) ? (ph >> 1) + head_dim / 2 : (ph >> 1);
    return p - ph + dim;
  }
  if (perm_kind == 2) {
    const int u = p >> 2, r = p & 3;
    return r < 2 ? 2 * u + r : F + 2 * u + (r - 2);
  }
  return p;
}

__global__ __launch_bounds__(256) void k_pack(const uint16_t* __restrict__ s0, const uint16_t* __restrict__ s1,
                                              const uint16_t* __restrict__ s2, int n0, int n1, int N, int K,
                                              int perm_kind, int head_dim, int n_rope_rows,
                                              uint16_t* __restrict__ dst) {
  const size_t chunk = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;  // 16-byte chunk
  const int Kt = K / 32;
  const size_t n_chunks = static_cast<size_t>(N) * K / 8;
  if (chunk >= n_chunks) return;
  const size_t tile = chunk / 64;
  const int lane = static_cast<int>(chunk % 64);
  const int nt = static_cast<int>(tile / Kt), kt = static_cast<int>(tile % Kt);
  const int p = 16 * nt + (lane & 15);
  const int k0 = 32 * kt + 8 * (lane >> 4);
  int lr = packed_to_logical(p, perm_kind, head_dim, n_rope_rows, n0);
  const uint16_t* src;
  if (lr < n0) {
    src = s0;
  } else if (lr < n0 + n1) {
    src = s1;
    lr -= n0;
  } else {
    src = s2;
    lr -= n0 + n1;
  }
  *reinterpret_cast<u32x4*>(dst + chunk * 8) = *reinterpret_cast<const u32x4*>(src + static_cast<size_t>(lr) * K + k0);
}

hipError_t launch_pack(const uint16_t* s0, const uint16_t* s1, const uint16_t* s2, int n0, int n1, int N, int K,
                       int perm_kind, int head_dim, int n_rope_rows, uint16_t* dst, hipStream_t s) {
  const size_t n_chunks = static_cast<size_t>(N) * K / 8;
  const unsigned blocks = static_cast<unsigned>((n_chunks + 255) / 256);
  hipLaunchKernelGGL(k_pack, dim3(blocks), dim3(256), 0, s, s0, s1, s2, n0, n1, N, K, perm_kind, head_dim,
                     n_rope_rows, dst);
  return hipGetLastError();
}

__global__ void k_copy16(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst, size_t n) {
  const size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

hipError_t launch_copy_bf16(const uint16_t* src, uint16_t* dst, size_t n, hipStream_t s) {
  hipLaunchKernelGGL(k_copy16, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

__global__ void k_zero(uint32_t* __restrict__ dst, size_t n) {
  const size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = 0u;
}

hipError_t launch_fill_zero(void* dst, size_t bytes, hipStream_t s) {
  const size_t n = bytes / 4;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_zero, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, s,
                     static_cast<uint32_t*>(dst), n);
  return hipGetLastError();
}

// ---------------------------------------------------------------- stream read (measurement)
// Reads `n16` 16-byte words once, four per thread per round in a grid-stride
// loop, and leaves one word per workgroup (an xor of what it read, so no load
// is dead): the achievable HBM read rate of a plain streaming kernel.
__global__ __launch_bounds__(256) void k_stream_read(const u32x4* __restrict__ src, size_t n16,
                                                     uint32_t* __restrict__ out) {
  __shared__ uint32_t s_x[4];
  const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
  size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  u32x4 acc = u32x4{0u, 0u, 0u, 0u};
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u32x4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    acc ^= a ^ b ^ c ^ d;
  }
  for (; i < n16; i += stride) acc ^= src[i];
  uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x ^= __shfl_xor(x, m, 64);
  if ((threadIdx.x & 63) == 0) s_x[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = s_x[0] ^ s_x[1] ^ s_x[2] ^ s_x[3];
}

hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* out, int wgs, hipStream_t s) {
  if (bytes % 16 != 0 || wgs < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_stream_read, dim3(wgs), dim3(256), 0, s, static_cast<const u32x4*>(src), bytes / 16, out);
  return hipGetLastError();
}

// ---------------------------------------------------------------- KV scatter / gather
// One thread per (token, kv head, dim); logical layout [n][Hkv][hd].
template <bool WRITE>
__global__ __launch_bounds__(256) void k_kv_move(uint16_t* __restrict__ pool, int layer, int n_blocks, int Hkv,
                                                 int hd, const int32_t* __restrict__ slots, int n,
                                                 uint16_t* __restrict__ k, uint16_t* __restrict__ v) {
  const size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const size_t total = static_cast<size_t>(n) * Hkv * hd;
  if (i >= total) return;
  const int e = static_cast<int>(i % hd);
  const int hk = static_cast<int>((i / hd) % Hkv);
  const int tok = static_cast<int>(i / (static_cast<size_t>(hd) * Hkv));
  const int sl = slots[tok];
  if (sl < 0 || sl >= n_blocks * kBlock) return;  // slots outside the pool are ignored
  const int blk = sl >> 4, t = sl & 15;
  const size_t kb = (((static_cast<size_t>(layer) * 2 + 0) * n_blocks + blk) * Hkv + hk) * kBlock * hd;
  const size_t vb = (((static_cast<size_t>(layer) * 2 + 1) * n_blocks + blk) * Hkv + hk) * kBlock * hd;
  if (WRITE) {
    pool[kb + kv_k_index(t, e)] = k[i];
    pool[vb + kv_v_index(t, e)] = v[i];
  } else {
    k[i] = pool[kb + kv_k_index(t, e)];
    v[i] = pool[vb + kv_v_index(t, e)];
  }
}

hipError_t launch_kv_move(bool write, uint16_t* pool, int layer, int n_blocks, int Hkv, int hd,
                          const int32_t* slots, int n, uint16_t* k, uint16_t* v, hipStream_t s) {
  const size_t total = static_cast<size_t>(n) * Hkv * hd;
  if (total == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>((total + 255) / 256);
  if (write)
    hipLaunchKernelGGL(k_kv_move<true>, dim3(blocks), dim3(256), 0, s, pool, layer, n_blocks, Hkv, hd, slots, n, k, v);
  else
    hipLaunchKernelGGL(k_kv_move<false>, dim3(blocks), dim3(256), 0, s, pool, layer, n_blocks, Hkv, hd, slots, n, k,
                       v);
  return hipGetLastError();
}

}  // namespace vsk
