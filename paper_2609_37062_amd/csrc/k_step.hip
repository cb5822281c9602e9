// The whole decode step as one persistent kernel.
//
// A pass is a chain of phases that each depend on all of the previous one:
// per layer QKV projection (+ rotary, q store, this layer's K,V write --
// Invariant 1), paged attention, O projection (+ residual), gate/up
// projection (+ SwiGLU), down projection (+ residual); then the final norm
// with the lm_head and the greedy argmax.  Launched as one kernel per phase,
// each phase pays a launch and a ramp of its weight stream while HBM idles
// (about 2-3 us each, ~140 times per step).  Here one workgroup per compute
// unit runs all phases, separated by grid synchronisation points, and before
// waiting at a point it already issues the first weight loads of the next
// projection: weights do not depend on the activations, so HBM keeps
// streaming while the slowest workgroup finishes (paper, appendix "The
// Switching Thresholds from the Roofline": below the ridge point decode is
// bound by weight bandwidth).
//
// Cross-workgroup data.  The L2 of each XCD is not coherent with the other
// XCDs' within a launch.  Every activation a phase hands on is stored
// write-through and lives at an address written once per launch (buffers
// are per layer), so no L2 holds a stale copy when it is read after the
// synchronisation point.  The attention split partials keep their
// agent-scope atomic accesses.
//
// Synchronisation.  A workgroup drains its stores, then counts its arrival
// at the point on one of eight counters; eight threads of every workgroup
// poll them until they reach the pass's epoch times the arrivals each
// expects.  Every wait is bounded: past the spin limit the
// workgroup records the epoch in the error word and all workgroups leave,
// so a fault in the protocol ends the kernel instead of hanging it.  The
// epoch lives in device memory and advances on the device, so a pass
// captured in a graph can be replayed.
//
// Projections.  A unit is one 16-column tile of W over all of K; the eight
// waves of a workgroup split K (wave w takes K steps w, w+8, ...), keep kPF
// weight tiles in flight in a register ring that runs on across unit
// boundaries, and are reduced in LDS in wave order, as the per-op projection
// kernel does.  The RMSNorm of a projection's input is a phase of its own:
// after the residual is complete every workgroup normalises a share of the
// 16 rows, h = bf16(x * g / sqrt(mean(x^2) + eps)) from the per-tile sums of
// x^2 the producing residual projection wrote, into the input frags of the
// projection; one more synchronisation point, and the projection streams
// them like any other input (the weight stream is already running across
// both points).
#include <climits>
#include <cmath>

#include "attn_core.hpp"
#include "dev.hpp"
#include "gemm.hpp"
#include "step.hpp"

namespace vsk {

namespace {

constexpr int kWaves = 8;                 // waves per workgroup (the K split of every projection)
constexpr int kPF = 8;                    // weight tiles in flight per wave
constexpr unsigned kSpinLimit = 1u << 21; // a few seconds of polling before a wait is declared failed
constexpr size_t kLdsRed = 2 * (kWaves - 1) * 1024;  // double-buffered cross-wave reduction
constexpr int kMaxParts = 256;            // sum-of-squares partials per row (hidden / 16, hidden <= 4096)

__device__ __forceinline__ unsigned ld_agent_u32(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ float silu_f(float v) { return v / (1.0f + expf(-v)); }

// ---------------------------------------------------------------- synchronisation
struct Sync {
  unsigned* flags;
  unsigned* err;
  unsigned epoch;
  uint64_t* trace;  // nullable: [points][gridDim.x][2] arrival and release times (100 MHz clock)
};

__device__ __forceinline__ void arrive(const Sync& s, int point) {
  __builtin_amdgcn_s_waitcnt(0);  // this wave's write-through stores have reached memory
  __syncthreads();
  if (threadIdx.x == 0) {
    if (s.trace) s.trace[(static_cast<size_t>(point) * gridDim.x + blockIdx.x) * 2] = __builtin_amdgcn_s_memrealtime();
    __hip_atomic_fetch_add(s.flags + (static_cast<size_t>(point) * kSyncCounters + (blockIdx.x % kSyncCounters)) *
                                         kFlagWords,
                           1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// True when every workgroup has arrived at `point`; false when some wait of
// this pass failed (the caller then leaves the kernel).  Counter c counts
// the arrivals of workgroups c, c+8, ... over all passes, so after this
// pass's arrivals it holds epoch times their number.  Eight threads poll
// (one counter each) with a pause between polls: polls go to memory, and
// hundreds of idle workgroups polling without pause would take a large share
// of the bandwidth the streaming workgroups need.
__device__ __forceinline__ bool await(const Sync& s, int point) {
  int bad = 0;
  if (threadIdx.x < kSyncCounters) {
    const unsigned n = (gridDim.x - threadIdx.x + kSyncCounters - 1) / kSyncCounters;
    const unsigned target = s.epoch * n;
    const unsigned* f = s.flags + (static_cast<size_t>(point) * kSyncCounters + threadIdx.x) * kFlagWords;
    unsigned spins = 0;
    while (n > 0 && static_cast<int>(ld_agent_u32(f) - target) < 0) {
      if ((spins & 15u) == 0u && ld_agent_u32(s.err) != 0u) {
        bad = 1;
        break;
      }
      if (++spins > kSpinLimit) {
        __hip_atomic_store(s.err, s.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        bad = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(8);
    }
  }
  const bool ok = !__syncthreads_or(bad);
  if (s.trace && threadIdx.x == 0)
    s.trace[(static_cast<size_t>(point) * gridDim.x + blockIdx.x) * 2 + 1] = __builtin_amdgcn_s_memrealtime();
  return ok;
}

// ---------------------------------------------------------------- projections
template <class T>
using gptr = const __attribute__((address_space(1))) T*;
template <class T>
__device__ __forceinline__ gptr<T> as_global(const T* p) {
  return reinterpret_cast<gptr<T>>(reinterpret_cast<uintptr_t>(p));
}
// global (not flat) loads: flat loads would also count on the LDS counter
// and make every LDS wait in the projection loop wait for memory too
__device__ __forceinline__ u32x4 ldg4(const void* p) { return *as_global(static_cast<const u32x4*>(p)); }
__device__ __forceinline__ u32x2 ldg2(const void* p) { return *as_global(static_cast<const u32x2*>(p)); }

struct GemmPh {
  const u32x4* W;  // packed tiles of the matrix
  int Kt;          // K / 32
  int u_lo, u_hi;  // this workgroup's units (16-column tiles)
  const u32x4* Xf; // input frags (16 rows) when the input is read from memory
};

__device__ __forceinline__ void unit_range(int U, int& lo, int& hi) {
  lo = static_cast<int>(static_cast<int64_t>(U) * blockIdx.x / gridDim.x);
  hi = static_cast<int>(static_cast<int64_t>(U) * (blockIdx.x + 1) / gridDim.x);
}

// Input of a projection that is normalised while it is staged
struct NormIn {
  const float* x;
  const uint16_t* gain;
  const double* ssq;
  int parts;
};

// The normalised input of a projection, h = bf16(x g r) with
// r = 1/sqrt(sum x^2 / H + eps), written as B-operand frags of the 16 rows
// ([K / 32][64 lanes] of 8 bf16) to memory, each workgroup its share of the
// frags' lanes.  r is summed from `parts` per-tile partials in a fixed order
// (the same order and arithmetic as the per-op norm kernel): every
// workgroup takes the sums of all 16 rows, wave w those of rows 2w and 2w+1.
// The first element loads are issued before the partials are summed, so
// the phase costs about one memory round trip.
__device__ __forceinline__ void norm_slice(const NormIn& ni, int R, int H, float eps, uint16_t* __restrict__ xf,
                                           unsigned char* lds) {
  const int tid = opaque_tid();
  const int lane = tid & 63, w = tid >> 6;
  double* s_r = reinterpret_cast<double*>(lds + kLdsRed);
  const int n_tasks = (H / 32) * 64;  // one per lane of every frag
  const int lo = static_cast<int>(static_cast<int64_t>(n_tasks) * blockIdx.x / gridDim.x);
  const int hi = static_cast<int>(static_cast<int64_t>(n_tasks) * (blockIdx.x + 1) / gridDim.x);
  float4 va, vb;
  u32x4 gv;
  int t = lo + tid;
  auto load = [&]() {
    const int fl = t & 63, kt = t >> 6;
    const int row = fl & 15, c = 32 * kt + 8 * (fl >> 4);
    const bool ok = t < hi && row < R;
    const float* xp = ni.x + static_cast<size_t>(ok ? row : 0) * H + (ok ? c : 0);
    va = __builtin_bit_cast(float4, ldg4(xp));
    vb = __builtin_bit_cast(float4, ldg4(xp + 4));
    gv = ldg4(ni.gain + (t < hi ? c : 0));
  };
  load();
  // this wave's two rows: every partial this lane adds is loaded before the
  // first sum (at most kParts / 64 per row), then added in partial order
  constexpr int kPl = kMaxParts / 64;
  double pv[2][kPl];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int row = 2 * w + k;
#pragma unroll
    for (int q = 0; q < kPl; ++q) {
      const int p = lane + 64 * q;
      pv[k][q] = (row < R && p < ni.parts) ? as_global(ni.ssq)[static_cast<size_t>(p) * R + row] : 0.0;
    }
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int row = 2 * w + k;
    double s = 0.0;
#pragma unroll
    for (int q = 0; q < kPl; ++q)
      if (lane + 64 * q < ni.parts) s += pv[k][q];
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
    if (lane == 0 && row < R) s_r[row] = 1.0 / sqrt(s / static_cast<double>(H) + static_cast<double>(eps));
  }
  __syncthreads();
  while (t < hi) {
    const int row = t & 15;
    u32x4 o = u32x4{0u, 0u, 0u, 0u};
    if (row < R) {
      const double rr = s_r[row];
      const float e[8] = {va.x, va.y, va.z, va.w, vb.x, vb.y, vb.z, vb.w};
#pragma unroll
      for (int q = 0; q < 4; ++q)
        o[q] = d2bf(static_cast<double>(e[2 * q]) * bf2f(gv[q] & 0xffffu) * rr) |
               (d2bf(static_cast<double>(e[2 * q + 1]) * bf2f(gv[q] >> 16) * rr) << 16);
    }
    store_wt(xf + static_cast<size_t>(t) * 8, o);
    t += blockDim.x;
    if (t < hi) load();
  }
}

// Epilogue inputs and outputs of one projection phase.
struct Epi {
  int N, R;
  // RESID
  const float* x_in;
  float* x_out;
  double* ssq_out;  // [tiles][R]
  // QKV
  uint16_t* q;
  uint16_t* pool;
  int layer, n_blocks, Hkv, hd, Nq, Nkv;
  const float2* rope;
  const int32_t* slot;  // [R] KV slot of each row
  const int32_t* pos;   // [R] position of each row
  // SWIGLU
  uint16_t* a_out;  // frags (16 rows)
  // LOGITS
  uint16_t* logits;
  float* am_val;
  int* am_idx;
};

// What wave 0 loads for a unit's epilogue ahead of the unit's sums.
struct EpiPre {
  float4 xv;
  float2 cs0, cs1;
  int slot;
};

template <int EPI>
__device__ __forceinline__ void epi_pre(const Epi& e, int unit, EpiPre& p) {
  const int lane = threadIdx.x & 63;
  const int row = lane & 15;
  const int n0 = 16 * unit + 4 * (lane >> 4);
  if constexpr (EPI == EPI_RESID) {
    p.xv = row < e.R ? __builtin_bit_cast(float4, ldg4(e.x_in + static_cast<size_t>(row) * e.N + n0))
                     : make_float4(0.f, 0.f, 0.f, 0.f);
  } else if constexpr (EPI == EPI_QKV) {
    const bool rot = row < e.R && n0 < e.Nq + e.Nkv;
    const int half = e.hd >> 1;
    const int j0 = (n0 % e.hd) >> 1;
    const int pos = row < e.R ? e.pos[row] : 0;
    p.slot = row < e.R ? e.slot[row] : 0;
    const float2* rp = e.rope + static_cast<size_t>(pos) * half + j0;
    p.cs0 = rot ? __builtin_bit_cast(float2, ldg2(rp)) : make_float2(1.f, 0.f);
    p.cs1 = rot ? __builtin_bit_cast(float2, ldg2(rp + 1)) : make_float2(1.f, 0.f);
  }
}

template <int EPI>
__device__ __forceinline__ void epilogue(const Epi& e, int unit, const f32x4 v, const EpiPre& p) {
  const int lane = threadIdx.x & 63;
  const int row = lane & 15;
  const int n0 = 16 * unit + 4 * (lane >> 4);
  if constexpr (EPI == EPI_RESID) {
    double ss = 0.0;
    if (row < e.R) {
      float4 x = p.xv;
      x.x += v[0];
      x.y += v[1];
      x.z += v[2];
      x.w += v[3];
      store_wt(e.x_out + static_cast<size_t>(row) * e.N + n0, __builtin_bit_cast(u32x4, x));
      ss = static_cast<double>(x.x) * x.x + static_cast<double>(x.y) * x.y + static_cast<double>(x.z) * x.z +
           static_cast<double>(x.w) * x.w;
    }
    // the four lane groups hold the same row
    ss += __shfl_xor(ss, 16, 64);
    ss += __shfl_xor(ss, 32, 64);
    if (lane < 16 && row < e.R) store_wt(e.ssq_out + static_cast<size_t>(unit) * e.R + row, ss);
  } else if constexpr (EPI == EPI_QKV) {
    if (row >= e.R) return;
    const int hd = e.hd, half = hd >> 1;
    const int blk = p.slot >> 4, t = p.slot & 15;
    if (n0 < e.Nq + e.Nkv) {
      const int ph = n0 % hd;   // packed row inside the head (multiple of 4)
      const int hb = n0 - ph;   // first packed row of the head
      const int j0 = ph >> 1;   // dims j0, j0+half, j0+1, j0+1+half
      const float y0 = v[0] * p.cs0.x - v[1] * p.cs0.y;
      const float y1 = v[1] * p.cs0.x + v[0] * p.cs0.y;
      const float y2 = v[2] * p.cs1.x - v[3] * p.cs1.y;
      const float y3 = v[3] * p.cs1.x + v[2] * p.cs1.y;
      if (n0 < e.Nq) {
        uint16_t* q = e.q + static_cast<size_t>(row) * e.Nq + hb;
        store_wt16(q + j0, f2bf(y0));
        store_wt16(q + j0 + half, f2bf(y1));
        store_wt16(q + j0 + 1, f2bf(y2));
        store_wt16(q + j0 + 1 + half, f2bf(y3));
      } else {
        const int hk = (hb - e.Nq) / hd;
        uint16_t* kb = e.pool + ((((static_cast<size_t>(e.layer) * 2 + 0) * e.n_blocks + blk) * e.Hkv + hk) *
                                 kBlock * hd);
        store_wt16(kb + kv_k_index(t, j0), f2bf(y0));
        store_wt16(kb + kv_k_index(t, j0 + half), f2bf(y1));
        store_wt16(kb + kv_k_index(t, j0 + 1), f2bf(y2));
        store_wt16(kb + kv_k_index(t, j0 + 1 + half), f2bf(y3));
      }
    } else {
      const int nv = n0 - e.Nq - e.Nkv;
      const int hk = nv / hd, e0 = nv % hd;
      uint16_t* vb = e.pool + ((((static_cast<size_t>(e.layer) * 2 + 1) * e.n_blocks + blk) * e.Hkv + hk) *
                               kBlock * hd);
#pragma unroll
      for (int r = 0; r < 4; ++r) store_wt16(vb + kv_v_index(t, e0 + r), f2bf(v[r]));
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    if (row >= e.R) return;
    const int u = 4 * unit + (lane >> 4);  // output columns 2u, 2u+1
    const float a0 = silu_f(v[0]) * v[2];
    const float a1 = silu_f(v[1]) * v[3];
    store_wt(e.a_out + frag_index(row, 2 * u, 1), pack_bf2(a0, a1));
  } else {  // EPI_LOGITS
    float bv = -INFINITY;
    int bi = INT_MAX;
    if (row < e.R) {
      u32x2 packed;
      packed[0] = pack_bf2(v[0], v[1]);
      packed[1] = pack_bf2(v[2], v[3]);
      *reinterpret_cast<u32x2*>(e.logits + static_cast<size_t>(row) * e.N + n0) = packed;
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (!(v[r] != v[r])) am_merge(bv, bi, v[r], n0 + r);
    }
    // lanes l, l^16, l^32, l^48 hold the same row
#pragma unroll
    for (int m = 16; m <= 32; m <<= 1) {
      const float v2 = shfl_xor(bv, m);
      const int i2 = shfl_xor(bi, m);
      am_merge(bv, bi, v2, i2);
    }
    if (lane < 16 && row < e.R) {
      store_wt(e.am_val + static_cast<size_t>(unit) * e.R + row, __float_as_uint(bv));
      store_wt(e.am_idx + static_cast<size_t>(unit) * e.R + row, static_cast<uint32_t>(bi));
    }
  }
}

// One projection phase of this workgroup, entered right after the previous
// phase's work: arrive at `point`, start the weight stream (the first kPF
// tiles of each wave do not depend on the input), wait for every workgroup;
// XN: arrive at `point` and wait, write this workgroup's share of the
// normalised input frags to g.Xf, arrive at `point + 1`, start the weight
// stream and wait again; then run the units, the input frags streaming from
// g.Xf beside the weights.  Returns false when a wait of this pass failed.
template <int EPI, bool XN>
__device__ __forceinline__ bool gemm_phase(const GemmPh& g, const Epi& e, const NormIn& ni, float eps, unsigned char* lds,
                           const Sync& sy, int point) {
  const int tid = opaque_tid();
  const int lane = tid & 63, w = tid >> 6;
  const int S = g.Kt / kWaves;
  const bool has = g.u_lo < g.u_hi;
  const gptr<u32x4> Wg = as_global(g.W) + static_cast<size_t>(w) * 64 + lane;
  const gptr<u32x4> Xg = as_global(g.Xf) + static_cast<size_t>(w) * 64 + lane;
  u32x4 wr[kPF], xr[kPF];
  int lu = g.u_lo, li = 0, xi = 0;  // next position to load: unit, K step; next input K step
  // Load the next position's weight tile into slot s (and its input frag).
  // Positions past the last unit re-read the last tile (a cached address;
  // the result is never used), so the loads of a full round are unconditional.
#define VSK_RING_LOAD(s, WITH_X)                                              \
  do {                                                                        \
    const bool past_ = lu >= g.u_hi;                                          \
    const int u_ = past_ ? g.u_hi - 1 : lu;                                   \
    const int i_ = past_ ? S - 1 : li;                                        \
    wr[s] = Wg[(static_cast<size_t>(u_) * g.Kt + kWaves * i_) * 64];          \
    if (WITH_X) {                                                             \
      xr[s] = Xg[static_cast<size_t>(kWaves * xi) * 64];                      \
      if (++xi == S) xi = 0;                                                  \
    }                                                                         \
    if (++li == S) {                                                          \
      li = 0;                                                                 \
      ++lu;                                                                   \
    }                                                                         \
  } while (0)

  // the first weight tiles go out before the wait that precedes the input
  // (with XN after the norm's stores: an arrival drains every outstanding
  // load, and the ring would hold up the norm phase's arrival)
  auto prefetch = [&]() {
    if (has) {
#pragma unroll
      for (int s = 0; s < kPF; ++s) VSK_RING_LOAD(s, false);
    }
  };
  arrive(sy, point);
  if constexpr (!XN) prefetch();
  if (!await(sy, point)) return false;
  if constexpr (XN) {
    norm_slice(ni, e.R, g.Kt * 32, eps, reinterpret_cast<uint16_t*>(const_cast<u32x4*>(g.Xf)), lds);
    arrive(sy, point + 1);
    prefetch();
    if (!await(sy, point + 1)) return false;
  }
  if (!has) return true;
#pragma unroll
  for (int s = 0; s < kPF; ++s) {
    xr[s] = Xg[static_cast<size_t>(kWaves * xi) * 64];
    if (++xi == S) xi = 0;
  }
  f32x4* red = reinterpret_cast<f32x4*>(lds);
  const int J = (g.u_hi - g.u_lo) * S;  // positions of this wave
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f}, done = acc;
  int cu = g.u_lo, ci = 0, pend = -1;
  EpiPre pre;
  if (w == 0) epi_pre<EPI>(e, cu, pre);

  // consume the position in slot s: one MFMA; at the end of a unit the
  // wave's sum goes to LDS (wave 0 keeps its own)
#define VSK_CONSUME(s) acc = mfma_16x16x32(wr[s], xr[s], acc)
#define VSK_UNIT_END()                                                        \
  do {                                                                        \
    if (++ci == S) {                                                          \
      ci = 0;                                                                 \
      if (w > 0) red[((cu & 1) * (kWaves - 1) + w - 1) * 64 + lane] = acc;     \
      else done = acc;                                                        \
      acc = f32x4{0.f, 0.f, 0.f, 0.f};                                        \
      pend = cu;                                                              \
      ++cu;                                                                   \
    }                                                                         \
  } while (0)
  // a unit ends at most once per round (S >= kPF): reduce it in wave order
  auto finish = [&]() {
    if (pend < 0) return;
    __syncthreads();
    if (w == 0) {
      f32x4 v = done;
      for (int w2 = 1; w2 < kWaves; ++w2) v += red[((pend & 1) * (kWaves - 1) + w2 - 1) * 64 + lane];
      epilogue<EPI>(e, pend, v, pre);
      if (cu < g.u_hi) epi_pre<EPI>(e, cu, pre);
    }
    pend = -1;
  };

  int j = 0;
  for (; j + kPF <= J; j += kPF) {
#pragma unroll
    for (int s = 0; s < kPF; ++s) {
      VSK_CONSUME(s);
      VSK_RING_LOAD(s, true);
      VSK_UNIT_END();
      // keep each refill next to its use
      __builtin_amdgcn_sched_barrier(0);
    }
    finish();
  }
#pragma unroll
  for (int s = 0; s < kPF; ++s) {
    if (j + s < J) {
      VSK_CONSUME(s);
      VSK_UNIT_END();
    }
  }
  finish();
#undef VSK_RING_LOAD
#undef VSK_CONSUME
#undef VSK_UNIT_END
  return true;
}

// ---------------------------------------------------------------- small phases
// x[0] = float(E[id]) and one partial of sum x^2 per row (the per-op
// embedding kernel's arithmetic and order, on its first 256 threads).
__device__ __forceinline__ void embed_phase(const StepArgs& a, unsigned char* lds) {
  double* s_ss = reinterpret_cast<double*>(lds);
  for (int r = blockIdx.x; r < a.R; r += gridDim.x) {
    double ss = 0.0;
    if (threadIdx.x < 256) {
      const int id = a.ids[r];
      const bool valid = id >= 0 && id < a.V;
      const size_t base = valid ? static_cast<size_t>(id) * a.H : 0;
      for (int c = threadIdx.x * 8; c < a.H; c += 256 * 8) {
        const u32x4 v = valid ? *reinterpret_cast<const u32x4*>(a.embed + base + c) : u32x4{0u, 0u, 0u, 0u};
        float e[8];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          e[2 * k] = bf2f(v[k] & 0xffffu);
          e[2 * k + 1] = bf2f(v[k] >> 16);
        }
        float* dst = a.xs + static_cast<size_t>(r) * a.H + c;
        store_wt(dst, __builtin_bit_cast(u32x4, make_float4(e[0], e[1], e[2], e[3])));
        store_wt(dst + 4, __builtin_bit_cast(u32x4, make_float4(e[4], e[5], e[6], e[7])));
#pragma unroll
        for (int k = 0; k < 8; ++k) ss += static_cast<double>(e[k]) * e[k];
      }
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
      if ((threadIdx.x & 63) == 0) s_ss[threadIdx.x >> 6] = ss;
    }
    __syncthreads();
    if (threadIdx.x == 0) store_wt(a.ssq + r, (s_ss[0] + s_ss[1]) + (s_ss[2] + s_ss[3]));
    __syncthreads();
  }
}

// Greedy ids from the lm_head partials ([tiles][R]), lowest index of the
// maximum; and the final residual copied out for inspection.
__device__ __forceinline__ void argmax_phase(const StepArgs& a, const float* x_fin, unsigned char* lds) {
  float* s_v = reinterpret_cast<float*>(lds);
  int* s_i = reinterpret_cast<int*>(lds + 64);
  const int tiles = a.V / 16;
  for (int r = blockIdx.x; r < a.R; r += gridDim.x) {
    float bv = -INFINITY;
    int bi = INT_MAX;
    // eight partials per lane loaded before any is merged (the merge is a
    // total order on (value, -index), so its order does not matter)
    for (int t0 = threadIdx.x; t0 < tiles; t0 += 8 * blockDim.x) {
      float v[8];
      int ix[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int t = t0 + u * blockDim.x;
        v[u] = t < tiles ? a.am_val[static_cast<size_t>(t) * a.R + r] : -INFINITY;
        ix[u] = t < tiles ? a.am_idx[static_cast<size_t>(t) * a.R + r] : INT_MAX;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) am_merge(bv, bi, v[u], ix[u]);
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const float v2 = shfl_xor(bv, m);
      const int i2 = shfl_xor(bi, m);
      am_merge(bv, bi, v2, i2);
    }
    if ((threadIdx.x & 63) == 0) {
      s_v[threadIdx.x >> 6] = bv;
      s_i[threadIdx.x >> 6] = bi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      for (int i = 1; i < kWaves; ++i) am_merge(bv, bi, s_v[i], s_i[i]);
      if (a.next_ids) a.next_ids[r] = (bi == INT_MAX) ? 0 : bi;
    }
    __syncthreads();
  }
  const size_t n4 = static_cast<size_t>(a.R) * a.H / 4;
  for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n4;
       i += static_cast<size_t>(gridDim.x) * blockDim.x)
    reinterpret_cast<float4*>(a.x_out)[i] = reinterpret_cast<const float4*>(x_fin)[i];
}

// ---------------------------------------------------------------- the kernel
template <int D>
__global__ __launch_bounds__(64 * kWaves) void k_step(StepArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const Sync sy{a.flags, a.err, ld_agent_u32(a.epoch_ctr) + 1u, a.trace};
  const int R = a.R, H = a.H;
  const int parts = H / 16;
  auto xbuf = [&](int b) { return a.xs + static_cast<size_t>(b) * R * H; };
  auto sbuf = [&](int b) { return a.ssq + static_cast<size_t>(b) * parts * R; };
  auto nbuf = [&](int b) { return a.ns + static_cast<size_t>(b) * kStepMaxRows * H; };
  auto layer = [&](int l) { return a.P + a.layer_bytes * l; };
  auto gemm = [&](const uint8_t* W, int Kt, int N, const uint16_t* Xf) {
    GemmPh g{reinterpret_cast<const u32x4*>(W), Kt, 0, 0, reinterpret_cast<const u32x4*>(Xf)};
    unit_range(N / 16, g.u_lo, g.u_hi);
    return g;
  };

  Epi e{};
  e.R = R;
  e.pool = a.pool;
  e.n_blocks = a.n_blocks;
  e.Hkv = a.Hkv;
  e.hd = a.hd;
  e.Nq = a.Nq;
  e.Nkv = a.Nkv;
  e.rope = a.rope;
  e.slot = a.slot;
  e.pos = a.pos;

  int point = 0;
  embed_phase(a, lds);

  for (int l = 0; l < a.n_run; ++l) {
    const uint8_t* Lw = layer(l);
    // ---- QKV + rotary + q and this layer's K,V (waits for the embedding or the last down projection)
    e.N = a.Nq + 2 * a.Nkv;
    e.q = a.qs + static_cast<size_t>(l) * R * a.Nq;
    e.layer = l;
    if (!gemm_phase<EPI_QKV, true>(gemm(Lw + a.lo.wqkv, H / 32, e.N, nbuf(2 * l)), e,
                                   NormIn{xbuf(2 * l), reinterpret_cast<const uint16_t*>(Lw + a.lo.attn_norm),
                                          sbuf(2 * l), l == 0 ? 1 : parts},
                                   a.eps, lds, sy, point))
      return;
    point += 2;
    // ---- attention
    arrive(sy, point);
    if (!await(sy, point++)) return;
    {
      AttnArgs aa{};
      aa.q = a.qs + static_cast<size_t>(l) * R * a.Nq;
      aa.pool = a.pool;
      aa.layer = l;
      aa.n_blocks = a.n_blocks;
      aa.Hkv = a.Hkv;
      aa.hd = a.hd;
      aa.G = a.G;
      aa.Nq = a.Nq;
      aa.block_table = a.block_table;
      aa.max_blocks = a.max_blocks;
      aa.row_seq = a.row_seq;
      aa.pos = a.pos;
      aa.scale_log2 = a.scale_log2;
      aa.bps = a.bps;
      aa.max_splits = a.max_splits;
      aa.split_stride = a.max_splits;
      aa.part_o = a.part_o;
      aa.part_ml = a.part_ml;
      aa.counter = a.att_cnt;
      aa.out = a.os + static_cast<size_t>(l) * 16 * a.Nq;
      aa.out_Rg = 1;
      // work items (split, row, KV head), strided over the workgroups; items
      // past a row's splits return at once (the per-op kernel's grid)
      const int n_items = a.max_splits * a.Hkv * R;
      for (int v = blockIdx.x; v < n_items; v += gridDim.x) {
        const int rem = v % (a.Hkv * R);
        __syncthreads();
        attn_unit<D, true, kWaves>(aa, rem / a.Hkv, rem % a.Hkv, v / (a.Hkv * R),
                                                        *reinterpret_cast<AttnLds<D, kWaves>*>(lds));
      }
    }
    // ---- O projection + residual
    e.N = H;
    e.x_in = xbuf(2 * l);
    e.x_out = xbuf(2 * l + 1);
    e.ssq_out = sbuf(2 * l + 1);
    if (!gemm_phase<EPI_RESID, false>(gemm(Lw + a.lo.wo, a.Nq / 32, H, a.os + static_cast<size_t>(l) * 16 * a.Nq), e,
                                      NormIn{}, a.eps, lds, sy, point++))
      return;
    // ---- gate/up + SwiGLU
    e.N = 2 * a.F;
    e.a_out = a.as + static_cast<size_t>(l) * 16 * a.F;
    if (!gemm_phase<EPI_SWIGLU, true>(gemm(Lw + a.lo.wgu, H / 32, 2 * a.F, nbuf(2 * l + 1)), e,
                                      NormIn{xbuf(2 * l + 1), reinterpret_cast<const uint16_t*>(Lw + a.lo.mlp_norm),
                                             sbuf(2 * l + 1), parts},
                                      a.eps, lds, sy, point))
      return;
    point += 2;
    // ---- down + residual
    e.N = H;
    e.x_in = xbuf(2 * l + 1);
    e.x_out = xbuf(2 * l + 2);
    e.ssq_out = sbuf(2 * l + 2);
    if (!gemm_phase<EPI_RESID, false>(gemm(Lw + a.lo.wd, a.F / 32, H, a.as + static_cast<size_t>(l) * 16 * a.F), e,
                                      NormIn{}, a.eps, lds, sy, point++))
      return;
  }

  // a pass that runs fewer layers still counts its arrival at the points of
  // the layers it skips: every counter then holds the pass's epoch times its
  // arrivals, which the next pass's waits rely on (no workgroup waits at
  // these points)
  if (threadIdx.x == 0)
    for (int pt = point; pt < kLayerSyncs * a.n_layers; ++pt)
      __hip_atomic_fetch_add(a.flags + (static_cast<size_t>(pt) * kSyncCounters + (blockIdx.x % kSyncCounters)) *
                                           kFlagWords,
                             1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  point = kLayerSyncs * a.n_layers;

  // ---- final norm + lm_head + argmax partials
  const int nb = 2 * a.n_run;
  e.N = a.V;
  e.logits = a.logits;
  e.am_val = a.am_val;
  e.am_idx = a.am_idx;
  if (!gemm_phase<EPI_LOGITS, true>(gemm(reinterpret_cast<const uint8_t*>(a.lm_head), H / 32, a.V, nbuf(nb)), e,
                                    NormIn{xbuf(nb), a.final_gain, sbuf(nb), a.n_run == 0 ? 1 : parts}, a.eps, lds,
                                    sy, point))
    return;
  point += 2;
  arrive(sy, point);
  if (!await(sy, point++)) return;
  argmax_phase(a, xbuf(nb), lds);
  if (blockIdx.x == 0 && threadIdx.x == 0) store_wt(a.epoch_ctr, sy.epoch);
}

}  // namespace

bool step_shape_ok(const vsk_model_cfg& c) {
  const int Nq = c.n_q_heads * c.head_dim;
  auto k_ok = [](int K) { return K % 256 == 0 && K / 256 >= kPF; };
  return k_ok(c.hidden) && k_ok(Nq) && k_ok(c.ffn) && c.hidden <= 4096 && (c.head_dim == 64 || c.head_dim == 128) &&
         c.vocab % 16 == 0 && (c.n_kv_heads * c.head_dim) % 16 == 0;
}

size_t step_lds_bytes(const vsk_model_cfg& c) {
  const size_t gemm = kLdsRed + kStepMaxRows * 8;
  const size_t attn = c.head_dim == 128 ? sizeof(AttnLds<128, kWaves>) : sizeof(AttnLds<64, kWaves>);
  return std::max<size_t>(std::max(gemm, attn), 256);
}

int step_occupancy(const vsk_model_cfg& c) {
  const size_t lds = step_lds_bytes(c);
  const void* f = c.head_dim == 128 ? reinterpret_cast<const void*>(&k_step<128>)
                                    : reinterpret_cast<const void*>(&k_step<64>);
  if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)) != hipSuccess)
    return 0;
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, 64 * kWaves, lds) != hipSuccess) return 0;
  return n;
}

hipError_t launch_step(const StepArgs& a, int n_wgs, size_t lds_bytes, hipStream_t s) {
  if (n_wgs < 1 || n_wgs > kStepMaxWgs) return hipErrorInvalidValue;
  StepArgs arg = a;
  void* args[] = {&arg};
  const void* f = a.hd == 128 ? reinterpret_cast<const void*>(&k_step<128>)
                              : reinterpret_cast<const void*>(&k_step<64>);
  return hipLaunchCooperativeKernel(f, dim3(n_wgs), dim3(64 * kWaves), args, static_cast<unsigned>(lds_bytes), s);
}

}  // namespace vsk
