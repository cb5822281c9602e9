// Weight-streaming projections on the matrix cores, with fused epilogues and
// the RMSNorm folded in.
//
// Y[R][N] = X[R][K] W[N][K]^T for the rows of a pass.  Below the ridge point
// the pass is bound by reading W once (paper, appendix "The Switching
// Thresholds from the Roofline": for M rows the arithmetic intensity of a
// weight-stationary decode GEMM is M flops per weight byte), so the kernel is
// organised around streaming W: every wave reads whole 1 KiB tiles with one
// 16-byte load per lane, several tiles in flight, and feeds them straight
// to v_mfma_f32_16x16x32_bf16 with W as the A operand (16 output columns)
// and a 16-row group of X as the B operand.  K is split across the waves of
// a workgroup and reduced in LDS in a fixed order.
//
// RMSNorm.  The residual projections (O, down) end by updating the fp32
// residual x and writing per-workgroup partial sums of x^2 of the updated
// rows, so the normalisation that follows (k_rmsnorm_frags) is one pass over
// x with no reduction of its own.
//
// Epilogues (the tensors stored between kernels are rounded to bf16):
//   RESID  : x[r][n] += y; sum of x^2 partials
//   QKV    : rotary on q,k; q -> bf16 buffer; k,v -> this layer's KV slot
//            (Invariant 1: every row writes its own-layer KV)
//   SWIGLU : a = silu(gate) * up -> bf16 frags for the down projection
//            (the SwiGLU product of Algorithm 1's RUN cohort step)
//   LOGITS : bf16 logits + per-workgroup (max, lowest index)
#include <algorithm>
#include <climits>
#include <utility>

#include <hip/hip_ext.h>

#include "dev.hpp"
#include "gemm.hpp"

namespace vsk {

__device__ __forceinline__ float silu_f(float v) { return v / (1.0f + expf(-v)); }

// The QKV epilogue of one row and four consecutive packed output columns
// n0..n0+3 (n0 a multiple of 4): rotary on q and k heads with the factors of
// packed rows n0, n0 + 2 (cs0, cs1), q to the bf16 buffer, k and v into this
// layer's KV slot `sl` of the row.
__device__ __forceinline__ void qkv_store(const GemmArgs& a, int row, int n0, const f32x4 v, int sl, float2 cs0,
                                          float2 cs1) {
  const int hd = a.hd, half = hd >> 1;
  const int blk = sl >> 4, t = sl & 15;
  if (n0 < a.Nq + a.Nkv) {
    const int ph = n0 % hd;          // packed row inside the head (multiple of 4)
    const int hb = n0 - ph;          // first packed row of the head
    const int j0 = ph >> 1;          // dims j0, j0+half, j0+1, j0+1+half
    const float y0 = v[0] * cs0.x - v[1] * cs0.y;
    const float y1 = v[1] * cs0.x + v[0] * cs0.y;
    const float y2 = v[2] * cs1.x - v[3] * cs1.y;
    const float y3 = v[3] * cs1.x + v[2] * cs1.y;
    if (n0 < a.Nq) {
      uint16_t* q = a.out + static_cast<size_t>(row) * a.Nq + hb;
      q[j0] = f2bf(y0);
      q[j0 + half] = f2bf(y1);
      q[j0 + 1] = f2bf(y2);
      q[j0 + 1 + half] = f2bf(y3);
    } else {
      const int hk = (hb - a.Nq) / hd;
      uint16_t* kb =
          a.pool + ((((static_cast<size_t>(a.layer) * 2 + 0) * a.n_blocks + blk) * a.Hkv + hk) * kBlock * hd);
      kb[kv_k_index(t, j0)] = f2bf(y0);
      kb[kv_k_index(t, j0 + half)] = f2bf(y1);
      kb[kv_k_index(t, j0 + 1)] = f2bf(y2);
      kb[kv_k_index(t, j0 + 1 + half)] = f2bf(y3);
    }
  } else {
    const int nv = n0 - a.Nq - a.Nkv;
    const int hk = nv / hd, e0 = nv % hd;
    uint16_t* vb = a.pool + ((((static_cast<size_t>(a.layer) * 2 + 1) * a.n_blocks + blk) * a.Hkv + hk) * kBlock * hd);
#pragma unroll
    for (int r = 0; r < 4; ++r) vb[kv_v_index(t, e0 + r)] = f2bf(v[r]);
  }
}

template <int MG, int NT, int WN, int WK, int PF, int EPI, bool XL>
__global__ __launch_bounds__(64 * (WN * WK + (XL ? 1 : 0))) void k_gemm(GemmArgs a) {
  static_assert(!XL || (WN * WK == 8 && (WK == 1 || WK == 2 || WK == 4)), "X in LDS: 8 compute waves");
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ float s_amv[WN][MG][16];
  __shared__ int s_ami[WN][MG][16];
  __shared__ double s_ss[WN][MG][16];  // RESID: per-wave sum of x^2

  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  // XL: wave WN * WK only loads X into LDS (wk = -1 keeps it out of every
  // K-split role: it holds no sums and runs no epilogue)
  const bool loader = XL && w == WN * WK;
  const int wn = w % WN, wk = loader ? -1 : w / WN;
  // Workgroup -> (N group, K split, row tile).  Workgroups are dispatched to
  // the 8 XCDs in turn (linear id modulo 8), each XCD with its own L2.  In a
  // row-tiled pass every row tile re-reads the same weights, so with
  // a.xcd_remap the linear ids an XCD receives are renumbered consecutively
  // and the row tile varies fastest: the row tiles of one N group run at the
  // same time on one XCD and read that weight slice from HBM once, the rest
  // from its L2.
  int ng = blockIdx.x, ks = blockIdx.y, mt = blockIdx.z;
  if (a.xcd_remap) {
    const int nwg = gridDim.x * gridDim.y * gridDim.z;
    const int bid = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
    const int xcd = bid & 7, slot = bid >> 3;
    const int lid = xcd * (nwg >> 3) + min(xcd, nwg & 7) + slot;  // a bijection of [0, nwg)
    mt = lid % gridDim.z;
    const int rest = lid / gridDim.z;
    ks = rest % gridDim.y;
    ng = rest / gridDim.y;
  }
  const int n_tiles = a.N >> 4;
  // RESID with K split over workgroups (gridDim.y splits): this workgroup
  // takes K steps [k_lo, k_hi) and stores its product, unreduced
  const bool split_out = EPI == EPI_RESID && a.ypart != nullptr;
  const int nt0 = (ng * WN + wn) * NT;
  const int g0 = mt * MG;
  // rows of this launch: the pass's rows, or a cohort's count read on the
  // device (Algorithm 1's count-bounded GEMMs: the grid is sized for the
  // capacity and a tile starting at or beyond the count exits at once)
  const int Rv = a.count != nullptr ? min(a.R, *a.count) : a.R;
  if (16 * g0 >= Rv) return;
  const int rsub = lane & 15;
  const int nq = 4 * (lane >> 4);

  f32x4 acc[NT][MG];
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int g = 0; g < MG; ++g) acc[j][g] = f32x4{0.f, 0.f, 0.f, 0.f};

  bool tvalid[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) tvalid[j] = (nt0 + j) < n_tiles;

  const int kc = (a.Kt + gridDim.y - 1) / gridDim.y;
  const int k_lo = ks * kc, k_hi = min(a.Kt, k_lo + kc);
  const int first = k_lo + wk;
  const int n_it = first < k_hi ? (k_hi - first + WK - 1) / WK : 0;
  // Out-of-range tiles and rows read a valid one (their sums are never
  // stored) and the stream past the last K step re-reads the last one, so
  // every load in the main loop is unconditional: the compiler can then keep
  // PF steps in flight instead of draining the queue each round.
  int ntc[NT], gc[MG];
#pragma unroll
  for (int j = 0; j < NT; ++j) ntc[j] = min(nt0 + j, n_tiles - 1);
#pragma unroll
  for (int g = 0; g < MG; ++g) gc[g] = min(g0 + g, a.Rg - 1);
  const u32x4* Wbase = a.W + lane;
  const u32x4* Xbase = a.X + lane;

  u32x4 fa[PF][NT], fb[PF][MG];
  auto load = [&](u32x4 (&ra)[NT], u32x4 (&rb)[MG], int i) {
    const int kt = first + min(i, n_it - 1) * WK;
#pragma unroll
    for (int j = 0; j < NT; ++j) ra[j] = Wbase[(static_cast<size_t>(ntc[j]) * a.Kt + kt) * 64];
#pragma unroll
    for (int g = 0; g < MG; ++g) rb[g] = Xbase[(static_cast<size_t>(kt) * a.Rg + gc[g]) * 64];
  };

  // ---- loads the epilogue needs.  They are all issued before the first
  // store of the epilogue: behind a store to a buffer the compiler cannot
  // prove disjoint, each would otherwise wait for a full memory round trip
  // of its own.  Small tiles issue them ahead of the weight stream, so that
  // their latency hides under it; larger ones (more registers) right after
  // the stream, before the cross-wave reduction.
  constexpr bool kHoist = MG * NT <= 2;
  float4 xv[NT][MG];          // RESID: the residual
  int q_slot[MG], q_pos[MG];  // QKV: KV slot and position of the rows
  float2 q_cs[NT][MG][2];     // QKV: rotary factors
  auto epi_loads_a = [&]() {
    if (wk != 0) return;
    if constexpr (EPI == EPI_RESID) {
      if (split_out) return;
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const int n0 = 16 * (nt0 + j) + nq;
#pragma unroll
        for (int g = 0; g < MG; ++g) {
          const int row = 16 * (g0 + g) + rsub;
          xv[j][g] = (tvalid[j] && row < Rv) ? *reinterpret_cast<const float4*>(a.x + static_cast<size_t>(row) * a.N + n0)
                                              : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
    } else if constexpr (EPI == EPI_QKV) {
#pragma unroll
      for (int g = 0; g < MG; ++g) {
        const int row = 16 * (g0 + g) + rsub;
        q_slot[g] = row < Rv ? a.slot[row] : 0;
        q_pos[g] = row < Rv ? a.pos[row] : 0;
      }
    }
  };
  auto epi_loads_b = [&]() {  // rotary factors, after the positions
    if (wk != 0) return;
    if constexpr (EPI == EPI_QKV) {
      const int half = a.hd >> 1;
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const int n0 = 16 * (nt0 + j) + nq;
        const int j0 = (n0 % a.hd) >> 1;
        const bool rot = tvalid[j] && n0 < a.Nq + a.Nkv;
#pragma unroll
        for (int g = 0; g < MG; ++g) {
          const int row = 16 * (g0 + g) + rsub;
          const bool ok = rot && row < Rv;
          const float2* rp = a.rope + static_cast<size_t>(q_pos[g]) * half + j0;
          q_cs[j][g][0] = ok ? rp[0] : make_float2(1.f, 0.f);
          q_cs[j][g][1] = ok ? rp[1] : make_float2(1.f, 0.f);
        }
      }
    }
  };
  if constexpr (kHoist) epi_loads_a();

  if constexpr (!XL) {
    if (n_it > 0) {
  #pragma unroll
      for (int st = 0; st < PF; ++st) load(fa[st], fb[st], st);
    }

    if constexpr (kHoist) epi_loads_b();

    auto step = [&](int st) {
  #pragma unroll
      for (int j = 0; j < NT; ++j)
  #pragma unroll
        for (int g = 0; g < MG; ++g) acc[j][g] = mfma_16x16x32(fa[st][j], fb[st][g], acc[j][g]);
    };

    int it = 0;
    for (; it + PF < n_it; it += PF) {
  #pragma unroll
      for (int st = 0; st < PF; ++st) {
        step(st);
        load(fa[st], fb[st], it + st + PF);
        // keep each step's refill next to its use instead of batching a
        // whole round of loads at the end of the loop body
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  #pragma unroll
    for (int st = 0; st < PF; ++st)
      if (it + st < n_it) step(st);
  } else {
    // ---- X staged in LDS by a loader wave.  The WN waves of a K parity
    // class take the same K steps for different N tiles, so each X chunk
    // (kCK K steps x MG row groups) is loaded once per workgroup.  All vector
    // loads of a wave complete in issue order, so X loads mixed into the
    // weight stream would make every X wait drain the weight ring; here a
    // ninth wave issues only X loads (global -> LDS, no registers) into LDS
    // buffers, and the eight compute waves issue only
    // weight loads, PF tiles ahead, and read X from LDS.  One workgroup
    // barrier per chunk; the loader runs two chunks ahead (three buffers), so
    // a chunk's X latency is hidden behind two chunks of weight streaming.
    constexpr int kCK = MG <= 4 ? 8 : 4;       // K steps per X chunk (32 KiB)
    constexpr int SPW = kCK / WK;              // a compute wave's K steps per chunk
    constexpr int NR = PF / SPW;               // chunks per round of the weight ring
    constexpr int kLead = 2;                   // chunks the loader runs ahead
    constexpr int kBuf = kLead + 1;            // X chunk buffers in LDS
    constexpr int kLPC = kCK * MG;             // loads per chunk (at most 63 may stay outstanding)
    static_assert(PF % SPW == 0, "weight ring spans whole chunks");
    static_assert((kLead - 1) * kLPC <= 63, "outstanding loads beyond the wait counter");
    u32x4* xs = reinterpret_cast<u32x4*>(smem);  // [kBuf][kCK][MG][64]
    const int n_chunks = (k_hi - k_lo + kCK - 1) / kCK;
    if (loader) {
      // chunk c -> buffer c % kBuf: one 1 KiB load per (K step, row group),
      // lane l's 16 bytes landing at LDS piece l
      auto xload = [&](int c) {
        const int buf = c % kBuf;
#pragma unroll
        for (int kc = 0; kc < kCK; ++kc) {
          const int kt = min(k_lo + c * kCK + kc, k_hi - 1);
#pragma unroll
          for (int g = 0; g < MG; ++g)
            lds_load16(a.X + (static_cast<size_t>(kt) * a.Rg + gc[g]) * 64 + lane,
                       xs + (static_cast<size_t>(buf * kCK + kc) * MG + g) * 64);
        }
      };
      // wait until chunk c has landed: the chunks issued after it may stay
      // in flight when there are kLead - 1 of them, else wait for all
      auto wait_for = [&](int c) {
        if (c + kLead - 1 < n_chunks) asm volatile("s_waitcnt vmcnt(%0)" ::"n"((kLead - 1) * kLPC) : "memory");
        else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      };
#pragma unroll
      for (int d = 0; d < kLead; ++d)
        if (d < n_chunks) xload(d);
      wait_for(0);
      barrier_no_fence();
      for (int c = 0; c < n_chunks; ++c) {
        // buffer (c + kLead) % kBuf was last read in chunk c - 1
        if (c + kLead < n_chunks) xload(c + kLead);
        if (c + 1 < n_chunks) wait_for(c + 1);
        barrier_no_fence();
      }
    } else {
      auto wload = [&](u32x4 (&r)[NT], int i) {
        const int kt = first + min(i, n_it - 1) * WK;
#pragma unroll
        for (int j = 0; j < NT; ++j) r[j] = Wbase[(static_cast<size_t>(ntc[j]) * a.Kt + kt) * 64];
      };
      if (n_it > 0) {
#pragma unroll
        for (int st = 0; st < PF; ++st) wload(fa[st], st);
      }
      __syncthreads();
      // one chunk from ring slots st0.. (compile-time: the ring lives in
      // registers); FULL: every wave has all SPW steps, so nothing in it is
      // conditional (a condition would make the compiler drain the load
      // queue before each step)
      auto chunk = [&](int c, auto st0_c, auto full_c) {
        constexpr int st0 = decltype(st0_c)::value;
        constexpr bool FULL = decltype(full_c)::value;
#pragma unroll
        for (int i = 0; i < SPW; ++i) {
          const int it = c * SPW + i;
          if (FULL || it < n_it) {
            const u32x4* xb = xs + (static_cast<size_t>((c % kBuf) * kCK + wk + i * WK) * MG) * 64 + lane;
            // all reads of a batch before its MFMAs: one LDS wait per batch
            // instead of one per row group.  Up to 8 row groups the step is
            // one batch; taller tiles read theirs four at a time (at 11 row
            // groups with two N tiles per wave, two batches spill)
            constexpr int XB = MG > 8 ? 4 : MG;
#pragma unroll
            for (int gb = 0; gb < MG; gb += XB) {
              u32x4 xv[XB];
#pragma unroll
              for (int g = 0; g < XB; ++g)
                if (gb + g < MG) xv[g] = xb[(gb + g) * 64];
#pragma unroll
              for (int j = 0; j < NT; ++j)
#pragma unroll
                for (int g = 0; g < XB; ++g)
                  if (gb + g < MG) acc[j][gb + g] = mfma_16x16x32(fa[st0 + i][j], xv[g], acc[j][gb + g]);
            }
            wload(fa[st0 + i], it + PF);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
        barrier_after_lds_reads();
      };
      const int n_full = (k_hi - k_lo) / kCK;  // chunks in which every wave has SPW steps
      int c = 0;
      for (; c + NR <= n_full; c += NR) {
        [&]<int... CC>(std::integer_sequence<int, CC...>) {
          (chunk(c + CC, std::integral_constant<int, CC * SPW>{}, std::true_type{}), ...);
        }(std::make_integer_sequence<int, NR>{});
      }
      // the rest of the chunks (fewer than a round), guarded
      [&]<int... CC>(std::integer_sequence<int, CC...>) {
        ((c + CC < n_chunks ? chunk(c + CC, std::integral_constant<int, CC * SPW>{}, std::false_type{}) : void()),
         ...);
      }(std::make_integer_sequence<int, NR>{});
    }
  }

  if constexpr (!kHoist) {
    epi_loads_a();
    epi_loads_b();
  }

  // ---- reduce the K-split waves of this workgroup (fixed order)
  if constexpr (WK > 1) {
    f32x4* red = reinterpret_cast<f32x4*>(smem);
    if (wk > 0) {
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int g = 0; g < MG; ++g) red[((((wk - 1) * WN + wn) * NT + j) * MG + g) * 64 + lane] = acc[j][g];
    }
    __syncthreads();
    if (wk == 0) {
      // one partner wave at a time: unrolled, the LDS reads of all seven
      // would be hoisted and hold 28 registers per output tile
#pragma unroll 1
      for (int w2 = 1; w2 < WK; ++w2)
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
          for (int g = 0; g < MG; ++g) acc[j][g] += red[((((w2 - 1) * WN + wn) * NT + j) * MG + g) * 64 + lane];
    }
  }

  // ---- epilogues (waves with wk == 0 hold the sums)
  if constexpr (EPI == EPI_RESID) {
    if (split_out) {
      if (wk == 0) {
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
          for (int g = 0; g < MG; ++g) {
            const int row = 16 * (g0 + g) + rsub;
            if (!tvalid[j] || row >= Rv) continue;
            const int n0 = 16 * (nt0 + j) + nq;
            *reinterpret_cast<f32x4*>(a.ypart + (static_cast<size_t>(ks) * a.R + row) * a.N + n0) = acc[j][g];
          }
      }
      return;
    }
    // x += y; this workgroup's share of sum x^2 per row
    if (wk == 0) {
#pragma unroll
      for (int g = 0; g < MG; ++g) {
        const int row = 16 * (g0 + g) + rsub;
        double ss = 0.0;
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          if (!tvalid[j] || row >= Rv) continue;
          const int n0 = 16 * (nt0 + j) + nq;
          float4* px = reinterpret_cast<float4*>(a.x + static_cast<size_t>(row) * a.N + n0);
          float4 v = xv[j][g];
          v.x += acc[j][g][0];
          v.y += acc[j][g][1];
          v.z += acc[j][g][2];
          v.w += acc[j][g][3];
          *px = v;
          ss += static_cast<double>(v.x) * v.x + static_cast<double>(v.y) * v.y +
                static_cast<double>(v.z) * v.z + static_cast<double>(v.w) * v.w;
        }
        // the four lane groups hold the same row
        ss += __shfl_xor(ss, 16, 64);
        ss += __shfl_xor(ss, 32, 64);
        if (lane < 16) s_ss[wn][g][lane] = ss;
      }
    }
    if (a.ssq_out != nullptr) {
      __syncthreads();
      if (threadIdx.x < MG * 16) {
        const int g = threadIdx.x >> 4, l = threadIdx.x & 15;
        double ss = s_ss[0][g][l];
#pragma unroll
        for (int w2 = 1; w2 < WN; ++w2) ss += s_ss[w2][g][l];
        const int row = 16 * (g0 + g) + l;
        if (row < Rv) a.ssq_out[static_cast<size_t>(row) * gridDim.x + ng] = ss;  // [row][workgroup]
      }
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    if (wk == 0) {
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        if (!tvalid[j]) continue;
        const int u = 4 * (nt0 + j) + (lane >> 4);  // output columns 2u, 2u+1
#pragma unroll
        for (int g = 0; g < MG; ++g) {
          const int row = 16 * (g0 + g) + rsub;
          if (row >= Rv) continue;
          const float a0 = silu_f(acc[j][g][0]) * acc[j][g][2];
          const float a1 = silu_f(acc[j][g][1]) * acc[j][g][3];
          *reinterpret_cast<uint32_t*>(a.out + frag_index(row, 2 * u, a.out_Rg)) = pack_bf2(a0, a1);
        }
      }
    }
  } else if constexpr (EPI == EPI_QKV) {
    if (wk == 0) {
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        if (!tvalid[j]) continue;
        const int n0 = 16 * (nt0 + j) + nq;
#pragma unroll
        for (int g = 0; g < MG; ++g) {
          const int row = 16 * (g0 + g) + rsub;
          if (row >= Rv) continue;
          qkv_store(a, row, n0, acc[j][g], q_slot[g], q_cs[j][g][0], q_cs[j][g][1]);
        }
      }
    }
  } else if constexpr (EPI == EPI_LOGITS) {
    if (wk == 0) {
#pragma unroll
      for (int g = 0; g < MG; ++g) {
        const int row = 16 * (g0 + g) + rsub;
        float bv = -INFINITY;
        int bi = INT_MAX;
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          if (!tvalid[j] || row >= Rv) continue;
          const int n0 = 16 * (nt0 + j) + nq;
          const f32x4 v = acc[j][g];
          uint2 packed;
          packed.x = pack_bf2(v[0], v[1]);
          packed.y = pack_bf2(v[2], v[3]);
          *reinterpret_cast<uint2*>(a.out + static_cast<size_t>(row) * a.N + n0) = packed;
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
        if (lane < 16) {
          s_amv[wn][g][lane] = bv;
          s_ami[wn][g][lane] = bi;
        }
      }
    }
    __syncthreads();
    if (threadIdx.x < MG * 16) {
      const int g = threadIdx.x >> 4, l = threadIdx.x & 15;
      float bv = s_amv[0][g][l];
      int bi = s_ami[0][g][l];
#pragma unroll
      for (int w2 = 1; w2 < WN; ++w2) am_merge(bv, bi, s_amv[w2][g][l], s_ami[w2][g][l]);
      const int row = 16 * (g0 + g) + l;
      if (row < Rv) {
        a.am_val[static_cast<size_t>(ng) * a.R + row] = bv;
        a.am_idx[static_cast<size_t>(ng) * a.R + row] = bi;
      }
    }
  }
}

// ---------------------------------------------------------------- launcher
template <int MG, int NT, int WN, int WK, int PF, int EPI, bool XL = false>
static hipError_t launch_cfg(const GemmArgs& a_in, int m_tiles, int ksplit, hipStream_t s, const LaunchEvents& ev) {
  GemmArgs a = a_in;
  a.xcd_remap = a_in.xcd_remap && m_tiles > 1 ? 1 : 0;
  const int n_groups = (a.N / 16 + NT * WN - 1) / (NT * WN);
  dim3 grid(n_groups, ksplit, m_tiles);
  // cross-wave reduction; with X in LDS the same space first holds the X chunks
  size_t smem = (WK > 1 ? (WK - 1) : 0) * WN * NT * MG * 64 * sizeof(f32x4);
  if constexpr (XL) {
    smem = std::max<size_t>(smem, 3 * (MG <= 4 ? 8 : 4) * MG * 64 * sizeof(u32x4));
    // with the static arrays this is more than 64 KiB of LDS: allow it once
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&k_gemm<MG, NT, WN, WK, PF, EPI, XL>),
        hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
    if (attr != hipSuccess) return attr;
  }
  const dim3 block(64 * (WN * WK + (XL ? 1 : 0)));
  if (ev.start != nullptr || ev.stop != nullptr) {
    // events bound to this dispatch: they take its start and end times
    hipExtLaunchKernelGGL((k_gemm<MG, NT, WN, WK, PF, EPI, XL>), grid, block, static_cast<uint32_t>(smem), s, ev.start,
                          ev.stop, 0u, a);
  } else {
    hipLaunchKernelGGL((k_gemm<MG, NT, WN, WK, PF, EPI, XL>), grid, block, smem, s, a);
  }
  return hipGetLastError();
}

// Launch shapes.  mg = 16-row groups of X per tile.  For mg == 1:
//  narrow  one 16-column N tile per wave, 8 K-split waves, 4 K steps in
//          flight (residual projections: N = hidden);
//  pair    two N tiles per wave, 4 K steps in flight (QKV, gate/up);
//  wide    four N tiles per wave (lm_head).
// For 2..8 row groups (2 takes the 4-row-group layouts) the default
// (shape 0) is, with one row tile: X staged
// in LDS by a ninth wave for gate/up (four N tiles; at 8 row groups eight,
// two per wave) and lm_head (sixteen, two per wave, the eight waves side by
// side), for the residual projections and QKV the four-tile (4 row groups)
// or eight-tile (8) LDS layout with K split over workgroups (unsplit QKV:
// two N tiles per workgroup).  A row-tiled pass (more than 128 rows) takes
// the LDS layout with the eight waves side by side (16 N tiles; 8 for QKV).
// Shape 1 takes one N tile per wave column everywhere, shape 2 two, shape 3
// is a 2 x 2 wave grid over four N tiles, shape 4 stages X in LDS for four N
// tiles (two for QKV) everywhere, shape 5 for eight (two per wave) at 8 row
// groups with QKV and 4 row groups on the 2 x 2 grid, shape 6 the default's
// LDS layouts for every projection but the residual ones, whatever the row
// tiling.
// Row-tiled passes whose launch rounds another tile height fills better
// than 8 row groups (see plan_gemm): staged X, the eight waves side by side,
// as at 8 (QKV keeps one N tile per wave: two spill 147 registers in its
// rotary epilogue at 11 row groups; the residual epilogue, holding the
// residual beside the sums, spills 53 at 11 and stays at 8 or below).
template <int MG, int EPI>
static hipError_t launch_row_tiled(const GemmArgs& a, const GemmPlan& p, hipStream_t s, const LaunchEvents& ev) {
  if constexpr (EPI == EPI_QKV) return launch_cfg<MG, 1, 8, 1, 4, EPI, true>(a, p.m_tiles, p.ksplit, s, ev);
  else if constexpr (EPI == EPI_LOGITS || (EPI == EPI_RESID && MG > 8)) return hipErrorInvalidValue;
  else return launch_cfg<MG, 2, 8, 1, 4, EPI, true>(a, p.m_tiles, p.ksplit, s, ev);
}

template <int EPI>
static hipError_t launch_epi(const GemmArgs& a, const GemmPlan& p, hipStream_t s, const LaunchEvents& ev) {
  switch (p.mg) {
    case 1:
      if (p.nt == 4) return launch_cfg<1, 4, 1, 8, 4, EPI>(a, p.m_tiles, p.ksplit, s, ev);
      if (p.nt == 2) return launch_cfg<1, 2, 1, 8, 4, EPI>(a, p.m_tiles, p.ksplit, s, ev);
      return launch_cfg<1, 1, 1, 8, 4, EPI>(a, p.m_tiles, p.ksplit, s, ev);
    case 4:
      if (p.xl) {
        // weight rings of 4 and 2 K steps: shallower rings measured faster
        // with X in LDS (16 steps: batch-64 pass 3.06 ms, these 2.90)
        if constexpr (EPI == EPI_LOGITS)
          if (p.nt == 2) return launch_cfg<4, 2, 8, 1, 8, EPI, true>(a, p.m_tiles, p.ksplit, s, ev);
        if (p.wn == 4) return launch_cfg<4, 1, 4, 2, 4, EPI, true>(a, p.m_tiles, p.ksplit, s, ev);
        return launch_cfg<4, 1, 2, 4, 2, EPI, true>(a, p.m_tiles, p.ksplit, s, ev);
      }
      if (p.wn == 2) return launch_cfg<4, 2, 2, 2, 2, EPI>(a, p.m_tiles, p.ksplit, s, ev);
      if (p.nt == 2) return launch_cfg<4, 2, 1, 8, 4, EPI>(a, p.m_tiles, p.ksplit, s, ev);
      return launch_cfg<4, 1, 1, 8, 4, EPI>(a, p.m_tiles, p.ksplit, s, ev);
    case 6: return launch_row_tiled<6, EPI>(a, p, s, ev);
    case 7: return launch_row_tiled<7, EPI>(a, p, s, ev);
    case 11: return launch_row_tiled<11, EPI>(a, p, s, ev);
    default:
      if (p.xl) {
        // (QKV takes one N tile per wave: see plan_gemm)
        // eight waves side by side (no K split inside the workgroup)
        if (p.wn == 8) {
          if constexpr (EPI == EPI_QKV) return launch_cfg<8, 1, 8, 1, 4, EPI, true>(a, p.m_tiles, p.ksplit, s, ev);
          else return launch_cfg<8, 2, 8, 1, 4, EPI, true>(a, p.m_tiles, p.ksplit, s, ev);
        }
        if constexpr (EPI != EPI_QKV)
          // (a 4-step weight ring here measured no faster: 8B batch-128
          // pass 7.60 against 7.65 ms, gate/up 55.8 against 55.9 us)
          if (p.nt == 2) return launch_cfg<8, 2, 4, 2, 2, EPI, true>(a, p.m_tiles, p.ksplit, s, ev);
        if (p.wn == 4) return launch_cfg<8, 1, 4, 2, 16, EPI, true>(a, p.m_tiles, p.ksplit, s, ev);
        return launch_cfg<8, 1, 2, 4, 4, EPI, true>(a, p.m_tiles, p.ksplit, s, ev);
      }
      if (p.wn == 2) return launch_cfg<8, 2, 2, 2, 2, EPI>(a, p.m_tiles, p.ksplit, s, ev);
      if (p.nt == 2) return launch_cfg<8, 2, 1, 4, 2, EPI>(a, p.m_tiles, p.ksplit, s, ev);
      return launch_cfg<8, 1, 1, 8, 4, EPI>(a, p.m_tiles, p.ksplit, s, ev);
  }
}

GemmPlan plan_gemm(int N, int K, int R, int epi, int shape, int resid_target, int row_tile) {
  GemmPlan p;
  const int Rg = (R + 15) / 16;
  // 17..32 rows take the 4-row-group layouts (the padding groups re-read the
  // last one): against one column of K-split waves over 2 row groups the 8B
  // step at 24 and 32 rows went from 5.15 / 5.24 to 4.58 / 4.67 ms
  p.mg = Rg <= 1 ? 1 : Rg <= 4 ? 4 : 8;
  p.m_tiles = (Rg + p.mg - 1) / p.mg;
  p.nt = 1;
  p.wn = 1;
  int wk = 8;
  if (p.mg == 1) {
    // (QKV with one tile per wave, 320 workgroups at batch 16 instead of
    // 160, measured slower: 12.2 against 11.0 us)
    if (epi != EPI_RESID) p.nt = epi == EPI_LOGITS ? 4 : 2;
    // a residual projection with K > N (down): two N tiles per workgroup,
    // half the X reads per weight byte, with K split in two (below) to keep
    // the workgroup count (batch 16: 15.5 -> 13.3 us, the pass 2.149 ->
    // 2.125 ms)
    else if (K > N) p.nt = 2;
  } else if (p.mg >= 4) {
    const bool wide_n = epi == EPI_SWIGLU || epi == EPI_LOGITS;
    const bool auto_shape = shape == 0;
    const bool one_tile = p.m_tiles == 1;
    if ((auto_shape || shape == 5 || shape == 6) && p.mg == 8 && epi != EPI_QKV) {
      // X in LDS, two N tiles per wave: eight N tiles per workgroup, each X
      // chunk read once from L2 for all of them (measured the fastest for 8
      // row groups, one row tile or several)
      p.xl = true;
      p.nt = 2;
      p.wn = 4;
      wk = 2;
      // lm_head, and every projection of a row-tiled pass (workgroups to
      // spare): the eight waves side by side, 16 N tiles per workgroup
      // (half the X reads per weight byte; lm_head 242 -> 222 us at batch
      // 128, the 2,080-row pass 21.0 -> 16.6 ms with QKV below)
      if (epi == EPI_LOGITS || (epi != EPI_QKV && !one_tile)) {
        p.wn = 8;
        wk = 1;
      }
    } else if (auto_shape && !one_tile && p.mg == 8 && epi == EPI_QKV) {
      // QKV of a row-tiled pass: X in LDS, eight waves side by side with one
      // N tile each (two per wave compile without spills but measured slower
      // at 2,080 rows: 112 against 108 us per launch)
      p.xl = true;
      p.wn = 8;
      wk = 1;
    } else if (shape == 3 || shape == 5 || (auto_shape && !one_tile)) {
      // a row-tiled pass (more than 128 rows) re-streams the weights once per
      // row tile: there the 2 x 2 wave grid, each X chunk feeding four N
      // tiles, is the faster default
      p.nt = 2;
      p.wn = 2;
      wk = 2;
    } else if (shape == 4 || ((shape == 6 || auto_shape) && epi != EPI_RESID) || auto_shape) {
      // X in LDS: four N tiles per workgroup (two for QKV, whose N is small);
      // the default for every projection of one row tile at 4 row groups
      // (the residual ones with K split over workgroups)
      p.xl = true;
      p.wn = epi == EPI_QKV ? 2 : 4;
      wk = 8 / p.wn;
      // lm_head (N = vocab: workgroups to spare) at 4 row groups: two N
      // tiles per wave and the eight waves side by side (no K split inside
      // the workgroup), a quarter of the X reads per weight byte (170 -> 152
      // us at batch 64 with four waves side by side, 151 -> 147 with eight)
      if (epi == EPI_LOGITS && p.mg == 4) {
        p.nt = 2;
        p.wn = 8;
        wk = 1;
      }
    } else {
      // one column of K-split waves (N = hidden gives 192-256 workgroups)
      p.nt = shape == 1 ? 1 : shape == 2 ? 2 : (wide_n ? 2 : 1);
      wk = p.mg == 8 && p.nt == 2 ? 4 : 8;
    }
  }
  const int cols_per_group = 16 * p.nt * p.wn;
  p.n_groups = (N / 16 * 16 + cols_per_group - 1) / cols_per_group;
  // Tile height of a row-tiled projection.  One staged workgroup fills a
  // compute unit (LDS), so a launch runs in rounds of kComputeUnits
  // workgroups and a partly filled last round costs a whole one.  A round
  // of mg-row-group tiles costs, relative to 8 (measured per round on the
  // 3B and 8B projections at 768-2,080 rows): 6 groups 0.85, 7 0.94, 11
  // 1.40 -- a shorter tile keeps its weight stream and epilogue, a taller
  // one reads its X fragments in batches.  6, 7 or 11 row groups replace 8
  // where rounds x that cost comes out lower, e.g. at 2,080 rows (130
  // groups): gate/up 12 tiles of 11 (3 rounds, 4.2) instead of 17 of 8 (5
  // rounds), QKV 12 of 11 (2 rounds, 2.8; 3 at 8), O and down 19 tiles of 7
  // in one round (0.94).  Launches that split K (at most
  // kRowTiledSplitBelow workgroups, below) keep 8.
  if (p.xl && p.wn == 8 && p.m_tiles > 1 && epi != EPI_LOGITS && row_tile != 8) {
    auto tiles_at = [&](int mg) { return (Rg + mg - 1) / mg * p.n_groups; };
    auto cost = [&](int mg) {
      const int per_round = mg == 6 ? 85 : mg == 7 ? 94 : mg == 11 ? 140 : 100;
      return (tiles_at(mg) + kComputeUnits - 1) / kComputeUnits * per_round;
    };
    const int tallest = epi == EPI_RESID ? 7 : 11;  // the residual epilogue spills at 11
    int best = 8;
    if (row_tile != 0) {
      best = row_tile <= tallest ? row_tile : 8;
    } else if (tiles_at(8) > kRowTiledSplitBelow) {
      for (const int mg : {6, 7, 11})
        if (mg <= tallest && tiles_at(mg) > kRowTiledSplitBelow && cost(mg) < cost(best)) best = mg;
    }
    p.mg = best;
    p.m_tiles = (Rg + best - 1) / best;
  }
  // a residual projection of one row tile splits K until the workgroups
  // reach resid_target, keeping at least 4 K steps per wave; k_resid_norm
  // then adds the splits' products into the residual.  With X in LDS the
  // default target is 192 workgroups at 4 row groups (4 splits at hidden
  // 3072) and 384 at 8 (measured best of 96-384 and 128-384).
  const int target = resid_target < 0            ? 0
                     : resid_target > 0          ? resid_target
                     : p.xl                      ? (p.mg == 4 ? 192 : 384)
                     : p.mg == 1 && p.nt == 2    ? 192
                                                 : kResidTargetWgs;
  // A row-tiled pass with few workgroups (n_groups x m_tiles at most
  // kRowTiledSplitBelow: 129 to about a thousand rows at hidden 4096, where
  // 16 N groups per row tile left 32-128 workgroups streaming the weights)
  // splits K too, into as many splits as keep the workgroups within
  // kRowTiledTarget (one per compute unit: a launch of one round).
  const int tiles = p.n_groups * p.m_tiles;
  const bool row_tiled_split = p.m_tiles > 1 && tiles <= kRowTiledSplitBelow;
  if (epi == EPI_RESID && target > 0 && (p.m_tiles == 1 || row_tiled_split)) {
    const int Kt = K / 32;
    const int want = p.m_tiles == 1 ? (target + tiles - 1) / tiles : kRowTiledTarget / tiles;
    int ks = std::min({want, kMaxResidSplits, std::max(1, Kt / (4 * wk))});
    ks = std::max(ks, 1);
    const int kc = (Kt + ks - 1) / ks;  // equal splits
    p.ksplit = (Kt + kc - 1) / kc;
  }
  return p;
}

hipError_t launch_gemm(GemmArgs a, const GemmPlan& p, int epi, hipStream_t s, LaunchEvents ev) {
  switch (epi) {
    case EPI_RESID: return launch_epi<EPI_RESID>(a, p, s, ev);
    case EPI_QKV: return launch_epi<EPI_QKV>(a, p, s, ev);
    case EPI_SWIGLU: return launch_epi<EPI_SWIGLU>(a, p, s, ev);
    default: return launch_epi<EPI_LOGITS>(a, p, s, ev);
  }
}

// ---------------------------------------------------------------- QKV, K split
// The QKV projection with K split over workgroups: the projection kernel
// stores each split's product (RESID layout, ypart[split][R][N]); this kernel
// adds them in split order and applies the QKV epilogue.  One thread per row
// and four packed columns; its loads (position, slot, every split) are all
// issued before the first add.  NS > 0: exactly NS splits (every load
// unconditional).
template <int NS>
__global__ __launch_bounds__(256) void k_qkv_reduce(GemmArgs a, int splits) {
  if constexpr (NS > 0) splits = NS;
  constexpr int kMax = NS > 0 ? NS : kMaxResidSplits;
  const int row = blockIdx.y;
  const int n0 = 4 * (blockIdx.x * blockDim.x + threadIdx.x);
  if (n0 >= a.N) return;
  const int sl = a.slot[row], p = a.pos[row];
  const float* y = a.ypart + static_cast<size_t>(row) * a.N + n0;
  const size_t stride = static_cast<size_t>(a.R) * a.N;
  f32x4 ys[kMax];
#pragma unroll
  for (int sp = 0; sp < kMax; ++sp)
    if (NS > 0 || sp < splits) ys[sp] = *reinterpret_cast<const f32x4*>(y + sp * stride);
  float2 cs0 = make_float2(1.f, 0.f), cs1 = make_float2(1.f, 0.f);
  if (n0 < a.Nq + a.Nkv) {
    const float2* rp = a.rope + static_cast<size_t>(p) * (a.hd >> 1) + ((n0 % a.hd) >> 1);
    cs0 = rp[0];
    cs1 = rp[1];
  }
  f32x4 v = ys[0];
#pragma unroll
  for (int sp = 1; sp < kMax; ++sp)
    if (NS > 0 || sp < splits) v += ys[sp];
  qkv_store(a, row, n0, v, sl, cs0, cs1);
}

hipError_t launch_qkv_reduce(const GemmArgs& a, int splits, hipStream_t s) {
  if (splits < 2 || splits > kMaxResidSplits || a.N % 16 != 0 || a.ypart == nullptr) return hipErrorInvalidValue;
  const dim3 grid((a.N / 4 + 255) / 256, a.R);
  switch (splits) {
    case 2: hipLaunchKernelGGL(k_qkv_reduce<2>, grid, dim3(256), 0, s, a, splits); break;
    case 3: hipLaunchKernelGGL(k_qkv_reduce<3>, grid, dim3(256), 0, s, a, splits); break;
    case 4: hipLaunchKernelGGL(k_qkv_reduce<4>, grid, dim3(256), 0, s, a, splits); break;
    default: hipLaunchKernelGGL(k_qkv_reduce<0>, grid, dim3(256), 0, s, a, splits);
  }
  return hipGetLastError();
}

}  // namespace vsk
