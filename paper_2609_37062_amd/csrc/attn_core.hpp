// One work item of paged-attention decode: (row, KV head, split of the
// context), processed by a workgroup of NW waves.  Shared by the
// per-op attention kernel (k_attn.hip) and the persistent step kernel
// (k_step.hip).
//
// For every row (one token at position p of its sequence) and KV head, the
// query heads of that KV head's group attend to keys 0..p read through the
// sequence's block table (paper, "Invariants": each layer reads its own
// cached K,V; Algorithm 1 keeps attention's launch shape).  The NW waves
// take the split's 16-token blocks as contiguous ranges.  The split's
// block-table entries are staged in LDS first; each wave then keeps NB
// blocks of K/V loads in flight ahead of the block it processes.  Per block
// a wave computes S = K q with v_mfma_f32_16x16x32_bf16 (16 tokens x up to
// 16 heads), an online softmax in the base-2 domain, and O^T += V^T P^T with
// v_mfma_f32_16x16x16_bf16, so the softmax row lives in the same lanes as the
// output it rescales.  The waves merge in LDS; with several splits the last
// workgroup to finish a (row, KV head) merges the splits' (m, l, O) partials
// in split order.  Decode attention reads about group-size flops per byte of
// KV, so it is bound by HBM, not by the matrix cores.
#pragma once

#include <cmath>

#include "attn.hpp"
#include "dev.hpp"

namespace vsk {

constexpr int kAttnWaves = 4;  // waves of a per-op decode work item (the persistent kernel uses 8)

// LDS of one work item (the persistent kernel overlays it on the space its
// projections use)
template <int D, int NW>
struct AttnLds {
  float m[NW][16];
  float l[NW][16];
  f32x4 o[NW - 1][D / 16][64];
  int32_t tbl[kAttnMaxBps];
  int last;
};

// agent-scope (all XCDs) coherent accesses for the split partials
__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Splits of a row: n_splits(kv_len) for the row's kv_len = pos + 1.
__device__ __forceinline__ int attn_row_splits(int kv_len, int bps) {
  const int nb = (kv_len + kBlock - 1) / kBlock;
  return (nb + bps - 1) / bps;
}

// WT: the attention output is stored write-through (sc1), so that other
// workgroups of the same launch read it from memory, not from a stale L2.
// FOLD2: a wave loads two shared-prefix partials before folding either (one
// round trip per two; 186 instead of 167 registers at head_dim 128), for
// passes with more prefix partials per row than waves.
template <int D, int NB, bool WT, int NW, bool FOLD2 = false>
__device__ __forceinline__ void attn_unit(const AttnArgs& a, int row, int hk, int split, AttnLds<D, NW>& sm) {
  constexpr int KC = D / 32;  // K chunks (1 KiB) per block
  constexpr int VC = D / 16;  // V chunks (512 B) per block

  const int tid = opaque_tid();
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int G = a.G;
  const int kv_len = a.pos[row] + 1;
  const int nb = (kv_len + kBlock - 1) / kBlock;
  // a shared prefix of P blocks is read by the prefix work items; this row's
  // splits cover blocks P.. and follow the prefix partials
  const int P = a.pfx_blocks != nullptr ? a.pfx_blocks[row] : 0;
  const int n_ps = P > 0 ? a.pfx_splits[row] : 0;
  const int n_splits = (nb - P + a.bps - 1) / a.bps;
  if (split >= n_splits) return;
  const int seq = a.row_seq[row];
  const int32_t* table = a.block_table + static_cast<size_t>(seq) * a.max_blocks;
  const int b_lo = P + split * a.bps;
  const int b_hi = min(nb, b_lo + a.bps);
  // the split's block-table entries, staged once for all waves
  for (int i = tid; i < b_hi - b_lo; i += blockDim.x) sm.tbl[i] = table[b_lo + i];
  const int h = lane & 15;       // query head within the group (valid if h < G)
  const int quad = lane >> 4;    // token quarter / k sub-range
  // q as the B operand of S = K q: lane holds q[h][32c + 8*quad .. +7]
  u32x4 qf[KC];
  {
    const uint16_t* qrow = a.q + static_cast<size_t>(row) * a.Nq + static_cast<size_t>(hk * G + h) * D;
#pragma unroll
    for (int c = 0; c < KC; ++c)
      qf[c] = (h < G) ? *reinterpret_cast<const u32x4*>(qrow + 32 * c + 8 * quad) : u32x4{0u, 0u, 0u, 0u};
  }
  const float sc = a.scale_log2;  // log2(e) / sqrt(D)
  float m = -INFINITY, l = 0.f;
  f32x4 o[VC];
#pragma unroll
  for (int c = 0; c < VC; ++c) o[c] = f32x4{0.f, 0.f, 0.f, 0.f};

  const size_t kv_stride = static_cast<size_t>(a.Hkv) * kBlock * D;  // one block, all heads
  const uint16_t* kbase = a.pool + (static_cast<size_t>(a.layer) * 2 + 0) * a.n_blocks * kv_stride +
                          static_cast<size_t>(hk) * kBlock * D;
  const uint16_t* vbase = a.pool + (static_cast<size_t>(a.layer) * 2 + 1) * a.n_blocks * kv_stride +
                          static_cast<size_t>(hk) * kBlock * D;

  // one 16-token block: S = K q, online softmax, O^T += V^T P^T
  auto process = [&](const u32x4 (&kf)[KC], u32x2 (&vf)[VC], int b) {
    // slots past kv_len in the last block hold whatever was there: zero their
    // V (a masked probability of 0 times a NaN pattern would still be NaN)
    const int t_lane = b * kBlock + 4 * quad;  // first token of this lane's quarter
    if (t_lane + 3 >= kv_len) {
      const uint32_t m01 = (t_lane + 0 < kv_len ? 0x0000ffffu : 0u) | (t_lane + 1 < kv_len ? 0xffff0000u : 0u);
      const uint32_t m23 = (t_lane + 2 < kv_len ? 0x0000ffffu : 0u) | (t_lane + 3 < kv_len ? 0xffff0000u : 0u);
#pragma unroll
      for (int c = 0; c < VC; ++c) {
        vf[c][0] &= m01;
        vf[c][1] &= m23;
      }
    }
    f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < KC; ++c) s = mfma_16x16x32(kf[c], qf[c], s);
    // lane holds S[token 4*quad + r][head h]
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      s[r] = (t_lane + r < kv_len) ? s[r] * sc : -INFINITY;
      mx = fmaxf(mx, s[r]);
    }
    mx = fmaxf(mx, shfl_xor(mx, 16));
    mx = fmaxf(mx, shfl_xor(mx, 32));
    const float m_new = fmaxf(m, mx);
    const float alpha = exp2f(m - m_new);
    float p[4], ps = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      p[r] = exp2f(s[r] - m_new);
      ps += p[r];
    }
    ps += shfl_xor(ps, 16);
    ps += shfl_xor(ps, 32);
    l = l * alpha + ps;
    m = m_new;
    // P = P_hi + P_lo with both parts bf16 (about 16 significant bits), so the
    // probabilities are not cut to bf16 precision before P V
    u32x2 pf, pl;
    pf[0] = pack_bf2(p[0], p[1]);
    pf[1] = pack_bf2(p[2], p[3]);
    pl[0] = pack_bf2(p[0] - bf2f(pf[0] & 0xffffu), p[1] - bf2f(pf[0] >> 16));
    pl[1] = pack_bf2(p[2] - bf2f(pf[1] & 0xffffu), p[3] - bf2f(pf[1] >> 16));
#pragma unroll
    for (int c = 0; c < VC; ++c) {
      o[c] *= alpha;
      o[c] = mfma_16x16x16(vf[c], pf, o[c]);  // lane holds O[head h][dim 16c + 4*quad + r]
      o[c] = mfma_16x16x16(vf[c], pl, o[c]);
    }
  };
  auto load = [&](u32x4 (&kf)[KC], u32x2 (&vf)[VC], int32_t tb) {
    const size_t blk = static_cast<size_t>(tb);
    const u32x4* kp = reinterpret_cast<const u32x4*>(kbase + blk * kv_stride) + lane;
    const u32x2* vp = reinterpret_cast<const u32x2*>(vbase + blk * kv_stride) + lane;
#pragma unroll
    for (int c = 0; c < KC; ++c) kf[c] = kp[c * 64];
#pragma unroll
    for (int c = 0; c < VC; ++c) vf[c] = vp[c * 64];
  };

  __syncthreads();  // sm.tbl
  // this wave's blocks: a contiguous range of the split, kept NB blocks ahead.
  // Loads past the range re-read its last block and the final round is
  // peeled, so the loop's loads are unconditional and stay in flight.
  const int per = (b_hi - b_lo + NW - 1) / NW;
  const int w_lo = min(b_hi - b_lo, w * per);
  const int cnt = min(b_hi - b_lo, w_lo + per) - w_lo;
  u32x4 kf[NB][KC];
  u32x2 vf[NB][VC];
  if (cnt > 0) {
#pragma unroll
    for (int i = 0; i < NB; ++i) load(kf[i], vf[i], sm.tbl[w_lo + min(i, cnt - 1)]);
  }
  // the first split starts from the group's shared-prefix partials: wave w
  // folds in partials w, w + NW, ... (their loads wait behind the K/V loads
  // just issued, whose latency they share)
  if (split == 0 && n_ps > 0 && h < G) {
    const size_t rh0 = static_cast<size_t>(row) * a.Hkv + hk;
    auto fold = [&](const f32x4 (&op)[VC], float2 ml) {
      const float M = fmaxf(m, ml.x);
      const float f0 = m == -INFINITY ? 0.f : exp2f(m - M);
      const float f1 = exp2f(ml.x - M);
      l = l * f0 + ml.y * f1;
#pragma unroll
      for (int c = 0; c < VC; ++c) o[c] = o[c] * f0 + op[c] * f1;
      m = M;
    };
    for (int sp = w; sp < n_ps; sp += (FOLD2 ? 2 : 1) * NW) {
      const bool two = FOLD2 && sp + NW < n_ps;
      const float* po0 = a.part_o + ((rh0 * a.split_stride + sp) * G + h) * D;
      const float* po1 = po0 + (two ? static_cast<size_t>(NW) * G * D : 0);
      const float2 ml0 = a.part_ml[(rh0 * a.split_stride + sp) * G + h];
      const float2 ml1 = a.part_ml[(rh0 * a.split_stride + sp + (two ? NW : 0)) * G + h];
      f32x4 op0[VC], op1[VC];
#pragma unroll
      for (int c = 0; c < VC; ++c) op0[c] = *reinterpret_cast<const f32x4*>(po0 + 16 * c + 4 * quad);
      if constexpr (FOLD2) {
#pragma unroll
        for (int c = 0; c < VC; ++c) op1[c] = *reinterpret_cast<const f32x4*>(po1 + 16 * c + 4 * quad);
      }
      fold(op0, ml0);
      if constexpr (FOLD2)
        if (two) fold(op1, ml1);
    }
  }
  if (cnt > 0) {
    int base = 0;
    for (; base + NB < cnt; base += NB) {
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        process(kf[i], vf[i], b_lo + w_lo + base + i);
        load(kf[i], vf[i], sm.tbl[w_lo + min(base + i + NB, cnt - 1)]);
      }
    }
#pragma unroll
    for (int i = 0; i < NB; ++i)
      if (base + i < cnt) process(kf[i], vf[i], b_lo + w_lo + base + i);
  }

  // ---- merge the waves of this workgroup
  if (lane < 16) {
    sm.m[w][lane] = m;
    sm.l[w][lane] = l;
  }
  if (w > 0) {
#pragma unroll
    for (int c = 0; c < VC; ++c) sm.o[w - 1][c][lane] = o[c];
  }
  __syncthreads();
  if (w == 0) {
    float M = sm.m[0][h];
#pragma unroll
    for (int w2 = 1; w2 < NW; ++w2) M = fmaxf(M, sm.m[w2][h]);
    const float f0 = exp2f(sm.m[0][h] - M);
    float L = sm.l[0][h] * f0;
#pragma unroll
    for (int c = 0; c < VC; ++c) o[c] *= f0;
    for (int w2 = 1; w2 < NW; ++w2) {
      const float mw = sm.m[w2][h];
      const float f = (mw == -INFINITY) ? 0.f : exp2f(mw - M);
      L += sm.l[w2][h] * f;
#pragma unroll
      for (int c = 0; c < VC; ++c) o[c] += sm.o[w2 - 1][c][lane] * f;
    }
    m = M;
    l = L;
  }

  if (n_splits == 1) {
    if (w == 0 && h < G) {
      const float inv = 1.f / l;
      const int col0 = (hk * G + h) * D;
#pragma unroll
      for (int c = 0; c < VC; ++c) {
        const int e = 16 * c + 4 * quad;
        const size_t i0 = frag_index(row, col0 + e, a.out_Rg);  // 4 consecutive dims, same 8-group
        u32x2 pk;
        pk[0] = pack_bf2(o[c][0] * inv, o[c][1] * inv);
        pk[1] = pack_bf2(o[c][2] * inv, o[c][3] * inv);
        if constexpr (WT) store_wt(a.out + i0, pk);
        else *reinterpret_cast<u32x2*>(a.out + i0) = pk;
      }
    }
    return;
  }

  // ---- several splits: publish this split's (m, l, O); the workgroup that
  // completes a (row, KV head) last merges all of them in split order.
  // Partials are written and read with agent-scope atomic accesses, which
  // bypass the non-coherent per-XCD L2 copies; a store is complete (visible
  // at agent scope) once the wave's memory counter has drained, and only
  // then is the arrival counted.  No workgroup waits for another.
  const size_t rh = static_cast<size_t>(row) * a.Hkv + hk;
  if (w == 0 && h < G) {
    float* po = a.part_o + ((rh * a.split_stride + n_ps + split) * G + h) * D;
#pragma unroll
    for (int c = 0; c < VC; ++c)
#pragma unroll
      for (int r = 0; r < 4; ++r) st_agent(po + 16 * c + 4 * quad + r, o[c][r]);
    if (quad == 0) {
      float* pm = reinterpret_cast<float*>(a.part_ml + (rh * a.split_stride + n_ps + split) * G + h);
      st_agent(pm, m);
      st_agent(pm + 1, l);
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    const int prev = __hip_atomic_fetch_add(a.counter + rh, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    sm.last = prev == n_splits - 1;
  }
  __syncthreads();
  if (!sm.last) return;

  // merge: O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s, in split order
  // (this row's own splits, which follow its group's prefix partials)
  constexpr int kC = 8;  // splits read with one round of independent loads
  const int n_all = n_splits;
  const float* pml = reinterpret_cast<const float*>(a.part_ml + (rh * a.split_stride + n_ps) * G);
  const float* pob = a.part_o + (rh * a.split_stride + n_ps) * G * D;
  for (int idx = tid; idx < G * D; idx += blockDim.x) {
    const int hh = idx / D, e = idx % D;
    float acc = 0.f, L = 0.f, M = -INFINITY;
    for (int s0 = 0; s0 < n_all; s0 += kC) {
      float mv[kC];
#pragma unroll
      for (int j = 0; j < kC; ++j)
        mv[j] = s0 + j < n_all ? ld_agent(pml + 2 * ((s0 + j) * G + hh)) : -INFINITY;
#pragma unroll
      for (int j = 0; j < kC; ++j) M = fmaxf(M, mv[j]);
    }
    for (int s0 = 0; s0 < n_all; s0 += kC) {
      float mv[kC], lv[kC], ov[kC];
#pragma unroll
      for (int j = 0; j < kC; ++j) {
        const bool ok = s0 + j < n_all;
        const int sj = s0 + j;
        mv[j] = ok ? ld_agent(pml + 2 * (sj * G + hh)) : -INFINITY;
        lv[j] = ok ? ld_agent(pml + 2 * (sj * G + hh) + 1) : 0.f;
        ov[j] = ok ? ld_agent(pob + (static_cast<size_t>(sj) * G + hh) * D + e) : 0.f;
      }
#pragma unroll
      for (int j = 0; j < kC; ++j) {
        if (s0 + j < n_all) {
          const float f = exp2f(mv[j] - M);
          L += lv[j] * f;
          acc += ov[j] * f;
        }
      }
    }
    const uint32_t ob = f2bf(acc * (1.f / L));
    uint16_t* dst = a.out + frag_index(row, (hk * G + hh) * D + e, a.out_Rg);
    if constexpr (WT) store_wt16(dst, ob);
    else *dst = static_cast<uint16_t>(ob);
  }
  // ready for the next pass (or the next layer of a persistent pass)
  if (threadIdx.x == 0) __hip_atomic_store(a.counter + rh, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace vsk
