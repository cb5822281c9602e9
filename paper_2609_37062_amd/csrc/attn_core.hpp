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
// block-table entries are staged in LDS first; each wave then walks its
// range two blocks (32 keys) at a time, the next pair's K and V loads issued
// while the current pair is processed.  Per pair a wave computes S = K q with
// v_mfma_f32_16x16x32_bf16 (two groups of 16 keys x up to 16 heads), an
// online softmax in the base-2 domain, and O^T += V^T P^T with
// v_mfma_f32_16x16x32_bf16 over the 32 keys, so the softmax row lives in the
// same lanes as the output it rescales.  The waves merge in LDS; with several
// splits the last workgroup to finish a (row, KV head) merges the splits'
// (m, l, O) partials in split order.  Decode attention reads about
// group-size flops per byte of KV; on this chip the matrix-core and softmax
// instructions per byte still set its pace (measured: the same kernel without
// them ran in less than half the time), hence 32-key steps.
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

// agent-scope (all XCDs) coherent loads of the split partials
__device__ __forceinline__ float ld_agent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Splits of a row: n_splits(kv_len) for the row's kv_len = pos + 1.
__device__ __forceinline__ int attn_row_splits(int kv_len, int bps) {
  const int nb = (kv_len + kBlock - 1) / kBlock;
  return (nb + bps - 1) / bps;
}

// ---- 32-key steps.  Two 16-token blocks, A (keys 0..15 of the step) and B
// (keys 16..31), are processed together, so that O^T += V^T P^T runs on
// v_mfma_f32_16x16x32_bf16 (32 keys per MFMA) instead of two
// v_mfma_f32_16x16x16_bf16, which take as many cycles each.  S = K q is taken
// in two MFMA groups whose 16 rows are the step's keys 8 (r / 4) + r % 4
// (group 0) and 8 (r / 4) + 4 + r % 4 (group 1): lane (column h, quarter q)
// then holds S of keys 8q .. 8q + 3 and 8q + 4 .. 8q + 7, exactly the eight
// probabilities P^T's operand asks of that lane, with no exchange between
// lanes.  The softmax's cross-lane max and sum and the rescale of O run once
// per 32 keys.
//
// K operand of group G: the block (0: A, 1: B) and the 16-byte index within
// each 1 KiB K chunk (stored in the 16 x 16 x 32 A-operand order of one block:
// piece key + 16 x dim-group) of the row this lane feeds.
__device__ __forceinline__ int pair_k_block(int lane) { return (lane & 15) >> 3; }
__device__ __forceinline__ int pair_k_index(int lane, int grp) {
  return 8 * ((lane >> 2) & 1) + 4 * grp + (lane & 3) + 16 * (lane >> 4);
}
// V^T operand: lane (dim i, quarter q) takes keys 8q .. 8q + 7, i.e. block
// q / 2, as two 8-byte pieces of each 512-byte V chunk (stored in the
// 16 x 16 x 16 A-operand order of one block): index below, and index + 16.
__device__ __forceinline__ int pair_v_block(int lane) { return lane >> 5; }
__device__ __forceinline__ int pair_v_index(int lane) { return (lane & 15) + 32 * ((lane >> 4) & 1); }

// The probabilities of a step as the B operand of P V, split into kPTerms
// bf16 terms whose sum is the float32 probability to about 8 kPTerms
// significant bits (each term is the bf16 rounding of what the previous
// ones left over); the products of the terms are accumulated in float32.
constexpr int kPTerms = 3;
struct PTerms {
  u32x4 t[kPTerms];
};

// One step over the keys at positions t0 .. t0 + 31, in two phases so that a
// caller streaming K and V through registers can reload K as soon as the
// scores are taken and V as soon as P V is issued.
// pair_scores: S = K q from kg[G][c] (the K operands of group G), the online
// softmax update of (m, l), and P as the bf16 terms pp (so the probabilities
// are not cut to bf16 precision before P V); alpha rescales O.  Keys at
// t >= t_end do not
// count; with MASK a key also needs t <= lim.  Base 2 (sc = log2(e) /
// sqrt(D)).  A column with no valid key yet keeps m = -inf and contributes
// nothing.
template <int D, bool MASK>
__device__ __forceinline__ void pair_scores(const u32x4 (&qf)[D / 32], const u32x4 (&kg)[2][D / 32], int t0,
                                            int t_end, int lim, float sc, float& m, float& l, PTerms& pp,
                                            float& alpha) {
  constexpr int KC = D / 32;
  const int tv = t0 + 8 * ((threadIdx.x & 63) >> 4);  // this lane's first key (of 8)
  f32x4 s0 = f32x4{0.f, 0.f, 0.f, 0.f}, s1 = s0;
#pragma unroll
  for (int c = 0; c < KC; ++c) s0 = mfma_16x16x32(kg[0][c], qf[c], s0);
#pragma unroll
  for (int c = 0; c < KC; ++c) s1 = mfma_16x16x32(kg[1][c], qf[c], s1);
  float mx = -INFINITY;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int ta = tv + r, tb = tv + 4 + r;
    bool va = ta < t_end, vb = tb < t_end;
    if constexpr (MASK) {
      va = va && ta <= lim;
      vb = vb && tb <= lim;
    }
    s0[r] = va ? s0[r] * sc : -INFINITY;
    s1[r] = vb ? s1[r] * sc : -INFINITY;
    mx = fmaxf(mx, fmaxf(s0[r], s1[r]));
  }
  mx = max_xor32(max_xor16(mx));
  const float m_new = fmaxf(m, mx);
  // v_exp_f32 directly: arguments are <= 0, and a probability below 2^-126
  // (flushed to 0) is negligible beside the maximum's 1; both results are
  // computed and selected, so there is no branch per exponential
  const bool none = m_new == -INFINITY;
  alpha = none ? 1.f : __builtin_amdgcn_exp2f(m - m_new);
  float p[8], ps = 0.f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    p[r] = none ? 0.f : __builtin_amdgcn_exp2f(s0[r] - m_new);
    p[4 + r] = none ? 0.f : __builtin_amdgcn_exp2f(s1[r] - m_new);
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) ps += p[j];
  ps = add_xor32(add_xor16(ps));
  l = l * alpha + ps;
  m = m_new;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float r0 = p[2 * j], r1 = p[2 * j + 1];
#pragma unroll
    for (int t = 0; t < kPTerms; ++t) {
      pp.t[t][j] = pack_bf2(r0, r1);
      r0 -= bf2f(pp.t[t][j] & 0xffffu);
      r1 -= bf2f(pp.t[t][j] >> 16);
    }
  }
}

// pair_pv: O = alpha O + V^T P^T from vt[c] (the V^T operands).  V rows of
// keys at t >= t_end are zeroed first: a slot past the end of a sequence may
// hold a NaN pattern, and a zero probability times NaN is NaN.
template <int D>
__device__ __forceinline__ void pair_pv(u32x4 (&vt)[D / 16], int t0, int t_end, const PTerms& pp, float alpha,
                                        f32x4 (&o)[D / 16]) {
  constexpr int VC = D / 16;
  const int tv = t0 + 8 * ((threadIdx.x & 63) >> 4);
  if (tv + 7 >= t_end) {
    uint32_t mk[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      mk[j] = (tv + 2 * j < t_end ? 0x0000ffffu : 0u) | (tv + 2 * j + 1 < t_end ? 0xffff0000u : 0u);
#pragma unroll
    for (int c = 0; c < VC; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j) vt[c][j] &= mk[j];
  }
#pragma unroll
  for (int c = 0; c < VC; ++c) {
    o[c] *= alpha;
    // lane holds O[column lane % 16][dim 16c + 4 (lane / 16) + r]
#pragma unroll
    for (int t = 0; t < kPTerms; ++t) o[c] = mfma_16x16x32(vt[c], pp.t[t], o[c]);
  }
}

// WT: the attention output is stored write-through (sc1), so that other
// workgroups of the same launch read it from memory, not from a stale L2.
// FOLD2: a wave loads two shared-prefix partials before folding either (one
// round trip per two; 186 instead of 167 registers at head_dim 128), for
// passes with more prefix partials per row than waves.
template <int D, bool WT, int NW, bool FOLD2 = false>
__device__ __forceinline__ void attn_unit(const AttnArgs& a, int row, int hk, int split, AttnLds<D, NW>& sm) {
  constexpr int KC = D / 32;  // K chunks (1 KiB) per block
  constexpr int VC = D / 16;  // V chunks (512 B) per block

  const int tid = opaque_tid();
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int G = a.G;
  // routed layer: a Project-Only row reads no KV and emits zero (its own K,V
  // were written by the projection like every row's); split 0 stores it
  if (a.run_mask != nullptr && a.run_mask[row] == 0) {
    const int hz = lane & 15, qz = lane >> 4;
    if (split == 0 && w == 0 && hz < G) {
      const int col0 = (hk * G + hz) * D;
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const size_t i0 = frag_index(row, col0 + 16 * c + 4 * qz, a.out_Rg);
        const u32x2 zero = u32x2{0u, 0u};
        if constexpr (WT) store_wt(a.out + i0, zero);
        else *reinterpret_cast<u32x2*>(a.out + i0) = zero;
      }
    }
    return;
  }
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

  // K and V operands of blocks 2p, 2p + 1 of this wave's range (a block past
  // the range: its last block again, whose keys the step then masks)
  auto pair_blocks = [&](int p, int cnt, int w_lo, size_t& bA, size_t& bB) {
    bA = static_cast<size_t>(sm.tbl[w_lo + min(2 * p, cnt - 1)]);
    bB = static_cast<size_t>(sm.tbl[w_lo + min(2 * p + 1, cnt - 1)]);
  };
  auto load_k = [&](u32x4 (&kg)[2][KC], int p, int cnt, int w_lo) {
    size_t bA, bB;
    pair_blocks(p, cnt, w_lo, bA, bB);
    const u32x4* kp = reinterpret_cast<const u32x4*>(kbase + (pair_k_block(lane) ? bB : bA) * kv_stride);
    const int k0 = pair_k_index(lane, 0), k1 = pair_k_index(lane, 1);
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      kg[0][c] = kp[c * 64 + k0];
      kg[1][c] = kp[c * 64 + k1];
    }
  };
  auto load_v = [&](u32x4 (&vt)[VC], int p, int cnt, int w_lo) {
    size_t bA, bB;
    pair_blocks(p, cnt, w_lo, bA, bB);
    const u32x2* vp =
        reinterpret_cast<const u32x2*>(vbase + (pair_v_block(lane) ? bB : bA) * kv_stride) + pair_v_index(lane);
#pragma unroll
    for (int c = 0; c < VC; ++c) {
      const u32x2 lo = vp[c * 64], hi = vp[c * 64 + 16];
      vt[c] = u32x4{lo[0], lo[1], hi[0], hi[1]};
    }
  };

  __syncthreads();  // sm.tbl
  // this wave's blocks: a contiguous range of the split, taken two at a time.
  // One pair's K and V live in registers: the next pair's K is loaded as soon
  // as the scores are taken and its V as soon as P V is issued, so a load is
  // always in flight.  Loads past the range re-read its last block, so the
  // loop's loads are unconditional.
  const int per = (b_hi - b_lo + NW - 1) / NW;
  const int w_lo = min(b_hi - b_lo, w * per);
  const int cnt = min(b_hi - b_lo, w_lo + per) - w_lo;
  const int n_pairs = (cnt + 1) / 2;
  const int t_first = kBlock * (b_lo + w_lo);                   // first key of the range
  const int t_end = min(kv_len, kBlock * (b_lo + w_lo + cnt));  // keys past it belong to others
  u32x4 kg[2][KC];
  u32x4 vt[VC], vt2[VC];  // V of the even and the odd pairs
  if (cnt > 0) {
    load_k(kg, 0, cnt, w_lo);
    load_v(vt, 0, cnt, w_lo);
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
  // Pair p + 1's K and V are both issued right after the scores of pair p
  // (its V into the other of two V buffers), so both have pair p's P V to
  // land in: the compiler waits for every outstanding load at the top of
  // the walk loop, so a V issued after P V would be waited for in full
  // there.  Two pairs per iteration keep the buffers compile-time; the
  // loop's loads are unconditional, the last one or two pairs are peeled.
  auto step = [&](u32x4 (&vc)[VC], u32x4 (&vn)[VC], int p, bool more) {
    const int t0 = t_first + 2 * kBlock * p;
    PTerms pp;
    float alpha;
    pair_scores<D, false>(qf, kg, t0, t_end, 0, sc, m, l, pp, alpha);
    if (more) {
      load_k(kg, p + 1, cnt, w_lo);
      load_v(vn, p + 1, cnt, w_lo);
    }
    pair_pv<D>(vc, t0, t_end, pp, alpha, o);
  };
  int p = 0;
  for (; p + 2 < n_pairs; p += 2) {
    step(vt, vt2, p, true);
    step(vt2, vt, p + 1, true);
  }
  if (p < n_pairs) {
    step(vt, vt2, p, p + 1 < n_pairs);
    if (p + 1 < n_pairs) step(vt2, vt, p + 1, false);
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
  // Partials are written with write-through stores (sc1, 16 bytes per lane)
  // and read with agent-scope loads, which bypass the non-coherent per-XCD
  // L2 copies; a store is complete (visible at agent scope) once the wave's
  // memory counter has drained, and only then is the arrival counted.  No
  // workgroup waits for another.
  const size_t rh = static_cast<size_t>(row) * a.Hkv + hk;
  if (w == 0 && h < G) {
    float* po = a.part_o + ((rh * a.split_stride + n_ps + split) * G + h) * D;
#pragma unroll
    for (int c = 0; c < VC; ++c) store_wt(po + 16 * c + 4 * quad, __builtin_bit_cast(u32x4, o[c]));
    if (quad == 0)
      store_wt(a.part_ml + (rh * a.split_stride + n_ps + split) * G + h,
               u32x2{__float_as_uint(m), __float_as_uint(l)});
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
  // (this row's own splits, which follow its group's prefix partials).  A
  // thread takes outputs idx = tid, tid + blockDim.x, ... two at a time, and
  // issues every load of a round of up to kC splits (both outputs' m, l and
  // O) before the first is used: one memory round trip per round.
  constexpr int kC = 8;  // splits per round
  const int n_all = n_splits;
  const float* pml = reinterpret_cast<const float*>(a.part_ml + (rh * a.split_stride + n_ps) * G);
  const float* pob = a.part_o + (rh * a.split_stride + n_ps) * G * D;
  for (int i0 = tid; i0 < G * D; i0 += 2 * blockDim.x) {
    const int i1 = i0 + blockDim.x;
    const bool two = i1 < G * D;
    const int hh[2] = {i0 / D, two ? i1 / D : i0 / D};
    const int ee[2] = {i0 % D, two ? i1 % D : i0 % D};
    float acc[2] = {0.f, 0.f}, L[2] = {0.f, 0.f}, M[2] = {-INFINITY, -INFINITY};
    for (int s0 = 0; s0 < n_all; s0 += kC) {
      float mv[2][kC], lv[2][kC], ov[2][kC];
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int j = 0; j < kC; ++j) {
          const int sj = min(s0 + j, n_all - 1);
          mv[u][j] = ld_agent(pml + 2 * (sj * G + hh[u]));
          lv[u][j] = ld_agent(pml + 2 * (sj * G + hh[u]) + 1);
          ov[u][j] = ld_agent(pob + (static_cast<size_t>(sj) * G + hh[u]) * D + ee[u]);
        }
      // rescale what earlier rounds summed to this round's running maximum
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        float Mn = M[u];
#pragma unroll
        for (int j = 0; j < kC; ++j)
          if (s0 + j < n_all) Mn = fmaxf(Mn, mv[u][j]);
        const float f0 = M[u] == -INFINITY ? 0.f : exp2f(M[u] - Mn);
        L[u] *= f0;
        acc[u] *= f0;
#pragma unroll
        for (int j = 0; j < kC; ++j) {
          if (s0 + j < n_all) {
            const float f = exp2f(mv[u][j] - Mn);
            L[u] += lv[u][j] * f;
            acc[u] += ov[u][j] * f;
          }
        }
        M[u] = Mn;
      }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      if (u == 1 && !two) break;
      const uint32_t ob = f2bf(acc[u] * (1.f / L[u]));
      uint16_t* dst = a.out + frag_index(row, (hk * G + hh[u]) * D + ee[u], a.out_Rg);
      if constexpr (WT) store_wt16(dst, ob);
      else *dst = static_cast<uint16_t>(ob);
    }
  }
  // ready for the next pass (or the next layer of a persistent pass)
  if (threadIdx.x == 0) __hip_atomic_store(a.counter + rh, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace vsk
