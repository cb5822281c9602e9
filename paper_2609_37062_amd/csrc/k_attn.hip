// Paged-attention decode over the block-table KV cache, split-K over context.
//
// For every row (one token at position p of its sequence) and KV head, the
// query heads of that KV head's group attend to keys 0..p read through the
// sequence's block table (paper, "Invariants": each layer reads its own
// cached K,V; Algorithm 1 keeps attention's launch shape).  A workgroup owns
// one (row, KV head, split) and its eight waves take the split's 16-token
// blocks in turn.  Per block a wave computes S = K q with
// v_mfma_f32_16x16x32_bf16 (16 tokens x up to 16 heads), an online softmax in
// the base-2 domain, and O^T += V^T P^T with v_mfma_f32_16x16x16_bf16, so the
// softmax row lives in the same lanes as the output it rescales.  The waves
// merge in LDS; splits write (m, l, O) partials that a second small kernel
// merges in split order.
// Decode attention reads about group-size flops per byte of KV, so it is
// bound by HBM, not by the matrix cores.
#include <cmath>

#include "attn.hpp"
#include "dev.hpp"

namespace vsk {

constexpr int kAttnWaves = 8;

template <int D>
__global__ __launch_bounds__(64 * kAttnWaves) void k_attn_decode(AttnArgs a) {
  constexpr int KC = D / 32;  // K chunks (1 KiB) per block
  constexpr int VC = D / 16;  // V chunks (512 B) per block
  __shared__ float s_m[kAttnWaves][16];
  __shared__ float s_l[kAttnWaves][16];
  __shared__ f32x4 s_o[kAttnWaves - 1][VC][64];

  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int row = blockIdx.z, hk = blockIdx.y, split = blockIdx.x;
  const int G = a.G;
  const int kv_len = a.pos[row] + 1;
  const int nb = (kv_len + kBlock - 1) / kBlock;
  const int n_splits = (nb + a.bps - 1) / a.bps;
  if (split >= n_splits) return;
  const int seq = a.row_seq[row];
  const int32_t* table = a.block_table + static_cast<size_t>(seq) * a.max_blocks;
  const int b_lo = split * a.bps;
  const int b_hi = min(nb, b_lo + a.bps);

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
  auto load = [&](u32x4 (&kf)[KC], u32x2 (&vf)[VC], int b) {
    const size_t blk = static_cast<size_t>(table[b]);
    const u32x4* kp = reinterpret_cast<const u32x4*>(kbase + blk * kv_stride) + lane;
    const u32x2* vp = reinterpret_cast<const u32x2*>(vbase + blk * kv_stride) + lane;
#pragma unroll
    for (int c = 0; c < KC; ++c) kf[c] = kp[c * 64];
#pragma unroll
    for (int c = 0; c < VC; ++c) vf[c] = vp[c * 64];
  };

  // this wave's blocks b_lo + w, + kAttnWaves, ...: two blocks in flight
  u32x4 kA[KC], kB[KC];
  u32x2 vA[VC], vB[VC];
  int b = b_lo + w;
  if (b < b_hi) load(kA, vA, b);
  for (; b < b_hi; b += 2 * kAttnWaves) {
    const int bn = b + kAttnWaves;
    if (bn < b_hi) load(kB, vB, bn);
    process(kA, vA, b);
    if (bn >= b_hi) break;
    if (bn + kAttnWaves < b_hi) load(kA, vA, bn + kAttnWaves);
    process(kB, vB, bn);
  }

  // ---- merge the waves of this workgroup
  if (lane < 16) {
    s_m[w][lane] = m;
    s_l[w][lane] = l;
  }
  if (w > 0) {
#pragma unroll
    for (int c = 0; c < VC; ++c) s_o[w - 1][c][lane] = o[c];
  }
  __syncthreads();
  if (w == 0) {
    float M = s_m[0][h];
#pragma unroll
    for (int w2 = 1; w2 < kAttnWaves; ++w2) M = fmaxf(M, s_m[w2][h]);
    const float f0 = exp2f(s_m[0][h] - M);
    float L = s_l[0][h] * f0;
#pragma unroll
    for (int c = 0; c < VC; ++c) o[c] *= f0;
    for (int w2 = 1; w2 < kAttnWaves; ++w2) {
      const float mw = s_m[w2][h];
      const float f = (mw == -INFINITY) ? 0.f : exp2f(mw - M);
      L += s_l[w2][h] * f;
#pragma unroll
      for (int c = 0; c < VC; ++c) o[c] += s_o[w2 - 1][c][lane] * f;
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
        uint2 pk;
        pk.x = pack_bf2(o[c][0] * inv, o[c][1] * inv);
        pk.y = pack_bf2(o[c][2] * inv, o[c][3] * inv);
        *reinterpret_cast<uint2*>(a.out + i0) = pk;
      }
    }
    return;
  }

  // ---- several splits: publish this split's (m, l, O); k_attn_combine merges them
  const size_t rh = static_cast<size_t>(row) * a.Hkv + hk;
  if (w == 0 && h < G) {
    float* po = a.part_o + ((rh * a.max_splits + split) * G + h) * D;
#pragma unroll
    for (int c = 0; c < VC; ++c)
      *reinterpret_cast<float4*>(po + 16 * c + 4 * quad) = make_float4(o[c][0], o[c][1], o[c][2], o[c][3]);
    if (quad == 0) a.part_ml[(rh * a.max_splits + split) * G + h] = make_float2(m, l);
  }
}

// Merge the split partials of rows with more than one split, in split order:
// O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s.  One workgroup per (KV head, row).
constexpr int kMaxSplits = 128;  // max_pos <= 16384 with at least 8 blocks per split
__global__ __launch_bounds__(256) void k_attn_combine(AttnArgs a) {
  __shared__ float s_f[kMaxSplits][16];  // per split and head: 2^(m_s - M)
  __shared__ float s_invL[16];
  const int hk = blockIdx.x, row = blockIdx.y;
  const int kv_len = a.pos[row] + 1;
  const int n_splits = (((kv_len + kBlock - 1) / kBlock) + a.bps - 1) / a.bps;
  if (n_splits <= 1) return;
  const int G = a.G, D = a.hd;
  const size_t rh = static_cast<size_t>(row) * a.Hkv + hk;
  const float2* ml = a.part_ml + rh * a.max_splits * G;
  if (threadIdx.x < G) {
    const int hh = threadIdx.x;
    float M = -INFINITY;
    for (int s = 0; s < n_splits; ++s) M = fmaxf(M, ml[s * G + hh].x);
    float L = 0.f;
    for (int s = 0; s < n_splits; ++s) {
      const float2 v = ml[s * G + hh];
      const float f = exp2f(v.x - M);
      s_f[s][hh] = f;
      L += v.y * f;
    }
    s_invL[hh] = 1.f / L;
  }
  __syncthreads();
  const float* po = a.part_o + rh * a.max_splits * G * D;
  for (int idx = threadIdx.x; idx < G * D; idx += blockDim.x) {
    const int hh = idx / D, e = idx % D;
    float acc = 0.f;
    int s = 0;
    for (; s + 4 <= n_splits; s += 4) {
      const float v0 = po[(static_cast<size_t>(s + 0) * G + hh) * D + e];
      const float v1 = po[(static_cast<size_t>(s + 1) * G + hh) * D + e];
      const float v2 = po[(static_cast<size_t>(s + 2) * G + hh) * D + e];
      const float v3 = po[(static_cast<size_t>(s + 3) * G + hh) * D + e];
      acc += v0 * s_f[s][hh];
      acc += v1 * s_f[s + 1][hh];
      acc += v2 * s_f[s + 2][hh];
      acc += v3 * s_f[s + 3][hh];
    }
    for (; s < n_splits; ++s) acc += po[(static_cast<size_t>(s) * G + hh) * D + e] * s_f[s][hh];
    a.out[frag_index(row, (hk * G + hh) * D + e, a.out_Rg)] = static_cast<uint16_t>(f2bf(acc * s_invL[hh]));
  }
}

hipError_t launch_attn_decode(const AttnArgs& a, int n_rows, hipStream_t s) {
  dim3 grid(a.max_splits, a.Hkv, n_rows);
  if (a.hd == 128) {
    hipLaunchKernelGGL(k_attn_decode<128>, grid, dim3(64 * kAttnWaves), 0, s, a);
  } else if (a.hd == 64) {
    hipLaunchKernelGGL(k_attn_decode<64>, grid, dim3(64 * kAttnWaves), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.max_splits <= 1) return e;
  hipLaunchKernelGGL(k_attn_combine, dim3(a.Hkv, n_rows), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace vsk
