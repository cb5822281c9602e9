// Paged-attention decode over the block-table KV cache, split-K over context:
// one workgroup per (split, KV head, row); the work item itself is
// attn_unit (attn_core.hpp).
//
// Shared prefixes.  When several sequences of a decode pass hold the same
// leading blocks (a common prompt prefix stored once in the paged cache),
// k_attn_prefix reads each such block once per work item for up to 64
// (row, query head) pairs of the group instead of once per sequence: the 16
// columns of each MFMA tile are 16 such pairs, four tiles per workgroup, each
// walked by two waves over alternate block pairs.  Each work item leaves, per
// pair, the (max, sum, unnormalised output) of its run of prefix blocks as
// one split partial; the decode kernel then reads only the blocks after the
// prefix, its waves starting their online softmax from the prefix partials.
// Softmax over the union of key sets is exactly the merge of the per-set
// partials, so this only changes the summation order.
#include <hip/hip_ext.h>

#include "attn_core.hpp"

namespace vsk {

constexpr int kPfxTiles = kPfxCols / 16;  // 16-column tiles of a shared-prefix work item
constexpr int kPfxHalves = 2;              // waves per tile (each walks half of the block pairs)
constexpr int kPfxWaves = kPfxTiles * kPfxHalves;
constexpr int kPreTiles = kPreCols / 16;   // 16-column tiles (one wave each) of a prefill work item

template <int D, bool FOLD2>
__global__ __launch_bounds__(64 * kAttnWaves) void k_attn_decode(AttnArgs a) {
  __shared__ AttnLds<D, kAttnWaves> sm;
  attn_unit<D, false, kAttnWaves, FOLD2>(
      a, a.rows != nullptr ? a.rows[blockIdx.z] : static_cast<int>(blockIdx.z), blockIdx.y, blockIdx.x, sm);
}

template <int D, bool FOLD2>
static void launch_decode_k(const AttnArgs& a, dim3 grid, hipStream_t s, const LaunchEvents& ev) {
  if (ev.start != nullptr || ev.stop != nullptr)  // events bound to this dispatch
    hipExtLaunchKernelGGL((k_attn_decode<D, FOLD2>), grid, dim3(64 * kAttnWaves), 0u, s, ev.start, ev.stop, 0u, a);
  else
    hipLaunchKernelGGL((k_attn_decode<D, FOLD2>), grid, dim3(64 * kAttnWaves), 0, s, a);
}

template <int D>
static void launch_decode_d(const AttnArgs& a, dim3 grid, bool fold2, hipStream_t s, const LaunchEvents& ev) {
  if (fold2) launch_decode_k<D, true>(a, grid, s, ev);
  else launch_decode_k<D, false>(a, grid, s, ev);
}

hipError_t launch_attn_decode(const AttnArgs& a, int n_rows, int grid_splits, int max_pfx_splits, hipStream_t s,
                              LaunchEvents ev) {
  if (grid_splits < 1 || grid_splits > a.max_splits) return hipErrorInvalidValue;
  dim3 grid(grid_splits, a.Hkv, n_rows);
  const bool fold2 = a.pfx_splits != nullptr && max_pfx_splits > kAttnWaves;
  if (a.hd == 128) launch_decode_d<128>(a, grid, fold2, s, ev);
  else if (a.hd == 64) launch_decode_d<64>(a, grid, fold2, s, ev);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

// Walk of a workgroup over a run of 16-token blocks: NCT x NH compute waves,
// wave w taking query-column tile w % NCT (16 columns, each lane's column
// h = lane % 16) and half w / NCT of the run's block pairs, and one loader
// wave (wave NCT x NH).  A compute wave takes 32-key steps (pair_scores and
// pair_pv); with NH halves, half hh takes pairs hh, hh + NH, ..., and the
// halves of a tile are merged in LDS at the end, so a tile's run is walked
// in 1 / NH of the steps.  The block ids are tbl[0..cnt) (in LDS), block
// tbl[i] holding key positions 16 (b0 + i) ..; every wave of the workgroup
// calls this with the same cnt.  The loader brings each step's NH pairs of
// K and V (2 x D / 16 chunks of 1 KiB per block) once for the workgroup
// straight into a ring of kWalkSlots LDS slots, kWalkLead steps ahead; one
// workgroup barrier per step hands the landed pairs to the compute waves and
// the slot they read in the previous step back to the loader.  (The compute
// waves issue no global-to-LDS loads themselves: the compiler would then
// drain every outstanding one before each LDS read.)  A compute wave
// computes only the pairs holding its tile's first my_cnt blocks.  Keys at
// t >= t_end do not count (their V is zeroed: stale slots may hold NaN
// patterns); with MASK a key also needs t <= lim.  Returns true on the waves
// that hold a tile's result (half 0).
constexpr int kWalkLead = 2;
constexpr int kWalkSlots = kWalkLead + 1;
template <int D, int NH>
struct WalkLds {
  // per slot, pair and block: D / 32 chunks of K, then D / 32 of V
  u32x4 ring[kWalkSlots][NH][2][D / 16][64];
};

template <int D, int NCT, int NH, bool MASK>
__device__ __forceinline__ bool mq_walk(const u32x4 (&qf)[D / 32], const uint16_t* kbase, const uint16_t* vbase,
                                        size_t kv_stride, const int32_t* tbl, int cnt, int my_cnt, int b0, int lim,
                                        int t_end, float sc, float& m, float& l, f32x4 (&o)[D / 16],
                                        WalkLds<D, NH>& sm) {
  constexpr int KC = D / 32;   // K chunks (1 KiB) per block
  constexpr int VC = D / 16;   // V chunks (512 B) per block
  constexpr int NCH = 2 * KC;  // 1 KiB chunks per block
  constexpr int NW = NCT * NH;  // compute waves
  static_assert((kWalkLead - 1) * NH * 2 * NCH <= 63, "outstanding loads beyond the wait counter");
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int ct = w % NCT, hh = w / NCT;
  const int n_pairs = (cnt + 1) / 2;
  const int n_steps = (n_pairs + NH - 1) / NH;
  if (cnt > 0) {
    if (w == NW) {
      // step st (past the run: its last block again, into a slot nobody
      // reads or a pair whose keys are masked) -> slot st % kWalkSlots
      auto issue = [&](int st) {
#pragma unroll
        for (int hp = 0; hp < NH; ++hp)
#pragma unroll
          for (int hb = 0; hb < 2; ++hb) {
            const size_t blk = static_cast<size_t>(tbl[min(2 * (st * NH + hp) + hb, cnt - 1)]);
            // block B's K pieces land swizzled (piece j at slot j ^ 4): a
            // compute wave's 16 lanes of one LDS read phase then take 16
            // distinct 16-byte bank groups (8 from each block) instead of
            // the same 8 twice
            const u32x4* kp = reinterpret_cast<const u32x4*>(kbase + blk * kv_stride) + (lane ^ (hb ? 4 : 0));
            const u32x4* vp = reinterpret_cast<const u32x4*>(vbase + blk * kv_stride) + lane;
#pragma unroll
            for (int g = 0; g < NCH; ++g)
              lds_load16((g < KC ? kp : vp) + (g % KC) * 64, &sm.ring[st % kWalkSlots][hp][hb][g][0]);
          }
      };
#pragma unroll
      for (int st = 0; st < kWalkLead; ++st) issue(st);
      for (int st = 0; st < n_steps; ++st) {
        // step st has landed once at most the loads of the kWalkLead - 1
        // steps after it are outstanding; the barrier then publishes it and
        // frees the slot of step st - 1 for step st + kWalkLead
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"((kWalkLead - 1) * NH * 2 * NCH) : "memory");
        barrier_no_fence();
        issue(st + kWalkLead);
      }
      // the loads past the run must land before the workgroup ends or the
      // ring is reused
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    } else {
      const int my_pairs = (my_cnt + 1) / 2;
      const int kb = pair_k_block(lane), k0 = pair_k_index(lane, 0), k1 = pair_k_index(lane, 1);
      const int ksw = kb ? 4 : 0;  // block B's K pieces are stored swizzled (see the loader)
      const int vb = pair_v_block(lane), vi = pair_v_index(lane);
      for (int st = 0; st < n_steps; ++st) {
        barrier_after_lds_reads();
        const int p = st * NH + hh;
        if (p < my_pairs) {
          const u32x4* kp = &sm.ring[st % kWalkSlots][hh][kb][0][0];
          const u32x2* vp = reinterpret_cast<const u32x2*>(&sm.ring[st % kWalkSlots][hh][vb][KC][0]) + vi;
          u32x4 kg[2][KC];
          u32x4 vt[VC];
#pragma unroll
          for (int c = 0; c < KC; ++c) {
            kg[0][c] = kp[c * 64 + (k0 ^ ksw)];
            kg[1][c] = kp[c * 64 + (k1 ^ ksw)];
          }
#pragma unroll
          for (int c = 0; c < VC; ++c) {
            const u32x2 lo = vp[c * 64], hi = vp[c * 64 + 16];
            vt[c] = u32x4{lo[0], lo[1], hi[0], hi[1]};
          }
          const int t0 = kBlock * (b0 + 2 * p);
          PTerms pp;
          float alpha;
          pair_scores<D, MASK>(qf, kg, t0, t_end, lim, sc, m, l, pp, alpha);
          pair_pv<D>(vt, t0, t_end, pp, alpha, o);
        }
      }
    }
  }
  if constexpr (NH > 1) {
    // merge the halves of each tile in a fixed order: halves 1.. hand their
    // (m, l, O) over through the ring's space once every wave is done with it
    f32x4* so = reinterpret_cast<f32x4*>(&sm.ring[0][0][0][0][0]);  // [NH - 1][NCT][VC][64]
    float* sml = reinterpret_cast<float*>(so + (NH - 1) * NCT * VC * 64);  // [NH - 1][NCT][2][16]
    __syncthreads();
    if (w < NW && hh > 0) {
#pragma unroll
      for (int c = 0; c < VC; ++c) so[(((hh - 1) * NCT + ct) * VC + c) * 64 + lane] = o[c];
      if (lane < 16) {
        sml[(((hh - 1) * NCT + ct) * 2 + 0) * 16 + lane] = m;
        sml[(((hh - 1) * NCT + ct) * 2 + 1) * 16 + lane] = l;
      }
    }
    __syncthreads();
    if (w < NCT) {
      const int h = lane & 15;
#pragma unroll
      for (int h2 = 1; h2 < NH; ++h2) {
        const float m2 = sml[(((h2 - 1) * NCT + ct) * 2 + 0) * 16 + h];
        const float l2 = sml[(((h2 - 1) * NCT + ct) * 2 + 1) * 16 + h];
        const float M = fmaxf(m, m2);
        const float f0 = m == -INFINITY ? 0.f : exp2f(m - M);
        const float f1 = m2 == -INFINITY ? 0.f : exp2f(m2 - M);
        l = l * f0 + l2 * f1;
#pragma unroll
        for (int c = 0; c < VC; ++c) o[c] = o[c] * f0 + so[(((h2 - 1) * NCT + ct) * VC + c) * 64 + lane] * f1;
        m = M;
      }
    }
  }
  return w < NCT;
}

template <int D>
__global__ __launch_bounds__(64 * (kPfxWaves + 1)) void k_attn_prefix(AttnPrefixArgs a) {
  constexpr int KC = D / 32;
  constexpr int VC = D / 16;
  __shared__ int32_t tbl[kMaxPfxBps];
  __shared__ WalkLds<D, kPfxHalves> ring;

  const int hk = blockIdx.y;
  const int32_t* it = a.items + static_cast<size_t>(blockIdx.x) * 5;
  const int grp = it[0], col0 = it[1], b_lo = it[2], b_hi = it[3], split = it[4];
  const int roff = a.grp_info[4 * grp], n_cols = a.grp_info[4 * grp + 1] * a.G;
  const int32_t* ptbl = a.pfx_tbl + a.grp_info[4 * grp + 3];
  const int G = a.G;
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int h = lane & 15, quad = lane >> 4;
  for (int i = tid; i < b_hi - b_lo; i += blockDim.x) tbl[i] = ptbl[b_lo + i];

  // this lane's column: pair (group row c / G, query head c % G); both
  // halves of a tile hold its columns (wave kPfxWaves only loads blocks)
  const int ct = w % kPfxTiles;
  const int c = col0 + 16 * ct + h;
  const bool cvalid = w < kPfxWaves && c < n_cols;
  const int row = cvalid ? a.grp_rows[roff + c / G] : 0;
  const int qh = cvalid ? c % G : 0;
  u32x4 qf[KC];
  {
    const uint16_t* qrow = a.q + static_cast<size_t>(row) * a.Nq + static_cast<size_t>(hk * G + qh) * D;
#pragma unroll
    for (int k = 0; k < KC; ++k)
      qf[k] = cvalid ? *reinterpret_cast<const u32x4*>(qrow + 32 * k + 8 * quad) : u32x4{0u, 0u, 0u, 0u};
  }
  float m = -INFINITY, l = 0.f;
  f32x4 o[VC];
#pragma unroll
  for (int k = 0; k < VC; ++k) o[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  const size_t kv_stride = static_cast<size_t>(a.Hkv) * kBlock * D;
  const uint16_t* kbase = a.pool + (static_cast<size_t>(a.layer) * 2 + 0) * a.n_blocks * kv_stride +
                          static_cast<size_t>(hk) * kBlock * D;
  const uint16_t* vbase = a.pool + (static_cast<size_t>(a.layer) * 2 + 1) * a.n_blocks * kv_stride +
                          static_cast<size_t>(hk) * kBlock * D;

  __syncthreads();  // tbl
  // every wave walks all blocks of the item (all keys lie inside the prefix);
  // a wave with no column in the group only loads its share of the blocks
  const int cnt = b_hi - b_lo;
  const int my_cnt = w < kPfxWaves && col0 + 16 * ct < n_cols ? cnt : 0;
  const bool owner = mq_walk<D, kPfxTiles, kPfxHalves, false>(qf, kbase, vbase, kv_stride, tbl, cnt, my_cnt, b_lo, 0,
                                                              kBlock * b_hi, a.scale_log2, m, l, o, ring);

  // this item's partial of each valid column, as split `split` of its row;
  // the decode kernel, launched after this one, reads them
  if (owner && cvalid) {
    const size_t rh = static_cast<size_t>(row) * a.Hkv + hk;
    float* po = a.part_o + ((rh * a.split_stride + split) * G + qh) * D;
#pragma unroll
    for (int k = 0; k < VC; ++k)
      *reinterpret_cast<float4*>(po + 16 * k + 4 * quad) = make_float4(o[k][0], o[k][1], o[k][2], o[k][3]);
    if (quad == 0) a.part_ml[(rh * a.split_stride + split) * G + qh] = make_float2(m, l);
  }
}

// Causal attention of a prefill chunk: one work item per (run of a
// sequence's consecutive new rows, KV head), its columns the (row, query
// head) pairs of the run, 16 per wave.  Row r at position p attends keys
// 0..p of its sequence; its own chunk's keys were written by the QKV
// projection before this kernel runs (every layer writes its own KV).  A
// wave walks the blocks up to its last row's position; each lane masks the
// keys past its own row.  The output is normalised and stored as the O
// projection's input frags.
template <int D>
__global__ __launch_bounds__(64 * (kPreTiles + 1)) void k_attn_prefill(AttnPrefillArgs a) {
  constexpr int KC = D / 32;
  constexpr int VC = D / 16;
  __shared__ int32_t tbl[kMaxPrefillBlocks];
  __shared__ WalkLds<D, 1> ring;

  // one-dimensional grid, an item's KV heads consecutive (items come
  // longest walk first)
  const int hk = blockIdx.x % a.Hkv;
  const int32_t* it = a.items + static_cast<size_t>(blockIdx.x / a.Hkv) * 3;
  const int seq = it[0], row0 = it[1], n_rows = it[2];
  const int G = a.G;
  const int n_cols = n_rows * G;
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int h = lane & 15, quad = lane >> 4;
  const int kv_end = a.kv_len[seq];
  const int p_last = a.pos[row0 + n_rows - 1];
  const int nb = p_last / kBlock + 1;  // blocks any row of the item reads
  const int32_t* table = a.block_table + static_cast<size_t>(seq) * a.max_blocks;
  for (int i = tid; i < nb; i += blockDim.x) tbl[i] = table[i];

  const int c = 16 * w + h;
  const bool cvalid = w < kPreTiles && c < n_cols;  // (wave kPreTiles only loads blocks)
  const int row = row0 + (cvalid ? c / G : 0);
  const int qh = cvalid ? c % G : 0;
  const int lim = cvalid ? a.pos[row] : -1;
  u32x4 qf[KC];
  {
    const uint16_t* qrow = a.q + static_cast<size_t>(row) * a.Nq + static_cast<size_t>(hk * G + qh) * D;
#pragma unroll
    for (int k = 0; k < KC; ++k)
      qf[k] = cvalid ? *reinterpret_cast<const u32x4*>(qrow + 32 * k + 8 * quad) : u32x4{0u, 0u, 0u, 0u};
  }
  float m = -INFINITY, l = 0.f;
  f32x4 o[VC];
#pragma unroll
  for (int k = 0; k < VC; ++k) o[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  const size_t kv_stride = static_cast<size_t>(a.Hkv) * kBlock * D;
  const uint16_t* kbase = a.pool + (static_cast<size_t>(a.layer) * 2 + 0) * a.n_blocks * kv_stride +
                          static_cast<size_t>(hk) * kBlock * D;
  const uint16_t* vbase = a.pool + (static_cast<size_t>(a.layer) * 2 + 1) * a.n_blocks * kv_stride +
                          static_cast<size_t>(hk) * kBlock * D;

  __syncthreads();  // tbl
  // the workgroup walks the blocks of its last row; each wave computes up to
  // its own last column's block (none if it has no column)
  const int c_last = min(16 * w + 15, n_cols - 1);
  const int w_blocks = w < kPreTiles && 16 * w < n_cols ? a.pos[row0 + c_last / G] / kBlock + 1 : 0;
  mq_walk<D, kPreTiles, 1, true>(qf, kbase, vbase, kv_stride, tbl, nb, w_blocks, 0, lim, min(kv_end, kBlock * nb),
                                 a.scale_log2, m, l, o, ring);
  if (!(w < kPreTiles && 16 * w < n_cols)) return;

  if (cvalid) {
    // a Project-Only row of a routed layer emits zero
    const bool po = a.run_mask != nullptr && a.run_mask[row] == 0;
    const float inv = 1.f / l;
    const int col0 = (hk * G + qh) * D;
#pragma unroll
    for (int k = 0; k < VC; ++k) {
      const int e = 16 * k + 4 * quad;
      u32x2 pk = u32x2{0u, 0u};
      if (!po) {
        pk[0] = pack_bf2(o[k][0] * inv, o[k][1] * inv);
        pk[1] = pack_bf2(o[k][2] * inv, o[k][3] * inv);
      }
      *reinterpret_cast<u32x2*>(a.out + frag_index(row, col0 + e, a.out_Rg)) = pk;
    }
  }
}

hipError_t launch_attn_prefill(const AttnPrefillArgs& a, int n_items, int head_dim, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  dim3 grid(n_items * a.Hkv);
  if (head_dim == 128) {
    hipLaunchKernelGGL((k_attn_prefill<128>), grid, dim3(64 * (kPreTiles + 1)), 0, s, a);
  } else if (head_dim == 64) {
    hipLaunchKernelGGL((k_attn_prefill<64>), grid, dim3(64 * (kPreTiles + 1)), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attn_prefix(const AttnPrefixArgs& a, int n_items, int head_dim, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  dim3 grid(n_items, a.Hkv);
  if (head_dim == 128) {
    hipLaunchKernelGGL((k_attn_prefix<128>), grid, dim3(64 * (kPfxWaves + 1)), 0, s, a);
  } else if (head_dim == 64) {
    hipLaunchKernelGGL((k_attn_prefix<64>), grid, dim3(64 * (kPfxWaves + 1)), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace vsk
