// Internal declarations shared by the C ABI (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/vsk.h"
#include "alloc.hpp"

namespace vsk {

constexpr int kBlock = 16;     // tokens per KV block
constexpr size_t kAlign = 256;

inline size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }

// ---------------------------------------------------------------- packed weights
// Every matrix W[N][K] is stored as 1 KiB tiles: tile (nt, kt) covers rows
// 16nt..16nt+15 and columns 32kt..32kt+31 and sits at tile index nt*(K/32)+kt.
// Inside a tile, lane l (0..63) owns 16 bytes: row l%16, columns
// 32kt + 8*(l/16) .. +7 -- the A-operand order of the 16x16x32 bf16 MFMA.
//
// Row permutations applied while packing:
//  * QKV (q heads, then k heads, then v heads): inside every q and k head the
//    packed row 2j holds dim j and 2j+1 holds dim j+d/2, so the rotary pairs
//    of a head end up in one lane's accumulator registers.
//  * gate/up: packed row 4u+0,1 = gate rows 2u,2u+1; 4u+2,3 = up rows 2u,2u+1.
struct LayerOffsets {
  size_t attn_norm, mlp_norm, wqkv, wo, wgu, wd;
};

struct PackedLayout {
  size_t layer_bytes = 0;
  LayerOffsets l;          // offsets inside one layer record
  size_t head_base = 0;    // start of the global record
  size_t final_norm = 0, embed = 0, lm_head = 0, rope = 0;  // absolute offsets
  size_t total = 0;
};

PackedLayout packed_layout(const vsk_model_cfg& c);

// ---------------------------------------------------------------- activation frags
// Activations feeding a projection are bf16 X[R][K] stored in "frag" order:
// chunk (kt, g) = 1 KiB at ((kt*Rg + g) * 1024) bytes, Rg = ceil(R/16); lane l
// owns X[16g + l%16][32kt + 8*(l/16) .. +7] -- the B-operand order of the
// 16x16x32 MFMA.  Padding rows (R..16*Rg) are kept at zero.
__host__ __device__ inline size_t frag_index(int row, int k, int Rg) {
  const int kt = k >> 5, kk = k & 31;
  const int lane = (row & 15) + 16 * (kk >> 3);
  return ((static_cast<size_t>(kt) * Rg + (row >> 4)) * 64 + lane) * 8 + (kk & 7);
}

// ---------------------------------------------------------------- KV pool
// Pool = [L][2][n_blocks][n_kv_heads][block of 16 tokens x head_dim] bf16.
// K block: chunk c = dim/32 (1 KiB each): lane t + 16*((dim%32)/8), elem dim%8
//          (A-operand order of the 16x16x32 MFMA for S = K q).
// V block: chunk c = dim/16 (512 B each): lane dim%16 + 16*(t/4), elem t%4
//          (A-operand order of the 16x16x16 MFMA for O^T = V^T P^T).
__host__ __device__ inline int kv_k_index(int t, int e) {
  const int c = e >> 5, ee = e & 31;
  return ((c * 64) + t + 16 * (ee >> 3)) * 8 + (ee & 7);
}
__host__ __device__ inline int kv_v_index(int t, int e) {
  const int c = e >> 4;
  return ((c * 64) + (e & 15) + 16 * (t >> 2)) * 4 + (t & 3);
}

// ---------------------------------------------------------------- device batch
struct BatchDev {
  int32_t n_seqs = 0, n_rows = 0, max_blocks = 0, max_kv_len = 0, max_q_len = 0;
  const int32_t* block_table = nullptr;  // [n_seqs][max_blocks]
  const int32_t* kv_len = nullptr;
  const int32_t* cu_q = nullptr;
  const int32_t* row_seq = nullptr;
  const int32_t* pos = nullptr;
  const int32_t* slot = nullptr;
  // shared prefixes (decode passes): see BatchHost
  const int32_t* pfx_blocks = nullptr;
  const int32_t* pfx_splits = nullptr;
  const int32_t* pfx_items = nullptr;
  const int32_t* grp_rows = nullptr;
  const int32_t* grp_info = nullptr;
  const int32_t* pfx_tbl = nullptr;
  int32_t n_pfx_items = 0, max_pfx_splits = 0;
  // prefill rows: causal work items, and the rows left to the decode kernel
  const int32_t* pre_items = nullptr;
  const int32_t* dec_rows = nullptr;
  int32_t n_pre_items = 0, n_dec_rows = 0;
};

// ---------------------------------------------------------------- workspace
// Timing probes: events bound to one dispatch (hipExtLaunchKernel), which
// take that kernel's own start and end times; null for an ordinary launch.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};

struct WsLayout {
  int32_t max_rows = 0, max_seqs = 0, max_kv_len = 0, Rg = 0, max_splits = 0;
  size_t x, x_c, fa, fb, fc, q, att_o, att_ml, att_cnt, ssq, ssq_c, am_part, total;
  size_t ypart = 0;  // products of residual projections with K split over workgroups
  // routed layers (present when `routed`): Project-Only cohort frags of the
  // MLP input and of the SwiGLU product, both cohorts' down-projection
  // products, and Algorithm 1's maps per layer (run, proj, inv [L][rows],
  // counts [L][2])
  bool routed = false;
  size_t fb_po = 0, fc_po = 0, y_run = 0, y_po = 0, r_run = 0, r_proj = 0, r_inv = 0, r_cnt = 0;
  // persistent decode step (present when max_rows <= kStepMaxRows and the
  // model shape is covered): per-layer activations, sync flags, error word, epoch
  bool step = false;
  size_t s_x, s_ssq, s_q, s_o, s_a, s_n, s_am, s_flags, s_err, s_epoch;
};

// attention split: 16-token blocks per split-K work item (tunable, >= kAttnMinBps)
constexpr int kAttnMinBps = 8;
constexpr int kAttnMaxBps = 512;
inline int attn_splits(int kv_len, int bps) {
  const int nb = (kv_len + kBlock - 1) / kBlock;
  return (nb + bps - 1) / bps;
}
// Default split size (4-wave work items, two per compute unit).  With few
// (row, KV head) pairs long contexts are cut into 512-token splits to spread
// them over the compute units; once the pairs alone fill the chip,
// 1536-token splits still cut the longest contexts of a heavy-tailed batch
// (dispatched first, longest walk first) while most rows need no merge
// (measured: batch 16 at 512-1024 tokens; batch 128 at lognormal lengths,
// 96 and 128 blocks best, 64 and 160 or more slower).
inline int attn_auto_bps(int n_rows, int n_kv_heads) { return n_rows * n_kv_heads >= 256 ? 96 : 32; }

struct Handle {
  vsk_model_cfg cfg{};
  std::string err;
  // weights
  uint8_t* packed = nullptr;
  size_t packed_bytes = 0;
  PackedLayout pl;
  // kv
  uint16_t* pool = nullptr;
  int32_t n_blocks = 0;
  BlockAllocator alloc;
  bool alloc_ready = false;
  // batch
  BatchHost bh;
  bool batch_built = false;
  BatchDev bd;
  bool batch_uploaded = false;
  // metadata upload: two pinned host staging buffers used in turn, each with
  // an event recorded after the copy that reads it, so an upload only waits
  // when the copy issued two uploads earlier is still running
  struct Staging {
    void* host = nullptr;
    size_t cap = 0;
    hipEvent_t done = nullptr;
    bool pending = false;
  };
  Staging stage[2];
  int stage_next = 0;
  ~Handle();
  // tuning
  int attn_bps = 0;  // 0: attn_auto_bps
  int layers_run = 0;  // inspection: run only the first layers_run layers (0 = all)
  int exec_mode = 0;   // 0 automatic, 1 one kernel per operation, 2 persistent step kernel
  int gemm_shape = 0;  // projection launch shape for 4 or 8 row groups (0 default)
  int shared_prefix = 1;  // read shared prefixes once per group (decode passes)
  int pfx_target = 192;   // workgroups the shared-prefix work items of a pass aim for
  int resid_target = 0;   // residual projections: split-K workgroup target (0 default, -1 no split)
  int qkv_target = 0;     // QKV at 4..8 row groups: split-K workgroup target (0 default, -1 no split)
  int prefill_attn = 1;   // prefill rows through the causal multi-row kernel (0: one row per work item)
  int xcd_remap = 1;      // row-tiled projections: XCD-aware workgroup order (0: dispatch order)
  int row_tile = 0;       // row-tiled projections: 16-row groups per tile (0 auto; 6, 7, 8 or 11)
  int step_wgs = -1;   // workgroups of a persistent launch on this device (0: not runnable; -1: not queried)
  uint64_t* step_trace = nullptr;  // measurement: timestamp buffer of the persistent kernel
  size_t step_trace_cap = 0;       // its capacity in uint64
  // workspace
  uint8_t* ws = nullptr;
  size_t ws_bytes = 0;
  WsLayout wl;
  // routed mode (Algorithm 1): the routed layers are first_routed..n_layers-1,
  // each with a SwiGLU projector of width proj_ffn packed at `routed_w`
  // (per routed layer: [gate/up interleaved 2*proj_ffn x hidden | down
  // hidden x proj_ffn], each 256-byte aligned)
  uint8_t* routed_w = nullptr;
  int32_t first_routed = -1, proj_ffn = 0;
  size_t routed_layer_bytes = 0, routed_pgu = 0, routed_pd = 0;
  // timing probes per kernel class
  static constexpr int kProbeClasses = 6;
  std::vector<hipEvent_t> probe_b[kProbeClasses], probe_e[kProbeClasses];
  size_t probe_i[kProbeClasses] = {0};
  // counters
  int64_t counters[8] = {0};
};

// with_step: include the persistent step kernel's region when the capacity
// and the model shape allow it
WsLayout ws_layout(const vsk_model_cfg& c, int32_t max_rows, int32_t max_seqs, int32_t max_kv_len,
                   bool with_step = true, bool routed = false);


// ---------------------------------------------------------------- launchers
// Each returns hipSuccess or the launch error.
hipError_t launch_pack_matrix(const uint16_t* src, uint16_t* dst, int N, int K, int perm_kind, int head_dim,
                              int n_rope_rows, hipStream_t s);
hipError_t launch_copy_bf16(const uint16_t* src, uint16_t* dst, size_t n, hipStream_t s);
hipError_t launch_fill_zero(void* dst, size_t bytes, hipStream_t s);
hipError_t launch_kv_write(const Handle& h, int layer, const int32_t* slots, int n, const uint16_t* k,
                           const uint16_t* v, hipStream_t s);
hipError_t launch_kv_read(const Handle& h, int layer, const int32_t* slots, int n, uint16_t* k, uint16_t* v,
                          hipStream_t s);
hipError_t launch_argmax_logits(const void* logits, int dtype, int rows, int vocab, int32_t* ids, int32_t* no_value,
                                hipStream_t s);

struct PassArgs {
  const int32_t* ids;
  const int32_t* logit_rows;  // nullable = every row
  int32_t n_logit_rows;
  uint16_t* logits;
  int32_t* next_ids;
  uint8_t* ws;
  WsLayout wl;
  // routed pass (nullable): route tape of the routed layers, run [L_r][rows]
  // (1 RUN, 0 Project-Only) and weights w [L_r][rows]
  const uint8_t* tape_run = nullptr;
  const float* tape_w = nullptr;
};
hipError_t run_pass(Handle& h, const PassArgs& a, hipStream_t s);
// True when run_pass would take the persistent step kernel for this pass.
bool step_eligible(Handle& h, const PassArgs& a);

}  // namespace vsk
