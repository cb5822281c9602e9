// Paged-attention decode interface (see k_attn.hip).
#pragma once

#include "internal.hpp"

namespace vsk {

struct AttnArgs {
  const uint16_t* q;  // [R][Nq] bf16
  const uint16_t* pool;
  int layer, n_blocks, Hkv, hd, G, Nq;
  const int32_t* block_table;  // [n_seqs][max_blocks]
  int max_blocks;
  const int32_t* row_seq;
  const int32_t* pos;
  float scale_log2;  // log2(e) / sqrt(hd)
  int bps;         // 16-token blocks per split (multiple of 8)
  int max_splits;  // split work items per (row, KV head) launched
  int split_stride;  // partials per (row, KV head) in the partial buffers
  float* part_o;   // [R][Hkv][split_stride][G][hd]
  float2* part_ml; // [R][Hkv][split_stride][G]
  int* counter;    // [R][Hkv] arrivals of splits, zero between passes
  uint16_t* out;   // o frags (K = Nq)
  int out_Rg;
  // shared prefixes (nullable): a row whose group prefix has P blocks reads
  // only blocks P.. itself; its group's prefix partials sit at split indices
  // 0..pfx_splits[row]-1 and its first split starts from them
  const int32_t* pfx_blocks;  // [R]
  const int32_t* pfx_splits;  // [R]
  const int32_t* rows;        // nullable: the rows of the launch (grid z indexes it), else all rows
  // routed layer (nullable): per row 1 RUN, 0 Project-Only; a Project-Only
  // row reads no KV and its attention output is zero (Algorithm 1)
  const uint8_t* run_mask;
};

// Causal attention of prefill rows (see k_attn_prefill).
constexpr int kMaxPrefillBlocks = 512;  // key blocks a prefill work item can stage (8192 positions)
struct AttnPrefillArgs {
  const uint16_t* q;  // [R][Nq] bf16
  const uint16_t* pool;
  int layer, n_blocks, Hkv, G, Nq;
  const int32_t* block_table;  // [n_seqs][max_blocks]
  int max_blocks;
  const int32_t* kv_len;       // [n_seqs]
  const int32_t* pos;          // [R]
  const int32_t* items;        // [n_items][3]: sequence, first row, rows
  float scale_log2;
  uint16_t* out;  // o frags (K = Nq)
  int out_Rg;
  const uint8_t* run_mask;  // routed layer (nullable): as in AttnArgs
};

// Shared-prefix attention: each work item reads a run of a group's prefix
// blocks once for up to kPfxCols (row, query head) columns of the group.
struct AttnPrefixArgs {
  const uint16_t* q;  // [R][Nq] bf16
  const uint16_t* pool;
  int layer, n_blocks, Hkv, G, Nq;
  const int32_t* block_table;  // [n_seqs][max_blocks]
  int max_blocks;
  const int32_t* row_seq;
  const int32_t* items;     // [n_items][5]: group, first column, first block, end block, split
  const int32_t* grp_rows;  // rows of every group
  const int32_t* grp_info;  // [n_groups][4]: first entry in grp_rows, rows, prefix blocks, first entry in pfx_tbl
  const int32_t* pfx_tbl;   // every group's prefix block ids
  float scale_log2;
  int split_stride;
  float* part_o;
  float2* part_ml;
};

// grid_splits: split work items launched per (row, KV head), at least the
// most any row has after its shared prefix and at most a.max_splits.
// max_pfx_splits: the most prefix partials any row folds in.
hipError_t launch_attn_decode(const AttnArgs& a, int n_rows, int grid_splits, int max_pfx_splits, hipStream_t s,
                              LaunchEvents ev = {});
hipError_t launch_attn_prefix(const AttnPrefixArgs& a, int n_items, int head_dim, hipStream_t s);
hipError_t launch_attn_prefill(const AttnPrefillArgs& a, int n_items, int head_dim, hipStream_t s);

}  // namespace vsk
