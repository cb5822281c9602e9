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
  int max_splits;  // split stride of the partial buffers
  float* part_o;   // [R][Hkv][max_splits][G][hd]
  float2* part_ml; // [R][Hkv][max_splits][G]
  int* counter;    // [R][Hkv] arrivals of splits, zero between passes
  uint16_t* out;   // o frags (K = Nq)
  int out_Rg;
};

hipError_t launch_attn_decode(const AttnArgs& a, int n_rows, hipStream_t s);

}  // namespace vsk
