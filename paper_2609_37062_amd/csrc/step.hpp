// Persistent decode-step kernel interface (see k_step.hip).
#pragma once

#include "internal.hpp"

namespace vsk {

constexpr int kStepMaxRows = 16;   // rows of a persistent pass: one 16-row MFMA group
constexpr int kStepMaxWgs = 1024;  // workgroups of a persistent launch
constexpr int kSyncCounters = 8;   // arrival counters per synchronisation point
constexpr int kFlagWords = 16;     // 64 bytes between two counters

// Synchronisation points of a persistent pass over n layers: after the
// embedding, after each of a layer's seven phases (attention norm, QKV,
// attention, O, MLP norm, gate/up, down), after the final norm and after
// the lm_head.
constexpr int kLayerSyncs = 7;
inline int step_syncs(int n_layers) { return kLayerSyncs * n_layers + 3; }

struct StepArgs {
  // model
  int n_run;     // layers to run
  int n_layers;  // layers of the model (synchronisation points are numbered for all of them)
  int H, Nq, Nkv, F, V, hd, G, Hkv;
  float eps;
  // packed weights
  const uint8_t* P;
  size_t layer_bytes;
  LayerOffsets lo;
  const uint16_t* embed;       // [V][H]
  const uint32_t __attribute__((ext_vector_type(4)))* lm_head;
  const uint16_t* final_gain;  // [H]
  const float2* rope;          // [max_pos][hd/2]
  // KV pool and batch
  uint16_t* pool;
  int n_blocks;
  int R;
  const int32_t* ids;
  const int32_t* pos;
  const int32_t* slot;
  const int32_t* row_seq;
  const int32_t* block_table;
  int max_blocks;
  float scale_log2;
  int bps, max_splits;
  float* part_o;
  float2* part_ml;
  int* att_cnt;
  // per-layer activation buffers: each address is written once and read
  // after a synchronisation point within one launch
  float* xs;       // [2L+1][R][H] residual after the embedding and after each half layer
  double* ssq;     // [2L+1][H/16][R] per-16-column sums of x^2 (buffer 0: one part per row)
  uint16_t* qs;    // [L][R][Nq] rotated q
  uint16_t* os;    // [L] attention output frags (16 rows, Nq wide)
  uint16_t* as;    // [L] SwiGLU output frags (16 rows, F wide)
  uint16_t* ns;    // [2L+1] normalised projection-input frags (16 rows, H wide), one per residual buffer
  float* am_val;   // [V/16][R] lm_head argmax partials
  int* am_idx;
  unsigned* flags;      // [syncs][kSyncCounters][kFlagWords] arrival counters
  unsigned* err;        // epoch of a pass whose synchronisation timed out (0: none)
  unsigned* epoch_ctr;  // epoch of the last completed pass
  uint64_t* trace;      // nullable: per point and workgroup, arrival and release times
  // outputs
  float* x_out;         // final residual [R][H] (inspection)
  uint16_t* logits;     // [R][V]
  int32_t* next_ids;    // nullable
};

// Shapes the persistent kernel covers: every projection's K a multiple of
// 256 with at least 8 K steps per wave, hidden at most 4096 (at most 256
// sum-of-squares partials per row), head_dim 64 or 128.
bool step_shape_ok(const vsk_model_cfg& c);
// LDS bytes of one persistent workgroup for this model.
size_t step_lds_bytes(const vsk_model_cfg& c);
// Co-resident workgroups per CU at that LDS size (0: the kernel cannot run).
int step_occupancy(const vsk_model_cfg& c);
hipError_t launch_step(const StepArgs& a, int n_wgs, size_t lds_bytes, hipStream_t s);

}  // namespace vsk
