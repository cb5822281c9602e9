/*
 * vsk.h -- C ABI of the MI355X (gfx950) batched decode step.
 *
 * One forward pass of a Llama-style GQA decoder over the rows of a batch:
 * paged-attention decode over a block-table KV cache, bf16 weight-streaming
 * projections with a SwiGLU MLP, fused RMSNorm and rotary positions, and a
 * greedy argmax.  It is the paper's dense mode, which takes every layer for
 * every row (Section 3, "Design and Implementation", Vocabulary paragraph).
 * Each row of a pass carries one token through the layers: the next token of
 * its sequence in a decode pass, one prompt token in a prefill chunk.
 *
 * Conventions
 *  - Every function returns an int status (VSK_OK or a negative VSK_E_*).
 *    On error nothing is launched and no state changes; vsk_last_error()
 *    holds a message.  No exceptions cross this boundary.
 *  - "dev" pointers are device (HBM) pointers, "host" pointers are host
 *    memory.  The library never allocates or frees device memory: every
 *    device buffer (weights, packed weights, KV pool, batch metadata,
 *    workspace, outputs) belongs to the caller and must outlive its use.
 *    Host arrays are copied, never retained.  (The library's own host
 *    memory includes two pinned staging buffers for vsk_batch_upload.)
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Device work is enqueued asynchronously on it.  The calls that wait for
 *    the device are: vsk_weights_pack_head (setup; it waits for its rotary
 *    table copy), vsk_device_status (by definition), and vsk_batch_upload
 *    only when the staging buffer it takes is still being read by the copy
 *    it issued two uploads earlier.  Nothing else synchronises.
 *  - bf16 tensors are IEEE bfloat16 bit patterns (uint16), row-major unless
 *    stated otherwise.  Matrices are [out][in].
 *  - A handle is not thread-safe.  Device faults surface at the caller's
 *    next synchronisation (and as VSK_E_HIP from a later call).
 */
#ifndef VSK_H
#define VSK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  VSK_OK = 0,
  VSK_E_ARG = -1,          /* bad argument, shape or size */
  VSK_E_NOMEM = -2,        /* KV pool has too few free blocks */
  VSK_E_RANGE = -3,        /* block id, slot or position out of range */
  VSK_E_SHARED_WRITE = -4, /* a new position falls in a block shared by several sequences */
  VSK_E_STATE = -5,        /* call out of order (unknown/duplicate sequence, nothing bound) */
  VSK_E_HIP = -6,          /* the HIP runtime reported an error */
  VSK_E_UNSUPPORTED = -7   /* shape the library has no kernel for */
};

/* Model shape.  block_size must be 16; head_dim 64 or 128; n_q_heads a
 * multiple of n_kv_heads with at most 16 query heads per KV head; hidden,
 * n_q_heads*head_dim and ffn multiples of 64; vocab a multiple of 16.
 * max_pos bounds positions (rotary table length). */
typedef struct vsk_model_cfg {
  int32_t n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn, vocab;
  int32_t block_size, max_pos;
  float rope_theta, rms_eps;
} vsk_model_cfg;

typedef struct vsk_handle vsk_handle;

const char* vsk_status_str(int status);
const char* vsk_last_error(const vsk_handle* h);

/* Validate cfg and create a handle (host memory only; touches no device). */
int vsk_create(const vsk_model_cfg* cfg, vsk_handle** out);
int vsk_destroy(vsk_handle* h);

/* ----------------------------------------------------------------- weights
 * The projections stream every weight byte once per pass; below the ridge
 * point decode is bound by that weight bandwidth (paper, appendix "The
 * Switching Thresholds from the Roofline", decode rule).  The library
 * repacks each [out][in] matrix once into 1 KiB tiles laid out as the matrix
 * cores consume them, so a pass reads each tile with one coalesced 16-byte
 * load per lane. */
typedef struct vsk_layer_weights {
  const void* attn_norm; /* dev bf16 [hidden] */
  const void* wq;        /* dev bf16 [n_q_heads*head_dim][hidden] */
  const void* wk;        /* dev bf16 [n_kv_heads*head_dim][hidden] */
  const void* wv;        /* dev bf16 [n_kv_heads*head_dim][hidden] */
  const void* wo;        /* dev bf16 [hidden][n_q_heads*head_dim] */
  const void* mlp_norm;  /* dev bf16 [hidden] */
  const void* w_gate;    /* dev bf16 [ffn][hidden] */
  const void* w_up;      /* dev bf16 [ffn][hidden] */
  const void* w_down;    /* dev bf16 [hidden][ffn] */
} vsk_layer_weights;

/* Bytes of the packed weight buffer (all layers, embedding, lm_head, norms,
 * rotary table). */
size_t vsk_packed_weight_bytes(const vsk_model_cfg* cfg);
/* Bind a caller-owned device buffer of at least vsk_packed_weight_bytes(). */
int vsk_weights_bind(vsk_handle* h, void* packed_dev, size_t bytes);
/* Repack one layer from logical [out][in] bf16 (source may be freed after
 * the stream passes this point).  Not part of the timed pass. */
int vsk_weights_pack_layer(vsk_handle* h, int32_t layer, const vsk_layer_weights* w, void* stream);
/* Repack embedding [vocab][hidden], lm_head [vocab][hidden] (untied),
 * final norm gain [hidden]; also writes the rotary cos/sin table. */
int vsk_weights_pack_head(vsk_handle* h, const void* embed_dev, const void* lm_head_dev,
                          const void* final_norm_dev, void* stream);

/* ----------------------------------------------------------------- KV cache
 * Paged KV cache (paper, "Invariants for Correct Mixed-Depth Execution":
 * position t of layer l holds that layer's own K and V, Invariant 1; every
 * row-to-memory map is rebuilt from the current row set, Invariant 2).
 * The pool holds n_blocks blocks of 16 tokens for every layer, K and V.
 * Its internal layout is private to the library; use vsk_kv_write /
 * vsk_kv_read to move logical [n][n_kv_heads][head_dim] bf16 values.
 * Position p of a sequence lives at slot table[p/16]*16 + p%16. */
size_t vsk_kv_pool_bytes(const vsk_model_cfg* cfg, int32_t n_blocks);
/* Bind a pool of n_blocks blocks.  pool_dev may be NULL, in which case only
 * the host allocator exists (device calls that need the pool return
 * VSK_E_STATE).  Resets the allocator: every block free, no sequences. */
int vsk_kv_init(vsk_handle* h, void* pool_dev, int32_t n_blocks);

int vsk_seq_create(vsk_handle* h, int64_t seq);
/* Drop the sequence; blocks whose reference count reaches 0 become free. */
int vsk_seq_release(vsk_handle* h, int64_t seq);
/* Install a caller-chosen block table (host int32[n]) holding ctx_len
 * resident tokens; each listed block gains a reference.  The same block may
 * appear in several sequences' tables (a shared prefix).  Requires an empty
 * sequence, distinct in-range ids and n*16 >= ctx_len. */
int vsk_seq_set_blocks(vsk_handle* h, int64_t seq, const int32_t* blocks_host, int32_t n,
                       int32_t ctx_len);
/* dst (empty) shares the first n_tokens (a multiple of 16, <= src length)
 * of src's blocks. */
int vsk_seq_share_prefix(vsk_handle* h, int64_t dst, int64_t src, int32_t n_tokens);
/* Append n_new positions to seq.  A position that starts a block beyond the
 * table takes the lowest-numbered free block.  Writing into a block with more
 * than one reference is VSK_E_SHARED_WRITE (no copy-on-write); too few free
 * blocks is VSK_E_NOMEM.  All or nothing.  slots_host (nullable, int32[n_new])
 * receives the new positions' slots. */
int vsk_kv_reserve(vsk_handle* h, int64_t seq, int32_t n_new, int32_t* slots_host);
/* Length and block table of seq: *len, *n_blocks, and up to cap ids. */
int vsk_seq_info(const vsk_handle* h, int64_t seq, int32_t* len, int32_t* n_blocks,
                 int32_t* blocks_host, int32_t cap);
int vsk_kv_free_blocks(const vsk_handle* h, int32_t* n_free);
/* Scatter logical k, v (dev bf16 [n][n_kv_heads][head_dim]) of one layer to
 * the given slots (dev int32[n]) / gather them back.  Setup and inspection. */
int vsk_kv_write(vsk_handle* h, int32_t layer, const int32_t* slots_dev, int32_t n,
                 const void* k_dev, const void* v_dev, void* stream);
int vsk_kv_read(vsk_handle* h, int32_t layer, const int32_t* slots_dev, int32_t n,
                void* k_dev, void* v_dev, void* stream);

/* ----------------------------------------------------------------- batch
 * Per-pass metadata, rebuilt from the current row set every pass
 * (Invariant 2).  For sequences seqs[0..n) with q_lens new rows each (the
 * rows are the last q_len resident positions, already reserved):
 *   block_table [n][max_blocks] int32 (unused entries -1)
 *   kv_len [n], cu_q [n+1], and per row r: row_seq[r], pos[r], slot[r].
 * Rows are numbered sequence by sequence.  vsk_batch_build validates and
 * keeps the host copy in the handle; vsk_batch_host_* reads it back. */
int vsk_batch_build(vsk_handle* h, const int64_t* seqs_host, const int32_t* q_lens_host,
                    int32_t n_seqs);
int vsk_batch_shape(const vsk_handle* h, int32_t* n_seqs, int32_t* n_rows, int32_t* max_blocks);
int vsk_batch_host_copy(const vsk_handle* h, int32_t* block_table, int32_t* kv_len, int32_t* cu_q,
                        int32_t* row_seq, int32_t* pos, int32_t* slot);
/* Shared prefixes of the built batch (decode passes only; paper, "Invariants
 * for Correct Mixed-Depth Execution": the page mappings are rebuilt per pass).
 * Sequences whose block tables start with the same blocks form a group when
 * at least two share at least 4 full blocks before their current tokens; the
 * group's prefix is the longest such run.  The pass then reads each prefix
 * block once per group instead of once per sequence (unless tuning key 4
 * turns it off).  pfx_blocks_host (nullable) int32[n_rows]: prefix blocks of
 * each row's group, 0 for a row in no group; n_groups (nullable). */
int vsk_batch_prefix_info(const vsk_handle* h, int32_t* pfx_blocks_host, int32_t* n_groups);
/* Device bytes needed by vsk_batch_upload for the current batch. */
size_t vsk_batch_device_bytes(const vsk_handle* h);
/* Copy the metadata into caller device memory (H2D on stream) and make it
 * the batch of the following passes.  The buffer must stay valid and
 * unmodified while those passes run. */
int vsk_batch_upload(vsk_handle* h, void* meta_dev, size_t bytes, void* stream);

/* ----------------------------------------------------------------- passes
 * Workspace: caller-owned device scratch sized for a capacity (max rows,
 * sequences and resident length of any pass that will use it).
 * vsk_workspace_init binds it to the handle and clears it on `stream`
 * (cross-workgroup arrival counters start at zero and every pass leaves them
 * at zero again).  Passes must then be given the bound buffer and fit its
 * capacity.  One workspace must not serve two passes that run concurrently. */
size_t vsk_workspace_bytes(const vsk_handle* h, int32_t max_rows, int32_t max_seqs,
                           int32_t max_kv_len);
int vsk_workspace_init(vsk_handle* h, void* ws_dev, size_t bytes, int32_t max_rows,
                       int32_t max_seqs, int32_t max_kv_len, void* stream);

/* One decode step over the uploaded batch (every q_len must be 1), the
 * dense-mode decode pass (Section 3, "Design and Implementation": dense mode
 * runs every layer for every row; Section 3.2, Invariant 1: every layer
 * writes its own K,V for every row; greedy decoding as in the paper's
 * measurements, Section 2 and appendix "Natural Stopping and the Output
 * Lengths").  Below the ridge point it is bound by streaming the weights
 * once (appendix "The Switching Thresholds from the Roofline", decode rule).
 * The batch metadata must have been uploaded; the workspace must be the one
 * bound by vsk_workspace_init and large enough for the batch (else
 * VSK_E_ARG / VSK_E_STATE before any launch).
 * ids_dev int32[n_rows] input tokens; writes every layer's K,V of every row
 * at its slot; logits_dev bf16 [n_rows][vocab]; next_ids_dev (nullable)
 * int32[n_rows] = lowest index of the maximum fp32 logit (greedy).
 * Replaying the same batch and ids rewrites the same slots with the same
 * bytes, so the step is idempotent. */
int vsk_decode_step(vsk_handle* h, const int32_t* ids_dev, void* logits_dev, int32_t* next_ids_dev,
                    void* ws_dev, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * decode step as vsk_decode_step, computing the same values with the same
 * kernels, but with its workspace taken from a fixed device array inside
 * the library (VSK_SCRATCH_BYTES per GPU, held from library load until the
 * process ends) instead of a caller's buffer.  It allocates and frees
 * nothing.  The batch must fit: a batch whose workspace would exceed
 * VSK_SCRATCH_BYTES (many rows with long contexts) is rejected with
 * VSK_E_ARG before any launch.  The array belongs to the device current at
 * the call (the stream must be on it) and keeps the last call's contents;
 * every call on a GPU shares it, so calls that overlap on one GPU (several
 * streams, threads or handles) race.  vsk_residual_copy reads the bound
 * workspace, not this array. */
#define VSK_SCRATCH_BYTES (64u * 1024u * 1024u)
int vsk_decode_step_scratch(vsk_handle* h, const int32_t* ids_dev, void* logits_dev, int32_t* next_ids_dev,
                            void* stream);

/* One ragged pass over the uploaded batch (any q_lens: chunked prefill rows
 * and decode rows together).  The paper's prefill passes carry one row per
 * prompt token (Section 3.1, Prefill paragraph) and are compute-bound
 * (Section 2); the engine it builds on runs chunked prefill beside decode
 * (appendix "The Switching Thresholds from the Roofline", prefill floor).  Prefill row at position p attends to keys
 * 0..p of its sequence; all of a layer's new K,V are written before that
 * layer's attention reads them.  Logits (bf16 [n_logit_rows][vocab]) and
 * next ids are produced only for the rows listed in logit_rows_dev
 * (int32[n_logit_rows]). */
int vsk_prefill_chunk(vsk_handle* h, const int32_t* ids_dev, const int32_t* logit_rows_dev,
                      int32_t n_logit_rows, void* logits_dev, int32_t* next_ids_dev,
                      void* ws_dev, size_t ws_bytes, void* stream);

/* Greedy sampling (the decoding the paper measures with, Section 2 and
 * appendix "Natural Stopping and the Output Lengths") over given logits: logits_dev
 * row-major [rows][vocab] of dtype 0 = bf16 or 1 = fp32; ids_dev int32[rows]
 * receives, per row, the lowest index of the maximum value.  NaN never wins;
 * a row with no non-NaN value gives 0 and is flagged in no_value_dev
 * (nullable int32[rows]: 1 for such a row, else 0); a row of -inf gives 0
 * (unflagged: -inf is a value).  rows >= 1, vocab >= 1 (any size), every
 * pointer device memory owned by the caller.  Uses no workspace beyond its
 * arguments.  VSK_E_ARG on a null logits or ids pointer, a non-positive
 * size or an unknown dtype. */
int vsk_argmax_sample(const void* logits_dev, int32_t dtype, int32_t rows, int32_t vocab,
                      int32_t* ids_dev, int32_t* no_value_dev, void* stream);

/* ----------------------------------------------------------------- routed mode
 * One routed layer per Algorithm 1 (Section 3.1, "Route-Guided Cohort
 * Execution"; appendix "Route-Guided Cohort Execution at the Kernel Level").
 * The routed layers are first_routed..n_layers-1 (the paper's skipper routes
 * the last 16 of 32).  Each has a projector: a SwiGLU block of width proj_ffn
 * (p_gate, p_up [proj_ffn][hidden], p_down [hidden][proj_ffn]) that a
 * Project-Only row runs instead of the MLP.
 *
 * A routed pass takes a route tape (device memory, caller-owned): run
 * uint8 [n_routed][n_rows] (1 RUN, 0 Project-Only) and w float
 * [n_routed][n_rows].  In a routed layer every row writes its own K,V
 * (Invariant 1); a Project-Only row reads no KV and its attention output is
 * zero (the attention launch keeps its shape); then, with X the layer's
 * normalised MLP input, a RUN row adds w * MLP(X) and a Project-Only row
 * (1 - w) * projector(X) to the residual.  The device builds the cohort maps
 * and counts from the tape on every pass (Invariant 2); each cohort's GEMMs
 * are launched for the whole batch and every tile at or beyond the cohort's
 * count exits at once, so a cohort with no rows reads no weights.  A RUN row
 * with w = 1 computes what the dense pass computes.  Layers before
 * first_routed run dense.  The persistent step kernel (tuning key 2 = 2)
 * has no routed mode (VSK_E_UNSUPPORTED). */
size_t vsk_routed_weight_bytes(const vsk_model_cfg* cfg, int32_t first_routed, int32_t proj_ffn);
/* Bind the projector weights' packed buffer (device, caller-owned, at least
 * vsk_routed_weight_bytes; 256-byte aligned).  first_routed in
 * [0, n_layers); proj_ffn a multiple of 64 in [64, ffn].  The workspace must
 * then be sized (vsk_workspace_bytes) and initialised again: a routed
 * workspace holds the Project-Only cohort's operands, both cohorts'
 * products and the maps. */
int vsk_routed_bind(vsk_handle* h, int32_t first_routed, int32_t proj_ffn, void* packed_dev, size_t bytes);
/* Repack one routed layer's projector from logical [out][in] bf16. */
int vsk_routed_pack_layer(vsk_handle* h, int32_t layer, const void* p_gate_dev, const void* p_up_dev,
                          const void* p_down_dev, void* stream);
/* vsk_decode_step / vsk_prefill_chunk in routed mode (arguments as there, plus
 * the route tape run_dev, w_dev described above). */
int vsk_decode_step_routed(vsk_handle* h, const int32_t* ids_dev, const uint8_t* run_dev, const float* w_dev,
                           void* logits_dev, int32_t* next_ids_dev, void* ws_dev, size_t ws_bytes, void* stream);
int vsk_prefill_chunk_routed(vsk_handle* h, const int32_t* ids_dev, const uint8_t* run_dev, const float* w_dev,
                             const int32_t* logit_rows_dev, int32_t n_logit_rows, void* logits_dev,
                             int32_t* next_ids_dev, void* ws_dev, size_t ws_bytes, void* stream);
/* Inspection: copy the maps the last routed pass built (device pointers,
 * each nullable): run_dev and proj_dev int32 [n_routed][n_rows] (the rows of
 * each cohort in row order, first n_r / n_p entries valid), inv_dev int32
 * [n_routed][n_rows] (each row's position in its cohort), cnt_dev int32
 * [n_routed][2] (n_r, n_p). */
int vsk_route_maps_read(vsk_handle* h, int32_t* run_dev, int32_t* proj_dev, int32_t* inv_dev, int32_t* cnt_dev,
                        void* stream);

/* ----------------------------------------------------------------- mode switch
 * Profitability-aware mode switching (Section 3.3; appendix "The Switching
 * Thresholds from the Roofline", decode rule and served thresholds).  Host
 * pure functions: no handle, no device, no state beyond their arguments.
 *
 * Routed mode pays a fixed cost tau per step; in decode below the ridge point
 * a Project-Only row saves only its attention read of the layer's KV, b bytes
 * per resident token.  With a fraction s of the routed decisions projecting
 * over L_r routed layers, routing pays when the resident tokens V exceed
 *   V* = tau_eff * BW / (s * L_r * b),  tau_eff = tau * L_r / tau_layers
 * (tau is measured once over tau_layers routed layers and reused as a
 * per-routed-layer coefficient).  Thresholds: exit = V*, enter =
 * enter_factor * V* (1.25 in the paper), each rounded to the nearest
 * multiple of round_tokens (10000 reproduces the printed thresholds; 0
 * rounds to the nearest token). */
typedef struct vsk_switch_params {
  double tau_s;                    /* fixed per-step cost of routed mode, seconds (> 0) */
  int32_t tau_layers;              /* routed layers tau was measured over (>= 1) */
  double bw_bytes_per_s;           /* device memory bandwidth, bytes/s (> 0) */
  double skip;                     /* s in (0, 1]: fraction of decisions projecting */
  int32_t routed_layers;           /* L_r (>= 1) */
  double kv_bytes_per_token_layer; /* b (> 0): K and V bytes of one token at one layer */
  double enter_factor;             /* >= 1 */
  double round_tokens;             /* >= 0 */
} vsk_switch_params;

typedef struct vsk_switch_band {
  double v_star;        /* the crossover V*, tokens (unrounded) */
  int64_t exit_tokens;  /* routing turns off at V <= exit_tokens */
  int64_t enter_tokens; /* routing turns on at V >= enter_tokens */
} vsk_switch_band;

/* Thresholds of the decode rule.  VSK_E_ARG on a parameter out of range. */
int vsk_switch_thresholds(const vsk_switch_params* p, vsk_switch_band* out);
/* One observation of the resident tokens V: the switching state (0 dense,
 * 1 routing) moves to 1 at V >= enter, to 0 at V <= exit, and is kept in
 * between.  *promote (nullable) = 1 exactly when the state went from 0 to 1:
 * that crossing promotes the requests already decoding in dense mode. */
int vsk_switch_step(const vsk_switch_band* t, int32_t routing_in, int64_t resident_tokens,
                    int32_t* routing_out, int32_t* promote);
/* Decode mode of one request after an observation: mode_in -1 (the request
 * starts decoding now: it takes the current state `routing`), 0 dense (it
 * becomes routed if `promote`), 1 routed (it stays routed: one-way). */
int vsk_switch_decode_mode(int32_t mode_in, int32_t routing, int32_t promote, int32_t* mode_out);
/* Prefill mode, fixed at admission: routed (1) iff the batch's prompt tokens
 * reach floor_tokens (1536 in the paper) and the estimated Project-Only
 * share exceeds share_min (0.35 in the paper). */
int vsk_switch_prefill(int64_t prompt_tokens, double po_share, int64_t floor_tokens, double share_min,
                       int32_t* routed);

/* Measurement: read `bytes` (a multiple of 16, 16-byte aligned device
 * memory) once with a plain streaming kernel of `workgroups` workgroups of
 * 256 threads, writing one uint32 per workgroup to out_dev: timed around, it
 * gives the device's achievable stream-read bandwidth, the ceiling beside
 * the 8 TB/s HBM peak. */
int vsk_stream_read(const void* src_dev, size_t bytes, uint32_t* out_dev, int32_t workgroups, void* stream);

/* Timing probes (measurement only).  While set, the first n_pairs launches
 * of kernel class `which` in the following passes are each launched with
 * hipExtLaunchKernel bound to (begin_events[i], end_events[i]), in launch
 * order: the events take that kernel's own start and end times on the pass
 * stream (hipEventElapsedTime then gives its execution time, without the
 * dispatch gap before it).  Classes: 0 gate/up projection, 1 down
 * projection, 2 QKV projection, 3 O projection, 4 decode attention, 5
 * lm_head projection.  Events are caller-created hipEvent_t handles (with
 * timing); n_pairs = 0 clears the probe.  Do not set probes while a pass is
 * being captured into a graph. */
int vsk_set_probe(vsk_handle* h, int32_t which, void* const* begin_events,
                  void* const* end_events, int32_t n_pairs);

/* Launch-shape tuning (the analogue of a device-tuned tile table).  Results
 * do not depend on it beyond floating-point summation order.
 * key 0: attention 16-token blocks per split-K work item (multiple of 8 in
 *        8..512), or 0 (the default) for automatic: 32 when fewer than 256
 *        (row, KV head) pairs are in the pass, else 96; with 128..255 pairs
 *        whose walks are within 20% of each other, one split per pair (the
 *        longest walk rounded up to a multiple of 8 blocks).
 * key 1: inspection only -- run just the first `value` layers before the
 *        final norm and lm_head (0 = all layers), for layer-local checks.
 * key 2: execution path.  0 (default) and 1: one kernel per operation.
 *        2: the whole pass as one persistent kernel (one workgroup per
 *        compute unit, grid synchronisation between the phases of a layer,
 *        the next projection's weight stream started before each wait); it
 *        covers decode passes of at most 16 rows (workspace sized for at most
 *        16 rows) whose every projection K is a multiple of 256 and at least
 *        2048, with hidden at most 4096, and returns VSK_E_UNSUPPORTED for
 *        other passes.  Both paths compute the same values.
 * key 3: launch shape of the per-operation projections for 17..128 rows
 *        (and longer row-tiled passes).  0 (default): with one row tile the
 *        activation chunks are staged in LDS by a ninth wave and shared by
 *        eight weight-streaming waves for QKV (K split over workgroups in
 *        the residual projections' staging, key 7; unsplit, two 16-column
 *        tiles per workgroup), gate/up (four; eight, two per wave, for 65
 *        rows or more) and lm_head (sixteen, two per wave, no K split in
 *        the workgroup), residual projections taking the four-tile (17..64
 *        rows) or eight-tile (65..128 rows) staging with K split over
 *        workgroups (key 5); passes of more than 128 rows
 *        take the staging with the eight waves side by side (16 tiles, 8
 *        for QKV).  1 one column of K-split waves, one tile, every
 *        projection; 2 the same with two tiles; 3 the 2 x 2 grid everywhere;
 *        4 staging with four tiles (two for QKV) everywhere, residual
 *        projections with K split over workgroups; 5 for 65 rows or more
 *        (QKV aside) staging with eight tiles, everything else shape 3; 6 the
 *        default's staging for every projection but the residual ones,
 *        whatever the row tiling.
 * key 4: shared prefixes of a decode pass (vsk_batch_prefix_info): 1 (the
 *        default) reads each group's prefix blocks once for the group, 0 reads
 *        them once per sequence.
 * key 5: residual projections (O, down) of passes of at most 128 rows: the
 *        workgroup count their K split aims for (1..4096); 0 (the default):
 *        192 workgroups in the activation-staged layout at 17..64 rows, 384
 *        at 65..128, 192 for the down projection at 1..16 rows (two tiles
 *        per workgroup), no split for O at 1..16 rows (measured no faster);
 *        -1: no split.  Split products are added to the residual in
 *        split order by the RMSNorm that follows.  Passes of more than 128
 *        rows whose residual projections have at most 128 workgroups (N
 *        groups x row tiles) split K into as many splits as keep them within
 *        256, unless the key is -1.
 * key 6: rows of a sequence with several new rows (a prefill chunk): 1 (the
 *        default) one causal work item per run of up to 128 (row, query
 *        head) pairs reading each key block once for all of them; 0 one
 *        work item per row, as for decode rows.
 * key 7: the QKV projection of passes of 17..128 rows: the workgroup count
 *        its K split aims for (1..4096); 0 (the default): 192; -1: no split
 *        (two 16-column tiles per workgroup with the epilogue in the
 *        projection).  Split products are added in split order by a kernel
 *        that then applies rotary and writes q and the KV slots.  Passes of
 *        more than 128 rows split QKV the same way when the residual
 *        layout would give it at most 128 workgroups (within 256 after the
 *        split), unless the key is -1.
 * key 8: projections of a row-tiled pass (more than 128 rows): 1 (the
 *        default) orders the workgroups so that the row tiles of one weight
 *        slice run together on one XCD and share its L2; 0 keeps the
 *        dispatch order.
 * key 9: the workgroup count the shared-prefix work items of a decode pass
 *        aim for when a group's prefix is split (1..4096, default 192); it
 *        applies to batches built after the call (vsk_batch_build).
 * key 10: 16-row groups per tile of the projections of a row-tiled pass
 *        (lm_head aside).  0 (the default): 6, 7 or 11 (residual
 *        projections: 6 or 7) where the launch then takes fewer rounds x
 *        tile height than at 8 (one workgroup per compute unit, 256 per
 *        round; launches that split K keep 8), else 8; 6, 7, 8 or 11 force
 *        that height (11 gives 8 for the residual projections). */
int vsk_set_tuning(vsk_handle* h, int32_t key, int32_t value);

/* Inspection: copy the fp32 residual stream x [n_rows][hidden] left in the
 * bound workspace by the last decode or prefill pass (all rows) to dst_dev. */
int vsk_residual_copy(vsk_handle* h, void* dst_dev, int32_t n_rows, void* stream);

/* Counters of what the last pass executed (kernel variants, split factors),
 * for attestation in tests and benchmarks.  Writes up to cap int64 values:
 * [0] passes run, [1] projection phases, [2] attention phases, [3] attention
 * splits (max per row), [4] workgroups per 16-column tile of the last down
 * projection, [5] 1 if the last pass ran as the persistent kernel, else 0. */
int vsk_exec_counters(const vsk_handle* h, int64_t* out, int32_t cap);

/* Measurement: while buf_dev is set (NULL clears it), each persistent pass
 * writes, per synchronisation point and workgroup, two uint64 timestamps of
 * the device's constant 100 MHz clock: when the workgroup arrived at the
 * point and when it was released from it ([points][workgroups][2]; a
 * buffer too small for the pass is ignored).  *n_wgs and *n_points
 * (nullable) receive the workgroup count of a persistent launch on the
 * current device (0: the kernel cannot run there) and the points of a pass. */
int vsk_set_step_trace(vsk_handle* h, void* buf_dev, size_t bytes, int32_t* n_wgs, int32_t* n_points);

/* Synchronise `stream`, then report whether a persistent pass on the bound
 * workspace failed: VSK_OK, or VSK_E_HIP when one of its grid
 * synchronisation waits exceeded its spin limit (the kernel then ended
 * without finishing the pass; the error stays recorded until
 * vsk_workspace_init) or the stream reported a HIP error. */
int vsk_device_status(vsk_handle* h, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* VSK_H */
