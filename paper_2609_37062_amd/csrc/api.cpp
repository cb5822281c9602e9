// The C ABI (include/vsk.h): validation, host allocator, layouts and the
// orchestration of one forward pass over the rows of a batch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "attn.hpp"
#include "gemm.hpp"
#include "internal.hpp"
#include "misc.hpp"
#include "step.hpp"

using namespace vsk;

struct vsk_handle : public Handle {};

vsk::Handle::~Handle() {
  for (Staging& st : stage) {
    if (st.pending && st.done) (void)hipEventSynchronize(st.done);
    if (st.done) (void)hipEventDestroy(st.done);
    if (st.host) (void)hipHostFree(st.host);
  }
}

namespace vsk {
static int step_workgroups(Handle& h);
}

namespace vsk {

PackedLayout packed_layout(const vsk_model_cfg& c) {
  PackedLayout p;
  const size_t H = c.hidden, F = c.ffn, Nq = static_cast<size_t>(c.n_q_heads) * c.head_dim,
               Nkv = static_cast<size_t>(c.n_kv_heads) * c.head_dim, V = c.vocab;
  size_t o = 0;
  p.l.attn_norm = o; o = align_up(o + H * 2);
  p.l.mlp_norm = o; o = align_up(o + H * 2);
  p.l.wqkv = o; o = align_up(o + (Nq + 2 * Nkv) * H * 2);
  p.l.wo = o; o = align_up(o + H * Nq * 2);
  p.l.wgu = o; o = align_up(o + 2 * F * H * 2);
  p.l.wd = o; o = align_up(o + H * F * 2);
  p.layer_bytes = o;
  p.head_base = p.layer_bytes * c.n_layers;
  o = p.head_base;
  p.final_norm = o; o = align_up(o + H * 2);
  p.embed = o; o = align_up(o + V * H * 2);
  p.lm_head = o; o = align_up(o + V * H * 2);
  p.rope = o; o = align_up(o + static_cast<size_t>(c.max_pos) * (c.head_dim / 2) * 8);
  p.total = o;
  return p;
}

static int ceil_div(int a, int b) { return (a + b - 1) / b; }

WsLayout ws_layout(const vsk_model_cfg& c, int32_t max_rows, int32_t max_seqs, int32_t max_kv_len, bool with_step,
                   bool routed) {
  WsLayout w;
  w.max_rows = max_rows;
  w.max_seqs = max_seqs;
  w.max_kv_len = max_kv_len;
  w.Rg = ceil_div(max_rows, 16);
  // a row's own splits, and the prefix splits of its group ahead of them
  w.max_splits = attn_splits(max_kv_len, kAttnMinBps) + kMaxPfxSplits;
  const size_t H = c.hidden, F = c.ffn, Nq = static_cast<size_t>(c.n_q_heads) * c.head_dim;
  const size_t Rp = static_cast<size_t>(w.Rg) * 16;
  const int G = c.n_q_heads / c.n_kv_heads;
  size_t o = 0;
  w.x = o; o = align_up(o + static_cast<size_t>(max_rows) * H * 4);
  w.x_c = o; o = align_up(o + static_cast<size_t>(max_rows) * H * 4);
  w.fa = o; o = align_up(o + Rp * Nq * 2);
  w.fb = o; o = align_up(o + Rp * H * 2);
  w.fc = o; o = align_up(o + Rp * F * 2);
  w.q = o; o = align_up(o + static_cast<size_t>(max_rows) * Nq * 2);
  const size_t rh = static_cast<size_t>(max_rows) * c.n_kv_heads;
  w.att_o = o; o = align_up(o + rh * w.max_splits * G * c.head_dim * 4);
  w.att_ml = o; o = align_up(o + rh * w.max_splits * G * 8);
  w.att_cnt = o; o = align_up(o + rh * 4);  // zeroed at init, left zero by every pass
  // x^2 partials: at most one per 16 columns of the hidden size, per row
  w.ssq = o; o = align_up(o + (H / 16) * static_cast<size_t>(max_rows) * 8);
  w.ssq_c = o; o = align_up(o + (H / 16) * static_cast<size_t>(max_rows) * 8);
  // residual projections with K split over workgroups: one product per split
  // and row (and the QKV projection's, N = Nq + 2 Nkv); row-tiled passes with
  // few workgroups split too
  const size_t y_cols = std::max<size_t>(H, static_cast<size_t>(Nq) + 2 * static_cast<size_t>(c.n_kv_heads) * c.head_dim);
  w.ypart = o; o = align_up(o + static_cast<size_t>(kMaxResidSplits) * max_rows * y_cols * 4);
  // lm_head argmax partials: n_groups x rows
  const size_t lm_groups = static_cast<size_t>(ceil_div(c.vocab, 16));  // upper bound over plans
  w.am_part = o; o = align_up(o + lm_groups * max_rows * 8);
  // routed layers: the Project-Only cohort's operands (the projector is at
  // most ffn wide), both cohorts' down-projection products, and the maps
  w.routed = routed;
  if (routed) {
    const size_t L = c.n_layers, R = max_rows;
    const size_t yrows = static_cast<size_t>(kMaxResidSplits) * R;  // a product per K split of every row
    w.fb_po = o; o = align_up(o + Rp * H * 2);
    w.fc_po = o; o = align_up(o + Rp * F * 2);
    w.y_run = o; o = align_up(o + yrows * H * 4);
    w.y_po = o; o = align_up(o + yrows * H * 4);
    w.r_run = o; o = align_up(o + L * R * 4);
    w.r_proj = o; o = align_up(o + L * R * 4);
    w.r_inv = o; o = align_up(o + L * R * 4);
    w.r_cnt = o; o = align_up(o + L * 2 * 4);
  }
  // persistent decode step: every per-layer buffer is written once per launch
  w.step = with_step && max_rows <= kStepMaxRows && step_shape_ok(c);
  if (w.step) {
    const size_t L = c.n_layers, nx = 2 * L + 1, R = max_rows;
    w.s_x = o; o = align_up(o + nx * R * H * 4);
    w.s_ssq = o; o = align_up(o + nx * (H / 16) * R * 8);
    w.s_q = o; o = align_up(o + L * R * Nq * 2);
    w.s_o = o; o = align_up(o + L * kStepMaxRows * Nq * 2);
    w.s_a = o; o = align_up(o + L * kStepMaxRows * F * 2);
    w.s_n = o; o = align_up(o + nx * kStepMaxRows * H * 2);
    w.s_am = o; o = align_up(o + static_cast<size_t>(c.vocab / 16) * R * 8);
    w.s_flags = o; o = align_up(o + static_cast<size_t>(step_syncs(c.n_layers)) * kSyncCounters * kFlagWords * 4);
    w.s_err = o; o = align_up(o + 4);
    w.s_epoch = o; o = align_up(o + 4);
  }
  w.total = o;
  return w;
}

}  // namespace vsk

// ------------------------------------------------------------------ helpers
static int fail(vsk_handle* h, int code, const std::string& msg) {
  if (h) h->err = msg;
  return code;
}

static int hip_check(vsk_handle* h, hipError_t e, const char* what) {
  if (e == hipSuccess) return VSK_OK;
  return fail(h, VSK_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

static bool cfg_ok(const vsk_model_cfg* c, std::string& why) {
  if (!c) { why = "null config"; return false; }
  if (c->n_layers < 1 || c->hidden < 64 || c->n_q_heads < 1 || c->n_kv_heads < 1 || c->ffn < 64 ||
      c->vocab < 16 || c->max_pos < 1) { why = "non-positive dimension"; return false; }
  if (c->block_size != kBlock) { why = "block_size must be 16"; return false; }
  if (c->head_dim != 64 && c->head_dim != 128) { why = "head_dim must be 64 or 128"; return false; }
  if (c->n_q_heads % c->n_kv_heads != 0 || c->n_q_heads / c->n_kv_heads > 16) {
    why = "n_q_heads must be a multiple of n_kv_heads, at most 16 per group"; return false;
  }
  if (c->hidden > 8192) { why = "hidden must be at most 8192"; return false; }
  if (c->max_pos > 16384) { why = "max_pos must be at most 16384"; return false; }
  if (c->hidden % 64 || (c->n_q_heads * c->head_dim) % 64 || c->ffn % 64 || c->vocab % 64) {
    why = "hidden, n_q_heads*head_dim, ffn and vocab must be multiples of 64"; return false;
  }
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f)) { why = "bad eps or rope theta"; return false; }
  return true;
}

extern "C" {

const char* vsk_status_str(int s) {
  switch (s) {
    case VSK_OK: return "ok";
    case VSK_E_ARG: return "bad argument";
    case VSK_E_NOMEM: return "KV pool exhausted";
    case VSK_E_RANGE: return "out of range";
    case VSK_E_SHARED_WRITE: return "write into a shared block";
    case VSK_E_STATE: return "invalid state";
    case VSK_E_HIP: return "HIP runtime error";
    case VSK_E_UNSUPPORTED: return "unsupported shape";
    default: return "unknown status";
  }
}

const char* vsk_last_error(const vsk_handle* h) { return h ? h->err.c_str() : "null handle"; }

int vsk_create(const vsk_model_cfg* cfg, vsk_handle** out) {
  if (!out) return VSK_E_ARG;
  *out = nullptr;
  std::string why;
  if (!cfg_ok(cfg, why)) return VSK_E_ARG;
  vsk_handle* h = new (std::nothrow) vsk_handle();
  if (!h) return VSK_E_ARG;
  h->cfg = *cfg;
  h->pl = packed_layout(*cfg);
  *out = h;
  return VSK_OK;
}

int vsk_destroy(vsk_handle* h) {
  delete h;
  return VSK_OK;
}

size_t vsk_packed_weight_bytes(const vsk_model_cfg* cfg) {
  std::string why;
  if (!cfg_ok(cfg, why)) return 0;
  return packed_layout(*cfg).total;
}

int vsk_weights_bind(vsk_handle* h, void* packed_dev, size_t bytes) {
  if (!h) return VSK_E_ARG;
  if (!packed_dev || bytes < h->pl.total) return fail(h, VSK_E_ARG, "packed weight buffer too small");
  if (reinterpret_cast<uintptr_t>(packed_dev) % kAlign) return fail(h, VSK_E_ARG, "packed buffer not 256-byte aligned");
  h->packed = static_cast<uint8_t*>(packed_dev);
  h->packed_bytes = bytes;
  return VSK_OK;
}

int vsk_weights_pack_layer(vsk_handle* h, int32_t layer, const vsk_layer_weights* w, void* stream) {
  if (!h || !w) return VSK_E_ARG;
  if (!h->packed) return fail(h, VSK_E_STATE, "no packed weight buffer bound");
  const vsk_model_cfg& c = h->cfg;
  if (layer < 0 || layer >= c.n_layers) return fail(h, VSK_E_RANGE, "layer out of range");
  if (!w->attn_norm || !w->wq || !w->wk || !w->wv || !w->wo || !w->mlp_norm || !w->w_gate || !w->w_up || !w->w_down)
    return fail(h, VSK_E_ARG, "null weight pointer");
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* base = h->packed + h->pl.layer_bytes * layer;
  const int H = c.hidden, F = c.ffn, d = c.head_dim, Nq = c.n_q_heads * d, Nkv = c.n_kv_heads * d;
  auto u16 = [](const void* p) { return static_cast<const uint16_t*>(p); };
  auto dst = [&](size_t off) { return reinterpret_cast<uint16_t*>(base + off); };
  hipError_t e;
  if ((e = launch_copy_bf16(u16(w->attn_norm), dst(h->pl.l.attn_norm), H, s)) != hipSuccess) return hip_check(h, e, "pack");
  if ((e = launch_copy_bf16(u16(w->mlp_norm), dst(h->pl.l.mlp_norm), H, s)) != hipSuccess) return hip_check(h, e, "pack");
  if ((e = launch_pack(u16(w->wq), u16(w->wk), u16(w->wv), Nq, Nkv, Nq + 2 * Nkv, H, 1, d, Nq + Nkv,
                       dst(h->pl.l.wqkv), s)) != hipSuccess) return hip_check(h, e, "pack qkv");
  if ((e = launch_pack(u16(w->wo), nullptr, nullptr, H, 0, H, Nq, 0, d, 0, dst(h->pl.l.wo), s)) != hipSuccess)
    return hip_check(h, e, "pack o");
  if ((e = launch_pack(u16(w->w_gate), u16(w->w_up), nullptr, F, F, 2 * F, H, 2, d, 0, dst(h->pl.l.wgu), s)) !=
      hipSuccess) return hip_check(h, e, "pack gate/up");
  if ((e = launch_pack(u16(w->w_down), nullptr, nullptr, H, 0, H, F, 0, d, 0, dst(h->pl.l.wd), s)) != hipSuccess)
    return hip_check(h, e, "pack down");
  return VSK_OK;
}

int vsk_weights_pack_head(vsk_handle* h, const void* embed_dev, const void* lm_head_dev, const void* final_norm_dev,
                          void* stream) {
  if (!h) return VSK_E_ARG;
  if (!h->packed) return fail(h, VSK_E_STATE, "no packed weight buffer bound");
  if (!embed_dev || !lm_head_dev || !final_norm_dev) return fail(h, VSK_E_ARG, "null weight pointer");
  const vsk_model_cfg& c = h->cfg;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t VH = static_cast<size_t>(c.vocab) * c.hidden;
  auto u16 = [](const void* p) { return static_cast<const uint16_t*>(p); };
  hipError_t e;
  if ((e = launch_copy_bf16(u16(final_norm_dev), reinterpret_cast<uint16_t*>(h->packed + h->pl.final_norm), c.hidden,
                            s)) != hipSuccess) return hip_check(h, e, "pack final norm");
  if ((e = hipMemcpyAsync(h->packed + h->pl.embed, embed_dev, VH * 2, hipMemcpyDeviceToDevice, s)) != hipSuccess)
    return hip_check(h, e, "copy embedding");
  if ((e = launch_pack(u16(lm_head_dev), nullptr, nullptr, c.vocab, 0, c.vocab, c.hidden, 0, c.head_dim, 0,
                       reinterpret_cast<uint16_t*>(h->packed + h->pl.lm_head), s)) != hipSuccess)
    return hip_check(h, e, "pack lm_head");
  // rotary table: (cos, sin) of pos * theta^(-2j/d) in double, stored as float
  const int half = c.head_dim / 2;
  std::vector<float> tab(static_cast<size_t>(c.max_pos) * half * 2);
  for (int p = 0; p < c.max_pos; ++p)
    for (int j = 0; j < half; ++j) {
      const double inv = std::pow(static_cast<double>(c.rope_theta), -2.0 * j / c.head_dim);
      const double ang = static_cast<double>(p) * inv;
      tab[(static_cast<size_t>(p) * half + j) * 2 + 0] = static_cast<float>(std::cos(ang));
      tab[(static_cast<size_t>(p) * half + j) * 2 + 1] = static_cast<float>(std::sin(ang));
    }
  if ((e = hipMemcpyAsync(h->packed + h->pl.rope, tab.data(), tab.size() * 4, hipMemcpyHostToDevice, s)) != hipSuccess)
    return hip_check(h, e, "copy rotary table");
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return hip_check(h, e, "sync");
  return VSK_OK;
}

// ------------------------------------------------------------------ KV
size_t vsk_kv_pool_bytes(const vsk_model_cfg* cfg, int32_t n_blocks) {
  std::string why;
  if (!cfg_ok(cfg, why) || n_blocks <= 0) return 0;
  return static_cast<size_t>(cfg->n_layers) * 2 * n_blocks * cfg->n_kv_heads * kBlock * cfg->head_dim * 2;
}

int vsk_kv_init(vsk_handle* h, void* pool_dev, int32_t n_blocks) {
  if (!h) return VSK_E_ARG;
  if (n_blocks <= 0) return fail(h, VSK_E_ARG, "n_blocks must be positive");
  if (static_cast<int64_t>(n_blocks) * kBlock > INT32_MAX) return fail(h, VSK_E_ARG, "pool too large for int32 slots");
  h->pool = static_cast<uint16_t*>(pool_dev);
  h->n_blocks = n_blocks;
  h->alloc = BlockAllocator(n_blocks, kBlock);
  h->alloc_ready = true;
  h->batch_built = false;
  h->batch_uploaded = false;
  return VSK_OK;
}

#define NEED_ALLOC(h)                                                   \
  do {                                                                  \
    if (!(h)) return VSK_E_ARG;                                         \
    if (!(h)->alloc_ready) return fail((h), VSK_E_STATE, "kv_init not called"); \
  } while (0)

int vsk_seq_create(vsk_handle* h, int64_t seq) {
  NEED_ALLOC(h);
  return h->alloc.seq_create(seq, h->err);
}

int vsk_seq_release(vsk_handle* h, int64_t seq) {
  NEED_ALLOC(h);
  return h->alloc.seq_release(seq, h->err);
}

int vsk_seq_set_blocks(vsk_handle* h, int64_t seq, const int32_t* blocks_host, int32_t n, int32_t ctx_len) {
  NEED_ALLOC(h);
  return h->alloc.seq_set_blocks(seq, blocks_host, n, ctx_len, h->err);
}

int vsk_seq_share_prefix(vsk_handle* h, int64_t dst, int64_t src, int32_t n_tokens) {
  NEED_ALLOC(h);
  return h->alloc.seq_share_prefix(dst, src, n_tokens, h->err);
}

int vsk_kv_reserve(vsk_handle* h, int64_t seq, int32_t n_new, int32_t* slots_host) {
  NEED_ALLOC(h);
  const SeqState* s = h->alloc.find(seq);
  if (s && static_cast<int64_t>(s->len) + n_new > h->cfg.max_pos)
    return fail(h, VSK_E_RANGE, "positions would exceed max_pos");
  return h->alloc.reserve(seq, n_new, slots_host, h->err);
}

int vsk_seq_info(const vsk_handle* h, int64_t seq, int32_t* len, int32_t* n_blocks, int32_t* blocks_host,
                 int32_t cap) {
  if (!h || !h->alloc_ready) return VSK_E_STATE;
  const SeqState* s = h->alloc.find(seq);
  if (!s) return VSK_E_STATE;
  if (len) *len = s->len;
  if (n_blocks) *n_blocks = static_cast<int32_t>(s->blocks.size());
  if (blocks_host)
    for (int32_t i = 0; i < cap && i < static_cast<int32_t>(s->blocks.size()); ++i) blocks_host[i] = s->blocks[i];
  return VSK_OK;
}

int vsk_kv_free_blocks(const vsk_handle* h, int32_t* n_free) {
  if (!h || !h->alloc_ready || !n_free) return VSK_E_STATE;
  *n_free = h->alloc.free_count();
  return VSK_OK;
}

static int kv_move(vsk_handle* h, bool write, int32_t layer, const int32_t* slots, int32_t n, const void* k,
                   const void* v, void* stream) {
  if (!h) return VSK_E_ARG;
  if (!h->pool) return fail(h, VSK_E_STATE, "no KV pool bound");
  if (layer < 0 || layer >= h->cfg.n_layers) return fail(h, VSK_E_RANGE, "layer out of range");
  if (n < 0 || (n > 0 && (!slots || !k || !v))) return fail(h, VSK_E_ARG, "bad KV transfer arguments");
  hipError_t e = launch_kv_move(write, h->pool, layer, h->n_blocks, h->cfg.n_kv_heads, h->cfg.head_dim, slots, n,
                                const_cast<uint16_t*>(static_cast<const uint16_t*>(k)),
                                const_cast<uint16_t*>(static_cast<const uint16_t*>(v)),
                                static_cast<hipStream_t>(stream));
  return hip_check(h, e, "kv transfer");
}

int vsk_kv_write(vsk_handle* h, int32_t layer, const int32_t* slots_dev, int32_t n, const void* k_dev,
                 const void* v_dev, void* stream) {
  return kv_move(h, true, layer, slots_dev, n, k_dev, v_dev, stream);
}

int vsk_kv_read(vsk_handle* h, int32_t layer, const int32_t* slots_dev, int32_t n, void* k_dev, void* v_dev,
                void* stream) {
  return kv_move(h, false, layer, slots_dev, n, k_dev, v_dev, stream);
}

// ------------------------------------------------------------------ batch
int vsk_batch_build(vsk_handle* h, const int64_t* seqs_host, const int32_t* q_lens_host, int32_t n_seqs) {
  NEED_ALLOC(h);
  BatchHost b;
  int st = build_batch(h->alloc, seqs_host, q_lens_host, n_seqs, b, h->err);
  if (st != VSK_OK) return st;
  plan_prefix_items(b, h->cfg.n_q_heads / h->cfg.n_kv_heads, h->cfg.n_kv_heads, h->pfx_target);
  plan_prefill_items(b, h->cfg.n_q_heads / h->cfg.n_kv_heads, kBlock);
  h->bh = std::move(b);
  h->batch_built = true;
  h->batch_uploaded = false;
  return VSK_OK;
}

int vsk_batch_shape(const vsk_handle* h, int32_t* n_seqs, int32_t* n_rows, int32_t* max_blocks) {
  if (!h || !h->batch_built) return VSK_E_STATE;
  if (n_seqs) *n_seqs = h->bh.n_seqs;
  if (n_rows) *n_rows = h->bh.n_rows;
  if (max_blocks) *max_blocks = h->bh.max_blocks;
  return VSK_OK;
}

int vsk_batch_host_copy(const vsk_handle* h, int32_t* block_table, int32_t* kv_len, int32_t* cu_q, int32_t* row_seq,
                        int32_t* pos, int32_t* slot) {
  if (!h || !h->batch_built) return VSK_E_STATE;
  const BatchHost& b = h->bh;
  auto cp = [](int32_t* d, const std::vector<int32_t>& s) {
    if (d) std::memcpy(d, s.data(), s.size() * 4);
  };
  cp(block_table, b.block_table);
  cp(kv_len, b.kv_len);
  cp(cu_q, b.cu_q);
  cp(row_seq, b.row_seq);
  cp(pos, b.pos);
  cp(slot, b.slot);
  return VSK_OK;
}

int vsk_batch_prefix_info(const vsk_handle* h, int32_t* pfx_blocks_host, int32_t* n_groups) {
  if (!h || !h->batch_built) return VSK_E_STATE;
  if (pfx_blocks_host) std::memcpy(pfx_blocks_host, h->bh.pfx_blocks.data(), h->bh.pfx_blocks.size() * 4);
  if (n_groups) *n_groups = h->bh.n_groups();
  return VSK_OK;
}

static size_t meta_bytes(const BatchHost& b) {
  auto sz = [](const std::vector<int32_t>& v) { return align_up(std::max<size_t>(v.size(), 1) * 4); };
  return sz(b.block_table) + sz(b.kv_len) + sz(b.cu_q) + sz(b.row_seq) + sz(b.pos) + sz(b.slot) +
         sz(b.pfx_blocks) + sz(b.pfx_splits) + sz(b.pfx_items) + sz(b.grp_rows) + sz(b.grp_info) + sz(b.pfx_tbl) +
         sz(b.pre_items) + sz(b.dec_rows);
}

size_t vsk_batch_device_bytes(const vsk_handle* h) {
  if (!h || !h->batch_built) return 0;
  return meta_bytes(h->bh);
}

int vsk_batch_upload(vsk_handle* h, void* meta_dev, size_t bytes, void* stream) {
  if (!h) return VSK_E_ARG;
  if (!h->batch_built) return fail(h, VSK_E_STATE, "no batch built");
  const BatchHost& b = h->bh;
  if (!meta_dev || bytes < meta_bytes(b)) return fail(h, VSK_E_ARG, "metadata buffer too small");
  if (reinterpret_cast<uintptr_t>(meta_dev) % kAlign) return fail(h, VSK_E_ARG, "metadata buffer not aligned");
  std::vector<uint8_t> staging(meta_bytes(b), 0);
  size_t o = 0;
  BatchDev d;
  uint8_t* base = static_cast<uint8_t*>(meta_dev);
  auto put = [&](const std::vector<int32_t>& v, const int32_t** dp) {
    std::memcpy(staging.data() + o, v.data(), v.size() * 4);
    *dp = reinterpret_cast<const int32_t*>(base + o);
    o += align_up(std::max<size_t>(v.size(), 1) * 4);
  };
  put(b.block_table, &d.block_table);
  put(b.kv_len, &d.kv_len);
  put(b.cu_q, &d.cu_q);
  put(b.row_seq, &d.row_seq);
  put(b.pos, &d.pos);
  put(b.slot, &d.slot);
  put(b.pfx_blocks, &d.pfx_blocks);
  put(b.pfx_splits, &d.pfx_splits);
  put(b.pfx_items, &d.pfx_items);
  put(b.grp_rows, &d.grp_rows);
  put(b.grp_info, &d.grp_info);
  put(b.pfx_tbl, &d.pfx_tbl);
  put(b.pre_items, &d.pre_items);
  put(b.dec_rows, &d.dec_rows);
  d.n_pre_items = b.n_pre_items();
  d.n_dec_rows = static_cast<int32_t>(b.dec_rows.size());
  d.n_pfx_items = b.n_pfx_items();
  d.max_pfx_splits = b.max_pfx_splits;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // copy from a pinned staging buffer: the transfer runs asynchronously and
  // the host returns at once, unless this buffer's previous copy (issued two
  // uploads ago) has not finished yet
  Handle::Staging& st = h->stage[h->stage_next];
  hipError_t e = hipSuccess;
  if (st.pending) {
    e = hipEventSynchronize(st.done);
    if (e != hipSuccess) return hip_check(h, e, "metadata staging wait");
    st.pending = false;
  }
  if (st.cap < staging.size()) {
    if (st.host) (void)hipHostFree(st.host);
    st.host = nullptr;
    st.cap = 0;
    const size_t cap = std::max<size_t>(align_up(staging.size(), 1 << 16), 1 << 16);
    e = hipHostMalloc(&st.host, cap, hipHostMallocDefault);
    if (e != hipSuccess) return hip_check(h, e, "metadata staging buffer");
    st.cap = cap;
  }
  if (!st.done) {
    e = hipEventCreateWithFlags(&st.done, hipEventDisableTiming);
    if (e != hipSuccess) return hip_check(h, e, "metadata staging event");
  }
  std::memcpy(st.host, staging.data(), staging.size());
  e = hipMemcpyAsync(meta_dev, st.host, staging.size(), hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipEventRecord(st.done, s);
  if (e != hipSuccess) return hip_check(h, e, "metadata upload");
  st.pending = true;
  h->stage_next ^= 1;
  d.n_seqs = b.n_seqs;
  d.n_rows = b.n_rows;
  d.max_blocks = b.max_blocks;
  d.max_kv_len = b.max_kv_len;
  d.max_q_len = b.max_q_len;
  h->bd = d;
  h->batch_uploaded = true;
  return VSK_OK;
}

// ------------------------------------------------------------------ passes
size_t vsk_workspace_bytes(const vsk_handle* h, int32_t max_rows, int32_t max_seqs, int32_t max_kv_len) {
  if (!h || max_rows <= 0 || max_seqs <= 0 || max_kv_len <= 0) return 0;
  return ws_layout(h->cfg, max_rows, max_seqs, max_kv_len, true, h->routed_w != nullptr).total;
}

int vsk_workspace_init(vsk_handle* h, void* ws_dev, size_t bytes, int32_t max_rows, int32_t max_seqs,
                       int32_t max_kv_len, void* stream) {
  if (!h || !ws_dev) return VSK_E_ARG;
  if (max_rows <= 0 || max_seqs <= 0 || max_kv_len <= 0) return fail(h, VSK_E_ARG, "capacity must be positive");
  if (reinterpret_cast<uintptr_t>(ws_dev) % kAlign) return fail(h, VSK_E_ARG, "workspace not aligned");
  const WsLayout wl = ws_layout(h->cfg, max_rows, max_seqs, max_kv_len, true, h->routed_w != nullptr);
  if (bytes < wl.total) return fail(h, VSK_E_ARG, "workspace smaller than vsk_workspace_bytes()");
  hipError_t e = launch_fill_zero(ws_dev, wl.total, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_check(h, e, "workspace init");
  h->ws = static_cast<uint8_t*>(ws_dev);
  h->ws_bytes = bytes;
  h->wl = wl;
  return VSK_OK;
}

static int pass_common(vsk_handle* h, const int32_t* ids, void* logits, void* ws, size_t ws_bytes) {
  if (!h) return VSK_E_ARG;
  if (!h->packed) return fail(h, VSK_E_STATE, "no weights bound");
  if (!h->pool) return fail(h, VSK_E_STATE, "no KV pool bound");
  if (!h->batch_uploaded) return fail(h, VSK_E_STATE, "no batch uploaded");
  if (!ids || !logits || !ws) return fail(h, VSK_E_ARG, "null buffer");
  if (ws != h->ws || ws_bytes != h->ws_bytes) return fail(h, VSK_E_STATE, "workspace not initialised with this handle");
  const BatchDev& b = h->bd;
  if (b.max_kv_len > h->cfg.max_pos) return fail(h, VSK_E_RANGE, "position beyond max_pos");
  if (b.n_rows > h->wl.max_rows || b.n_seqs > h->wl.max_seqs || b.max_kv_len > h->wl.max_kv_len)
    return fail(h, VSK_E_ARG, "batch exceeds the workspace capacity");
  return VSK_OK;
}

int vsk_decode_step(vsk_handle* h, const int32_t* ids_dev, void* logits_dev, int32_t* next_ids_dev, void* ws_dev,
                    size_t ws_bytes, void* stream) {
  int st = pass_common(h, ids_dev, logits_dev, ws_dev, ws_bytes);
  if (st != VSK_OK) return st;
  if (h->bd.max_q_len != 1) return fail(h, VSK_E_ARG, "decode_step needs one row per sequence");
  PassArgs a{ids_dev, nullptr, h->bd.n_rows, static_cast<uint16_t*>(logits_dev), next_ids_dev,
             static_cast<uint8_t*>(ws_dev), h->wl};
  if (h->exec_mode == 2 && !step_eligible(*h, a))
    return fail(h, VSK_E_UNSUPPORTED, "the persistent step kernel does not cover this pass (rows, shape or device)");
  return hip_check(h, run_pass(*h, a, static_cast<hipStream_t>(stream)), "decode step");
}

}  // extern "C"

// ------------------------------------------------------------------ scratch entry point
// vsk_decode_step_scratch takes its workspace from this file-scope device
// array instead of a caller's buffer.  Every GPU the library runs on holds
// its own copy (VSK_SCRATCH_BYTES, zero at load) until the process ends.  In
// host code `scratch` names a host-side stand-in, never the device memory:
// the device address is looked up once per device with hipGetSymbolAddress
// and only that pointer is handed to kernels.
static __device__ __align__(256) uint8_t scratch[VSK_SCRATCH_BYTES];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of the current device's scratch array (looked up on the
// first call on that device).
hipError_t scratch_base(uint8_t** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = static_cast<uint8_t*>(g_scratch_ptr[dev]);
  return hipSuccess;
}
}  // namespace

extern "C" {

int vsk_decode_step_scratch(vsk_handle* h, const int32_t* ids_dev, void* logits_dev, int32_t* next_ids_dev,
                            void* stream) {
  if (!h) return VSK_E_ARG;
  if (!h->packed) return fail(h, VSK_E_STATE, "no weights bound");
  if (!h->pool) return fail(h, VSK_E_STATE, "no KV pool bound");
  if (!h->batch_uploaded) return fail(h, VSK_E_STATE, "no batch uploaded");
  if (!ids_dev || !logits_dev) return fail(h, VSK_E_ARG, "null buffer");
  const BatchDev& b = h->bd;
  if (b.max_q_len != 1) return fail(h, VSK_E_ARG, "decode_step needs one row per sequence");
  if (b.max_kv_len > h->cfg.max_pos) return fail(h, VSK_E_RANGE, "position beyond max_pos");
  // the workspace of exactly this batch, without the persistent kernel's region
  const WsLayout wl = ws_layout(h->cfg, b.n_rows, b.n_seqs, b.max_kv_len, false);
  if (wl.total > static_cast<size_t>(VSK_SCRATCH_BYTES))
    return fail(h, VSK_E_ARG, "the batch needs " + std::to_string(wl.total) + " bytes of scratch, more than the " +
                                  std::to_string(static_cast<size_t>(VSK_SCRATCH_BYTES)) + " of vsk_decode_step_scratch");
  uint8_t* base = nullptr;
  hipError_t e = scratch_base(&base);
  if (e != hipSuccess) return hip_check(h, e, "scratch address");
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the attention arrival counters must start at zero; the layout (and so
  // their place) follows the batch, and the array keeps the last call's bytes
  e = launch_fill_zero(base + wl.att_cnt, static_cast<size_t>(b.n_rows) * h->cfg.n_kv_heads * 4, s);
  if (e != hipSuccess) return hip_check(h, e, "scratch counters");
  PassArgs a{ids_dev, nullptr, b.n_rows, static_cast<uint16_t*>(logits_dev), next_ids_dev, base, wl};
  return hip_check(h, run_pass(*h, a, s), "decode step (scratch)");
}

int vsk_prefill_chunk(vsk_handle* h, const int32_t* ids_dev, const int32_t* logit_rows_dev, int32_t n_logit_rows,
                      void* logits_dev, int32_t* next_ids_dev, void* ws_dev, size_t ws_bytes, void* stream) {
  int st = pass_common(h, ids_dev, logits_dev, ws_dev, ws_bytes);
  if (st != VSK_OK) return st;
  if (!logit_rows_dev || n_logit_rows < 1 || n_logit_rows > h->bd.n_rows)
    return fail(h, VSK_E_ARG, "logit rows must be 1..n_rows");
  PassArgs a{ids_dev, logit_rows_dev, n_logit_rows, static_cast<uint16_t*>(logits_dev), next_ids_dev,
             static_cast<uint8_t*>(ws_dev), h->wl};
  if (h->exec_mode == 2) return fail(h, VSK_E_UNSUPPORTED, "the persistent step kernel serves decode passes only");
  return hip_check(h, run_pass(*h, a, static_cast<hipStream_t>(stream)), "prefill chunk");
}

// ------------------------------------------------------------------ routed mode
static size_t routed_layer_bytes(const vsk_model_cfg& c, int32_t proj_ffn, size_t* pgu, size_t* pd) {
  const size_t H = c.hidden, Fp = proj_ffn;
  size_t o = 0;
  if (pgu) *pgu = o;
  o = align_up(o + 2 * Fp * H * 2);
  if (pd) *pd = o;
  o = align_up(o + H * Fp * 2);
  return o;
}

static bool routed_cfg_ok(const vsk_model_cfg& c, int32_t first_routed, int32_t proj_ffn, std::string& why) {
  if (first_routed < 0 || first_routed >= c.n_layers) { why = "first routed layer out of range"; return false; }
  if (proj_ffn < 64 || proj_ffn % 64 != 0 || proj_ffn > c.ffn) {
    why = "projector width must be a multiple of 64 in [64, ffn]";
    return false;
  }
  return true;
}

size_t vsk_routed_weight_bytes(const vsk_model_cfg* cfg, int32_t first_routed, int32_t proj_ffn) {
  std::string why;
  if (!cfg_ok(cfg, why) || !routed_cfg_ok(*cfg, first_routed, proj_ffn, why)) return 0;
  return routed_layer_bytes(*cfg, proj_ffn, nullptr, nullptr) * (cfg->n_layers - first_routed);
}

int vsk_routed_bind(vsk_handle* h, int32_t first_routed, int32_t proj_ffn, void* packed_dev, size_t bytes) {
  if (!h) return VSK_E_ARG;
  std::string why;
  if (!routed_cfg_ok(h->cfg, first_routed, proj_ffn, why)) return fail(h, VSK_E_ARG, why);
  const size_t need = vsk_routed_weight_bytes(&h->cfg, first_routed, proj_ffn);
  if (!packed_dev || bytes < need) return fail(h, VSK_E_ARG, "projector weight buffer too small");
  if (reinterpret_cast<uintptr_t>(packed_dev) % kAlign) return fail(h, VSK_E_ARG, "projector buffer not aligned");
  h->routed_w = static_cast<uint8_t*>(packed_dev);
  h->first_routed = first_routed;
  h->proj_ffn = proj_ffn;
  h->routed_layer_bytes = routed_layer_bytes(h->cfg, proj_ffn, &h->routed_pgu, &h->routed_pd);
  h->ws = nullptr;  // the workspace layout grows: it must be sized and bound again
  h->ws_bytes = 0;
  return VSK_OK;
}

int vsk_routed_pack_layer(vsk_handle* h, int32_t layer, const void* p_gate_dev, const void* p_up_dev,
                          const void* p_down_dev, void* stream) {
  if (!h) return VSK_E_ARG;
  if (!h->routed_w) return fail(h, VSK_E_STATE, "no projector weight buffer bound");
  if (layer < h->first_routed || layer >= h->cfg.n_layers) return fail(h, VSK_E_RANGE, "not a routed layer");
  if (!p_gate_dev || !p_up_dev || !p_down_dev) return fail(h, VSK_E_ARG, "null weight pointer");
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* base = h->routed_w + h->routed_layer_bytes * (layer - h->first_routed);
  const int H = h->cfg.hidden, Fp = h->proj_ffn;
  auto u16 = [](const void* p) { return static_cast<const uint16_t*>(p); };
  hipError_t e;
  if ((e = launch_pack(u16(p_gate_dev), u16(p_up_dev), nullptr, Fp, Fp, 2 * Fp, H, 2, h->cfg.head_dim, 0,
                       reinterpret_cast<uint16_t*>(base + h->routed_pgu), s)) != hipSuccess)
    return hip_check(h, e, "pack projector gate/up");
  if ((e = launch_pack(u16(p_down_dev), nullptr, nullptr, H, 0, H, Fp, 0, h->cfg.head_dim, 0,
                       reinterpret_cast<uint16_t*>(base + h->routed_pd), s)) != hipSuccess)
    return hip_check(h, e, "pack projector down");
  return VSK_OK;
}

static int routed_common(vsk_handle* h, const uint8_t* run_dev, const float* w_dev) {
  if (!h->routed_w) return fail(h, VSK_E_STATE, "no projector weights bound (vsk_routed_bind)");
  if (!h->wl.routed) return fail(h, VSK_E_STATE, "workspace sized before vsk_routed_bind: initialise it again");
  if (!run_dev || !w_dev) return fail(h, VSK_E_ARG, "null route tape");
  if (h->exec_mode == 2) return fail(h, VSK_E_UNSUPPORTED, "the persistent step kernel has no routed mode");
  return VSK_OK;
}

int vsk_decode_step_routed(vsk_handle* h, const int32_t* ids_dev, const uint8_t* run_dev, const float* w_dev,
                           void* logits_dev, int32_t* next_ids_dev, void* ws_dev, size_t ws_bytes, void* stream) {
  int st = pass_common(h, ids_dev, logits_dev, ws_dev, ws_bytes);
  if (st != VSK_OK) return st;
  if ((st = routed_common(h, run_dev, w_dev)) != VSK_OK) return st;
  if (h->bd.max_q_len != 1) return fail(h, VSK_E_ARG, "decode_step needs one row per sequence");
  PassArgs a{ids_dev, nullptr, h->bd.n_rows, static_cast<uint16_t*>(logits_dev), next_ids_dev,
             static_cast<uint8_t*>(ws_dev), h->wl, run_dev, w_dev};
  return hip_check(h, run_pass(*h, a, static_cast<hipStream_t>(stream)), "routed decode step");
}

int vsk_prefill_chunk_routed(vsk_handle* h, const int32_t* ids_dev, const uint8_t* run_dev, const float* w_dev,
                             const int32_t* logit_rows_dev, int32_t n_logit_rows, void* logits_dev,
                             int32_t* next_ids_dev, void* ws_dev, size_t ws_bytes, void* stream) {
  int st = pass_common(h, ids_dev, logits_dev, ws_dev, ws_bytes);
  if (st != VSK_OK) return st;
  if ((st = routed_common(h, run_dev, w_dev)) != VSK_OK) return st;
  if (!logit_rows_dev || n_logit_rows < 1 || n_logit_rows > h->bd.n_rows)
    return fail(h, VSK_E_ARG, "logit rows must be 1..n_rows");
  PassArgs a{ids_dev, logit_rows_dev, n_logit_rows, static_cast<uint16_t*>(logits_dev), next_ids_dev,
             static_cast<uint8_t*>(ws_dev), h->wl, run_dev, w_dev};
  return hip_check(h, run_pass(*h, a, static_cast<hipStream_t>(stream)), "routed prefill chunk");
}

int vsk_route_maps_read(vsk_handle* h, int32_t* run_dev, int32_t* proj_dev, int32_t* inv_dev, int32_t* cnt_dev,
                        void* stream) {
  if (!h) return VSK_E_ARG;
  if (!h->ws || !h->wl.routed) return fail(h, VSK_E_STATE, "no routed workspace bound");
  if (!h->batch_uploaded) return fail(h, VSK_E_STATE, "no batch uploaded");
  const size_t Lr = static_cast<size_t>(h->cfg.n_layers - h->first_routed), R = h->bd.n_rows;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the maps are stored with the pass's row count as the stride of each layer
  auto cp = [&](void* dst, size_t off, size_t n) {
    return dst ? hipMemcpyAsync(dst, h->ws + off, n, hipMemcpyDeviceToDevice, s) : hipSuccess;
  };
  hipError_t e = cp(run_dev, h->wl.r_run, Lr * R * 4);
  if (e == hipSuccess) e = cp(proj_dev, h->wl.r_proj, Lr * R * 4);
  if (e == hipSuccess) e = cp(inv_dev, h->wl.r_inv, Lr * R * 4);
  if (e == hipSuccess) e = cp(cnt_dev, h->wl.r_cnt, Lr * 2 * 4);
  return hip_check(h, e, "route maps copy");
}

int vsk_argmax_sample(const void* logits_dev, int32_t dtype, int32_t rows, int32_t vocab, int32_t* ids_dev,
                      int32_t* no_value_dev, void* stream) {
  if (!logits_dev || !ids_dev || rows < 1 || vocab < 1 || (dtype != 0 && dtype != 1)) return VSK_E_ARG;
  hipError_t e =
      launch_argmax_logits(logits_dev, dtype, rows, vocab, ids_dev, no_value_dev, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? VSK_OK : VSK_E_HIP;
}

int vsk_stream_read(const void* src_dev, size_t bytes, uint32_t* out_dev, int32_t workgroups, void* stream) {
  if (!src_dev || !out_dev || bytes == 0 || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(src_dev) % 16 ||
      workgroups < 1)
    return VSK_E_ARG;
  return launch_stream_read(src_dev, bytes, out_dev, workgroups, static_cast<hipStream_t>(stream)) == hipSuccess
             ? VSK_OK
             : VSK_E_HIP;
}

int vsk_set_probe(vsk_handle* h, int32_t which, void* const* begin_events, void* const* end_events, int32_t n_pairs) {
  if (!h) return VSK_E_ARG;
  if (which < 0 || which >= Handle::kProbeClasses) return fail(h, VSK_E_RANGE, "unknown probe class");
  if (n_pairs < 0 || (n_pairs > 0 && (!begin_events || !end_events))) return fail(h, VSK_E_ARG, "bad probe events");
  h->probe_b[which].assign(reinterpret_cast<const hipEvent_t*>(begin_events),
                           reinterpret_cast<const hipEvent_t*>(begin_events) + n_pairs);
  h->probe_e[which].assign(reinterpret_cast<const hipEvent_t*>(end_events),
                           reinterpret_cast<const hipEvent_t*>(end_events) + n_pairs);
  h->probe_i[which] = 0;
  return VSK_OK;
}

int vsk_set_tuning(vsk_handle* h, int32_t key, int32_t value) {
  if (!h) return VSK_E_ARG;
  switch (key) {
    case 0:
      if (value != 0 && (value < kAttnMinBps || value % 8 != 0 || value > kAttnMaxBps))
        return fail(h, VSK_E_ARG, "attention blocks per split must be 0 (auto) or a multiple of 8 in [8, 512]");
      h->attn_bps = value;
      return VSK_OK;
    case 1:
      if (value < 0 || value > h->cfg.n_layers) return fail(h, VSK_E_ARG, "layer count out of range");
      h->layers_run = value;
      return VSK_OK;
    case 2:
      if (value < 0 || value > 2) return fail(h, VSK_E_ARG, "execution mode must be 0, 1 or 2");
      h->exec_mode = value;
      return VSK_OK;
    case 3:
      if (value < 0 || value > 6) return fail(h, VSK_E_ARG, "projection shape must be 0..6");
      h->gemm_shape = value;
      return VSK_OK;
    case 4:
      if (value < 0 || value > 1) return fail(h, VSK_E_ARG, "shared-prefix switch must be 0 or 1");
      h->shared_prefix = value;
      return VSK_OK;
    case 6:
      if (value < 0 || value > 1) return fail(h, VSK_E_ARG, "prefill attention switch must be 0 or 1");
      h->prefill_attn = value;
      return VSK_OK;
    case 5:
      if (value < -1 || value > 4096)
        return fail(h, VSK_E_ARG, "residual split target must be -1 (no split), 0 (default) or 1..4096");
      h->resid_target = value;
      return VSK_OK;
    case 9:
      if (value < 1 || value > 4096) return fail(h, VSK_E_ARG, "shared-prefix work item target must be 1..4096");
      h->pfx_target = value;
      return VSK_OK;
    case 8:
      if (value < 0 || value > 1) return fail(h, VSK_E_ARG, "XCD remap switch must be 0 or 1");
      h->xcd_remap = value;
      return VSK_OK;
    case 10:
      if (value != 0 && value != 6 && value != 7 && value != 8 && value != 11)
        return fail(h, VSK_E_ARG, "row tile must be 0 (auto), 6, 7, 8 or 11");
      h->row_tile = value;
      return VSK_OK;
    case 7:
      if (value < -1 || value > 4096)
        return fail(h, VSK_E_ARG, "QKV split target must be -1 (no split), 0 (default) or 1..4096");
      h->qkv_target = value;
      return VSK_OK;
    default:
      return fail(h, VSK_E_ARG, "unknown tuning key");
  }
}

int vsk_residual_copy(vsk_handle* h, void* dst_dev, int32_t n_rows, void* stream) {
  if (!h || !dst_dev) return VSK_E_ARG;
  if (!h->ws) return fail(h, VSK_E_STATE, "no workspace bound");
  if (n_rows < 1 || n_rows > h->wl.max_rows) return fail(h, VSK_E_ARG, "row count out of range");
  const size_t bytes = static_cast<size_t>(n_rows) * h->cfg.hidden * 4;
  return hip_check(h, hipMemcpyAsync(dst_dev, h->ws + h->wl.x, bytes, hipMemcpyDeviceToDevice,
                                     static_cast<hipStream_t>(stream)), "residual copy");
}

int vsk_exec_counters(const vsk_handle* h, int64_t* out, int32_t cap) {
  if (!h || !out) return VSK_E_ARG;
  for (int i = 0; i < cap && i < 8; ++i) out[i] = h->counters[i];
  return VSK_OK;
}

int vsk_set_step_trace(vsk_handle* h, void* buf_dev, size_t bytes, int32_t* n_wgs, int32_t* n_points) {
  if (!h) return VSK_E_ARG;
  if (buf_dev && reinterpret_cast<uintptr_t>(buf_dev) % 8) return fail(h, VSK_E_ARG, "trace buffer not 8-byte aligned");
  h->step_trace = static_cast<uint64_t*>(buf_dev);
  h->step_trace_cap = buf_dev ? bytes / 8 : 0;
  const int wgs = step_workgroups(*h);
  if (n_wgs) *n_wgs = wgs;
  if (n_points) *n_points = step_syncs(h->layers_run > 0 ? h->layers_run : h->cfg.n_layers);
  return VSK_OK;
}

int vsk_device_status(vsk_handle* h, void* stream) {
  if (!h) return VSK_E_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_check(h, e, "stream");
  if (!h->ws || !h->wl.step) return VSK_OK;
  uint32_t err = 0;
  e = hipMemcpyAsync(&err, h->ws + h->wl.s_err, 4, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_check(h, e, "status read");
  if (err != 0)
    return fail(h, VSK_E_HIP, "a persistent pass (epoch " + std::to_string(err) +
                                  ") timed out at a grid synchronisation point; re-initialise the workspace");
  return VSK_OK;
}

}  // extern "C"

// ------------------------------------------------------------------ the pass
namespace vsk {

// Workgroups of a persistent launch on the current device: one per compute
// unit when the kernel fits there with its LDS (0 when it does not).
static int step_workgroups(Handle& h) {
  if (h.step_wgs < 0) {
    int dev = 0, cus = 0;
    h.step_wgs = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        step_occupancy(h.cfg) >= 1)
      h.step_wgs = std::min(cus, kStepMaxWgs);
  }
  return h.step_wgs;
}

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

static hipError_t run_step(Handle& h, const PassArgs& pa, int n_wgs, hipStream_t s) {
  const vsk_model_cfg& c = h.cfg;
  const BatchDev& b = h.bd;
  const WsLayout& wl = pa.wl;
  uint8_t* ws = pa.ws;
  const int d = c.head_dim;
  StepArgs a{};
  a.n_run = h.layers_run > 0 ? h.layers_run : c.n_layers;
  a.n_layers = c.n_layers;
  a.H = c.hidden;
  a.Nq = c.n_q_heads * d;
  a.Nkv = c.n_kv_heads * d;
  a.F = c.ffn;
  a.V = c.vocab;
  a.hd = d;
  a.G = c.n_q_heads / c.n_kv_heads;
  a.Hkv = c.n_kv_heads;
  a.eps = c.rms_eps;
  a.P = h.packed;
  a.layer_bytes = h.pl.layer_bytes;
  a.lo = h.pl.l;
  a.embed = reinterpret_cast<const uint16_t*>(h.packed + h.pl.embed);
  a.lm_head = reinterpret_cast<const u32x4_t*>(h.packed + h.pl.lm_head);
  a.final_gain = reinterpret_cast<const uint16_t*>(h.packed + h.pl.final_norm);
  a.rope = reinterpret_cast<const float2*>(h.packed + h.pl.rope);
  a.pool = h.pool;
  a.n_blocks = h.n_blocks;
  a.R = b.n_rows;
  a.ids = pa.ids;
  a.pos = b.pos;
  a.slot = b.slot;
  a.row_seq = b.row_seq;
  a.block_table = b.block_table;
  a.max_blocks = b.max_blocks;
  a.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(d)));
  a.bps = h.attn_bps > 0 ? h.attn_bps : attn_auto_bps(b.n_rows, c.n_kv_heads);
  a.max_splits = attn_splits(b.max_kv_len, a.bps);
  a.part_o = reinterpret_cast<float*>(ws + wl.att_o);
  a.part_ml = reinterpret_cast<float2*>(ws + wl.att_ml);
  a.att_cnt = reinterpret_cast<int*>(ws + wl.att_cnt);
  a.xs = reinterpret_cast<float*>(ws + wl.s_x);
  a.ssq = reinterpret_cast<double*>(ws + wl.s_ssq);
  a.qs = reinterpret_cast<uint16_t*>(ws + wl.s_q);
  a.os = reinterpret_cast<uint16_t*>(ws + wl.s_o);
  a.as = reinterpret_cast<uint16_t*>(ws + wl.s_a);
  a.ns = reinterpret_cast<uint16_t*>(ws + wl.s_n);
  a.am_val = reinterpret_cast<float*>(ws + wl.s_am);
  a.am_idx = reinterpret_cast<int*>(ws + wl.s_am + static_cast<size_t>(c.vocab / 16) * wl.max_rows * 4);
  a.flags = reinterpret_cast<unsigned*>(ws + wl.s_flags);
  a.err = reinterpret_cast<unsigned*>(ws + wl.s_err);
  a.epoch_ctr = reinterpret_cast<unsigned*>(ws + wl.s_epoch);
  a.x_out = reinterpret_cast<float*>(ws + wl.x);
  a.logits = pa.logits;
  a.next_ids = pa.next_ids;
  a.trace = h.step_trace_cap >= static_cast<size_t>(step_syncs(c.n_layers)) * n_wgs * 2 ? h.step_trace : nullptr;
  hipError_t e = launch_step(a, n_wgs, step_lds_bytes(c), s);
  if (e != hipSuccess) return e;
  h.counters[0] += 1;
  h.counters[1] += 4 * a.n_run + 1;
  h.counters[2] += a.n_run;
  h.counters[3] = a.max_splits;
  h.counters[4] = 1;
  h.counters[5] = 1;
  return hipSuccess;
}

bool step_eligible(Handle& h, const PassArgs& pa) {
  return h.exec_mode == 2 && pa.logit_rows == nullptr && h.bd.max_q_len == 1 && pa.wl.step &&
         h.bd.n_rows <= kStepMaxRows && step_workgroups(h) > 0;
}

hipError_t run_pass(Handle& h, const PassArgs& pa, hipStream_t s) {
  const vsk_model_cfg& c = h.cfg;
  const BatchDev& b = h.bd;
  const WsLayout& wl = pa.wl;
  const int R = b.n_rows;
  // the persistent step kernel serves decode passes of up to 16 rows
  if (step_eligible(h, pa)) return run_step(h, pa, step_workgroups(h), s);
  const int Rg = (R + 15) / 16;
  const int H = c.hidden, F = c.ffn, d = c.head_dim, Nq = c.n_q_heads * d, Nkv = c.n_kv_heads * d;
  uint8_t* ws = pa.ws;
  float* x = reinterpret_cast<float*>(ws + wl.x);
  // frag buffers: A = attention output (O input); B = normalised rows (QKV,
  // gate/up and lm_head input); C = SwiGLU output (down input)
  uint16_t* fa = reinterpret_cast<uint16_t*>(ws + wl.fa);
  uint16_t* fb = reinterpret_cast<uint16_t*>(ws + wl.fb);
  uint16_t* fc = reinterpret_cast<uint16_t*>(ws + wl.fc);
  uint16_t* q = reinterpret_cast<uint16_t*>(ws + wl.q);
  double* ssq = reinterpret_cast<double*>(ws + wl.ssq);
  const uint8_t* P = h.packed;
  typedef uint32_t u4 __attribute__((ext_vector_type(4)));
  const int n_run = h.layers_run > 0 ? h.layers_run : c.n_layers;
  auto norm_gain = [&](int layer, bool mlp) {
    return reinterpret_cast<const uint16_t*>(P + h.pl.layer_bytes * layer + (mlp ? h.pl.l.mlp_norm : h.pl.l.attn_norm));
  };
  const uint16_t* final_gain = reinterpret_cast<const uint16_t*>(P + h.pl.final_norm);
  hipError_t e;
#define TRY(call)                      \
  do {                                 \
    if ((e = (call)) != hipSuccess) return e; \
  } while (0)
  // probed launch of kernel class `cls`: while probe events remain, the
  // launch takes the next pair, bound to its dispatch (the kernel's own start
  // and end times)
  auto probed = [&](int cls, auto&& launch) -> hipError_t {
    LaunchEvents ev;
    if (h.probe_i[cls] < h.probe_b[cls].size()) {
      ev.start = h.probe_b[cls][h.probe_i[cls]];
      ev.stop = h.probe_e[cls][h.probe_i[cls]];
      ++h.probe_i[cls];
    }
    return launch(ev);
  };

  TRY(launch_embed(reinterpret_cast<const uint16_t*>(P + h.pl.embed), pa.ids, R, H, c.vocab, x, ssq, s));
  int ssq_parts = 1;

  GemmArgs ga{};
  ga.R = R;
  ga.Rg = Rg;
  ga.pool = h.pool;
  ga.n_blocks = h.n_blocks;
  ga.Hkv = c.n_kv_heads;
  ga.hd = d;
  ga.Nq = Nq;
  ga.Nkv = Nkv;
  ga.slot = b.slot;
  ga.pos = b.pos;
  ga.rope = reinterpret_cast<const float2*>(P + h.pl.rope);
  ga.x = x;
  ga.out_Rg = Rg;
  ga.xcd_remap = h.xcd_remap;

  AttnArgs aa{};
  aa.q = q;
  aa.pool = h.pool;
  aa.n_blocks = h.n_blocks;
  aa.Hkv = c.n_kv_heads;
  aa.hd = d;
  aa.G = c.n_q_heads / c.n_kv_heads;
  aa.Nq = Nq;
  aa.block_table = b.block_table;
  aa.max_blocks = b.max_blocks;
  aa.row_seq = b.row_seq;
  aa.pos = b.pos;
  aa.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(d)));
  // shared prefixes of a decode pass: read once per group by k_attn_prefix
  const bool cascade = h.shared_prefix != 0 && b.n_pfx_items > 0 && pa.logit_rows == nullptr;
  // the blocks each row of the decode kernel walks (after its shared prefix)
  int blk_min = INT_MAX, blk_max = 0, n_dec = 0;
  {
    const BatchHost& bh = h.bh;
    auto row_blocks = [&](int r) {
      const int nb = (bh.pos[r] + 1 + kBlock - 1) / kBlock - (cascade ? bh.pfx_blocks[r] : 0);
      blk_min = std::min(blk_min, nb);
      blk_max = std::max(blk_max, nb);
      ++n_dec;
    };
    if (h.prefill_attn != 0 && b.n_pre_items > 0 && b.max_kv_len <= kMaxPrefillBlocks * kBlock) {
      for (int32_t r : bh.dec_rows) row_blocks(r);
    } else {
      for (int r = 0; r < R; ++r) row_blocks(r);
    }
  }
  aa.bps = h.attn_bps > 0 ? h.attn_bps : attn_auto_bps(R, c.n_kv_heads);
  // 128..255 (row, KV head) pairs whose walks are within 20% of each other:
  // one split per pair (no merge, and the items are balanced already); a
  // wider spread keeps the split, the longest walk setting the time, and
  // fewer pairs keep it for the parallelism
  const int pairs = n_dec * c.n_kv_heads;
  if (h.attn_bps == 0 && pairs >= 128 && pairs < 256 && 5 * blk_min >= 4 * blk_max)
    aa.bps = std::clamp((blk_max + 7) / 8 * 8, kAttnMinBps, kAttnMaxBps);
  aa.max_splits = attn_splits(b.max_kv_len, aa.bps);
  aa.part_o = reinterpret_cast<float*>(ws + wl.att_o);
  aa.part_ml = reinterpret_cast<float2*>(ws + wl.att_ml);
  aa.counter = reinterpret_cast<int*>(ws + wl.att_cnt);
  aa.out = fa;
  aa.out_Rg = Rg;
  aa.split_stride = aa.max_splits + (cascade ? b.max_pfx_splits : 0);
  aa.pfx_blocks = cascade ? b.pfx_blocks : nullptr;
  aa.pfx_splits = cascade ? b.pfx_splits : nullptr;
  // decode work items launched per (row, KV head): the most splits any
  // decode row has after its shared prefix (the rest would exit at once)
  const int dec_splits = std::max(1, (blk_max + aa.bps - 1) / aa.bps);
  const int pfx_fold = cascade ? b.max_pfx_splits : 0;
  AttnPrefixArgs ap{};
  ap.q = q;
  ap.pool = h.pool;
  ap.n_blocks = h.n_blocks;
  ap.Hkv = c.n_kv_heads;
  ap.G = aa.G;
  ap.Nq = Nq;
  ap.block_table = b.block_table;
  ap.max_blocks = b.max_blocks;
  ap.row_seq = b.row_seq;
  ap.items = b.pfx_items;
  ap.grp_rows = b.grp_rows;
  ap.grp_info = b.grp_info;
  ap.pfx_tbl = b.pfx_tbl;
  ap.scale_log2 = aa.scale_log2;
  ap.split_stride = aa.split_stride;
  ap.part_o = aa.part_o;
  ap.part_ml = aa.part_ml;
  // prefill rows: causal multi-row work items (keys staged per item in LDS)
  const bool prefill = h.prefill_attn != 0 && b.n_pre_items > 0 && b.max_kv_len <= kMaxPrefillBlocks * kBlock;
  AttnPrefillArgs pf{};
  pf.q = q;
  pf.pool = h.pool;
  pf.n_blocks = h.n_blocks;
  pf.Hkv = c.n_kv_heads;
  pf.G = aa.G;
  pf.Nq = Nq;
  pf.block_table = b.block_table;
  pf.max_blocks = b.max_blocks;
  pf.kv_len = b.kv_len;
  pf.pos = b.pos;
  pf.items = b.pre_items;
  pf.scale_log2 = aa.scale_log2;
  pf.out = fa;
  pf.out_Rg = Rg;

  const int rt = h.resid_target;  // -1 no split, 0 the layout's default, else the target
  const GemmPlan p_qkv = plan_gemm(Nq + 2 * Nkv, H, R, EPI_QKV, h.gemm_shape, 0, h.row_tile);
  // QKV of one row tile at 4 or 8 row groups: K split over workgroups of
  // the residual projections' layout (4 or 8 N tiles each instead of 2, so
  // each activation chunk staged in LDS feeds two or four times the weight
  // bytes), the products added by k_qkv_reduce, which applies the epilogue
  GemmPlan p_qkv_split;
  if (h.qkv_target >= 0 && p_qkv.mg >= 4)
    p_qkv_split = plan_gemm(Nq + 2 * Nkv, H, R, EPI_RESID, h.gemm_shape, h.qkv_target > 0 ? h.qkv_target : kQkvTargetWgs);
  const GemmPlan p_o = plan_gemm(H, Nq, R, EPI_RESID, h.gemm_shape, rt, h.row_tile);
  const GemmPlan p_gu = plan_gemm(2 * F, H, R, EPI_SWIGLU, h.gemm_shape, 0, h.row_tile);
  const GemmPlan p_d = plan_gemm(H, F, R, EPI_RESID, h.gemm_shape, rt, h.row_tile);
  float* ypart = reinterpret_cast<float*>(ws + wl.ypart);

  // routed pass (Algorithm 1): the maps of every routed layer, built on the
  // device from the route tape before the first layer; per routed layer the
  // MLP input is written per cohort, the RUN cohort runs the MLP and the
  // Project-Only cohort the projector (count-bounded launches), and one
  // kernel scatters both weighted products into the residual
  const bool routed_pass = pa.tape_run != nullptr;
  const int first_routed = routed_pass ? h.first_routed : c.n_layers;
  const int Fp = h.proj_ffn;
  uint16_t* fb_po = routed_pass ? reinterpret_cast<uint16_t*>(ws + wl.fb_po) : nullptr;
  uint16_t* fc_po = routed_pass ? reinterpret_cast<uint16_t*>(ws + wl.fc_po) : nullptr;
  int32_t* r_run = reinterpret_cast<int32_t*>(ws + wl.r_run);
  int32_t* r_proj = reinterpret_cast<int32_t*>(ws + wl.r_proj);
  int32_t* r_inv = reinterpret_cast<int32_t*>(ws + wl.r_inv);
  int32_t* r_cnt = reinterpret_cast<int32_t*>(ws + wl.r_cnt);
  if (routed_pass) TRY(launch_route_maps(pa.tape_run, c.n_layers - first_routed, R, r_run, r_proj, r_inv, r_cnt, s));
  GemmPlan p_pgu, p_pd;
  if (routed_pass) {
    p_pgu = plan_gemm(2 * Fp, H, R, EPI_SWIGLU, h.gemm_shape, 0, h.row_tile);
    p_pd = plan_gemm(H, Fp, R, EPI_RESID, h.gemm_shape, rt, h.row_tile);
  }
  CohortOut cohort{};  // set for the MLP input of a routed layer

  // RMSNorm: one pass over x using the x^2 partials of the step that wrote it
  auto norm = [&](const uint16_t* gain, const float* xin, int rows, int rg, const double* sq, int parts) {
    return launch_rmsnorm_frags(xin, gain, sq, parts, rows, H, c.rms_eps, fb, rg, s, cohort);
  };
  // a residual projection: in place (x += y, with x^2 partials), or with K
  // split over workgroups and the splits added by k_resid_norm, which also
  // normalises the rows with `next_gain` (null: no norm follows here)
  bool normed = false;  // fb already holds the normalised input of the next projection
  auto resid = [&](int cls, const GemmPlan& p, const uint16_t* next_gain) -> hipError_t {
    hipError_t re;
    if (p.ksplit > 1) {
      ga.ypart = ypart;
      ga.ssq_out = nullptr;
      if ((re = probed(cls, [&](LaunchEvents ev) { return launch_gemm(ga, p, EPI_RESID, s, ev); })) != hipSuccess) return re;
      ga.ypart = nullptr;
      if ((re = launch_resid_norm(x, ypart, p.ksplit, R, H, next_gain, c.rms_eps, fb, Rg, s, cohort)) != hipSuccess)
        return re;
      normed = next_gain != nullptr;
    } else {
      ga.ypart = nullptr;
      ga.ssq_out = ssq;
      if ((re = probed(cls, [&](LaunchEvents ev) { return launch_gemm(ga, p, EPI_RESID, s, ev); })) != hipSuccess) return re;
      ssq_parts = p.n_groups;
      normed = false;
    }
    return hipSuccess;
  };
  ga.X = reinterpret_cast<const u4*>(fb);
  for (int l = 0; l < n_run; ++l) {
    const uint8_t* L = P + h.pl.layer_bytes * l;
    const bool routed = l >= first_routed;
    const int lr = l - first_routed;
    const uint8_t* mask = routed ? pa.tape_run + static_cast<size_t>(lr) * R : nullptr;
    aa.run_mask = mask;
    pf.run_mask = mask;
    // attention block
    if (!normed) TRY(norm(norm_gain(l, false), x, R, Rg, ssq, ssq_parts));
    ga.W = reinterpret_cast<const u4*>(L + h.pl.l.wqkv);
    ga.X = reinterpret_cast<const u4*>(fb);
    ga.Kt = H / 32;
    ga.N = Nq + 2 * Nkv;
    ga.ssq_out = nullptr;
    ga.out = q;
    ga.layer = l;
    if (p_qkv_split.ksplit > 1) {
      ga.ypart = ypart;
      TRY(probed(2, [&](LaunchEvents ev) { return launch_gemm(ga, p_qkv_split, EPI_RESID, s, ev); }));
      TRY(launch_qkv_reduce(ga, p_qkv_split.ksplit, s));
      ga.ypart = nullptr;
    } else {
      TRY(probed(2, [&](LaunchEvents ev) { return launch_gemm(ga, p_qkv, EPI_QKV, s, ev); }));
    }
    aa.layer = l;
    if (cascade) {
      ap.layer = l;
      TRY(launch_attn_prefix(ap, b.n_pfx_items, d, s));
    }
    if (prefill) {
      pf.layer = l;
      TRY(launch_attn_prefill(pf, b.n_pre_items, d, s));
      aa.rows = b.dec_rows;
      if (b.n_dec_rows > 0)
        TRY(probed(4, [&](LaunchEvents ev) { return launch_attn_decode(aa, b.n_dec_rows, dec_splits, pfx_fold, s, ev); }));
    } else if (b.n_pre_items == 0) {
      aa.rows = b.dec_rows;  // every row, longest walk first
      TRY(probed(4, [&](LaunchEvents ev) { return launch_attn_decode(aa, b.n_dec_rows, dec_splits, pfx_fold, s, ev); }));
    } else {
      aa.rows = nullptr;
      TRY(probed(4, [&](LaunchEvents ev) { return launch_attn_decode(aa, R, dec_splits, pfx_fold, s, ev); }));
    }
    // O projection: x += o Wo^T, then the MLP's RMSNorm
    ga.W = reinterpret_cast<const u4*>(L + h.pl.l.wo);
    ga.X = reinterpret_cast<const u4*>(fa);
    ga.Kt = Nq / 32;
    ga.N = H;
    // a routed layer's MLP input goes to its row's cohort, at its position there
    if (routed) cohort = CohortOut{mask, r_inv + static_cast<size_t>(lr) * R, fb_po};
    TRY(resid(3, p_o, norm_gain(l, true)));
    // MLP block
    if (!normed) TRY(norm(norm_gain(l, true), x, R, Rg, ssq, ssq_parts));
    cohort = CohortOut{};
    if (routed) {
      const int32_t* cnt = r_cnt + 2 * lr;
      const uint8_t* Q = h.routed_w + h.routed_layer_bytes * lr;
      const uint16_t* next_gain =
          l + 1 < n_run ? norm_gain(l + 1, false) : (pa.logit_rows == nullptr ? final_gain : nullptr);
      float* y_run = reinterpret_cast<float*>(ws + wl.y_run);
      float* y_po = reinterpret_cast<float*>(ws + wl.y_po);
      ga.ssq_out = nullptr;
      ga.Kt = H / 32;
      // RUN cohort: gate/up + SwiGLU over its n_r rows
      ga.W = reinterpret_cast<const u4*>(L + h.pl.l.wgu);
      ga.X = reinterpret_cast<const u4*>(fb);
      ga.N = 2 * F;
      ga.out = fc;
      ga.count = cnt;
      TRY(probed(0, [&](LaunchEvents ev) { return launch_gemm(ga, p_gu, EPI_SWIGLU, s, ev); }));
      // Project-Only cohort: the projector's gate/up + SwiGLU over its n_p rows
      ga.W = reinterpret_cast<const u4*>(Q + h.routed_pgu);
      ga.X = reinterpret_cast<const u4*>(fb_po);
      ga.N = 2 * Fp;
      ga.out = fc_po;
      ga.count = cnt + 1;
      TRY(launch_gemm(ga, p_pgu, EPI_SWIGLU, s));
      // both down projections store their products (cohort order)
      ga.W = reinterpret_cast<const u4*>(L + h.pl.l.wd);
      ga.X = reinterpret_cast<const u4*>(fc);
      ga.Kt = F / 32;
      ga.N = H;
      ga.ypart = y_run;
      ga.count = cnt;
      TRY(probed(1, [&](LaunchEvents ev) { return launch_gemm(ga, p_d, EPI_RESID, s, ev); }));
      ga.W = reinterpret_cast<const u4*>(Q + h.routed_pd);
      ga.X = reinterpret_cast<const u4*>(fc_po);
      ga.Kt = Fp / 32;
      ga.ypart = y_po;
      ga.count = cnt + 1;
      TRY(launch_gemm(ga, p_pd, EPI_RESID, s));
      ga.ypart = nullptr;
      ga.count = nullptr;
      // x[row] += w * y_run (RUN) or (1 - w) * y_po (Project-Only), then the next norm
      TRY(launch_route_reduce_norm(x, y_run, p_d.ksplit, y_po, p_pd.ksplit, mask, r_inv + static_cast<size_t>(lr) * R,
                                   pa.tape_w + static_cast<size_t>(lr) * R, R, H, next_gain, c.rms_eps, fb, Rg, s));
      normed = next_gain != nullptr;
      continue;
    }
    ga.W = reinterpret_cast<const u4*>(L + h.pl.l.wgu);
    ga.X = reinterpret_cast<const u4*>(fb);
    ga.Kt = H / 32;
    ga.N = 2 * F;
    ga.ssq_out = nullptr;
    ga.out = fc;
    TRY(probed(0, [&](LaunchEvents ev) { return launch_gemm(ga, p_gu, EPI_SWIGLU, s, ev); }));
    // down projection: x += a Wd^T, then the next layer's RMSNorm (or the
    // final one of a decode pass, whose rows all return logits)
    ga.W = reinterpret_cast<const u4*>(L + h.pl.l.wd);
    ga.X = reinterpret_cast<const u4*>(fc);
    ga.Kt = F / 32;
    ga.N = H;
    const uint16_t* next_gain =
        l + 1 < n_run ? norm_gain(l + 1, false) : (pa.logit_rows == nullptr ? final_gain : nullptr);
    TRY(resid(1, p_d, next_gain));
  }
  // final norm over the logit rows, lm_head, greedy argmax
  const int Ro = pa.n_logit_rows;
  const int Rgo = (Ro + 15) / 16;
  if (pa.logit_rows != nullptr) {
    float* x_c = reinterpret_cast<float*>(ws + wl.x_c);
    double* ssq_c = reinterpret_cast<double*>(ws + wl.ssq_c);
    TRY(launch_gather_rows(x, R, pa.logit_rows, Ro, H, x_c, ssq_c, s));
    TRY(norm(final_gain, x_c, Ro, Rgo, ssq_c, 1));
  } else if (!normed) {
    TRY(norm(final_gain, x, Ro, Rgo, ssq, ssq_parts));
  }
  const GemmPlan p_lm = plan_gemm(c.vocab, H, Ro, EPI_LOGITS, h.gemm_shape);
  ga.W = reinterpret_cast<const u4*>(P + h.pl.lm_head);
  ga.X = reinterpret_cast<const u4*>(fb);
  ga.Kt = H / 32;
  ga.N = c.vocab;
  ga.R = Ro;
  ga.Rg = Rgo;
  ga.ssq_out = nullptr;
  ga.out = pa.logits;
  ga.out_Rg = Rgo;
  ga.am_val = reinterpret_cast<float*>(ws + wl.am_part);
  ga.am_idx = reinterpret_cast<int*>(ws + wl.am_part + static_cast<size_t>((c.vocab + 15) / 16) * wl.max_rows * 4);
  TRY(probed(5, [&](LaunchEvents ev) { return launch_gemm(ga, p_lm, EPI_LOGITS, s, ev); }));
  if (pa.next_ids) TRY(launch_argmax_partials(ga.am_val, ga.am_idx, p_lm.n_groups, Ro, pa.next_ids, s));
#undef TRY
  h.counters[0] += 1;
  h.counters[1] += 4 * n_run + 1;
  h.counters[2] += n_run;
  h.counters[3] = aa.max_splits;
  h.counters[4] = p_d.n_groups;
  h.counters[5] = 0;
  return hipSuccess;
}

}  // namespace vsk
