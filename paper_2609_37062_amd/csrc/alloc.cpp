// Host-side KV block allocator and batch metadata builder (see alloc.hpp).
#include "alloc.hpp"

#include <climits>
#include <map>

#include <algorithm>
#include <unordered_set>

namespace vsk {

BlockAllocator::BlockAllocator(int32_t n_blocks, int32_t block)
    : block_(block), ref_(static_cast<size_t>(n_blocks > 0 ? n_blocks : 0), 0),
      free_count_(n_blocks > 0 ? n_blocks : 0) {}

const SeqState* BlockAllocator::find(int64_t seq) const {
  auto it = seqs_.find(seq);
  return it == seqs_.end() ? nullptr : &it->second;
}

int32_t BlockAllocator::next_free(int32_t from) const {
  for (int32_t b = from; b < n_blocks(); ++b)
    if (ref_[b] == 0) return b;
  return -1;
}

int BlockAllocator::seq_create(int64_t seq, std::string& err) {
  if (seqs_.count(seq)) {
    err = "sequence " + std::to_string(seq) + " already exists";
    return kErrState;
  }
  seqs_.emplace(seq, SeqState{});
  return kOk;
}

int BlockAllocator::seq_release(int64_t seq, std::string& err) {
  auto it = seqs_.find(seq);
  if (it == seqs_.end()) {
    err = "unknown sequence " + std::to_string(seq);
    return kErrState;
  }
  for (int32_t b : it->second.blocks) {
    if (--ref_[b] == 0) ++free_count_;
  }
  seqs_.erase(it);
  return kOk;
}

int BlockAllocator::seq_set_blocks(int64_t seq, const int32_t* blocks, int32_t n, int32_t ctx_len,
                                   std::string& err) {
  auto it = seqs_.find(seq);
  if (it == seqs_.end()) {
    err = "unknown sequence " + std::to_string(seq);
    return kErrState;
  }
  if (!it->second.blocks.empty() || it->second.len != 0) {
    err = "sequence already holds blocks";
    return kErrState;
  }
  if (n < 0 || ctx_len < 0 || static_cast<int64_t>(n) * block_ < ctx_len || (n > 0 && !blocks)) {
    err = "block table shorter than the context";
    return kErrArg;
  }
  std::unordered_set<int32_t> seen;
  for (int32_t i = 0; i < n; ++i) {
    if (blocks[i] < 0 || blocks[i] >= n_blocks()) {
      err = "block id " + std::to_string(blocks[i]) + " outside the pool";
      return kErrRange;
    }
    if (!seen.insert(blocks[i]).second) {
      err = "block listed twice";
      return kErrArg;
    }
  }
  for (int32_t i = 0; i < n; ++i) {
    if (ref_[blocks[i]]++ == 0) --free_count_;
  }
  it->second.blocks.assign(blocks, blocks + n);
  it->second.len = ctx_len;
  return kOk;
}

int BlockAllocator::seq_share_prefix(int64_t dst, int64_t src, int32_t n_tokens, std::string& err) {
  auto d = seqs_.find(dst);
  auto s = seqs_.find(src);
  if (d == seqs_.end() || s == seqs_.end()) {
    err = "unknown sequence";
    return kErrState;
  }
  if (!d->second.blocks.empty() || d->second.len != 0) {
    err = "destination sequence not empty";
    return kErrState;
  }
  if (n_tokens < 0 || n_tokens % block_ != 0 || n_tokens > s->second.len) {
    err = "shared prefix must be block aligned and resident";
    return kErrArg;
  }
  const int32_t nb = n_tokens / block_;
  d->second.blocks.assign(s->second.blocks.begin(), s->second.blocks.begin() + nb);
  for (int32_t b : d->second.blocks) ++ref_[b];
  d->second.len = n_tokens;
  return kOk;
}

int BlockAllocator::reserve(int64_t seq, int32_t n_new, int32_t* slots_out, std::string& err) {
  auto it = seqs_.find(seq);
  if (it == seqs_.end()) {
    err = "unknown sequence " + std::to_string(seq);
    return kErrState;
  }
  if (n_new < 0) {
    err = "negative count";
    return kErrArg;
  }
  SeqState& s = it->second;
  const int32_t L = s.len;
  const int32_t have = static_cast<int32_t>(s.blocks.size());
  const int32_t need_blocks = (L + n_new + block_ - 1) / block_;
  const int32_t extra = std::max(0, need_blocks - have);
  // positions are checked in order: those in already-held blocks come first
  for (int32_t p = L; p < L + n_new; ++p) {
    const int32_t bi = p / block_;
    if (bi >= have) break;
    if (ref_[s.blocks[bi]] > 1) {
      err = "position " + std::to_string(p) + " falls in shared block " + std::to_string(s.blocks[bi]);
      return kErrSharedWrite;
    }
  }
  if (extra > free_count_) {
    err = "KV pool exhausted: need " + std::to_string(extra) + " blocks, " +
          std::to_string(free_count_) + " free";
    return kErrNomem;
  }
  // commit: take the lowest free ids
  int32_t cursor = 0;
  for (int32_t e = 0; e < extra; ++e) {
    const int32_t b = next_free(cursor);
    ref_[b] = 1;
    --free_count_;
    s.blocks.push_back(b);
    cursor = b + 1;
  }
  if (slots_out) {
    for (int32_t p = L; p < L + n_new; ++p)
      slots_out[p - L] = s.blocks[p / block_] * block_ + p % block_;
  }
  s.len = L + n_new;
  return kOk;
}

int build_batch(const BlockAllocator& a, const int64_t* seqs, const int32_t* q_lens, int32_t n,
                BatchHost& out, std::string& err) {
  if (n <= 0 || !seqs || !q_lens) {
    err = "empty batch";
    return kErrArg;
  }
  BatchHost b;
  b.n_seqs = n;
  b.cu_q.assign(static_cast<size_t>(n) + 1, 0);
  b.kv_len.resize(n);
  std::unordered_set<int64_t> seen;
  int32_t max_blocks = 1;
  for (int32_t i = 0; i < n; ++i) {
    const SeqState* s = a.find(seqs[i]);
    if (!s) {
      err = "unknown sequence " + std::to_string(seqs[i]);
      return kErrState;
    }
    if (!seen.insert(seqs[i]).second) {
      err = "sequence listed twice in one pass";
      return kErrArg;
    }
    if (q_lens[i] < 1 || q_lens[i] > s->len) {
      err = "rows of a sequence must be 1..resident length";
      return kErrArg;
    }
    b.kv_len[i] = s->len;
    b.cu_q[i + 1] = b.cu_q[i] + q_lens[i];
    max_blocks = std::max<int32_t>(max_blocks, static_cast<int32_t>(s->blocks.size()));
    b.max_kv_len = std::max(b.max_kv_len, s->len);
    b.max_q_len = std::max(b.max_q_len, q_lens[i]);
  }
  b.max_blocks = max_blocks;
  b.n_rows = b.cu_q[n];
  b.block_table.assign(static_cast<size_t>(n) * max_blocks, -1);
  b.row_seq.resize(b.n_rows);
  b.pos.resize(b.n_rows);
  b.slot.resize(b.n_rows);
  const int32_t bs = a.block();
  for (int32_t i = 0; i < n; ++i) {
    const SeqState* s = a.find(seqs[i]);
    std::copy(s->blocks.begin(), s->blocks.end(), b.block_table.begin() + static_cast<size_t>(i) * max_blocks);
    for (int32_t r = b.cu_q[i]; r < b.cu_q[i + 1]; ++r) {
      const int32_t p = s->len - (b.cu_q[i + 1] - r);
      b.row_seq[r] = i;
      b.pos[r] = p;
      b.slot[r] = s->blocks[p / bs] * bs + p % bs;
    }
  }
  b.pfx_blocks.assign(b.n_rows, 0);
  if (b.max_q_len == 1) find_shared_prefixes(b, bs);
  out = std::move(b);
  return kOk;
}

void plan_prefix_items(BatchHost& b, int32_t group_size, int32_t n_kv_heads, int32_t target_wgs) {
  b.pfx_splits.assign(b.n_rows, 0);
  b.pfx_items.clear();
  b.max_pfx_splits = 0;
  const int32_t ng = b.n_groups();
  if (ng == 0) return;
  auto cdiv = [](int32_t x, int32_t y) { return (x + y - 1) / y; };
  int32_t chunks = 0;
  for (int32_t g = 0; g < ng; ++g) chunks += cdiv(b.grp_info[4 * g + 1] * group_size, kPfxCols);
  const int32_t want = std::max(1, cdiv(target_wgs, chunks * n_kv_heads));
  for (int32_t g = 0; g < ng; ++g) {
    const int32_t off = b.grp_info[4 * g], rows = b.grp_info[4 * g + 1], P = b.grp_info[4 * g + 2];
    const int32_t lo = cdiv(P, kMaxPfxBps), hi = std::min(kMaxPfxSplits, std::max(1, P / 2));
    int32_t splits = std::max(lo, std::min(want, hi));
    const int32_t bps = cdiv(P, splits);
    splits = cdiv(P, bps);
    b.max_pfx_splits = std::max(b.max_pfx_splits, splits);
    for (int32_t k = 0; k < rows; ++k) b.pfx_splits[b.grp_rows[off + k]] = splits;
    for (int32_t c0 = 0; c0 < rows * group_size; c0 += kPfxCols)
      for (int32_t sp = 0; sp < splits; ++sp) {
        const int32_t it[5] = {g, c0, sp * bps, std::min(P, (sp + 1) * bps), sp};
        b.pfx_items.insert(b.pfx_items.end(), it, it + 5);
      }
  }
}

void plan_prefill_items(BatchHost& b, int32_t group_size, int32_t block) {
  b.pre_items.clear();
  b.dec_rows.clear();
  const int32_t per = std::max(1, kPreCols / group_size);
  for (int32_t i = 0; i < b.n_seqs; ++i) {
    const int32_t r0 = b.cu_q[i], r1 = b.cu_q[i + 1];
    if (r1 - r0 == 1) {
      b.dec_rows.push_back(r0);
      continue;
    }
    for (int32_t r = r0; r < r1; r += per) {
      const int32_t it[3] = {i, r, std::min(per, r1 - r)};
      b.pre_items.insert(b.pre_items.end(), it, it + 3);
    }
  }
  // prefill items too in order of their walks (the blocks up to their last
  // row), longest first, ties in build order: the launch dispatches an
  // item's KV heads together, so the longest items start in the first round
  {
    const int32_t n = b.n_pre_items();
    std::vector<int32_t> order(n);
    for (int32_t k = 0; k < n; ++k) order[k] = k;
    auto blocks = [&](int32_t k) { return b.pos[b.pre_items[3 * k + 1] + b.pre_items[3 * k + 2] - 1] / block + 1; };
    std::stable_sort(order.begin(), order.end(), [&](int32_t x, int32_t y) { return blocks(x) > blocks(y); });
    std::vector<int32_t> sorted(b.pre_items.size());
    for (int32_t k = 0; k < n; ++k)
      for (int32_t j = 0; j < 3; ++j) sorted[3 * k + j] = b.pre_items[3 * order[k] + j];
    b.pre_items.swap(sorted);
  }
  // longest remaining walk first, ties in row order
  auto walk = [&](int32_t r) { return (b.pos[r] + block) / block - b.pfx_blocks[r]; };
  std::stable_sort(b.dec_rows.begin(), b.dec_rows.end(), [&](int32_t x, int32_t y) { return walk(x) > walk(y); });
}

void find_shared_prefixes(BatchHost& b, int32_t block, int32_t min_blocks) {
  b.pfx_blocks.assign(b.n_rows, 0);
  b.grp_rows.clear();
  b.grp_info.clear();
  b.pfx_tbl.clear();
  if (b.max_q_len != 1) return;
  // sequences by first block, in sequence order
  std::map<int32_t, std::vector<int32_t>> by_first;
  for (int32_t i = 0; i < b.n_seqs; ++i) {
    const int32_t full = (b.kv_len[i] - 1) / block;  // blocks before the current token's block
    if (full >= min_blocks) by_first[b.block_table[static_cast<size_t>(i) * b.max_blocks]].push_back(i);
  }
  for (const auto& kv : by_first) {
    const std::vector<int32_t>& m = kv.second;
    if (m.size() < 2) continue;
    int32_t lim = INT32_MAX;
    for (int32_t i : m) lim = std::min(lim, (b.kv_len[i] - 1) / block);
    const int32_t* t0 = b.block_table.data() + static_cast<size_t>(m[0]) * b.max_blocks;
    int32_t p = 0;
    for (; p < lim; ++p) {
      bool same = true;
      for (size_t k = 1; k < m.size() && same; ++k)
        same = b.block_table[static_cast<size_t>(m[k]) * b.max_blocks + p] == t0[p];
      if (!same) break;
    }
    if (p < min_blocks) continue;
    b.grp_info.push_back(static_cast<int32_t>(b.grp_rows.size()));
    b.grp_info.push_back(static_cast<int32_t>(m.size()));
    b.grp_info.push_back(p);
    b.grp_info.push_back(static_cast<int32_t>(b.pfx_tbl.size()));
    b.pfx_tbl.insert(b.pfx_tbl.end(), t0, t0 + p);
    for (int32_t i : m) {
      const int32_t r = b.cu_q[i];  // the sequence's one row
      b.grp_rows.push_back(r);
      b.pfx_blocks[r] = p;
    }
  }
}

}  // namespace vsk
