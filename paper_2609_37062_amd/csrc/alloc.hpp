// Host-side KV block allocator and per-pass batch metadata.
//
// Paged KV bookkeeping of the serving engine (paper, "Invariants for
// Correct Mixed-Depth Execution"): position t of a sequence lives at slot
// table[t/16]*16 + t%16 of every layer's cache (Invariant 1 keeps every
// layer's own K,V there) and the row-to-slot maps are rebuilt from the
// current row set for every pass (Invariant 2).  Plain C++17, no HIP.
#pragma once

#include <cstdint>
#include <string>
#include <unordered_map>
#include <vector>

namespace vsk {

enum Status : int {
  kOk = 0,
  kErrArg = -1,
  kErrNomem = -2,
  kErrRange = -3,
  kErrSharedWrite = -4,
  kErrState = -5,
  kErrHip = -6,
  kErrUnsupported = -7,
};

struct SeqState {
  std::vector<int32_t> blocks;
  int32_t len = 0;
};

// Reference-counted block pool.  Free blocks are handed out lowest id first.
// Every mutating call is all-or-nothing: on error the state is unchanged and
// `err` says why.
class BlockAllocator {
 public:
  BlockAllocator() = default;
  explicit BlockAllocator(int32_t n_blocks, int32_t block = 16);

  int seq_create(int64_t seq, std::string& err);
  int seq_release(int64_t seq, std::string& err);
  int seq_set_blocks(int64_t seq, const int32_t* blocks, int32_t n, int32_t ctx_len, std::string& err);
  int seq_share_prefix(int64_t dst, int64_t src, int32_t n_tokens, std::string& err);
  int reserve(int64_t seq, int32_t n_new, int32_t* slots_out, std::string& err);

  const SeqState* find(int64_t seq) const;
  int32_t n_blocks() const { return static_cast<int32_t>(ref_.size()); }
  int32_t block() const { return block_; }
  int32_t free_count() const { return free_count_; }

 private:
  // lowest free block id at or after `from`, or -1
  int32_t next_free(int32_t from) const;
  int32_t block_ = 16;
  std::vector<int32_t> ref_;
  int32_t free_count_ = 0;
  std::unordered_map<int64_t, SeqState> seqs_;
};

// Host copy of one pass's metadata (see vsk_batch_build in vsk.h).
struct BatchHost {
  int32_t n_seqs = 0, n_rows = 0, max_blocks = 0, max_kv_len = 0, max_q_len = 0;
  std::vector<int32_t> block_table;  // [n_seqs][max_blocks]
  std::vector<int32_t> kv_len;       // [n_seqs]
  std::vector<int32_t> cu_q;         // [n_seqs + 1]
  std::vector<int32_t> row_seq;      // [n_rows]
  std::vector<int32_t> pos;          // [n_rows]
  std::vector<int32_t> slot;         // [n_rows]
  // Shared prefixes of a decode pass: groups of sequences whose tables start
  // with the same full blocks before each member's current token.
  std::vector<int32_t> pfx_blocks;   // [n_rows] blocks of the row's group prefix (0: none)
  std::vector<int32_t> grp_rows;     // rows of every group, group by group
  std::vector<int32_t> grp_info;     // [n_groups][4]: first entry in grp_rows, rows, prefix blocks, first entry in pfx_tbl
  std::vector<int32_t> pfx_tbl;      // every group's prefix block ids, group by group
  int32_t n_groups() const { return static_cast<int32_t>(grp_info.size() / 4); }
  // Work items of the shared-prefix attention (plan_prefix_items)
  std::vector<int32_t> pfx_splits;   // [n_rows] prefix splits of the row's group (0: none)
  std::vector<int32_t> pfx_items;    // [n_items][5]: group, first column, first block, end block, split
  int32_t max_pfx_splits = 0;
  int32_t n_pfx_items() const { return static_cast<int32_t>(pfx_items.size() / 5); }
  // Attention work of a pass with prefill rows (plan_prefill_items)
  std::vector<int32_t> pre_items;    // [n][3]: sequence, first row, rows -- runs of a sequence's new rows
  std::vector<int32_t> dec_rows;     // rows of one-row sequences, longest walk first
  int32_t n_pre_items() const { return static_cast<int32_t>(pre_items.size() / 3); }
};

// Attention work items.  Each sequence with more than one new row has its
// rows cut into runs of at most kPreCols / group_size rows (one
// causal-attention work item each).  The rows of one-row sequences (every
// row of a decode pass) are listed for the decode attention, ordered by the
// blocks each reads after its shared prefix, most first (ties in row order):
// the decode grid dispatches its rows in that order, so the longest walks
// start first instead of finishing last.
void plan_prefill_items(BatchHost& b, int32_t group_size, int32_t block);

// Columns (row, query head) of one shared-prefix work item: 4 tiles of 16,
// each walked by two waves; of one prefill work item: 8 tiles of 16.
constexpr int32_t kPfxCols = 64;
constexpr int32_t kPreCols = 128;
// Most prefix splits of one group, and the largest split (blocks).
constexpr int32_t kMaxPfxSplits = 16;
constexpr int32_t kMaxPfxBps = 512;
// Split every group's prefix so that the work items of all groups and KV
// heads come to about target_wgs workgroups (at least 2 blocks per split).
void plan_prefix_items(BatchHost& b, int32_t group_size, int32_t n_kv_heads, int32_t target_wgs = 192);

// Smallest common prefix (in blocks) worth reading once for a group.
constexpr int32_t kMinSharedPrefixBlocks = 4;
// Fill the shared-prefix fields of a decode pass (one row per sequence):
// sequences are grouped by their first block; a group's prefix is the
// longest run of leading blocks that every member holds and that lies
// wholly before every member's current token.  Groups of one sequence and
// prefixes shorter than min_blocks are dropped.
void find_shared_prefixes(BatchHost& b, int32_t block, int32_t min_blocks = kMinSharedPrefixBlocks);

int build_batch(const BlockAllocator& a, const int64_t* seqs, const int32_t* q_lens, int32_t n,
                BatchHost& out, std::string& err);

}  // namespace vsk
