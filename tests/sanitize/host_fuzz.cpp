// Randomised exercise of the library's host code under AddressSanitizer and
// UndefinedBehaviorSanitizer (built by tests/test_host_sanitize.py with g++;
// no GPU code).  It drives the KV block allocator, the batch builder, the
// shared-prefix grouping and the attention work planners with random
// operation sequences, checks their invariants after every step, and runs
// the mode-switch functions on random parameters.  Exit status 0 when every
// check held; a sanitizer report or a failed check ends it with a non-zero
// status.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <random>
#include <set>
#include <string>
#include <vector>

#include "../../paper_2609_37062_amd/csrc/alloc.hpp"
#include "../../include/vsk.h"

using namespace vsk;

#define CHECK(c)                                                          \
  do {                                                                    \
    if (!(c)) {                                                           \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      std::exit(2);                                                       \
    }                                                                     \
  } while (0)

// the allocator's reference counts against the blocks every sequence holds
static void check_refs(const BlockAllocator& a, const std::map<int64_t, bool>& live) {
  std::vector<int32_t> refs(a.n_blocks(), 0);
  for (const auto& kv : live) {
    const SeqState* s = a.find(kv.first);
    CHECK(s != nullptr);
    CHECK(static_cast<int64_t>(s->blocks.size()) * a.block() >= s->len);
    std::set<int32_t> seen;
    for (int32_t b : s->blocks) {
      CHECK(b >= 0 && b < a.n_blocks());
      CHECK(seen.insert(b).second);
      ++refs[b];
    }
  }
  int32_t free_blocks = 0;
  for (int32_t r : refs) free_blocks += r == 0;
  CHECK(free_blocks == a.free_count());
}

static void check_batch(const BlockAllocator& a, const std::vector<int64_t>& seqs, const std::vector<int32_t>& q,
                        const BatchHost& b) {
  CHECK(b.n_seqs == static_cast<int32_t>(seqs.size()));
  int32_t rows = 0;
  for (int32_t x : q) rows += x;
  CHECK(b.n_rows == rows);
  CHECK(static_cast<int32_t>(b.cu_q.size()) == b.n_seqs + 1 && b.cu_q[0] == 0 && b.cu_q[b.n_seqs] == rows);
  std::set<int32_t> slots;
  for (int32_t i = 0; i < b.n_seqs; ++i) {
    const SeqState* s = a.find(seqs[i]);
    CHECK(s != nullptr && b.kv_len[i] == s->len);
    for (int32_t r = b.cu_q[i]; r < b.cu_q[i + 1]; ++r) {
      CHECK(b.row_seq[r] == i);
      const int32_t p = b.pos[r];
      CHECK(p >= 0 && p < s->len);
      CHECK(b.slot[r] == s->blocks[p / a.block()] * a.block() + p % a.block());
      CHECK(slots.insert(b.slot[r]).second);
    }
  }
}

static void check_prefixes(const BatchHost& b, int32_t block) {
  const int32_t ng = b.n_groups();
  for (int32_t g = 0; g < ng; ++g) {
    const int32_t off = b.grp_info[4 * g], n = b.grp_info[4 * g + 1], P = b.grp_info[4 * g + 2],
                  t0 = b.grp_info[4 * g + 3];
    CHECK(n >= 2 && P >= 1);
    for (int32_t k = 0; k < n; ++k) {
      const int32_t r = b.grp_rows[off + k];
      CHECK(b.pfx_blocks[r] == P);
      const int32_t seq = b.row_seq[r];
      CHECK(P * block <= b.pos[r]);  // the prefix lies wholly before the current token
      for (int32_t j = 0; j < P; ++j) CHECK(b.block_table[static_cast<size_t>(seq) * b.max_blocks + j] == b.pfx_tbl[t0 + j]);
    }
  }
}

int main(int argc, char** argv) {
  const int iters = argc > 1 ? std::atoi(argv[1]) : 300;
  std::mt19937_64 rng(12345);
  auto uni = [&](int lo, int hi) { return static_cast<int>(std::uniform_int_distribution<int>(lo, hi)(rng)); };
  std::string err;
  long n_passes = 0, n_groups = 0, n_pfx_items = 0, n_pre_items = 0;
  for (int it = 0; it < iters; ++it) {
    const int32_t n_blocks = uni(8, 160);
    BlockAllocator a(n_blocks, 16);
    std::map<int64_t, bool> live;
    int64_t next_id = 0;
    for (int op = 0; op < 60; ++op) {
      const int kind = uni(0, 6);
      if (kind == 6) {  // a group: a source of 64..200 tokens and 2..5 sequences sharing whole blocks of it
        const int64_t src = next_id++;
        CHECK(a.seq_create(src, err) == kOk);
        live[src] = true;
        const int32_t ctx = uni(64, 200);
        std::vector<int32_t> sl(ctx);
        if (a.reserve(src, ctx, sl.data(), err) != kOk) continue;
        const int32_t shared = 16 * uni(1, (ctx - 1) / 16);
        for (int k = uni(2, 5); k > 0; --k) {
          const int64_t id = next_id++;
          CHECK(a.seq_create(id, err) == kOk);
          live[id] = true;
          CHECK(a.seq_share_prefix(id, src, shared, err) == kOk);
        }
        check_refs(a, live);
        continue;
      }
      if (kind == 0 || live.empty()) {  // create, optionally with a chosen table
        const int64_t id = next_id++;
        CHECK(a.seq_create(id, err) == kOk);
        live[id] = true;
        if (uni(0, 1)) {
          const int32_t ctx = uni(0, 80);
          const int32_t nb = (ctx + 15) / 16;
          std::vector<int32_t> blocks;
          std::set<int32_t> used;
          while (static_cast<int32_t>(blocks.size()) < nb && static_cast<int32_t>(used.size()) < n_blocks) {
            const int32_t b = uni(0, n_blocks - 1);
            if (used.insert(b).second) blocks.push_back(b);
          }
          const int rc = a.seq_set_blocks(id, blocks.data(), static_cast<int32_t>(blocks.size()), ctx, err);
          CHECK(rc == kOk || rc == kErrArg);
        }
      } else if (kind == 1) {  // reserve new tokens (all-or-nothing)
        auto itr = live.begin();
        std::advance(itr, uni(0, static_cast<int>(live.size()) - 1));
        const int32_t n_new = uni(0, 40);
        std::vector<int32_t> slots(n_new > 0 ? n_new : 1);
        const int32_t free_before = a.free_count();
        const int32_t len_before = a.find(itr->first)->len;
        const int rc = a.reserve(itr->first, n_new, slots.data(), err);
        if (rc != kOk) {
          CHECK(a.free_count() == free_before && a.find(itr->first)->len == len_before);
        } else {
          CHECK(a.find(itr->first)->len == len_before + n_new);
        }
      } else if (kind == 2) {  // release
        auto itr = live.begin();
        std::advance(itr, uni(0, static_cast<int>(live.size()) - 1));
        CHECK(a.seq_release(itr->first, err) == kOk);
        live.erase(itr);
      } else if (kind == 3 && live.size() >= 1) {  // share a prefix into a fresh sequence
        auto itr = live.begin();
        std::advance(itr, uni(0, static_cast<int>(live.size()) - 1));
        const int64_t id = next_id++;
        CHECK(a.seq_create(id, err) == kOk);
        live[id] = true;
        const int32_t n_tok = uni(0, 3) == 0 ? uni(0, 40) : uni(48, 160);
        const int rc = a.seq_share_prefix(id, itr->first, n_tok, err);
        CHECK(rc == kOk || rc == kErrArg || rc == kErrRange || rc == kErrState);
      } else {  // a pass over some sequences: build, group, plan
        // as a serving step does: reserve each row's new token(s), then
        // build the pass over them (the rows' slots are then exclusive)
        std::vector<int64_t> seqs;
        std::vector<int32_t> q;
        std::vector<int32_t> reserved;
        for (const auto& kv : live) {
          if (uni(0, 2) == 0) continue;
          const int32_t n_new = uni(0, 3) == 0 ? uni(1, 5) : 1;
          std::vector<int32_t> sl(n_new);
          if (a.reserve(kv.first, n_new, sl.data(), err) != kOk) continue;
          seqs.push_back(kv.first);
          q.push_back(n_new);
          reserved.insert(reserved.end(), sl.begin(), sl.end());
        }
        if (seqs.empty()) continue;
        BatchHost b;
        const int rc = build_batch(a, seqs.data(), q.data(), static_cast<int32_t>(seqs.size()), b, err);
        CHECK(rc == kOk);
        check_batch(a, seqs, q, b);
        for (int32_t r = 0; r < b.n_rows; ++r) CHECK(b.slot[r] == reserved[r]);
        bool decode = true;
        for (int32_t x : q) decode = decode && x == 1;
        ++n_passes;
        if (decode) {
          find_shared_prefixes(b, 16, uni(1, 4));
          check_prefixes(b, 16);
          plan_prefix_items(b, uni(1, 8), uni(1, 8), uni(1, 400));
          n_groups += b.n_groups();
          n_pfx_items += b.n_pfx_items();
          for (int32_t i = 0; i < b.n_pfx_items(); ++i) {
            const int32_t* itm = &b.pfx_items[5 * i];
            CHECK(itm[0] >= 0 && itm[0] < b.n_groups());
            CHECK(itm[2] >= 0 && itm[2] < itm[3] && itm[3] <= b.grp_info[4 * itm[0] + 2]);
            CHECK(itm[4] >= 0 && itm[4] < b.max_pfx_splits);
          }
        }
        plan_prefill_items(b, uni(1, 8), 16);
        n_pre_items += b.n_pre_items();
        int32_t covered = 0;
        for (int32_t i = 0; i < b.n_pre_items(); ++i) covered += b.pre_items[3 * i + 2];
        CHECK(covered + static_cast<int32_t>(b.dec_rows.size()) == b.n_rows);
      }
      check_refs(a, live);
    }
  }
  // the mode switch on random parameters: bands ordered, steps consistent
  for (int it = 0; it < 2000; ++it) {
    vsk_switch_params p{};
    p.tau_s = std::uniform_real_distribution<double>(1e-4, 5e-3)(rng);
    p.tau_layers = uni(1, 40);
    p.bw_bytes_per_s = std::uniform_real_distribution<double>(1e12, 8e12)(rng);
    p.skip = std::uniform_real_distribution<double>(0.05, 1.0)(rng);
    p.routed_layers = uni(1, 40);
    p.kv_bytes_per_token_layer = uni(1, 8) * 1024.0;
    p.enter_factor = std::uniform_real_distribution<double>(1.0, 2.0)(rng);
    p.round_tokens = uni(0, 3) * 5000.0;
    vsk_switch_band band{};
    if (vsk_switch_thresholds(&p, &band) != VSK_OK) continue;
    CHECK(std::isfinite(band.v_star) && band.v_star > 0);
    CHECK(band.exit_tokens <= band.enter_tokens);
    int32_t routing = uni(0, 1), out = 0, promote = 0;
    for (int k = 0; k < 20; ++k) {
      const int64_t V = std::uniform_int_distribution<int64_t>(0, 3 * band.enter_tokens + 1)(rng);
      CHECK(vsk_switch_step(&band, routing, V, &out, &promote) == VSK_OK);
      if (V >= band.enter_tokens) CHECK(out == 1);  // (entering wins where exit == enter)
      else if (V <= band.exit_tokens) CHECK(out == 0);
      else CHECK(out == routing);
      routing = out;
    }
  }
  std::printf("host fuzz: %d allocator runs, %ld passes, %ld prefix groups, %ld prefix items, %ld prefill items; "
              "switch checks passed\n", iters, n_passes, n_groups, n_pfx_items, n_pre_items);
  return 0;
}
