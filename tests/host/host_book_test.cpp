// CPU tests of the host bookkeeping (paper_2606_12243_amd/csrc/host_book.cpp):
// the paged block allocator, window validation, row plans with lag rows and
// tree masks, commit validation, tree-compaction moves and the commit itself.
// Built with -fsanitize=address,undefined by tests/test_host_book.py.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "host_book.h"

using namespace via;

static int g_fail = 0;
#define CHECK(c)                                                          \
  do {                                                                    \
    if (!(c)) {                                                           \
      std::printf("FAIL %s:%d: %s (%s)\n", __FILE__, __LINE__, #c, last_error()); \
      ++g_fail;                                                           \
    }                                                                     \
  } while (0)

static const int V = 100;

// A window built from plain vectors (chain unless parents are given).
struct Win {
  std::vector<int32_t> seq, n_rows, row_tok, row_depth, n_drafts, draft_tok, draft_row, draft_parent, n_lag,
      lag_tok;
  std::vector<uint64_t> row_mask;
  via_window w{};
  void finish(int max_rows, int max_drafts, int max_lag, bool tree) {
    w.batch = (int)seq.size();
    w.max_rows = max_rows;
    w.max_drafts = max_drafts;
    w.max_lag = max_lag;
    w.seq_id = seq.data();
    w.n_rows = n_rows.data();
    w.row_tok = row_tok.data();
    w.row_depth = tree ? row_depth.data() : nullptr;
    w.row_mask = tree ? row_mask.data() : nullptr;
    w.n_drafts = n_drafts.data();
    w.draft_tok = draft_tok.data();
    w.draft_row = draft_row.data();
    w.draft_parent = tree ? draft_parent.data() : nullptr;
    w.n_lag = n_lag.empty() ? nullptr : n_lag.data();
    w.lag_tok = lag_tok.empty() ? nullptr : lag_tok.data();
  }
};

// Chain window: per sequence k drafts, rows [pending, d0..d_{k-2}].
static Win chain(const std::vector<int>& seqs, int k, int max_drafts = 8) {
  Win c;
  for (int s : seqs) {
    c.seq.push_back(s);
    c.n_rows.push_back(k);
    c.n_drafts.push_back(k);
    for (int r = 0; r < k; ++r) c.row_tok.push_back((s * 7 + r) % V);
    for (int r = k; r < k; ++r) c.row_tok.push_back(0);
    for (int j = 0; j < max_drafts; ++j) {
      c.draft_tok.push_back(j < k ? (s * 11 + j) % V : 0);
      c.draft_row.push_back(j < k ? j : 0);
    }
  }
  c.finish(k, max_drafts, 1, false);
  return c;
}

static bool owned_once(const KvBook& bk, int cache, int n_blocks) {
  std::vector<int> seen(n_blocks, 0);
  for (const SeqSt& S : bk.seqs)
    for (int b : S.table[cache]) {
      if (b < 0 || b >= n_blocks || seen[b]++) return false;
    }
  for (int b : bk.free_[cache]) {
    if (b < 0 || b >= n_blocks || seen[b]++) return false;
  }
  for (int v : seen)
    if (v != 1) return false;
  return true;
}

static void attach(KvBook& bk, int seq, int n) {
  bk.seqs[seq] = SeqSt();
  bk.seqs[seq].on = true;
  CHECK(book_alloc(bk, 0, {{seq, n}}, nullptr) == VIA_OK);
  CHECK(book_alloc(bk, 1, {{seq, n}}, nullptr) == VIA_OK);
  bk.seqs[seq].valid[0] = bk.seqs[seq].valid[1] = n;
}

static void test_allocator() {
  KvBook bk;
  book_init(bk, 3, 4, 8, 8);
  CHECK(book_alloc(bk, 0, {{0, 20}, {1, 16}}, nullptr) == VIA_OK);  // seq 0: 2 blocks, seq 1: 1
  CHECK((bk.seqs[0].table[0] == std::vector<int>{0, 1}) && (bk.seqs[1].table[0] == std::vector<int>{2}));
  book_trim(bk, 0, 0, 16);  // keeps block 0
  CHECK(bk.seqs[0].table[0] == std::vector<int>{0});
  CHECK(book_alloc(bk, 0, {{1, 48}}, nullptr) == VIA_OK);  // lowest free first: 1, 3
  CHECK((bk.seqs[1].table[0] == std::vector<int>{2, 1, 3}));
  // more than max_blocks_per_seq (4) or more than the pool holds: nothing taken
  KvBook before = bk;
  CHECK(book_alloc(bk, 0, {{0, 16 * 5}}, nullptr) == VIA_ENOMEM);
  CHECK(book_alloc(bk, 0, {{0, 64}, {2, 64}}, nullptr) == VIA_ENOMEM);  // 3 + 4 > 4 free
  CHECK(bk.seqs[0].table[0] == before.seqs[0].table[0] && bk.free_[0] == before.free_[0]);
  // release_taken undoes exactly what an allocation took
  std::vector<std::pair<int, int>> taken;
  CHECK(book_alloc(bk, 0, {{0, 40}, {2, 30}}, &taken) == VIA_OK);
  CHECK(taken.size() == 4);
  book_release_taken(bk, 0, taken);
  CHECK(bk.seqs[0].table[0] == before.seqs[0].table[0] && bk.seqs[2].table[0].empty());
  CHECK(bk.free_[0] == before.free_[0]);
  CHECK(owned_once(bk, 0, 8) && owned_once(bk, 1, 8));
}

static void test_window_validation() {
  KvBook bk;
  book_init(bk, 4, 8, 32, 32);
  attach(bk, 0, 10);
  attach(bk, 2, 33);
  WinCopy c;
  Win ok = chain({0, 2}, 4);
  CHECK(copy_window(bk, &ok.w, V, 4, 8, c) == VIA_OK);
  CHECK(c.batch == 2 && c.seq[1] == 2 && c.draft_tok[8 + 3] == (2 * 11 + 3) % V && !c.tree);
  CHECK(copy_window(bk, nullptr, V, 4, 8, c) == VIA_EINVAL);
  {
    Win w = chain({0, 1}, 4);  // 1 not attached
    CHECK(copy_window(bk, &w.w, V, 4, 8, c) == VIA_EINVAL);
  }
  {
    Win w = chain({0, 0}, 4);  // repeated
    CHECK(copy_window(bk, &w.w, V, 4, 8, c) == VIA_EINVAL);
  }
  {
    Win w = chain({0}, 4);
    CHECK(copy_window(bk, &w.w, V, 0, 8, c) == VIA_EINVAL);  // batch above max_batch
    CHECK(copy_window(bk, &w.w, V, 4, 4, c) == VIA_EINVAL);  // strides above the handle's max_drafts
  }
  {
    Win w = chain({0}, 4);
    w.row_tok[1] = V;  // token out of range
    CHECK(copy_window(bk, &w.w, V, 4, 8, c) == VIA_EINVAL);
  }
  {
    Win w = chain({0}, 4);
    w.draft_tok[2] = -1;
    CHECK(copy_window(bk, &w.w, V, 4, 8, c) == VIA_EINVAL);
  }
  {
    Win w = chain({0}, 4);
    w.draft_row[2] = 1;  // chain draft j must be verified by row j
    CHECK(copy_window(bk, &w.w, V, 4, 8, c) == VIA_EINVAL);
  }
  {
    Win w = chain({0}, 4);
    w.n_rows[0] = 5;  // more rows than the stride
    CHECK(copy_window(bk, &w.w, V, 4, 8, c) == VIA_EINVAL);
  }
  {
    Win w = chain({0}, 4);
    w.w.draft_tok = nullptr;
    CHECK(copy_window(bk, &w.w, V, 4, 8, c) == VIA_EINVAL);
  }
  // tree: root -> {0, 1}; 0 -> {2}; rows: root, node 0
  {
    Win w;
    w.seq = {2};
    w.n_rows = {2};
    w.row_tok = {5, 6};
    w.row_depth = {0, 1};
    w.row_mask = {1, 3};
    w.n_drafts = {3};
    w.draft_tok = {6, 7, 8, 0};
    w.draft_row = {0, 0, 1, 0};
    w.draft_parent = {-1, -1, 0, -1};
    w.finish(2, 4, 1, true);
    CHECK(copy_window(bk, &w.w, V, 4, 8, c) == VIA_OK && c.tree);
    Win bad = w;
    bad.row_mask = {1, 2};  // row 1 misses row 0
    bad.finish(2, 4, 1, true);
    CHECK(copy_window(bk, &bad.w, V, 4, 8, c) == VIA_EINVAL);
    bad = w;
    bad.draft_row = {0, 1, 1, 0};  // a child of the root verified by row 1
    bad.finish(2, 4, 1, true);
    CHECK(copy_window(bk, &bad.w, V, 4, 8, c) == VIA_EINVAL);
    bad = w;
    bad.draft_parent = {-1, -1, 2, -1};  // parent index not below j
    bad.finish(2, 4, 1, true);
    CHECK(copy_window(bk, &bad.w, V, 4, 8, c) == VIA_EINVAL);
    bad = w;
    bad.row_depth = {1, 1};  // row 0 must sit at depth 0
    bad.finish(2, 4, 1, true);
    CHECK(copy_window(bk, &bad.w, V, 4, 8, c) == VIA_EINVAL);
    bad = w;
    bad.w.row_mask = nullptr;  // half a tree
    CHECK(copy_window(bk, &bad.w, V, 4, 8, c) == VIA_EINVAL);
  }
}

static void test_plans() {
  KvBook bk;
  book_init(bk, 2, 8, 16, 16);
  attach(bk, 0, 20);
  attach(bk, 1, 5);
  bk.seqs[1].valid[0] = 3;  // full cache of seq 1 lags 2 tokens
  WinCopy c;
  Win w = chain({0, 1}, 4);
  w.n_lag = {0, 2};
  w.lag_tok = {0, 0, 41, 42};
  w.finish(4, 8, 2, false);
  CHECK(copy_window(bk, &w.w, V, 2, 8, c) == VIA_OK);
  // slim forward: window rows only, positions n-1 .. n+2, slots after the valid length
  Plan P;
  std::vector<std::pair<int, int>> taken;
  CHECK(build_verify_plan(bk, VIA_CACHE_SLIM, c, {0, 1}, &w.w, true, V, 4, P, &taken) == VIA_OK);
  CHECK(P.rows.size() == 8 && P.lm.size() == 8 && P.seqs.size() == 2);
  CHECK(P.rows[0].pos == 20 && P.rows[0].slot == 20 && P.rows[3].vis_len == 24 && P.rows[4].pos == 5);
  CHECK(P.rows[4].blk == bk.seqs[1].table[1][0]);
  CHECK(P.lm[5].out == 1 * 4 + 1 && P.lm[5].n_drafts == 1 && P.lm[5].draft_idx[0] == 8 + 1);
  CHECK(P.items.size() == 2);  // 4 rows x 4 heads = 16 queries per sequence: one item each
  CHECK(bk.seqs[0].table[1].size() == 2 && bk.seqs[1].table[1].size() == 1);
  book_release_taken(bk, VIA_CACHE_SLIM, taken);
  CHECK(owned_once(bk, 1, 16));
  // full forward of seq 1 only: 2 lag rows first, then the window
  Plan F;
  CHECK(build_verify_plan(bk, VIA_CACHE_FULL, c, {1}, &w.w, true, V, 4, F, nullptr) == VIA_OK);
  CHECK(F.rows.size() == 6 && F.rows[0].tok == 41 && F.rows[1].pos == 4 && F.rows[1].lm == -1);
  CHECK(F.rows[2].pos == 5 && F.rows[2].slot == 5 && F.rows[2].vis_len == 6 && F.seqs[0].kv_len == 9);
  CHECK(F.lm.size() == 4 && F.lm[0].row == 2);
  // a lag that disagrees with the cache: ESTATE, nothing allocated
  KvBook before = bk;
  w.n_lag = {0, 1};
  w.finish(4, 8, 2, false);
  Plan G;
  CHECK(build_verify_plan(bk, VIA_CACHE_FULL, c, {1}, &w.w, true, V, 4, G, nullptr) == VIA_ESTATE);
  CHECK(bk.free_[0] == before.free_[0]);
  // a lag token out of range
  w.n_lag = {0, 2};
  w.lag_tok[3] = V + 3;
  w.finish(4, 8, 2, false);
  CHECK(build_verify_plan(bk, VIA_CACHE_FULL, c, {1}, &w.w, true, V, 4, G, nullptr) == VIA_EINVAL);
  // pool exhaustion: nothing allocated
  KvBook small;
  book_init(small, 1, 8, 2, 2);
  attach(small, 0, 30);
  Win w2 = chain({0}, 4);
  WinCopy c2;
  CHECK(copy_window(small, &w2.w, V, 1, 8, c2) == VIA_OK);
  Plan H;
  CHECK(build_verify_plan(small, VIA_CACHE_SLIM, c2, {0}, &w2.w, true, V, 4, H, nullptr) == VIA_ENOMEM);
  CHECK(small.seqs[0].table[1].size() == 2 && small.free_[1].empty());
  // prefill plan rows [16, 20) of a 20-token prompt
  std::vector<int32_t> toks(20);
  for (int i = 0; i < 20; ++i) toks[i] = i;
  Plan Q;
  build_prefill_plan(bk.seqs[0], VIA_CACHE_FULL, toks.data(), 16, 20, 4, Q);
  CHECK(Q.rows.size() == 4 && Q.rows[0].slot == 16 && Q.rows[0].vis_len == 17 && Q.seqs[0].kv_len == 20);
  // attention items stop at the last key their rows see: rows [0, 20) of a
  // prompt with G = 4 queries per row make items of rows 0-7, 8-15 and 16-19
  CHECK(Q.items.size() == 1 && Q.items[0].kv_len == 20);
  Plan Q2;
  build_prefill_plan(bk.seqs[0], VIA_CACHE_FULL, toks.data(), 0, 20, 4, Q2);
  CHECK(Q2.items.size() == 3 && Q2.items[0].kv_len == 8 && Q2.items[1].kv_len == 16 && Q2.items[2].kv_len == 20);
  // a 10-row tree window shaped as a chain: the first item's rows see the
  // committed prefix and, through their mask bits, window slots up to row 7
  {
    KvBook tb;
    book_init(tb, 1, 8, 16, 16);
    attach(tb, 0, 30);
    Win t;
    t.seq = {0};
    t.n_rows = {10};
    t.n_drafts = {10};
    for (int i = 0; i < 10; ++i) {
      t.row_tok.push_back(i == 0 ? 5 : 10 + i - 1);
      t.row_depth.push_back(i);
      t.row_mask.push_back((2ull << i) - 1);
      t.draft_tok.push_back(10 + i);
      t.draft_row.push_back(i);
      t.draft_parent.push_back(i - 1);
    }
    t.finish(10, 10, 1, true);
    WinCopy tc;
    CHECK(copy_window(tb, &t.w, V, 1, 10, tc) == VIA_OK);
    Plan T;
    CHECK(build_verify_plan(tb, VIA_CACHE_SLIM, tc, {0}, &t.w, true, V, 4, T, nullptr) == VIA_OK);
    const int base = T.seqs[0].win_base;
    CHECK(T.items.size() == 2 && T.items[0].kv_len == base + 8 && T.items[1].kv_len == T.seqs[0].kv_len);
    CHECK(T.seqs[0].kv_len == base + 10 && T.rows[7].vis_len <= base + 8);
  }
}

// Decision block for B sequences, max_drafts D.
static std::vector<int32_t> decision(int B, int D) { return std::vector<int32_t>(4 * B + B * D, -1); }
static void set(std::vector<int32_t>& hp, int B, int D, int b, int st, int kappa, int emit, int nl,
                std::vector<int> path) {
  hp[b] = st;
  hp[B + b] = kappa;
  hp[2 * B + b] = emit;
  hp[3 * B + b] = nl;
  for (size_t i = 0; i < path.size(); ++i) hp[4 * B + b * D + i] = path[i];
}

static void test_commit() {
  KvBook bk;
  book_init(bk, 2, 8, 32, 32);
  attach(bk, 0, 30);
  attach(bk, 1, 14);
  Win w = chain({0, 1}, 4);
  WinCopy c;
  CHECK(copy_window(bk, &w.w, V, 2, 8, c) == VIA_OK);
  std::vector<std::pair<int, int>> t0, t1;
  Plan P;
  CHECK(build_verify_plan(bk, VIA_CACHE_SLIM, c, {0, 1}, &w.w, true, V, 4, P, nullptr) == VIA_OK);
  bk.seqs[0].full_ran = true;
  Plan F;
  CHECK(build_verify_plan(bk, VIA_CACHE_FULL, c, {0}, &w.w, true, V, 4, F, nullptr) == VIA_OK);
  const std::vector<int> step_n = {31, 15};
  const int B = 2, D = 8;
  CommitMoves cm;
  // malformed decisions are refused and change nothing
  auto hp = decision(B, D);
  set(hp, B, D, 0, 1, 0, -1, 31, {});
  set(hp, B, D, 1, 0, 0, 5, 16, {});
  CHECK(plan_commit(bk, c, step_n, hp.data(), V, cm) == VIA_ESTATE);  // still needs the full verifier
  set(hp, B, D, 0, 3, 0, -1, 31, {});
  CHECK(plan_commit(bk, c, step_n, hp.data(), V, cm) == VIA_EINVAL);  // bad status
  set(hp, B, D, 0, 0, 5, -1, 36, {0, 1, 2, 3, 4});
  CHECK(plan_commit(bk, c, step_n, hp.data(), V, cm) == VIA_EINVAL);  // kappa above n_drafts
  set(hp, B, D, 0, 0, 2, V, 34, {0, 1});
  CHECK(plan_commit(bk, c, step_n, hp.data(), V, cm) == VIA_EINVAL);  // emit out of range
  set(hp, B, D, 0, 0, 2, 7, 33, {0, 1});
  CHECK(plan_commit(bk, c, step_n, hp.data(), V, cm) == VIA_EINVAL);  // new_len inconsistent
  set(hp, B, D, 0, 0, 2, 7, 34, {1, 0});
  CHECK(plan_commit(bk, c, step_n, hp.data(), V, cm) == VIA_EINVAL);  // not a root path
  set(hp, B, D, 0, 2, 0, -1, 32, {});
  CHECK(plan_commit(bk, c, step_n, hp.data(), V, cm) == VIA_EINVAL);  // status 2 must keep n
  // a good decision: seq 0 accepts 2 drafts and emits (full ran), seq 1 status 2
  set(hp, B, D, 0, 0, 2, 7, 34, {0, 1});
  set(hp, B, D, 1, 2, 0, -1, 15, {});
  KvBook before = bk;
  CHECK(plan_commit(bk, c, step_n, hp.data(), V, cm) == VIA_OK);
  CHECK(cm.moves[0].empty() && cm.moves[1].empty());  // chain: nothing to compact
  CHECK(bk.seqs[0].valid[0] == before.seqs[0].valid[0]);  // validation alone changes nothing
  apply_commit(bk, c, hp.data());
  CHECK(bk.seqs[0].valid[1] == 33 && bk.seqs[0].valid[0] == 33 && bk.seqs[0].table[1].size() == 3);
  CHECK(bk.seqs[1].valid[1] == 14 && bk.seqs[1].valid[0] == 14 && bk.seqs[1].table[1].size() == 1);
  CHECK(!bk.seqs[0].full_ran && owned_once(bk, 0, 32) && owned_once(bk, 1, 32));
}

static void test_tree_moves() {
  KvBook bk;
  book_init(bk, 1, 8, 16, 16);
  attach(bk, 0, 15);
  // root -> {0, 1}; 1 -> {2, 3}; 3 -> {4}; rows: root, node 1, node 3
  Win w;
  w.seq = {0};
  w.n_rows = {3};
  w.row_tok = {5, 6, 7};
  w.row_depth = {0, 1, 2};
  w.row_mask = {1, 3, 7};
  w.n_drafts = {5};
  w.draft_tok = {1, 2, 3, 4, 5, 0, 0, 0};
  w.draft_row = {0, 0, 1, 1, 2, 0, 0, 0};
  w.draft_parent = {-1, -1, 1, 1, 3, -1, -1, -1};
  w.finish(3, 8, 1, true);
  WinCopy c;
  CHECK(copy_window(bk, &w.w, V, 1, 8, c) == VIA_OK);
  Plan P;
  CHECK(build_verify_plan(bk, VIA_CACHE_SLIM, c, {0}, &w.w, true, V, 4, P, nullptr) == VIA_OK);
  CHECK(P.rows[0].pos == 15 && P.rows[1].pos == 16 && P.rows[2].pos == 17 && P.rows[2].vis_len == 15 && P.rows[2].mask == 7);
  const std::vector<int> step_n = {16};
  auto hp = decision(1, 8);
  // path 1 -> 3 -> 4, all accepted, no emit: root stays at slot 15, node 1's row (1) to 16, node 3's row (2) to 17
  set(hp, 1, 8, 0, 0, 3, -1, 19, {1, 3, 4});
  CommitMoves cm;
  CHECK(plan_commit(bk, c, step_n, hp.data(), V, cm) == VIA_OK);
  CHECK(cm.moves[1].empty());  // slots 16 and 17 are rows 1 and 2 already
  // path 1 -> 2 (node 2 is a leaf, fed by no row): kept rows are root and node 1 only
  set(hp, 1, 8, 0, 0, 2, -1, 18, {1, 2});
  CHECK(plan_commit(bk, c, step_n, hp.data(), V, cm) == VIA_OK && cm.moves[1].empty());
  // path 0 (a leaf) then emit: node 0 has no row -> refused
  set(hp, 1, 8, 0, 0, 1, 9, 18, {0});
  CHECK(plan_commit(bk, c, step_n, hp.data(), V, cm) == VIA_EINVAL);
  // a tree where the accepted path skips a fed row: root -> {0, 1}; 0 -> {2}; 1 -> {3}; 3 -> {4}
  Win t = w;
  t.n_rows = {4};
  t.row_tok = {5, 6, 7, 8};
  t.row_depth = {0, 1, 1, 2};
  t.row_mask = {1, 3, 5, 13};
  t.draft_row = {0, 0, 1, 2, 3, 0, 0, 0};
  t.draft_parent = {-1, -1, 0, 1, 3, -1, -1, -1};
  t.finish(4, 8, 1, true);
  KvBook bk2;
  book_init(bk2, 1, 8, 16, 16);
  attach(bk2, 0, 15);
  CHECK(copy_window(bk2, &t.w, V, 1, 8, c) == VIA_OK);
  Plan P2;
  CHECK(build_verify_plan(bk2, VIA_CACHE_SLIM, c, {0}, &t.w, true, V, 4, P2, nullptr) == VIA_OK);
  bk2.seqs[0].full_ran = true;
  Plan F2;
  CHECK(build_verify_plan(bk2, VIA_CACHE_FULL, c, {0}, &t.w, true, V, 4, F2, nullptr) == VIA_OK);
  // path 1 -> 3 -> 4: node 1 is row 2 (slot 17 -> 16), node 3 is row 3 (slot 18 -> 17)
  set(hp, 1, 8, 0, 0, 3, -1, 19, {1, 3, 4});
  CHECK(plan_commit(bk2, c, step_n, hp.data(), V, cm) == VIA_OK);
  for (int cache = 0; cache < 2; ++cache) {
    CHECK(cm.moves[cache].size() == 2);
    if (cm.moves[cache].size() == 2) {
      CHECK(cm.moves[cache][0].src == 17 && cm.moves[cache][0].dst == 16);
      CHECK(cm.moves[cache][1].src == 18 && cm.moves[cache][1].dst == 17);
      CHECK(cm.btab[cache].size() == bk2.seqs[0].table[cache].size());
    }
  }
  apply_commit(bk2, c, hp.data());
  CHECK(bk2.seqs[0].valid[0] == 18 && bk2.seqs[0].valid[1] == 18);
}

// Random steps: windows of random sizes, random lag catch-up, random
// decisions; the pools stay partitioned and the tables fit the valid lengths.
static void test_random_steps() {
  std::mt19937 rng(7);
  const int NB = 40, S = 3;
  KvBook bk;
  book_init(bk, S, 16, NB, NB);
  for (int s = 0; s < S; ++s) attach(bk, s, 5 + 17 * s);
  for (int it = 0; it < 400; ++it) {
    std::vector<int> seqs;
    for (int s = 0; s < S; ++s)
      if (rng() % 3) seqs.push_back(s);
    if (seqs.empty()) seqs.push_back(it % S);
    const int k = 1 + rng() % 6;
    Win w = chain(seqs, k);
    std::vector<int32_t> lag(seqs.size()), lt(seqs.size() * 64, 1);
    int ml = 1;
    for (size_t b = 0; b < seqs.size(); ++b) {
      lag[b] = bk.seqs[seqs[b]].valid[1] - bk.seqs[seqs[b]].valid[0];
      ml = std::max(ml, (int)lag[b]);
    }
    if (ml > 64) continue;
    w.n_lag = lag;
    w.lag_tok = lt;
    w.finish(k, 8, 64, false);
    WinCopy c;
    CHECK(copy_window(bk, &w.w, V, S, 8, c) == VIA_OK);
    std::vector<int> run;
    for (size_t b = 0; b < seqs.size(); ++b) run.push_back((int)b);
    Plan P;
    KvBook before = bk;
    via_status st = build_verify_plan(bk, VIA_CACHE_SLIM, c, run, &w.w, true, V, 4, P, nullptr);
    if (st == VIA_ENOMEM) {
      CHECK(bk.free_[1] == before.free_[1]);
      // make room: drop the longest sequence back to a short context
      int big = 0;
      for (int s = 1; s < S; ++s)
        if (bk.seqs[s].valid[1] > bk.seqs[big].valid[1]) big = s;
      for (int cc = 0; cc < 2; ++cc) {
        bk.seqs[big].valid[cc] = 3;
        book_trim(bk, cc, big, 3);
      }
      continue;
    }
    CHECK(st == VIA_OK);
    std::vector<int> frun;
    for (size_t b = 0; b < seqs.size(); ++b)
      if (rng() % 2) frun.push_back((int)b);
    if (!frun.empty()) {
      Plan F;
      std::vector<std::pair<int, int>> taken;
      st = build_verify_plan(bk, VIA_CACHE_FULL, c, frun, &w.w, true, V, 4, F, &taken);
      if (st == VIA_ENOMEM) {
        frun.clear();
      } else {
        CHECK(st == VIA_OK);
        for (int b : frun) bk.seqs[seqs[b]].full_ran = true;
      }
    }
    std::vector<int> step_n;
    auto hp = decision((int)seqs.size(), 8);
    for (size_t b = 0; b < seqs.size(); ++b) {
      const int n = bk.seqs[seqs[b]].valid[1] + 1;
      step_n.push_back(n);
      const bool ran = bk.seqs[seqs[b]].full_ran;
      const int status = ran && rng() % 10 == 0 ? 2 : 0;
      const int kappa = status ? 0 : rng() % (k + 1);
      // every draft accepted: nothing is emitted (no bonus token)
      const int emit = status || kappa == k ? -1 : (int)(rng() % V);
      std::vector<int> path;
      for (int j = 0; j < kappa; ++j) path.push_back(j);
      set(hp, (int)seqs.size(), 8, (int)b, status, kappa, emit, status ? n : n + kappa + (emit >= 0), path);
    }
    CommitMoves cm;
    CHECK(plan_commit(bk, c, step_n, hp.data(), V, cm) == VIA_OK);
    apply_commit(bk, c, hp.data());
    for (int s = 0; s < S; ++s) {
      const SeqSt& Sq = bk.seqs[s];
      CHECK(Sq.valid[0] <= Sq.valid[1]);
      for (int cc = 0; cc < 2; ++cc) CHECK((int)Sq.table[cc].size() == blocks_for(Sq.valid[cc]));
    }
    CHECK(owned_once(bk, 0, NB) && owned_once(bk, 1, NB));
  }
}

static void test_step_window_and_tokens() {
  KvBook bk;
  book_init(bk, 2, 8, 32, 32);
  attach(bk, 0, 20);
  attach(bk, 1, 9);
  bk.seqs[1].valid[0] = 6;  // full cache lags 3 tokens
  for (int s = 0; s < 2; ++s) {
    bk.seqs[s].has_tokens = true;
    for (int i = 0; i <= bk.seqs[s].valid[1]; ++i) bk.seqs[s].tokens.push_back(100 + 10 * s + i % 10);
  }
  // chain: seq 0 drafts 4, seq 1 drafts 2
  std::vector<int32_t> sid = {0, 1}, nd = {4, 2}, tok = {1, 2, 3, 4, 5, 6, 0, 0};
  via_drafts d{2, 4, sid.data(), nd.data(), tok.data(), nullptr};
  StepWin sw;
  CHECK(build_step_window(bk, &d, true, sw) == VIA_OK);
  CHECK(sw.win.max_rows == 4 && sw.n_rows[0] == 4 && sw.n_rows[1] == 2);
  CHECK(sw.row_tok[0] == bk.seqs[0].tokens.back() && sw.row_tok[1] == 1 && sw.row_tok[3] == 3);
  CHECK(sw.row_tok[4] == bk.seqs[1].tokens.back() && sw.row_tok[5] == 5);
  CHECK(sw.draft_row[3] == 3 && sw.draft_row[4 + 1] == 1 && !sw.win.row_mask);
  CHECK(sw.n_lag[0] == 0 && sw.n_lag[1] == 3 && sw.win.max_lag == 3);
  CHECK(sw.lag_tok[3 + 0] == bk.seqs[1].tokens[6] && sw.lag_tok[3 + 2] == bk.seqs[1].tokens[8]);
  WinCopy c;
  CHECK(copy_window(bk, &sw.win, 200, 2, 8, c) == VIA_OK);
  Plan F;
  CHECK(build_verify_plan(bk, VIA_CACHE_FULL, c, {1}, &sw.win, true, 200, 4, F, nullptr) == VIA_OK);
  CHECK(F.rows.size() == 5 && F.rows[0].tok == bk.seqs[1].tokens[6]);
  // tree: root -> {0, 1}; 1 -> {2, 3}; 3 -> {4}
  std::vector<int32_t> sid1 = {0}, nd1 = {5}, tok1 = {7, 8, 9, 10, 11}, par1 = {-1, -1, 1, 1, 3};
  via_drafts t{1, 5, sid1.data(), nd1.data(), tok1.data(), par1.data()};
  StepWin tw;
  CHECK(build_step_window(bk, &t, false, tw) == VIA_OK);
  CHECK(tw.n_rows[0] == 3 && tw.row_tok[1] == 8 && tw.row_tok[2] == 10);
  CHECK(tw.row_depth[1] == 1 && tw.row_depth[2] == 2 && tw.row_mask[2] == 7 && tw.row_mask[1] == 3);
  CHECK(tw.draft_row[0] == 0 && tw.draft_row[2] == 1 && tw.draft_row[4] == 2);
  CHECK(copy_window(bk, &tw.win, 200, 2, 8, c) == VIA_OK && c.tree);
  // a sequence without tokens, bad parents, no drafts
  bk.seqs[1].has_tokens = false;
  CHECK(build_step_window(bk, &d, false, sw) == VIA_ESTATE);
  bk.seqs[1].has_tokens = true;
  par1[2] = 2;
  CHECK(build_step_window(bk, &t, false, tw) == VIA_EINVAL);
  par1[2] = 1;
  nd1[0] = 0;
  CHECK(build_step_window(bk, &t, false, tw) == VIA_EINVAL);
  nd1[0] = 5;
  // a commit appends the accepted drafts and the emitted token
  Plan P;
  CHECK(build_step_window(bk, &d, false, sw) == VIA_OK);
  CHECK(copy_window(bk, &sw.win, 200, 2, 8, c) == VIA_OK);
  CHECK(build_verify_plan(bk, VIA_CACHE_SLIM, c, {0, 1}, &sw.win, true, 200, 4, P, nullptr) == VIA_OK);
  auto hp = decision(2, 4);
  set(hp, 2, 4, 0, 0, 2, 77, 21 + 3, {0, 1});
  set(hp, 2, 4, 1, 0, 2, -1, 10 + 2, {0, 1});
  CommitMoves cm;
  const std::vector<int> step_n = {21, 10};
  CHECK(plan_commit(bk, c, step_n, hp.data(), 200, cm) == VIA_OK);
  const size_t n0 = bk.seqs[0].tokens.size(), n1 = bk.seqs[1].tokens.size();
  apply_commit(bk, c, hp.data());
  CHECK(bk.seqs[0].tokens.size() == n0 + 3 && bk.seqs[0].tokens[n0] == 1 && bk.seqs[0].tokens[n0 + 2] == 77);
  CHECK(bk.seqs[1].tokens.size() == n1 + 2 && bk.seqs[1].tokens.back() == 6);
  CHECK((int)bk.seqs[0].tokens.size() == bk.seqs[0].valid[1] + 1);
  CHECK((int)bk.seqs[1].tokens.size() == bk.seqs[1].valid[1] + 1);
}

// The state ring: ring rows of every planned row, the slim forward's
// overwrite check, the row map of a full forward that starts after the
// shared layers, and the commits that set and clear xs_ok.
static void test_state_ring() {
  KvBook bk;
  book_init(bk, 2, 16, 64, 64);
  attach(bk, 0, 20);
  attach(bk, 1, 130);
  Win w = chain({0, 1}, 4);
  WinCopy c;
  CHECK(copy_window(bk, &w.w, V, 2, 8, c) == VIA_OK);
  Plan P;
  CHECK(build_verify_plan(bk, VIA_CACHE_SLIM, c, {0, 1}, &w.w, true, V, 4, P, nullptr) == VIA_OK);
  CHECK(P.rows[0].xs == 20 && P.rows[3].xs == 23);                              // seq 0, slots 20..23
  CHECK(P.rows[4].xs == kStateRows + 130 % kStateRows && P.rows[7].xs == kStateRows + 133 % kStateRows);
  note_slim_forward(bk, c, {0, 1}, true);
  CHECK(bk.seqs[0].xs_ok && bk.seqs[1].xs_ok);
  // commit without the full verifier: seq 0 keeps pending + 2 drafts + emit (lag 3), seq 1 pending + emit
  const int B = 2, D = 8;
  auto hp = decision(B, D);
  set(hp, B, D, 0, 0, 2, 7, 24, {0, 1});
  set(hp, B, D, 1, 0, 0, 9, 132, {});
  CommitMoves cm;
  CHECK(plan_commit(bk, c, {21, 131}, hp.data(), V, cm) == VIA_OK);
  apply_commit(bk, c, hp.data());
  CHECK(bk.seqs[0].valid[VIA_CACHE_SLIM] == 23 && bk.seqs[0].valid[VIA_CACHE_FULL] == 20 && bk.seqs[0].xs_ok);
  // next step: seq 0 escalates; its full forward has lag rows 20..22 then window slots 23..26
  Win w2 = chain({0, 1}, 4);
  w2.n_lag = {3, 1};
  w2.lag_tok = {1, 2, 3, 4, 0, 0};
  w2.finish(4, 8, 3, false);
  WinCopy c2;
  CHECK(copy_window(bk, &w2.w, V, 2, 8, c2) == VIA_OK);
  Plan S2;
  CHECK(build_verify_plan(bk, VIA_CACHE_SLIM, c2, {0, 1}, &w2.w, true, V, 4, S2, nullptr) == VIA_OK);
  note_slim_forward(bk, c2, {0, 1}, true);
  CHECK(bk.seqs[0].xs_ok && bk.seqs[1].xs_ok);  // 23 + 4 - 20 and 131 + 4 - 130 slots fit the ring
  Plan F;
  CHECK(build_verify_plan(bk, VIA_CACHE_FULL, c2, {0}, &w2.w, true, V, 4, F, nullptr) == VIA_OK);
  CHECK(build_prefix_xfer(bk, c2, {0}, F));
  CHECK(F.xfer.size() == 7);
  if (F.xfer.size() == 7) {
    CHECK(F.xfer[0].src_row == 20 && F.xfer[0].t == 4 && F.xfer[0].src_blk == bk.seqs[0].table[VIA_CACHE_SLIM][1] &&
          F.xfer[0].dst_blk == bk.seqs[0].table[VIA_CACHE_FULL][1]);
    CHECK(F.xfer[3].src_row == 23 && F.xfer[6].src_row == 26 && F.xfer[6].t == 26 % 16);
  }
  // a window that would overwrite ring rows of lag slots: seq 1 lags 121 slots, 8 rows need 129
  bk.seqs[1].valid[VIA_CACHE_FULL] = 10;
  note_slim_forward(bk, c2, {1}, true);
  CHECK(bk.seqs[1].xs_ok);  // 131 + 4 - 10 = 125 slots
  Win w3 = chain({1}, 8);
  WinCopy c3;
  CHECK(copy_window(bk, &w3.w, V, 2, 8, c3) == VIA_OK);
  note_slim_forward(bk, c3, {0}, true);
  CHECK(!bk.seqs[1].xs_ok);
  Plan F3;
  F3.rows = F.rows;
  F3.xfer.push_back(PrefixXfer{0, 0, 0, 0});
  CHECK(!build_prefix_xfer(bk, c3, {0}, F3) && F3.xfer.empty());
  // a slim forward that saved nothing clears it too
  note_slim_forward(bk, c2, {0}, false);
  CHECK(!bk.seqs[0].xs_ok);
  // the full verifier's commit sets it again
  bk.seqs[0].full_ran = true;
  auto h2 = decision(1, 8);
  set(h2, 1, 8, 0, 0, 0, 5, 24, {});
  Win w4 = chain({0}, 4);
  WinCopy c4;
  CHECK(copy_window(bk, &w4.w, V, 2, 8, c4) == VIA_OK);
  apply_commit(bk, c4, h2.data());
  CHECK(bk.seqs[0].xs_ok && bk.seqs[0].valid[VIA_CACHE_FULL] == 23);
  // tree commits the full verifier did not see: keeping the root alone leaves the ring valid, keeping
  // more clears it (compaction moves cache slots, not ring rows)
  for (int keep_more = 0; keep_more < 2; ++keep_more) {
    KvBook tb;
    book_init(tb, 1, 8, 16, 16);
    attach(tb, 0, 15);
    Win t;
    t.seq = {0};
    t.n_rows = {3};
    t.row_tok = {5, 6, 7};
    t.row_depth = {0, 1, 2};
    t.row_mask = {1, 3, 7};
    t.n_drafts = {5};
    t.draft_tok = {1, 2, 3, 4, 5, 0, 0, 0};
    t.draft_row = {0, 0, 1, 1, 2, 0, 0, 0};
    t.draft_parent = {-1, -1, 1, 1, 3, -1, -1, -1};
    t.finish(3, 8, 1, true);
    WinCopy tc;
    CHECK(copy_window(tb, &t.w, V, 1, 8, tc) == VIA_OK);
    Plan TP;
    CHECK(build_verify_plan(tb, VIA_CACHE_SLIM, tc, {0}, &t.w, true, V, 4, TP, nullptr) == VIA_OK);
    note_slim_forward(tb, tc, {0}, true);
    auto th = decision(1, 8);
    if (keep_more)
      set(th, 1, 8, 0, 0, 2, -1, 18, {1, 2});  // root + node 1 kept
    else
      set(th, 1, 8, 0, 0, 0, 9, 17, {});  // root only
    CommitMoves tm;
    CHECK(plan_commit(tb, tc, {16}, th.data(), V, tm) == VIA_OK);
    apply_commit(tb, tc, th.data());
    CHECK(tb.seqs[0].xs_ok == !keep_more);
  }
}


// Attention split spans (plan_attention): the cfg3 shape, the one-round
// widening of a ragged long batch, the cap it must not undo, the split
// limit and the error for a sequence too long for any span.
// Prefill row map: the slim forward of a chunk takes row m's state from row m
// of its full forward and copies K/V between the pages of the same slot.
static void test_prefill_xfer() {
  KvBook bk;
  book_init(bk, 4, 16, 16, 16);
  bk.seqs[2] = SeqSt();
  bk.seqs[2].on = true;
  bk.seqs[0] = SeqSt();
  bk.seqs[0].on = true;
  bk.seqs[3] = SeqSt();
  bk.seqs[3].on = true;
  // the caches hand out different pages: take one extra full page first
  CHECK(book_alloc(bk, 0, {{3, 1}}, nullptr) == VIA_OK);
  for (int cache = 0; cache < 2; ++cache) CHECK(book_alloc(bk, cache, {{2, 37}, {0, 9}}, nullptr) == VIA_OK);
  const int32_t tok[64] = {0};
  Plan F, S;
  // chunk rows [16, 37) of seq 2, then [0, 9) of seq 0
  build_prefill_plan(bk.seqs[2], VIA_CACHE_FULL, tok, 16, 37, 4, F);
  build_prefill_plan(bk.seqs[0], VIA_CACHE_FULL, tok, 0, 9, 4, F);
  build_prefill_plan(bk.seqs[2], VIA_CACHE_SLIM, tok, 16, 37, 4, S);
  build_prefill_plan(bk.seqs[0], VIA_CACHE_SLIM, tok, 0, 9, 4, S);
  build_prefill_xfer(bk, {2, 0}, S);
  CHECK(S.xfer.size() == 30 && S.rows.size() == F.rows.size());
  for (size_t m = 0; m < S.rows.size(); ++m) {
    const PrefixXfer& x = S.xfer[m];
    CHECK(x.src_row == (int)m && F.rows[m].slot == S.rows[m].slot && x.t == S.rows[m].slot % kBlock);
    CHECK(x.src_blk == F.rows[m].blk && x.dst_blk == S.rows[m].blk);
  }
  // first row: seq 2, slot 16 (its second page); last row: seq 0, slot 8
  CHECK(S.xfer[0].src_blk == bk.seqs[2].table[VIA_CACHE_FULL][1] && S.xfer[0].dst_blk == bk.seqs[2].table[VIA_CACHE_SLIM][1]);
  CHECK(S.xfer[29].t == 8 && S.xfer[29].dst_blk == bk.seqs[0].table[VIA_CACHE_SLIM][0]);
  CHECK(S.xfer[0].src_blk != S.xfer[0].dst_blk);
}

static void test_attention_plan() {
  auto items = [](const std::vector<int>& kv) {
    std::vector<AttnItem> v;
    for (int k : kv) {
      AttnItem a{};
      a.kv_len = k;
      v.push_back(a);
    }
    return v;
  };
  auto groups = [](const std::vector<AttnItem>& v, int kvh, int span) {
    long long g = 0;
    for (const AttnItem& a : v) g += (long long)kvh * ((a.kv_len + span - 1) / span);
    return g;
  };
  int span = 0, mc = 0;
  // 4 sequences of 2056 keys, 8 KV heads, about 192 work-groups: 6 splits of 352 keys
  std::vector<AttnItem> c3 = items({2056, 2056, 2056, 2056});
  CHECK(plan_attention(c3.data(), 4, 8, 32, 192, 256, &span, &mc) == 0);
  CHECK(span == 352 && mc == 6 && c3[0].n_chunks == 6 && groups(c3, 8, span) == 192);
  // 15 sequences of 5000 keys and one of 9100: the target's span (3520) leaves 264 work-groups; the
  // planner widens it to the narrowest multiple of 32 that fits one round of 256
  std::vector<int> kv(15, 5000);
  kv.push_back(9100);
  std::vector<AttnItem> lg = items(kv);
  {
    std::vector<AttnItem> probe = lg;
    int s0 = 0, m0 = 0;
    CHECK(plan_attention(probe.data(), 16, 8, 32, 192, 1 << 20, &s0, &m0) == 0);  // no round limit
    CHECK(groups(probe, 8, s0) > 256);  // the case the widening is for
  }
  CHECK(plan_attention(lg.data(), 16, 8, 32, 192, 256, &span, &mc) == 0);
  CHECK(span % 32 == 0 && span <= 6144 && groups(lg, 8, span) <= 256 && groups(lg, 8, span - 32) > 256);
  long long n = 0;
  for (const AttnItem& a : lg) n += 8LL * a.n_chunks;
  CHECK(n == groups(lg, 8, span) && mc == (kv.back() + span - 1) / span && span == 4576 && mc == 2);
  // two query items per sequence of 8192 keys: one round cannot hold them below the cap, so the
  // 4096-key spans stay
  std::vector<AttnItem> two = items(std::vector<int>(32, 8192));
  CHECK(plan_attention(two.data(), 32, 8, 32, 192, 256, &span, &mc) == 0 && span == 4096 && mc == 2);
  // at most max_splits splits per sequence
  std::vector<AttnItem> one = items({9000});
  CHECK(plan_attention(one.data(), 1, 8, 2, 192, 256, &span, &mc) == 0 && mc <= 2 && span >= 4500);
  // a sequence longer than max_splits spans of kAttnMaxSpan keys
  std::vector<AttnItem> too = items({2 * kAttnMaxSpan + 32});
  CHECK(plan_attention(too.data(), 1, 8, 2, 192, 256, &span, &mc) == -1);
}

int main() {
  test_prefill_xfer();
  test_attention_plan();
  test_step_window_and_tokens();
  test_allocator();
  test_window_validation();
  test_plans();
  test_commit();
  test_tree_moves();
  test_state_ring();
  test_random_steps();
  if (g_fail) {
    std::printf("%d check(s) failed\n", g_fail);
    return 1;
  }
  std::printf("ALL OK\n");
  return 0;
}
