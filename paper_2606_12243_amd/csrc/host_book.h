// Host bookkeeping of the verification step: the paged block allocator of
// both caches, validation and copies of draft windows, the per-forward row
// plans, and the checks and tree-compaction moves of a commit.  Plain C++
// (no HIP), so that it builds and is tested on its own on the CPU; the
// runtime (runtime.cpp) owns the device side.
#pragma once
#include <stdint.h>

#include <set>
#include <string>
#include <utility>
#include <vector>

#include "../../include/via.h"
#include "plan.h"

namespace via {

// Records a thread-local message (via_last_error) and returns `s`.
via_status fail(via_status s, const char* fmt, ...);
const char* last_error();

int ceil_div(int a, int b);
// Blocks a sequence needs to hold `slots` cache slots.
int blocks_for(int slots);

// Logical KV state of one sequence: valid lengths and block tables of the
// full (index VIA_CACHE_FULL) and slim (VIA_CACHE_SLIM) caches.
struct SeqSt {
  bool on = false;
  int valid[2] = {0, 0};
  std::vector<int> table[2];
  bool full_ran = false;  // the full verifier ran for it in the open step
  // every slot in [valid full, valid slim) has its state after the shared
  // layers in the state ring (kStateRows rows per sequence, row slot %
  // kStateRows), so a full forward can start after those layers
  bool xs_ok = true;
  // committed tokens x[0..n-1] (n = slim valid length + 1) when the caller
  // gave them (via_kv_seq_set_tokens); commits then append to them
  bool has_tokens = false;
  std::vector<int32_t> tokens;
};

// Both caches' sequences and free block sets.  Blocks are handed out lowest
// id first (a min-ordered free set).
struct KvBook {
  int max_blocks_per_seq = 0;
  std::vector<SeqSt> seqs;
  std::set<int> free_[2];
};
void book_init(KvBook& bk, int max_seqs, int max_blocks_per_seq, int blocks_full, int blocks_slim);
// All-or-nothing: give every (seq, slots) of `need` the blocks it lacks in
// `cache`, lowest free id first, in the given order; taken (nullable)
// records every (seq, block) handed out.  ENOMEM (nothing taken) if the pool
// or a block table is too small.
via_status book_alloc(KvBook& bk, int cache, const std::vector<std::pair<int, int>>& need,
                      std::vector<std::pair<int, int>>* taken);
// Free the blocks of `seq` lying wholly at or past `valid` slots.
void book_trim(KvBook& bk, int cache, int seq, int valid);
// Undo a book_alloc (blocks back to the pool, tables shortened).
void book_release_taken(KvBook& bk, int cache, const std::vector<std::pair<int, int>>& taken);

// Validated copy of a draft window (include/via.h, via_window).
struct WinCopy {
  int batch = 0, max_rows = 0, max_drafts = 0;
  bool tree = false;
  std::vector<int> seq, n_rows, row_tok, row_depth, n_drafts, draft_tok, draft_row, draft_parent;
  std::vector<uint64_t> row_mask;
};
// EINVAL for every malformed window: batch and strides out of range, missing
// arrays, unattached or repeated sequences, tokens outside [0, vocab), bad
// depths or masks, drafts whose row is not their parent's row, more than
// kMaxChildren drafts on one row.
via_status copy_window(const KvBook& bk, const via_window* w, int vocab, int max_batch, int max_drafts,
                       WinCopy& c);

// Rows of one forward and everything the kernels index by them.
struct Plan {
  std::vector<RowInfo> rows;
  std::vector<SeqInfo> seqs;
  std::vector<int32_t> btab;
  std::vector<AttnItem> items;
  std::vector<LmRow> lm;
  std::vector<PrefixXfer> xfer;  // forwards that start after the shared layers
  std::vector<char> extra;       // bytes uploaded with the plan (the decision's step data)
};
// Plan of a verify forward of `cache` over the batch entries `run` of w: the
// full cache's lag rows (raw->n_lag / lag_tok, which must equal the cache's
// lag: ESTATE otherwise) and the window rows, their positions, cache slots
// and visibility, the head rows with the drafts each verifies (`head`), the
// attention items (kAttnQueries queries of G = H / KVH heads per item).
// Allocates the blocks the rows need (ENOMEM: nothing allocated).
via_status build_verify_plan(KvBook& bk, int cache, const WinCopy& w, const std::vector<int>& run,
                             const via_window* raw, bool head, int vocab, int G, Plan& P,
                             std::vector<std::pair<int, int>>* taken);
// After a slim forward over the batch entries `run` of w that saved (saved)
// or did not save its rows' states to the state ring: a sequence whose
// window rows, written at slots valid slim .. + n_rows - 1, overwrite ring
// rows of slots the full cache still lacks loses xs_ok.
void note_slim_forward(KvBook& bk, const WinCopy& w, const std::vector<int>& run, bool saved);
// Row map of a full forward (plan P of the entries `run` of w) that starts
// after the shared layers: one PrefixXfer per row of P (its state-ring row
// and the slim and full pages of its slot).  False, with P.xfer left empty,
// unless every running sequence has xs_ok.
bool build_prefix_xfer(const KvBook& bk, const WinCopy& w, const std::vector<int>& run, Plan& P);
// Append prefill rows [c0, c1) of one sequence to a plan (causal, positions
// = slots; the sequence's rows, table and attention items follow those
// already in P).
void build_prefill_plan(const SeqSt& S, int cache, const int32_t* tokens, int c0, int c1, int G, Plan& P);
// Row map of a prefill's slim forward (plan P, whose plan-sequence i is
// sequence id seq_of[i]) that starts after the shared layers from its full
// forward over the same rows: row m takes the full forward's state row m and
// the full and slim pages of its slot.
void build_prefill_xfer(const KvBook& bk, const std::vector<int>& seq_of, Plan& P);

// Commit of an open step from the host copy of a decision (the packed block
// of include/via.h).  Validation (nothing changes on error): no status 1,
// statuses 0 or 2, kappa in [0, n_drafts], emit in [-1, vocab), new_len
// consistent (n for status 2, n + kappa + [emit >= 0] otherwise), the
// accepted path a root path of the draft tree, every accepted node but the
// last with a fed row.  moves[cache] receives the tree-compaction copies
// (block-table offsets into btab[cache]); chain windows need none.
struct CommitMoves {
  std::vector<int32_t> btab[2];
  std::vector<KvMove> moves[2];
};
via_status plan_commit(const KvBook& bk, const WinCopy& w, const std::vector<int>& step_n, const int32_t* hp,
                       int vocab, CommitMoves& cm);
// Apply a validated commit: valid lengths (slim always, full where it ran),
// blocks past them freed, full_ran cleared, and the accepted drafts and the
// emitted token appended to the committed tokens of sequences that keep them.
// xs_ok: set where the full cache caught up; cleared where a tree commit
// that the full verifier did not see keeps more than the root row (the
// compaction moves cache slots, the state ring is not moved).
void apply_commit(KvBook& bk, const WinCopy& w, const int32_t* hp);

// The key-split span of a forward's attention items: about target_groups
// work-groups over all items and KV heads, at most max_splits splits per
// sequence, spans capped near kAttnPrefSpan, and widened so that the
// work-groups fit one round of max_groups (the device's compute units) when
// one split per item would.  Sets every item's n_chunks, *span_out and
// *max_chunks_out; returns -1 if a sequence needs a span above kAttnMaxSpan.
int plan_attention(AttnItem* items, int n_items, int KVH, int max_splits, int target_groups, int max_groups,
                   int* span_out, int* max_chunks_out);

// Draft window of a natively driven step (via_step): rows, draft rows,
// depths and ancestor masks built from each sequence's committed tokens (the
// pending token x[n-1] is row 0) and its drafts, plus the lag rows (the
// committed tokens x[valid_full .. n-2] the full cache is missing).  `win`
// points into the vectors of this object.
struct StepWin {
  std::vector<int32_t> seq, n_rows, row_tok, row_depth, n_drafts, draft_tok, draft_row, draft_parent, n_lag, lag_tok;
  std::vector<uint64_t> row_mask;
  via_window win{};
};
// EINVAL for malformed drafts (sizes, parents, more than VIA_MAX_TREE_ROWS
// fed rows), ESTATE for a sequence without committed tokens.
via_status build_step_window(const KvBook& bk, const via_drafts* d, bool with_lag, StepWin& sw);

}  // namespace via
