// Plan structures the host builds per call and uploads to the device, and the
// constants both sides share.  Plain C++: the host bookkeeping that fills
// them builds without HIP.
#pragma once
#include <stdint.h>

namespace via {

constexpr int kBlock = 16;        // tokens per KV page
constexpr int kMaxChildren = 8;   // drafts verified by one row
constexpr int kAttnMaxSplits = 32;  // key splits per sequence (partials one query's combine merges)
constexpr int kAttnMaxSpan = 8192;  // keys of one split (pages of a split's work-group, x16)
constexpr int kAttnPrefSpan = 4096;  // keys per work-group beyond which a forward takes more work-groups than the target
constexpr int kAttnTargetGroups = 192;  // attention work-groups a forward aims for (fewer, longer spans than one per compute unit: measured best at the 8B shapes)
constexpr int kAttnQueries = 32;  // (row, head-in-group) queries per attention work-group
constexpr int kNormChunk = 512;   // columns per partial sum of squares (RMSNorm)
// Per-sequence ring of post-shared-layer states: slot p of a sequence keeps
// its state in ring row p % kStateRows.
constexpr int kStateRows = 128;

// One fed row of a forward (lag row or window row).
struct RowInfo {
  int32_t tok;      // token id
  int32_t pos;      // RoPE position
  int32_t seq;      // index into the SeqInfo array of this forward
  int32_t slot;     // cache slot the row's K/V are written to
  int32_t vis_len;  // slots [0, vis_len) are visible
  int32_t lm;       // index into the head rows, -1 if the row has no head output
  int32_t blk;      // pool block holding `slot` (the sequence's block table entry slot / block size)
  int32_t xs;       // state-store row of (sequence, slot) the slim forward saves the row's state to, -1: none
  uint64_t mask;    // extra visible slots win_base + bit (tree rows)
};

struct SeqInfo {
  int32_t kv_len;     // slots written after the forward's K/V write
  int32_t row_start;  // first row of this sequence in the forward
  int32_t n_rows;     // rows of this sequence (lag + window)
  int32_t win_base;   // slot of window row 0 (tree masks are relative to it)
  int32_t bt;         // offset of the block table in the uploaded tables
  int32_t n_blocks;   // block-table length
  int32_t pad0, pad1;
};

// One attention work item: up to kAttnQueries (row, head-in-group) queries of a
// sequence, with the sequence's cache geometry inlined.
struct AttnItem {
  int32_t q0;       // first query (row * G + g) of the tile, within the sequence
  int32_t n_chunks; // key splits of this sequence: ceil(kv_len / span)
  int32_t kv_len, row_start, n_rows, win_base, bt, n_blocks;
};

// Head row: which forward row and where its statistics go.
struct LmRow {
  int32_t row;      // forward row
  int32_t out;      // b * max_rows + r in the caller's output arrays
  int32_t n_drafts; // drafts this row verifies (<= kMaxChildren)
  int32_t pad;
  int32_t draft_idx[kMaxChildren];  // b * max_drafts + j
  int32_t draft_tok[kMaxChildren];
};

// Per-sequence data of an open step, read by the tier decision.
struct StepSeq {
  int32_t n;          // committed length before the step
  int32_t n_drafts;
  int32_t full_ran;   // full forward ran this step
  int32_t pad;
};

// One row of a full forward that starts after the P layers the slim route
// shares with it (route layer i == i for i < P).
struct PrefixXfer {
  int32_t src_row;           // state row of (sequence, slot)
  int32_t t;                 // slot within the page (position % 16)
  int32_t src_blk, dst_blk;  // page of the position in the source and the destination cache
};

// Tree compaction: copy K/V of slot src -> dst for every layer slot.
struct KvMove {
  int32_t bt;      // offset of the block table in btab
  int32_t src, dst;
  int32_t pad;
};

}  // namespace via
