// Host bookkeeping of the verification step (host_book.h): plain C++, no HIP.
#include "host_book.h"

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>

namespace via {

namespace {
thread_local std::string g_err;
}

via_status fail(via_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

const char* last_error() { return g_err.c_str(); }

int ceil_div(int a, int b) { return (a + b - 1) / b; }

int blocks_for(int slots) { return ceil_div(slots, kBlock); }

void book_init(KvBook& bk, int max_seqs, int max_blocks_per_seq, int blocks_full, int blocks_slim) {
  bk.max_blocks_per_seq = max_blocks_per_seq;
  bk.seqs.assign(max_seqs, SeqSt());
  for (int c = 0; c < 2; ++c) {
    bk.free_[c].clear();
    const int nb = c == VIA_CACHE_FULL ? blocks_full : blocks_slim;
    for (int i = 0; i < nb; ++i) bk.free_[c].insert(bk.free_[c].end(), i);
  }
}

via_status book_alloc(KvBook& bk, int cache, const std::vector<std::pair<int, int>>& need,
                      std::vector<std::pair<int, int>>* taken) {
  size_t missing = 0;
  for (auto& pr : need) {
    const SeqSt& S = bk.seqs[pr.first];
    const int want = blocks_for(pr.second);
    if (want > bk.max_blocks_per_seq)
      return fail(VIA_ENOMEM, "sequence %d needs %d blocks > max_blocks_per_seq %d", pr.first, want,
                  bk.max_blocks_per_seq);
    if (want > (int)S.table[cache].size()) missing += want - S.table[cache].size();
  }
  if (missing > bk.free_[cache].size())
    return fail(VIA_ENOMEM, "%s KV pool exhausted: need %zu blocks, %zu free", cache == 0 ? "full" : "slim", missing,
                bk.free_[cache].size());
  for (auto& pr : need) {
    SeqSt& S = bk.seqs[pr.first];
    const int want = blocks_for(pr.second);
    while ((int)S.table[cache].size() < want) {
      const int blk = *bk.free_[cache].begin();
      bk.free_[cache].erase(bk.free_[cache].begin());
      S.table[cache].push_back(blk);
      if (taken) taken->push_back({pr.first, blk});
    }
  }
  return VIA_OK;
}

void book_trim(KvBook& bk, int cache, int seq, int valid) {
  SeqSt& S = bk.seqs[seq];
  const size_t keep = blocks_for(valid);
  while (S.table[cache].size() > keep) {
    bk.free_[cache].insert(S.table[cache].back());
    S.table[cache].pop_back();
  }
}

void book_release_taken(KvBook& bk, int cache, const std::vector<std::pair<int, int>>& taken) {
  for (auto it = taken.rbegin(); it != taken.rend(); ++it) {
    SeqSt& S = bk.seqs[it->first];
    if (!S.table[cache].empty() && S.table[cache].back() == it->second) S.table[cache].pop_back();
    bk.free_[cache].insert(it->second);
  }
}

via_status copy_window(const KvBook& bk, const via_window* w, int vocab, int max_batch, int max_drafts,
                       WinCopy& c) {
  if (!w) return fail(VIA_EINVAL, "null window");
  if (w->batch < 1 || w->batch > max_batch) return fail(VIA_EINVAL, "batch %d not in [1, %d]", w->batch, max_batch);
  if (w->max_rows < 1 || w->max_drafts < 1 || w->max_drafts > max_drafts)
    return fail(VIA_EINVAL, "window strides out of range (1 <= max_drafts <= %d)", max_drafts);
  if (!w->seq_id || !w->n_rows || !w->row_tok || !w->n_drafts || !w->draft_tok || !w->draft_row)
    return fail(VIA_EINVAL, "window arrays missing");
  const int max_seqs = (int)bk.seqs.size();
  c = WinCopy();
  c.batch = w->batch;
  c.max_rows = w->max_rows;
  c.max_drafts = w->max_drafts;
  c.tree = w->row_mask != nullptr || w->draft_parent != nullptr;
  if ((w->row_mask != nullptr) != (w->draft_parent != nullptr))
    return fail(VIA_EINVAL, "tree windows need both row_mask and draft_parent");
  std::set<int> seen;
  for (int b = 0; b < w->batch; ++b) {
    const int sid = w->seq_id[b];
    if (sid < 0 || sid >= max_seqs || !bk.seqs[sid].on) return fail(VIA_EINVAL, "sequence %d not attached", sid);
    if (!seen.insert(sid).second) return fail(VIA_EINVAL, "sequence %d appears twice", sid);
    const int R = w->n_rows[b], nd = w->n_drafts[b];
    if (R < 1 || R > w->max_rows) return fail(VIA_EINVAL, "n_rows[%d]=%d out of range", b, R);
    if (nd < 0 || nd > w->max_drafts) return fail(VIA_EINVAL, "n_drafts[%d]=%d out of range", b, nd);
    if (c.tree && R > VIA_MAX_TREE_ROWS) return fail(VIA_EINVAL, "tree windows hold at most %d rows", VIA_MAX_TREE_ROWS);
    c.seq.push_back(sid);
    c.n_rows.push_back(R);
    c.n_drafts.push_back(nd);
  }
  c.row_tok.assign((size_t)w->batch * w->max_rows, 0);
  c.row_depth.assign((size_t)w->batch * w->max_rows, 0);
  c.row_mask.assign((size_t)w->batch * w->max_rows, 0);
  c.draft_tok.assign((size_t)w->batch * w->max_drafts, 0);
  c.draft_row.assign((size_t)w->batch * w->max_drafts, 0);
  c.draft_parent.assign((size_t)w->batch * w->max_drafts, -1);
  for (int b = 0; b < w->batch; ++b) {
    const int R = c.n_rows[b], nd = c.n_drafts[b];
    for (int r = 0; r < R; ++r) {
      const size_t i = (size_t)b * w->max_rows + r;
      const int t = w->row_tok[i];
      if (t < 0 || t >= vocab) return fail(VIA_EINVAL, "row token %d out of range", t);
      c.row_tok[i] = t;
      const int dep = w->row_depth ? w->row_depth[i] : r;
      if (dep < 0 || (r == 0 && dep != 0)) return fail(VIA_EINVAL, "row depth must be >= 0 and 0 for row 0");
      c.row_depth[i] = dep;
      if (w->row_mask) {
        const uint64_t mk = w->row_mask[i];
        if (!((mk >> r) & 1) || !(mk & 1) || (r < 63 && (mk >> (r + 1))))
          return fail(VIA_EINVAL, "row_mask[%d][%d] must contain row 0, itself and no later row", b, r);
        c.row_mask[i] = mk;
      }
    }
    std::vector<int> node_row(nd, -1);
    for (int j = 0; j < nd; ++j) {
      const size_t i = (size_t)b * w->max_drafts + j;
      const int t = w->draft_tok[i], row = w->draft_row[i];
      const int par = w->draft_parent ? w->draft_parent[i] : j - 1;
      if (t < 0 || t >= vocab) return fail(VIA_EINVAL, "draft token %d out of range", t);
      if (row < 0 || row >= R) return fail(VIA_EINVAL, "draft_row[%d][%d]=%d out of range", b, j, row);
      if (par < -1 || par >= j) return fail(VIA_EINVAL, "draft_parent[%d][%d] must be -1 or < j", b, j);
      // the row verifying draft j is its parent's row (root row 0)
      if (par == -1 ? row != 0 : (node_row[par] >= 0 && node_row[par] != row))
        return fail(VIA_EINVAL, "draft_row[%d][%d] inconsistent with its parent", b, j);
      if (par >= 0) node_row[par] = row;
      if (!w->draft_parent && row != j) return fail(VIA_EINVAL, "chain draft j must be verified by row j");
      c.draft_tok[i] = t;
      c.draft_row[i] = row;
      c.draft_parent[i] = par;
    }
    // children per row bounded (head rows carry at most kMaxChildren drafts)
    std::vector<int> per_row(R, 0);
    for (int j = 0; j < nd; ++j)
      if (++per_row[c.draft_row[(size_t)b * w->max_drafts + j]] > kMaxChildren)
        return fail(VIA_EINVAL, "a row verifies more than %d drafts", kMaxChildren);
  }
  return VIA_OK;
}

// One item per kAttnQueries queries of the sequence.  An item streams keys
// up to the last one any of its rows sees (its causal prefix and tree-mask
// bits), not the whole sequence: the items of a long prefill then read
// about half the keys, and a block no row sees would add exactly nothing.
static void push_items(Plan& P, const SeqInfo& si, int G) {
  const int nq = si.n_rows * G;
  for (int q0 = 0; q0 < nq; q0 += kAttnQueries) {
    int kv = 1;
    const int r1 = std::min(si.n_rows, (q0 + kAttnQueries + G - 1) / G);
    for (int rl = q0 / G; rl < r1; ++rl) {
      const RowInfo& r = P.rows[si.row_start + rl];
      kv = std::max(kv, r.vis_len);
      if (r.mask) kv = std::max(kv, si.win_base + 64 - __builtin_clzll(r.mask));
    }
    P.items.push_back(AttnItem{q0, 0, std::min(kv, si.kv_len), si.row_start, si.n_rows, si.win_base, si.bt, si.n_blocks});
  }
}

via_status build_verify_plan(KvBook& bk, int cache, const WinCopy& w, const std::vector<int>& run,
                             const via_window* raw, bool head, int vocab, int G, Plan& P,
                             std::vector<std::pair<int, int>>* taken) {
  std::vector<std::pair<int, int>> need;
  for (int b : run) {
    const SeqSt& S = bk.seqs[w.seq[b]];
    int n_lag = 0;
    if (cache == VIA_CACHE_FULL) {
      const int lag = S.valid[VIA_CACHE_SLIM] - S.valid[VIA_CACHE_FULL];
      n_lag = (raw && raw->n_lag) ? raw->n_lag[b] : 0;
      if (n_lag != lag)
        return fail(VIA_ESTATE, "sequence %d: full cache lags %d tokens, window gives %d", w.seq[b], lag, n_lag);
      if (n_lag > 0 && (!raw->lag_tok || n_lag > raw->max_lag))
        return fail(VIA_EINVAL, "lag_tok missing or max_lag too small");
      for (int i = 0; i < n_lag; ++i) {
        const int t = raw->lag_tok[(size_t)b * raw->max_lag + i];
        if (t < 0 || t >= vocab) return fail(VIA_EINVAL, "lag token out of range");
      }
    }
    need.push_back({w.seq[b], S.valid[cache] + n_lag + w.n_rows[b]});
  }
  via_status st = book_alloc(bk, cache, need, taken);
  if (st) return st;
  int lm_i = 0;
  for (size_t q = 0; q < run.size(); ++q) {
    const int b = run[q];
    const SeqSt& S = bk.seqs[w.seq[b]];
    const int valid = S.valid[cache];
    const int n_lag = need[q].second - valid - w.n_rows[b];
    const int R = w.n_rows[b];
    const int win_base = valid + n_lag;
    const int npos = S.valid[VIA_CACHE_SLIM];  // position of the pending token, n - 1
    SeqInfo si{};
    si.row_start = (int)P.rows.size();
    si.n_rows = n_lag + R;
    si.kv_len = valid + n_lag + R;
    si.win_base = win_base;
    si.bt = (int)P.btab.size();
    si.n_blocks = (int)S.table[cache].size();
    for (int blk : S.table[cache]) P.btab.push_back(blk);
    const int sidx = (int)P.seqs.size();
    for (int i = 0; i < n_lag; ++i) {
      RowInfo r{};
      r.tok = raw->lag_tok[(size_t)b * raw->max_lag + i];
      r.pos = valid + i;
      r.seq = sidx;
      r.slot = valid + i;
      r.blk = S.table[cache][r.slot / kBlock];
      r.xs = w.seq[b] * kStateRows + r.slot % kStateRows;
      r.vis_len = valid + i + 1;
      r.lm = -1;
      P.rows.push_back(r);
    }
    for (int rr = 0; rr < R; ++rr) {
      const size_t i = (size_t)b * w.max_rows + rr;
      RowInfo r{};
      r.tok = w.row_tok[i];
      r.pos = npos + w.row_depth[i];
      r.seq = sidx;
      r.slot = win_base + rr;
      r.blk = S.table[cache][r.slot / kBlock];
      r.xs = w.seq[b] * kStateRows + r.slot % kStateRows;
      r.vis_len = w.tree ? win_base : win_base + rr + 1;
      r.mask = w.tree ? w.row_mask[i] : 0;
      r.lm = -1;
      if (head) {
        LmRow lr{};
        lr.row = (int)P.rows.size();
        lr.out = b * w.max_rows + rr;
        for (int j = 0; j < w.n_drafts[b]; ++j) {
          const size_t di = (size_t)b * w.max_drafts + j;
          if (w.draft_row[di] == rr) {
            lr.draft_idx[lr.n_drafts] = (int)di;
            lr.draft_tok[lr.n_drafts] = w.draft_tok[di];
            lr.n_drafts++;
          }
        }
        r.lm = lm_i++;
        P.lm.push_back(lr);
      }
      P.rows.push_back(r);
    }
    P.seqs.push_back(si);
    push_items(P, si, G);
  }
  return VIA_OK;
}

void note_slim_forward(KvBook& bk, const WinCopy& w, const std::vector<int>& run, bool saved) {
  for (int b : run) {
    SeqSt& S = bk.seqs[w.seq[b]];
    if (!saved || S.valid[VIA_CACHE_SLIM] + w.n_rows[b] - S.valid[VIA_CACHE_FULL] > kStateRows) S.xs_ok = false;
  }
}

bool build_prefix_xfer(const KvBook& bk, const WinCopy& w, const std::vector<int>& run, Plan& P) {
  P.xfer.clear();
  for (int b : run)
    if (!bk.seqs[w.seq[b]].xs_ok) return false;
  for (const RowInfo& r : P.rows) {
    const SeqSt& S = bk.seqs[w.seq[run[r.seq]]];
    P.xfer.push_back(PrefixXfer{r.xs, r.slot % kBlock, S.table[VIA_CACHE_SLIM][r.slot / kBlock],
                                S.table[VIA_CACHE_FULL][r.slot / kBlock]});
  }
  return true;
}

void build_prefill_plan(const SeqSt& S, int cache, const int32_t* tokens, int c0, int c1, int G, Plan& P) {
  SeqInfo si{};
  si.row_start = (int)P.rows.size();
  si.n_rows = c1 - c0;
  si.kv_len = c1;
  si.win_base = c0;
  si.bt = (int)P.btab.size();
  si.n_blocks = (int)S.table[cache].size();
  const int sidx = (int)P.seqs.size();
  for (int blk : S.table[cache]) P.btab.push_back(blk);
  for (int i = c0; i < c1; ++i) {
    RowInfo r{};
    r.tok = tokens[i];
    r.pos = i;
    r.seq = sidx;
    r.slot = i;
    r.blk = S.table[cache][i / kBlock];
    r.xs = -1;
    r.vis_len = i + 1;
    r.lm = -1;
    P.rows.push_back(r);
  }
  P.seqs.push_back(si);
  push_items(P, si, G);
}

void build_prefill_xfer(const KvBook& bk, const std::vector<int>& seq_of, Plan& P) {
  P.xfer.clear();
  for (size_t m = 0; m < P.rows.size(); ++m) {
    const RowInfo& r = P.rows[m];
    const SeqSt& S = bk.seqs[seq_of[r.seq]];
    P.xfer.push_back(PrefixXfer{(int32_t)m, r.slot % kBlock, S.table[VIA_CACHE_FULL][r.slot / kBlock],
                                S.table[VIA_CACHE_SLIM][r.slot / kBlock]});
  }
}

via_status plan_commit(const KvBook& bk, const WinCopy& w, const std::vector<int>& step_n, const int32_t* hp,
                       int vocab, CommitMoves& cm) {
  const int B = w.batch, Dd = std::max(1, w.max_drafts);
  std::vector<std::vector<int>> kept_rows(B);
  for (int b = 0; b < B; ++b) {
    const int status = hp[b], kappa = hp[B + b], emit = hp[2 * B + b], nl = hp[3 * B + b];
    const int* path = hp + 4 * B + b * Dd;
    const int n = step_n[b];
    if (status == 1) return fail(VIA_ESTATE, "sequence %d still needs the full verifier", w.seq[b]);
    if (status != 0 && status != 2) return fail(VIA_EINVAL, "bad status %d", status);
    if (kappa < 0 || kappa > w.n_drafts[b]) return fail(VIA_EINVAL, "kappa %d out of range", kappa);
    if (emit < -1 || emit >= vocab) return fail(VIA_EINVAL, "emit %d out of range", emit);
    if (status == 2) {
      if (nl != n) return fail(VIA_EINVAL, "new_len must equal n when the sequence is not advanced");
      continue;
    }
    if (nl != n + kappa + (emit >= 0 ? 1 : 0)) return fail(VIA_EINVAL, "new_len inconsistent with kappa/emit");
    int prev = -1;
    for (int i = 0; i < kappa; ++i) {
      const int j = path[i];
      if (j < 0 || j >= w.n_drafts[b] || w.draft_parent[(size_t)b * w.max_drafts + j] != prev)
        return fail(VIA_EINVAL, "accepted path of sequence %d is not a root path", w.seq[b]);
      prev = j;
    }
    // window rows that stay valid: root + the first (kept - 1) path nodes
    const int kept = kappa + (emit >= 0 ? 1 : 0);
    for (int i = 1; i < kept; ++i) {
      const int node = path[i - 1];
      int row = -1;
      for (int j = 0; j < w.n_drafts[b]; ++j)
        if (w.draft_parent[(size_t)b * w.max_drafts + j] == node) {
          row = w.draft_row[(size_t)b * w.max_drafts + j];
          break;
        }
      if (row < 0) return fail(VIA_EINVAL, "accepted node %d has no fed row", node);
      kept_rows[b].push_back(row);
    }
  }
  // tree compaction moves (slim cache always, full cache where it ran)
  for (int cache = 0; cache < 2; ++cache) {
    cm.btab[cache].clear();
    cm.moves[cache].clear();
    if (!w.tree) continue;
    for (int b = 0; b < B; ++b) {
      const SeqSt& S = bk.seqs[w.seq[b]];
      if (hp[b] != 0) continue;
      if (cache == VIA_CACHE_FULL && !S.full_ran) continue;
      const int base = step_n[b] - 1;
      const int off = (int)cm.btab[cache].size();
      bool any = false;
      for (size_t i = 0; i < kept_rows[b].size(); ++i) {
        const int src = base + kept_rows[b][i], dst = base + (int)i + 1;
        if (src != dst) {
          cm.moves[cache].push_back(KvMove{off, src, dst, 0});
          any = true;
        }
      }
      if (any)
        for (int blk : S.table[cache]) cm.btab[cache].push_back(blk);
    }
  }
  return VIA_OK;
}

void apply_commit(KvBook& bk, const WinCopy& w, const int32_t* hp) {
  const int B = w.batch, Dd = std::max(1, w.max_drafts);
  for (int b = 0; b < B; ++b) {
    SeqSt& S = bk.seqs[w.seq[b]];
    if (hp[b] == 0) {
      const int nv = hp[3 * B + b] - 1;
      const int kept = hp[B + b] + (hp[2 * B + b] >= 0 ? 1 : 0);
      S.valid[VIA_CACHE_SLIM] = nv;
      if (S.full_ran) {
        S.valid[VIA_CACHE_FULL] = nv;
        S.xs_ok = true;
      } else if (w.tree && kept >= 2) {
        S.xs_ok = false;
      }
      if (S.has_tokens) {
        const int kappa = hp[B + b], emit = hp[2 * B + b];
        for (int i = 0; i < kappa; ++i) S.tokens.push_back(w.draft_tok[(size_t)b * w.max_drafts + hp[4 * B + b * Dd + i]]);
        if (emit >= 0) S.tokens.push_back(emit);
      }
    }
    book_trim(bk, VIA_CACHE_SLIM, w.seq[b], S.valid[VIA_CACHE_SLIM]);
    book_trim(bk, VIA_CACHE_FULL, w.seq[b], S.valid[VIA_CACHE_FULL]);
    S.full_ran = false;
  }
}

via_status build_step_window(const KvBook& bk, const via_drafts* d, bool with_lag, StepWin& sw) {
  if (!d || !d->seq_id || !d->n_drafts || !d->draft_tok) return fail(VIA_EINVAL, "drafts: arrays missing");
  if (d->batch < 1 || d->max_drafts < 1 || d->max_drafts > VIA_MAX_DRAFTS)
    return fail(VIA_EINVAL, "drafts: batch >= 1 and 1 <= max_drafts <= %d", VIA_MAX_DRAFTS);
  const int B = d->batch, D = d->max_drafts;
  const bool tree = d->draft_parent != nullptr;
  sw = StepWin();
  // rows per sequence: chain k rows; tree the root and every node with children
  std::vector<std::vector<int>> rows_of(B);
  int R = 1, Lg = 1;
  for (int b = 0; b < B; ++b) {
    const int sid = d->seq_id[b], nd = d->n_drafts[b];
    if (sid < 0 || sid >= (int)bk.seqs.size() || !bk.seqs[sid].on) return fail(VIA_EINVAL, "sequence %d not attached", sid);
    const SeqSt& S = bk.seqs[sid];
    if (!S.has_tokens || (int)S.tokens.size() != S.valid[VIA_CACHE_SLIM] + 1)
      return fail(VIA_ESTATE, "sequence %d has no committed tokens (via_kv_seq_set_tokens)", sid);
    if (nd < 1 || nd > D) return fail(VIA_EINVAL, "n_drafts[%d] = %d outside [1, %d]", b, nd, D);
    std::vector<int>& rn = rows_of[b];
    rn.push_back(-1);
    if (tree) {
      std::vector<char> has_child(nd, 0);
      for (int j = 0; j < nd; ++j) {
        const int par = d->draft_parent[(size_t)b * D + j];
        if (par < -1 || par >= j) return fail(VIA_EINVAL, "draft_parent[%d][%d] must be -1 or < j", b, j);
        if (par >= 0) has_child[par] = 1;
      }
      for (int j = 0; j < nd; ++j)
        if (has_child[j]) rn.push_back(j);
      if ((int)rn.size() > VIA_MAX_TREE_ROWS) return fail(VIA_EINVAL, "tree windows hold at most %d rows", VIA_MAX_TREE_ROWS);
    } else {
      for (int j = 0; j + 1 < nd; ++j) rn.push_back(j);
    }
    R = std::max(R, (int)rn.size());
    Lg = std::max(Lg, S.valid[VIA_CACHE_SLIM] - S.valid[VIA_CACHE_FULL]);
  }
  sw.seq.assign(d->seq_id, d->seq_id + B);
  sw.n_rows.resize(B);
  sw.n_drafts.assign(d->n_drafts, d->n_drafts + B);
  sw.row_tok.assign((size_t)B * R, 0);
  sw.draft_tok.assign((size_t)B * D, 0);
  sw.draft_row.assign((size_t)B * D, 0);
  if (tree) {
    sw.row_depth.assign((size_t)B * R, 0);
    sw.row_mask.assign((size_t)B * R, 0);
    sw.draft_parent.assign((size_t)B * D, -1);
  }
  if (with_lag) {
    sw.n_lag.assign(B, 0);
    sw.lag_tok.assign((size_t)B * Lg, 0);
  }
  for (int b = 0; b < B; ++b) {
    const SeqSt& S = bk.seqs[d->seq_id[b]];
    const std::vector<int>& rn = rows_of[b];
    const int nd = d->n_drafts[b];
    sw.n_rows[b] = (int)rn.size();
    std::vector<int> row_of(nd, -1), depth(nd, 0);
    for (int r = 0; r < (int)rn.size(); ++r) {
      if (rn[r] >= 0) row_of[rn[r]] = r;
      sw.row_tok[(size_t)b * R + r] = rn[r] < 0 ? S.tokens.back() : d->draft_tok[(size_t)b * D + rn[r]];
    }
    for (int j = 0; j < nd; ++j) {
      const size_t i = (size_t)b * D + j;
      const int par = tree ? d->draft_parent[i] : j - 1;
      sw.draft_tok[i] = d->draft_tok[i];
      sw.draft_row[i] = par < 0 ? 0 : (tree ? row_of[par] : j);
      depth[j] = par < 0 ? 1 : depth[par] + 1;
      if (tree) sw.draft_parent[i] = par;
    }
    if (tree) {
      for (int r = 0; r < (int)rn.size(); ++r) {
        uint64_t mk = 1ull | (1ull << r);
        for (int u = rn[r]; u >= 0; u = d->draft_parent[(size_t)b * D + u]) mk |= 1ull << row_of[u];
        sw.row_mask[(size_t)b * R + r] = mk;
        sw.row_depth[(size_t)b * R + r] = rn[r] < 0 ? 0 : depth[rn[r]];
      }
    }
    if (with_lag) {
      const int vf = S.valid[VIA_CACHE_FULL], n1 = S.valid[VIA_CACHE_SLIM];
      sw.n_lag[b] = n1 - vf;
      for (int i = vf; i < n1; ++i) sw.lag_tok[(size_t)b * Lg + (i - vf)] = S.tokens[i];
    }
  }
  via_window& w = sw.win;
  w.batch = B;
  w.max_rows = R;
  w.max_drafts = D;
  w.max_lag = Lg;
  w.seq_id = sw.seq.data();
  w.n_rows = sw.n_rows.data();
  w.row_tok = sw.row_tok.data();
  w.row_depth = tree ? sw.row_depth.data() : nullptr;
  w.row_mask = tree ? sw.row_mask.data() : nullptr;
  w.n_drafts = sw.n_drafts.data();
  w.draft_tok = sw.draft_tok.data();
  w.draft_row = sw.draft_row.data();
  w.draft_parent = tree ? sw.draft_parent.data() : nullptr;
  w.n_lag = with_lag ? sw.n_lag.data() : nullptr;
  w.lag_tok = with_lag ? sw.lag_tok.data() : nullptr;
  return VIA_OK;
}

int plan_attention(AttnItem* items, int n_items, int KVH, int max_splits, int target_groups, int max_groups,
                   int* span_out, int* max_chunks_out) {
  long long blocks = 0;
  int max_kv = 0;
  for (int i = 0; i < n_items; ++i) {
    blocks += (long long)KVH * ((items[i].kv_len + 31) / 32);
    max_kv = std::max(max_kv, items[i].kv_len);
  }
  long long per = std::max<long long>(1, (blocks + target_groups - 1) / target_groups);
  int span = (int)std::min<long long>(per * 32, kAttnMaxSpan);
  // a forward whose spans would run well past kAttnPrefSpan keys (long
  // contexts with several query items per sequence) takes more work-groups
  if (span > kAttnPrefSpan * 3 / 2) span = kAttnPrefSpan;
  const int need = ((max_kv + 31) / 32 + max_splits - 1) / max_splits * 32;  // at most max_splits splits
  span = std::max(span, need);
  if (span > kAttnMaxSpan) return -1;
  // One round: when these spans leave more work-groups than the GPU has
  // compute units (ragged lengths round up to an extra split; a second
  // work-group on a compute unit halves the bandwidth of both) and one split
  // per item would fit, widen the span to the smallest multiple of 32 that
  // fits, up to the preferred cap.
  auto groups = [&](int sp) {
    long long g = 0;
    for (int i = 0; i < n_items; ++i) g += (long long)KVH * ((items[i].kv_len + sp - 1) / sp);
    return g;
  };
  const int cap = kAttnPrefSpan * 3 / 2;
  if (span < cap && (long long)n_items * KVH <= max_groups && groups(span) > max_groups) {
    int lo = span, hi = std::min(cap, (max_kv + 31) / 32 * 32);
    if (hi > lo && groups(hi) <= max_groups) {
      while (hi - lo > 32) {  // groups(lo) > max_groups >= groups(hi)
        const int mid = (lo + hi) / 64 * 32;
        if (groups(mid) <= max_groups)
          hi = mid;
        else
          lo = mid;
      }
      span = hi;
    }
  }
  int max_chunks = 0;
  for (int i = 0; i < n_items; ++i) {
    items[i].n_chunks = (items[i].kv_len + span - 1) / span;
    max_chunks = std::max(max_chunks, items[i].n_chunks);
  }
  *span_out = span;
  *max_chunks_out = max_chunks;
  return 0;
}

}  // namespace via
