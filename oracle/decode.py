"""Oracle verification step and decode loop — TEST INFRASTRUCTURE ONLY.

Written from the paper's hierarchical verification (Alg. 1 and its full form
in App. B.1, the regions B.1-B.3 of App. B.2, the pipeline Steps 3-4 of
Sec. 3.4) with greedy semantics.  Only the test suite, the smoke check and
the benchmark's CPU-baseline leg may use it.

Readings taken where the paper is silent or inconsistent:
  * Confidence of draft token d at a position is the ratio
    c = q'(d) / max_u q'(u) = exp((l'(d) - max_u l'(u)) / T), with q' the
    slim-verifier's distribution at temperature T (App. B.2 gates q'(v)
    against a fraction of M' = max_u q'(u)).
  * Tiers (regions A/B/C of App. B.2): accept "A" if c >= tau_acc; slim
    rewrite "S" if tau_full <= c < tau_acc; escalate "F" if c < tau_full.
    tau_acc plays 1 - alpha_1 and tau_full plays 1 - alpha_2 with
    tau_acc >= tau_full.
  * Greedy rules: a slim rewrite emits argmax q'; an escalated position is
    accepted iff d == argmax q, else argmax q is emitted; ties go to the
    lowest token id.  A slim rewrite ends the step without calling q.
  * Positions are walked in order; the first non-accepted position ends the
    step (longest accepted prefix kappa, Sec. 3.4 Step 4).  When every draft
    is accepted no extra token is emitted (t <- t + gamma in Alg. 1).
  * Rows fed: the pending token x[n-1] and the first k-1 drafts; the output
    of row j verifies draft j (App. B.1 runs q' on prefixes x_<t .. x_<t+gamma-1).
  * The full verifier's cache lags when q is not invoked; its next forward
    re-feeds the committed tokens it is missing ("lag rows").
  * Tree drafts: the fed rows are the root (pending token) and every draft
    node with children, in node order; a node's RoPE position is
    n - 1 + depth and it sees its ancestors and itself.  The walk descends
    into the accepted child with the largest confidence (lowest index on
    ties); if no child is accepted, a slim-tier child ends the step with a
    slim rewrite, otherwise q is consulted and the child equal to argmax q
    (lowest index) is taken, or argmax q is emitted.
  * KV pages: caches are paged in blocks; before a forward a sequence takes
    the lowest free block ids until its rows fit; after the commit every
    block lying wholly at or beyond the new valid length is freed.

Parity pins: tests/test_oracle_decode.py (forced-full == greedy decoding,
the lossless reduction of App. A; tier partition and monotonicity B.18-B.19;
brute-force agreement; KV index invariants; chain == tree of branching 1;
the tree walk against hand-worked walks, tests/golden/tree_walk_cases.json,
and against the brute-force tree walk with natural tiers).
"""
from __future__ import annotations

import heapq
import math
from dataclasses import dataclass, field

import numpy as np
import torch

from .model import OracleModel, SeqCache, causal, forward_window
from .sampling import accept_prob, inverse_cdf, residual, tempered

A, S, F = "A", "S", "F"
FORCED_NONE, FORCED_ACCEPT, FORCED_SLIM, FORCED_FULL = -1, 0, 1, 2
TIER_CODE = {A: 0, S: 1, F: 2}


@dataclass
class TierParams:
    tau_acc: float = 0.9
    tau_full: float = 0.5
    temperature: float = 1.0
    forced: int = FORCED_NONE


def row_stats(logits: torch.Tensor, T: float) -> dict:
    """Per-row max, argmax (lowest id on ties), sum exp((l - max)/T) and
    top-2 gap (max minus the largest other entry; 0 on a tie)."""
    mx, am = [], []
    for r in range(logits.shape[0]):
        row = logits[r]
        m = float(row.max())
        idx = int(torch.nonzero(row == m)[0, 0]) if math.isfinite(m) else 0
        mx.append(m)
        am.append(idx)
    mx_t = torch.tensor(mx, dtype=torch.float64)
    se = torch.exp((logits - mx_t[:, None]) / T).sum(dim=1)
    gaps = []
    for r in range(logits.shape[0]):
        row = logits[r].clone()
        row[am[r]] = float("-inf")
        gaps.append(mx[r] - float(row.max()))
    return dict(max=mx, argmax=am, sumexp=[float(v) for v in se], gap=gaps)


def confidence(l_d: float, l_max: float, T: float) -> float:
    """c = q'(d) / max_u q'(u) = exp((l'(d) - max l') / T)."""
    return math.exp((l_d - l_max) / T)


def tier_of(c: float, p: TierParams) -> str:
    """Region of App. B.2 for ratio confidence c (forced modes override)."""
    if p.forced == FORCED_ACCEPT:
        return A
    if p.forced == FORCED_SLIM:
        return S
    if p.forced == FORCED_FULL:
        return F
    if c >= p.tau_acc:
        return A
    if c >= p.tau_full:
        return S
    return F          # includes a NaN confidence


# ---------------------------------------------------------------- drafts
@dataclass
class Draft:
    """A draft block for one sequence.

    Chain: ``parent[j] = j - 1`` (``-1`` for the first).  Tree: node order is
    breadth-first; ``parent[j]`` is the parent node index or -1 (root).
    """
    tok: list
    parent: list

    @staticmethod
    def chain(tokens):
        return Draft(list(tokens), [j - 1 for j in range(len(tokens))])

    def depth(self, j):
        d = 1
        while self.parent[j] >= 0:
            j = self.parent[j]
            d += 1
        return d

    def children(self, u):
        """Draft indices whose parent is ``u`` (u = -1: children of the root)."""
        return [j for j, p in enumerate(self.parent) if p == u]

    def layout(self):
        """Fed rows: root then every node with a child, in node order.

        Returns (row_nodes, draft_row, row_depth, win_vis):
        row_nodes[r] = node index of row r (-1 for the root);
        draft_row[j] = row whose output verifies draft j (its parent's row);
        row_depth[r] = depth of row r (root 0); win_vis = ancestors-and-self mask.
        """
        has_child = set(p for p in self.parent if p >= 0)
        row_nodes = [-1] + [j for j in range(len(self.tok)) if j in has_child]
        row_of = {u: r for r, u in enumerate(row_nodes)}
        draft_row = [row_of[p] for p in self.parent]
        row_depth = [0] + [self.depth(u) for u in row_nodes[1:]]
        R = len(row_nodes)
        vis = np.zeros((R, R), dtype=bool)
        for r, u in enumerate(row_nodes):
            vis[r, 0] = True
            vis[r, r] = True
            while u >= 0:
                vis[r, row_of[u]] = True
                u = self.parent[u]
        return row_nodes, draft_row, row_depth, vis


# ---------------------------------------------------------------- paging
class PagedIndex:
    """Block allocator of one cache: lowest free id first."""

    def __init__(self, n_blocks: int, block_size: int):
        self.bs = block_size
        self.free = list(range(n_blocks))
        heapq.heapify(self.free)
        self.tables = {}

    def ensure(self, seq, n_slots: int):
        t = self.tables.setdefault(seq, [])
        need = (n_slots + self.bs - 1) // self.bs
        if need - len(t) > len(self.free):
            raise MemoryError("KV pool exhausted")
        while len(t) < need:
            t.append(heapq.heappop(self.free))

    def trim(self, seq, valid: int):
        t = self.tables.setdefault(seq, [])
        keep = (valid + self.bs - 1) // self.bs
        for blk in t[keep:]:
            heapq.heappush(self.free, blk)
        del t[keep:]

    def release(self, seq):
        self.trim(seq, 0)
        self.tables.pop(seq, None)


# ------------------------------------------------------------ sequences
@dataclass
class SeqState:
    tokens: list                 # committed tokens x[0..n-1]; x[n-1] is pending
    full: SeqCache
    slim: SeqCache
    n_ctx: int = 0
    full_ran: bool = False
    done: bool = False
    history: list = field(default_factory=list)

    @property
    def n(self):
        return len(self.tokens)


class Verifier:
    """Oracle decoding state for a batch of sequences sharing one verifier.

    ``route``: retained layer ids of the slim-verifier.  Both caches are
    paged with the same block size; ``n_blocks_*`` bound the pools.
    """

    def __init__(self, model: OracleModel, route, block_size=16, n_blocks_full=1 << 30,
                 n_blocks_slim=1 << 30):
        self.m = model
        self.route_full = list(range(model.L))
        self.route_slim = list(route)
        self.idx_full = PagedIndex(min(n_blocks_full, 1 << 20), block_size)
        self.idx_slim = PagedIndex(min(n_blocks_slim, 1 << 20), block_size)
        self.seqs = []

    def _new_seq(self, tokens, n_ctx):
        m = self.m
        st = SeqState(list(tokens), SeqCache(len(self.route_full), m.KVH, m.hd),
                      SeqCache(len(self.route_slim), m.KVH, m.hd), n_ctx=n_ctx)
        self.seqs.append(st)
        return len(self.seqs) - 1

    def prefill(self, tokens):
        """Cache the prompt x[0..n-2] in both caches; x[n-1] stays pending."""
        b = self._new_seq(tokens, len(tokens) - 1)
        st = self.seqs[b]
        ctx = st.tokens[:-1]
        for cache, route, idx in ((st.full, self.route_full, self.idx_full),
                                  (st.slim, self.route_slim, self.idx_slim)):
            idx.ensure(b, len(ctx))
            if ctx:
                forward_window(self.m, route, cache, ctx, range(len(ctx)), causal(len(ctx)))
            cache.valid = len(ctx)
        return b

    def attach_context(self, tokens, kv_full, kv_slim):
        """Sequence whose context K/V are given (synthetic context).

        ``tokens`` has n entries; slots [0, n-1) of each cache take the given
        K/V (lists over route layers of (K, V) fp64 tensors [n-1, KVH, hd]).
        """
        b = self._new_seq(tokens, len(tokens) - 1)
        st = self.seqs[b]
        n1 = len(tokens) - 1
        for cache, kv, idx in ((st.full, kv_full, self.idx_full), (st.slim, kv_slim, self.idx_slim)):
            idx.ensure(b, n1)
            for s, (k, v) in enumerate(kv):
                cache.set_context(s, k, v)
            cache.valid = n1
        return b

    # -------------------------------------------------------------- forwards
    def _slim_forward(self, b, draft: Draft):
        st = self.seqs[b]
        row_nodes, draft_row, row_depth, vis = draft.layout()
        toks = [st.tokens[-1]] + [draft.tok[u] for u in row_nodes[1:]]
        pos = [st.n - 1 + dd for dd in row_depth]
        self.idx_slim.ensure(b, st.slim.valid + len(toks))
        return forward_window(self.m, self.route_slim, st.slim, toks, pos, vis)

    def _full_forward(self, b, draft: Draft):
        st = self.seqs[b]
        row_nodes, draft_row, row_depth, vis = draft.layout()
        lag = st.tokens[st.full.valid: st.n - 1]
        nl = len(lag)
        toks = lag + [st.tokens[-1]] + [draft.tok[u] for u in row_nodes[1:]]
        pos = [st.full.valid + i for i in range(nl)] + [st.n - 1 + dd for dd in row_depth]
        R = len(toks)
        wv = np.zeros((R, R), dtype=bool)
        wv[:nl, :nl] = causal(nl)
        wv[nl:, :nl] = True
        wv[nl:, nl:] = vis
        self.idx_full.ensure(b, st.full.valid + R)
        logits = forward_window(self.m, self.route_full, st.full, toks, pos, wv)
        return logits[nl:]

    # ------------------------------------------------------------------ step
    def step(self, drafts: dict, p: TierParams, sampling: dict = None) -> dict:
        """One verification step for the active sequences.

        ``drafts``: {seq index: Draft}.  Returns {seq: decision dict} and
        commits every decision (tokens, cache lengths, tree compaction,
        block frees).

        ``sampling`` (chain drafts only) switches the rewrite and escalation
        rules to sampling (App. A, module ``sampling``): dict with ``alpha``,
        ``beta``, ``probs`` {seq: [k, V] drafter distributions p_j} and ``u``
        {seq: [k][3] uniforms: acceptance, slim sample, residual sample}.
        """
        order = sorted(drafts)
        T = p.temperature
        slim, dec = {}, {}
        for b in order:                               # slim-verifier pass
            lg = self._slim_forward(b, drafts[b])
            slim[b] = (lg, row_stats(lg, T))
        for b in order:
            d = drafts[b]
            _, draft_row, _, _ = d.layout()
            lg, stt = slim[b]
            conf = [confidence(float(lg[draft_row[j], d.tok[j]]), stt["max"][draft_row[j]], T)
                    for j in range(len(d.tok))]
            tiers = [tier_of(c, p) for c in conf]
            dec[b] = dict(conf=conf, tiers=tiers, slim_stats=stt, draft_row=draft_row, slim_logits=lg,
                          slim_draft_logit=[float(lg[draft_row[j], d.tok[j]]) for j in range(len(d.tok))])
            dec[b].update(self._walk_any(b, d, tiers, conf, slim[b], None, p, sampling))
            dec[b]["first_status"] = dec[b]["status"]
        full = {}
        for b in order:                               # escalation to q
            if dec[b]["needs_full"]:
                lg = self._full_forward(b, drafts[b])
                full[b] = (lg, row_stats(lg, 1.0))
                dec[b]["full_stats"] = full[b][1]
                dec[b]["full_logits"] = lg
                d = drafts[b]
                dec[b]["full_draft_logit"] = [float(lg[dec[b]["draft_row"][j], d.tok[j]])
                                              for j in range(len(d.tok))]
                dec[b].update(self._walk_any(b, d, dec[b]["tiers"], dec[b]["conf"], slim[b], full[b], p, sampling))
                dec[b]["full_ran"] = True
            else:
                dec[b]["full_ran"] = False
        for b in order:
            self._commit(b, drafts[b], dec[b])
        return dec

    def _walk_any(self, b, d: Draft, tiers, conf, slim, full, p: TierParams, sampling):
        if sampling is None:
            return self._walk(d, tiers, conf, slim[1], None if full is None else full[1])
        return self._walk_sampled(d, tiers, slim, full, p.temperature, sampling["alpha"], sampling["beta"],
                                  sampling["probs"][b], sampling["u"][b])

    @staticmethod
    def _walk_sampled(d: Draft, tiers, slim, full, T, alpha, beta, probs, u):
        """Chain walk with sampling rules: accept-tier drafts are kept; a
        slim-tier position emits a sample of q'_j (uniform u[j][1]); an
        escalated position keeps d_j with probability A.2 (accepted iff
        u[j][0] < that probability), else emits a sample of the A.3 residual
        (uniform u[j][2])."""
        if d.parent is not None and any(par != j - 1 for j, par in enumerate(d.parent)):
            raise ValueError("sampling mode takes chain drafts")
        path = []
        for j in range(len(d.tok)):
            if tiers[j] == A:
                path.append(j)
                continue
            if tiers[j] == S:
                qs = tempered(slim[0][j], T)
                return dict(kappa=len(path), emit=inverse_cdf(qs, float(u[j][1])), path=path,
                            needs_full=False, status=0)
            if full is None:
                return dict(kappa=len(path), emit=-1, path=path, needs_full=True, status=1)
            if not math.isfinite(full[1]["max"][j]):
                return dict(kappa=len(path), emit=-1, path=path, needs_full=False, status=2)
            q = tempered(full[0][j], T)
            pj = torch.as_tensor(probs[j], dtype=torch.float64)
            x = d.tok[j]
            if float(u[j][0]) < accept_prob(float(q[x]), float(pj[x]), alpha):
                path.append(j)
                continue
            return dict(kappa=len(path), emit=inverse_cdf(residual(q, pj, beta), float(u[j][2])), path=path,
                        needs_full=False, status=0)
        return dict(kappa=len(path), emit=-1, path=path, needs_full=False, status=0)

    @staticmethod
    def _walk(d: Draft, tiers, conf, slim_stats, full_stats):
        """Gate walk of App. B.1 over a chain or tree.

        Returns kappa, emit (-1 none), path (accepted draft indices), and
        needs_full (the walk reached an escalated position and q's logits are
        not given yet).  status 2 marks non-finite logits of q.
        """
        row_of_parent = d.layout()[1]
        path, u = [], -1
        while True:
            kids = d.children(u)
            if not kids:
                return dict(kappa=len(path), emit=-1, path=path, needs_full=False, status=0)
            r = row_of_parent[kids[0]]
            acc = [j for j in kids if tiers[j] == A]
            if acc:
                u = max(acc, key=lambda j: (conf[j], -j))
                path.append(u)
                continue
            if any(tiers[j] == S for j in kids):
                return dict(kappa=len(path), emit=slim_stats["argmax"][r], path=path,
                            needs_full=False, status=0)
            if full_stats is None:
                return dict(kappa=len(path), emit=-1, path=path, needs_full=True, status=1)
            if not math.isfinite(full_stats["max"][r]):
                return dict(kappa=len(path), emit=-1, path=path, needs_full=False, status=2)
            g = full_stats["argmax"][r]
            same = [j for j in kids if d.tok[j] == g]
            if same:
                u = same[0]
                path.append(u)
                continue
            return dict(kappa=len(path), emit=g, path=path, needs_full=False, status=0)

    def _commit(self, b, d: Draft, dec):
        st = self.seqs[b]
        n = st.n
        if dec["status"] == 2:
            # not advanced: both caches keep their valid lengths, and the blocks
            # this step's forwards took past them are freed like any others
            dec["new_len"] = n
            self.idx_slim.trim(b, st.slim.valid)
            self.idx_full.trim(b, st.full.valid)
            return
        new = [d.tok[j] for j in dec["path"]] + ([dec["emit"]] if dec["emit"] >= 0 else [])
        n2 = n + len(new)
        # tree compaction: K/V of accepted path nodes move to contiguous slots
        row_nodes = d.layout()[0]
        row_of = {u: r for r, u in enumerate(row_nodes)}
        kv_needed = n2 - 1 - (n - 1)          # window slots that stay valid after the root
        caches = [st.slim] + ([st.full] if dec["full_ran"] else [])
        for cache in caches:
            base = n - 1
            for i in range(1, kv_needed):
                src = base + row_of[dec["path"][i - 1]]
                if src != base + i:
                    cache.move(src, base + i)
        st.tokens.extend(new)
        st.slim.valid = n2 - 1
        if dec["full_ran"]:
            st.full.valid = n2 - 1
        self.idx_slim.trim(b, st.slim.valid)
        self.idx_full.trim(b, st.full.valid)
        dec["new_len"] = n2
        st.history.append(dict(kappa=dec["kappa"], emit=dec["emit"], full_ran=dec["full_ran"]))

    def block_table(self, which: str, b: int) -> list:
        idx = self.idx_full if which == "full" else self.idx_slim
        return list(idx.tables.get(b, []))


# -------------------------------------------------------------- drafters
class GreedyDrafter:
    """Synthetic drafter: the full verifier's greedy token on the draft's own
    prefix, with positions replaced at random (workload corruption draws).

    Keeps its own cache of the committed prefix (full route, no paging).
    """

    def __init__(self, model: OracleModel, corrupt_fn):
        self.m = model
        self.route = list(range(model.L))
        self.caches = {}
        self.corrupt_fn = corrupt_fn          # (b, step, j) -> (replace, token)

    def attach(self, b, kv_full=None):
        c = SeqCache(self.m.L, self.m.KVH, self.m.hd)
        if kv_full is not None:
            for s, (k, v) in enumerate(kv_full):
                c.set_context(s, k, v)
            c.valid = kv_full[0][0].shape[0]
        self.caches[b] = c

    def _catch_up(self, b, tokens):
        c = self.caches[b]
        todo = tokens[c.valid: len(tokens) - 1]
        if todo:
            forward_window(self.m, self.route, c, todo, range(c.valid, c.valid + len(todo)),
                           causal(len(todo)))
            c.valid += len(todo)

    def chain(self, b, tokens, k, step) -> Draft:
        self._catch_up(b, tokens)
        c = self.caches[b]
        keep = c.valid
        out, cur = [], tokens[-1]
        for j in range(k):
            lg = forward_window(self.m, self.route, c, [cur], [c.valid], [[True]])
            c.valid += 1
            g = int(torch.argmax(lg[0]))              # first index of the max
            rep, tok = self.corrupt_fn(b, step, j)
            cur = tok if rep else g
            out.append(cur)
        c.valid = keep
        return Draft.chain(out)

    def tree(self, b, tokens, budget, branch, step) -> Draft:
        """Token tree: per depth, earlier nodes expand first with up to
        ``branch`` children each; children are the parent's top tokens
        under q, each replaced at random."""
        self._catch_up(b, tokens)
        c = self.caches[b]
        toks, parents = [], []
        frontier = [-1]
        for depth, nb in enumerate(budget, start=1):
            # which frontier nodes expand and how many children each gets
            plan, left = [], nb
            for u in frontier:
                if left <= 0:
                    break
                take = min(branch, left)
                plan.append((u, take))
                left -= take
            # forward the tree so far (root + all existing nodes) to read q at the expanders
            cur = Draft(list(toks), list(parents))
            nodes = [-1] + list(range(len(toks)))
            row_of = {u: r for r, u in enumerate(nodes)}
            R = len(nodes)
            vis = np.zeros((R, R), dtype=bool)
            for r, u in enumerate(nodes):
                vis[r, 0] = True
                vis[r, r] = True
                while u >= 0:
                    vis[r, row_of[u]] = True
                    u = parents[u]
            row_toks = [tokens[-1]] + list(toks)
            row_pos = [len(tokens) - 1] + [len(tokens) - 1 + cur.depth(u) for u in range(len(toks))]
            lg = forward_window(self.m, self.route, c, row_toks, row_pos, vis)
            new_frontier = []
            for u, take in plan:
                row = lg[row_of[u]]
                order = sorted(range(row.shape[0]), key=lambda v: (-float(row[v]), v))[:take]
                for t in order:
                    j = len(toks)
                    rep, tok = self.corrupt_fn(b, step, j)
                    toks.append(tok if rep else int(t))
                    parents.append(u)
                    new_frontier.append(j)
            frontier = new_frontier
        return Draft(toks, parents)

    def committed(self, b, tokens):
        """Nothing to do: the next draft catches up from the committed tokens."""
        return None


def greedy_decode(model: OracleModel, tokens, G: int, route=None):
    """Plain autoregressive greedy decoding from q (cache-free forward)."""
    x = list(tokens)
    out = []
    for _ in range(G):
        lg = model.forward_sequence(x, route)
        g = int(torch.argmax(lg[-1]))
        x.append(g)
        out.append(g)
    return out
