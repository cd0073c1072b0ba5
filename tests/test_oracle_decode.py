"""Pins of the oracle's verification step and decode loop.

* hand-worked tier cases on the regions of App. B.2 (tests/golden/tier_cases.json);
* partition and monotonicity of the tiers in the thresholds (App. B.18-B.19,
  restated on tau_acc = 1 - alpha_1, tau_full = 1 - alpha_2);
* lossless reduction (App. A: with the full verifier deciding every
  position, decoding is plain greedy decoding from q);
* forced accept reproduces the draft stream; an accept threshold above 1
  with tau_full <= 0 gives slim-verifier greedy decoding, one token a step;
* the windowed, cached, lagging oracle against the brute-force per-position
  algorithm of App. B.1 (no cache at all);
* KV index invariants and the paged allocator rule; tree forward and tree
  compaction against chain forwards of each path.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import bruteforce
from oracle.decode import (A, F, FORCED_ACCEPT, FORCED_FULL, S, Draft, GreedyDrafter, PagedIndex,
                           TierParams, Verifier, confidence, greedy_decode, row_stats, tier_of)
from oracle.model import OracleModel, SeqCache, causal, forward_window
from workload import configs, gen

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def tiny():
    cfg = configs.get("tiny_fp32")
    return cfg, OracleModel(cfg["model"], gen.model_weights(cfg))


def _corrupt(cfg, p=None):
    p = cfg["corrupt"] if p is None else p
    V = cfg["model"]["vocab"]
    return lambda b, step, j: gen.corruption(cfg["seed_d"], b, step, j, p, V)


def run_decode(cfg, m, params, G, prompt_len=None, k=None, drafter_p=None, batch=1):
    ver = Verifier(m, cfg["route"], block_size=cfg.get("block_size", 16))
    dr = GreedyDrafter(m, _corrupt(cfg, drafter_p))
    n0 = prompt_len or cfg["ctx"][0]
    for b in range(batch):
        ver.prefill(gen.context_tokens(cfg, b, n0))
        dr.attach(b)
    k = k or cfg["k"]
    steps = []
    step = 0
    while True:
        active = [b for b in range(batch) if ver.seqs[b].n - n0 < G]
        if not active:
            break
        drafts = {b: dr.chain(b, ver.seqs[b].tokens, k, step) for b in active}
        dec = ver.step(drafts, params)
        steps.append((drafts, dec))
        for b in active:
            st = ver.seqs[b]
            assert st.slim.valid == st.n - 1
            if dec[b]["full_ran"]:
                assert st.full.valid == st.n - 1
            else:
                assert st.full.valid <= st.n - 1
        step += 1
    return ver, steps, n0


def test_golden_tier_cases():
    g = json.load(open(os.path.join(HERE, "golden", "tier_cases.json")))
    p = TierParams(g["tau_acc"], g["tau_full"], 1.0)
    for c in g["cases"]:
        l = torch.tensor(c["logits"], dtype=torch.float64)
        st = row_stats(l[None], 1.0)
        cc = confidence(c["logits"][c["draft"]], st["max"][0], 1.0)
        assert abs(cc - c["ratio"]) < 1e-15
        assert tier_of(cc, p) == c["tier"], c
    for c in g["boundary"]:
        assert tier_of(c["ratio"], p) == c["tier"], c


def test_tier_partition_and_monotonicity():
    rng = np.random.default_rng(0)
    codes = {A: 0, S: 1, F: 2}
    for _ in range(2000):
        t_full, t_acc = sorted(rng.uniform(0, 1, 2))
        c1, c2 = sorted(rng.uniform(0, 1, 2))
        p = TierParams(t_acc, t_full, 1.0)
        t1, t2 = tier_of(c1, p), tier_of(c2, p)
        # exactly one region (A u B u C = Omega, regions disjoint)
        regions = [c1 >= t_acc, t_full <= c1 < t_acc, c1 < t_full]
        assert sum(regions) == 1 and codes[t1] == regions.index(True)
        # lower confidence never gets a less escalated tier
        assert codes[t1] >= codes[t2]
        # raising tau_acc shrinks the accept set; raising tau_full grows the escalate set
        hi = TierParams(min(1.0, t_acc + rng.uniform(0, 0.5)), t_full, 1.0)
        if tier_of(c1, hi) == A:
            assert t1 == A
        hi2 = TierParams(max(t_acc, t_full + rng.uniform(0, 0.5)), t_full + 0, 1.0)
        hi2.tau_full = min(hi2.tau_acc, t_full + rng.uniform(0, 0.5))
        if t1 == F:
            assert tier_of(c1, hi2) == F


def test_ratio_is_one_iff_argmax():
    rng = np.random.default_rng(1)
    for _ in range(200):
        l = torch.tensor(np.round(rng.normal(size=50), 1), dtype=torch.float64)
        st = row_stats(l[None], 0.7)
        for v in range(50):
            c = confidence(float(l[v]), st["max"][0], 0.7)
            assert (c == 1.0) == (float(l[v]) == st["max"][0])
        assert float(l[st["argmax"][0]]) == st["max"][0]
        assert all(float(l[u]) < st["max"][0] for u in range(st["argmax"][0]))


def test_forced_full_is_greedy_decoding(tiny):
    cfg, m = tiny
    G = 24
    ver, steps, n0 = run_decode(cfg, m, TierParams(forced=FORCED_FULL), G)
    ref = greedy_decode(m, gen.context_tokens(cfg, 0, n0), G)
    assert ver.seqs[0].tokens[n0:n0 + G] == ref
    # q ran every step, so its cache never lags
    assert all(dec[0]["full_ran"] for _, dec in steps)


def test_forced_accept_is_draft_stream(tiny):
    cfg, m = tiny
    ver, steps, n0 = run_decode(cfg, m, TierParams(forced=FORCED_ACCEPT), 16)
    stream = []
    for drafts, dec in steps:
        assert dec[0]["kappa"] == cfg["k"] and dec[0]["emit"] == -1
        stream += drafts[0].tok
    assert ver.seqs[0].tokens[n0:] == stream


@pytest.mark.parametrize("taus", [(1.5, 0.0), (1.0, 0.0)])
def test_slim_greedy_limits(tiny, taus):
    cfg, m = tiny
    G = 12
    ver, steps, n0 = run_decode(cfg, m, TierParams(taus[0], taus[1], 1.0), G)
    ref = greedy_decode(m, gen.context_tokens(cfg, 0, n0), G, route=cfg["route"])
    assert ver.seqs[0].tokens[n0:n0 + G] == ref
    if taus[0] > 1:
        assert all(dec[0]["kappa"] == 0 and dec[0]["emit"] >= 0 for _, dec in steps)


def test_windowed_oracle_matches_bruteforce(tiny):
    cfg, m = tiny
    p = TierParams(0.9, 0.5, 1.0)
    ver, steps, n0 = run_decode(cfg, m, p, 20)
    x = gen.context_tokens(cfg, 0, n0)
    seen = set()
    for drafts, dec in steps:
        d = drafts[0].tok
        kappa, emit, tiers = bruteforce.verify_block(m, cfg["route"], x, d, p.tau_acc, p.tau_full, 1.0)
        assert (kappa, emit) == (dec[0]["kappa"], dec[0]["emit"])
        assert tiers == dec[0]["tiers"][:len(tiers)]
        seen.update(tiers)
        x = x + d[:kappa] + ([emit] if emit >= 0 else [])
    assert x == ver.seqs[0].tokens
    assert seen == {A, S, F}, seen            # every tier exercised


def test_lag_rows_and_kv_invariants(tiny):
    cfg, m = tiny
    ver, steps, n0 = run_decode(cfg, m, TierParams(0.9, 0.5, 1.0), 40, batch=2)
    lagged = False
    for drafts, dec in steps:
        for b in dec:
            lagged |= not dec[b]["full_ran"]
    assert lagged, "want at least one step without q so the full cache lags"
    for b in range(2):
        st = ver.seqs[b]
        for which, cache in (("full", st.full), ("slim", st.slim)):
            t = ver.block_table(which, b)
            assert len(t) == (cache.valid + 15) // 16
    # every block is owned at most once across sequences and caches of a kind
    for idx in (ver.idx_full, ver.idx_slim):
        owned = [blk for t in idx.tables.values() for blk in t]
        assert len(owned) == len(set(owned))
        assert not set(owned) & set(idx.free)


def test_paged_allocator_rule():
    idx = PagedIndex(8, 4)
    idx.ensure(0, 5)       # blocks 0,1
    idx.ensure(1, 4)       # block 2
    idx.ensure(0, 9)       # block 3
    assert idx.tables == {0: [0, 1, 3], 1: [2]}
    idx.trim(0, 4)         # keeps block 0 only
    assert idx.tables[0] == [0]
    idx.ensure(1, 12)      # lowest free first: 1, 3
    assert idx.tables[1] == [2, 1, 3]
    with pytest.raises(MemoryError):
        idx.ensure(0, 100)
    assert idx.tables[0] == [0]


def _chain_logits(m, route, prefix, path_toks):
    return m.forward_sequence(list(prefix) + list(path_toks), route)[len(prefix) - 1:]


def test_tree_forward_matches_chain_forward_per_path(tiny):
    cfg, m = tiny
    x = gen.context_tokens(cfg, 0, 20)
    # a small tree: root -> {0, 1}; 0 -> {2, 3}; 1 -> {4}; 3 -> {5}
    d = Draft([11, 12, 13, 14, 15, 16], [-1, -1, 0, 0, 1, 3])
    row_nodes, draft_row, depth, vis = d.layout()
    for route in (list(range(m.L)), cfg["route"]):
        c = SeqCache(len(route), m.KVH, m.hd)
        forward_window(m, route, c, x[:-1], range(len(x) - 1), causal(len(x) - 1))
        c.valid = len(x) - 1
        toks = [x[-1]] + [d.tok[u] for u in row_nodes[1:]]
        pos = [len(x) - 1 + dd for dd in depth]
        lg = forward_window(m, route, c, toks, pos, vis)
        for r, u in enumerate(row_nodes):
            path = []
            while u >= 0:
                path.append(d.tok[u])
                u = d.parent[u]
            ref = m.forward_sequence(x + path[::-1], route)[-1]
            assert torch.allclose(lg[r], ref, rtol=0, atol=1e-11)


def test_tree_compaction_equals_recompute(tiny):
    cfg, m = tiny
    ver = Verifier(m, cfg["route"])
    dr = GreedyDrafter(m, _corrupt(cfg, 0.2))
    x = gen.context_tokens(cfg, 0, 24)
    ver.prefill(x)
    dr.attach(0)
    found = False
    for step in range(6):
        tree = dr.tree(0, ver.seqs[0].tokens, [3, 4, 3], 2, step)
        dec = ver.step({0: tree}, TierParams(0.9, 0.5, 1.0, forced=FORCED_FULL))
        st = ver.seqs[0]
        # the compacted caches equal a fresh forward over the committed tokens
        for cache, route in ((st.slim, cfg["route"]),) + (((st.full, list(range(m.L))),) if dec[0]["full_ran"] else ()):
            ref = SeqCache(len(route), m.KVH, m.hd)
            toks = st.tokens[:-1]
            forward_window(m, route, ref, toks, range(len(toks)), causal(len(toks)))
            for s in range(len(route)):
                assert torch.allclose(cache.K[s][:cache.valid], ref.K[s][:cache.valid], rtol=0, atol=1e-11)
                assert torch.allclose(cache.V[s][:cache.valid], ref.V[s][:cache.valid], rtol=0, atol=1e-11)
        found |= any(u != j for j, u in enumerate(dec[0]["path"]))
    assert found, "want a step whose accepted path is not the first-child chain"
    # with the full verifier deciding, the tree walk is greedy decoding too
    ref = greedy_decode(m, x, len(ver.seqs[0].tokens) - len(x))
    assert ver.seqs[0].tokens[len(x):] == ref


def test_chain_as_tree_of_branching_one(tiny):
    cfg, m = tiny
    x = gen.context_tokens(cfg, 2, 16)
    d1 = Draft.chain([5, 6, 7, 8])
    d2 = Draft([5, 6, 7, 8], [-1, 0, 1, 2])
    outs = []
    for d in (d1, d2):
        ver = Verifier(m, cfg["route"])
        ver.prefill(x)
        dec = ver.step({0: d}, TierParams(0.9, 0.5, 1.0))[0]
        outs.append((dec["kappa"], dec["emit"], dec["tiers"], ver.seqs[0].tokens))
    assert outs[0] == outs[1]


def test_decode_is_deterministic(tiny):
    cfg, m = tiny
    a, _, _ = run_decode(cfg, m, TierParams(0.9, 0.5, 1.0), 10)
    b, _, _ = run_decode(cfg, m, TierParams(0.9, 0.5, 1.0), 10)
    assert a.seqs[0].tokens == b.seqs[0].tokens
    assert a.block_table("slim", 0) == b.block_table("slim", 0)


def _golden_tree():
    return json.load(open(os.path.join(HERE, "golden", "tree_walk_cases.json")))


@pytest.mark.parametrize("case", range(len(_golden_tree()["cases"])))
def test_golden_tree_walk_cases(case):
    """Hand-worked tree walks (tests/golden/tree_walk_cases.json) against both
    the windowed oracle's gate walk and the brute-force tree walk."""
    g = _golden_tree()
    c = g["cases"][case]
    rows = {k: torch.tensor(v, dtype=torch.float64) for k, v in g["rows"].items()}
    T = g["temperature"]
    p = TierParams(g["tau_acc"], g["tau_full"], T)
    d = Draft(list(c["tok"]), list(c["parent"]))
    row_nodes, draft_row, _, _ = d.layout()
    zero = rows["Z"]
    slim_rows = torch.stack([rows[c["slim"].get(str(u), "Z")] for u in row_nodes])
    full_rows = torch.stack([rows[c["full"].get(str(u), "Z")] for u in row_nodes])
    st = row_stats(slim_rows, T)
    conf = [confidence(float(slim_rows[draft_row[j], d.tok[j]]), st["max"][draft_row[j]], T)
            for j in range(len(d.tok))]
    tiers = [tier_of(x, p) for x in conf]
    want = c["expect"]
    first = Verifier._walk(d, tiers, conf, st, None)
    if want["full_used"]:
        assert first["needs_full"] and first["status"] == 1, c["name"]
        got = Verifier._walk(d, tiers, conf, st, row_stats(full_rows, 1.0))
    else:
        assert not first["needs_full"], c["name"]
        got = first
    assert (got["kappa"], got["path"], got["emit"], got["status"]) == \
        (want["kappa"], want["path"], want["emit"], want["status"]), c["name"]
    # the brute-force walk from probabilities (softmax of the same rows)
    sm = lambda v, t: torch.softmax(v / t, dim=0)
    bf = bruteforce.tree_walk(d.tok, d.parent, lambda u: sm(rows[c["slim"].get(str(u), "Z")], T),
                              lambda u: sm(rows[c["full"].get(str(u), "Z")], 1.0), p.tau_acc, p.tau_full)
    assert (bf["kappa"], bf["path"], bf["emit"], bf["status"], bf["full_used"]) == \
        (want["kappa"], want["path"], want["emit"], want["status"], want["full_used"]), c["name"]
    assert zero.abs().sum() == 0


# T = 1 reaches the escalation branches (descend into argmax q, rewrite with
# it) and slim rewrites; T = 8 accepts several siblings, so the choice by
# confidence matters.
@pytest.mark.parametrize("T,branches", [
    (1.0, {"slim-rewrite", "escalate-rewrite", "escalate-descend"}),
    (8.0, {"accept-first", "accept-by-confidence"}),
])
def test_tree_walk_natural_tiers_matches_bruteforce(tiny, T, branches):
    """The windowed oracle on token trees with natural tiers (slim cache, lag
    rows, tree mask, compaction) against the brute-force tree walk, which
    recomputes q' and q for every node from its root path without a cache."""
    cfg, m = tiny
    p = TierParams(0.9, 0.5, T)
    x = gen.context_tokens(cfg, 1, 24)
    ver = Verifier(m, cfg["route"])
    ver.prefill(x)
    dr = GreedyDrafter(m, _corrupt(cfg, 0.3))
    dr.attach(0)
    seen = set()
    for step in range(10):
        tree = dr.tree(0, ver.seqs[0].tokens, [3, 4, 3], 2, step)
        before = list(ver.seqs[0].tokens)
        dec = ver.step({0: tree}, p)[0]
        bf = bruteforce.verify_tree(m, cfg["route"], before, tree.tok, tree.parent, p.tau_acc, p.tau_full,
                                    p.temperature)
        assert (dec["kappa"], dec["path"], dec["emit"], dec["full_ran"]) == \
            (bf["kappa"], bf["path"], bf["emit"], bf["full_used"]), f"step {step}"
        # which branches of the rule this step took
        u = -1
        for j in dec["path"]:
            kids = tree.children(u)
            acc = [k for k in kids if dec["tiers"][k] == A]
            if acc:
                seen.add("accept-first" if j == kids[0] else "accept-by-confidence")
            else:
                seen.add("escalate-descend")
            u = j
        if dec["emit"] >= 0:
            kids = tree.children(u)
            seen.add("escalate-rewrite" if all(dec["tiers"][k] == F for k in kids) else "slim-rewrite")
        elif tree.children(u):
            raise AssertionError("walk stopped without a rewrite at a node with children")
        else:
            seen.add("leaf")
    assert branches <= seen, seen


def test_nonfinite_full_logits_not_committed():
    """A non-finite full-verifier row at an escalated position: status 2, the
    sequence is not advanced, both caches keep their valid lengths and the
    blocks the step took past them are free again; the slim verifier (which
    bypasses the poisoned layer) is unaffected."""
    cfg = configs.get("tiny_fp32")
    W = gen.model_weights(cfg)
    W["w_down"][1] = np.full_like(W["w_down"][1], np.inf)   # layer 1 is not in the slim route [0, 3]
    m = OracleModel(cfg["model"], W)
    ver = Verifier(m, cfg["route"])
    x = gen.context_tokens(cfg, 0, 31)                      # 30 cached slots: two blocks
    ver.prefill(x)
    tables = (ver.block_table("full", 0), ver.block_table("slim", 0))
    dec = ver.step({0: Draft.chain([1, 2, 3, 4])}, TierParams(0.9, 0.5, 1.0, FORCED_FULL))[0]
    assert (dec["status"], dec["kappa"], dec["emit"], dec["new_len"]) == (2, 0, -1, len(x))
    assert all(math.isfinite(v) for v in dec["slim_stats"]["max"])
    assert not math.isfinite(dec["full_stats"]["max"][0])
    st = ver.seqs[0]
    assert st.tokens == x and st.slim.valid == st.full.valid == len(x) - 1
    assert (ver.block_table("full", 0), ver.block_table("slim", 0)) == tables
    # a later step without q commits normally
    dec = ver.step({0: Draft.chain([1, 2, 3, 4])}, TierParams(0.9, 0.5, 1.0, FORCED_ACCEPT))[0]
    assert dec["status"] == 0 and ver.seqs[0].tokens == x + [1, 2, 3, 4]
