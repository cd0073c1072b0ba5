"""Brute-force hierarchical verification — TEST INFRASTRUCTURE ONLY.

One draft position at a time, in the order of the full algorithm of App. B.1,
with every distribution recomputed from scratch by the cache-free forward
(no KV cache, no window, no lag bookkeeping).  Used on tiny models to pin the
windowed oracle in ``decode.py``.

Per position j of a chain draft d (greedy semantics):
  q'_j = softmax(l'/T) of the slim-verifier on prefix x ++ d_<j, M' = max q'_j.
  If q'_j(d_j) >= tau_full * M' (no escalation):
      accept if q'_j(d_j) >= tau_acc * M', else rewrite with argmax q'_j and stop.
  Else (escalate): q_j = the full verifier on the same prefix; accept if
      d_j = argmax q_j, else rewrite with argmax q_j and stop.
It works with probabilities, not with the logit-difference form used by the
windowed oracle, so the two share no tier arithmetic.

``tree_walk`` / ``verify_tree`` apply the same per-position gate to token
trees (the reading for tree drafts, which the paper does not spell out:
stated in the comment above them), again from fresh forwards of every root
path.
"""
from __future__ import annotations

import torch

from .model import OracleModel


def _softmax(l: torch.Tensor, T: float) -> torch.Tensor:
    z = l / T
    e = torch.exp(z - z.max())
    return e / e.sum()


def verify_block(model: OracleModel, route_slim, x, drafts, tau_acc, tau_full, T, forced=-1):
    """Returns (kappa, emit, tiers) for one chain block; emit = -1 if none."""
    tiers = []
    for j, v in enumerate(drafts):
        prefix = list(x) + list(drafts[:j])
        lq = model.forward_sequence(prefix, route_slim)[-1]
        q1 = _softmax(lq, T)
        M1 = float(q1.max())
        pv = float(q1[v])
        if forced == 0:
            escalate, accept = False, True
        elif forced == 1:
            escalate, accept = False, False
        elif forced == 2:
            escalate, accept = True, False
        else:
            escalate = not (pv >= tau_full * M1)
            accept = pv >= tau_acc * M1
        if not escalate:
            if accept:
                tiers.append("A")
                continue
            tiers.append("S")
            return j, int(torch.argmax(q1)), tiers
        tiers.append("F")
        lfull = model.forward_sequence(prefix)[-1]
        g = int(torch.argmax(lfull))
        if g == v:
            continue
        return j, g, tiers
    return len(drafts), -1, tiers


# ------------------------------------------------------------------ trees
# A token tree generalises the block: each node is a draft token whose prefix
# is x followed by the tokens on its root path.  The per-position gate above
# is applied to every child of the node the walk stands on (all children
# share one prefix, hence one q' and one M'):
#   * children that q' accepts (q'(v) >= tau_acc M'): descend into the one
#     with the largest q'(v), the lowest node index on ties;
#   * else, if some child is confident but not accepted
#     (tau_full M' <= q'(v) < tau_acc M'): rewrite with argmax q' and stop;
#   * else every child escalates: q on the same prefix; descend into the
#     lowest-index child whose token is argmax q, or rewrite with argmax q and
#     stop (stop without a token when q's row is not finite);
#   * a node without children ends the walk with nothing rewritten.
# The walk takes its distributions from callables, so the same rule runs on a
# model (cache-free forwards of each root path) or on hand-written tables.

def _argmax_lowest(v: torch.Tensor) -> int:
    m = v.max()
    return int(torch.nonzero(v == m)[0, 0])


def tree_walk(tok, parent, slim_dist, full_dist, tau_acc, tau_full, forced=-1):
    """Walk one token tree.  ``slim_dist(u)`` / ``full_dist(u)`` give the
    probability vector of q' / q after node u's root path (u = -1: the
    root).  Returns dict(kappa, emit, path, full_used, status)."""
    path, u, full_used = [], -1, False
    while True:
        kids = [j for j in range(len(tok)) if parent[j] == u]
        if not kids:
            return dict(kappa=len(path), emit=-1, path=path, full_used=full_used, status=0)
        q1 = slim_dist(u)
        M1 = float(q1.max())
        acc, rew = [], []
        for j in kids:
            pv = float(q1[tok[j]])
            if forced == 0 or (forced == -1 and pv >= tau_acc * M1):
                acc.append((pv, j))
            elif forced == 1 or (forced == -1 and pv >= tau_full * M1):
                rew.append(j)
        if acc:
            best = max(pv for pv, _ in acc)
            u = min(j for pv, j in acc if pv == best)
            path.append(u)
            continue
        if rew:
            return dict(kappa=len(path), emit=_argmax_lowest(q1), path=path, full_used=full_used, status=0)
        full_used = True
        qf = full_dist(u)
        if not bool(torch.isfinite(qf).all()):
            return dict(kappa=len(path), emit=-1, path=path, full_used=True, status=2)
        g = _argmax_lowest(qf)
        same = [j for j in kids if tok[j] == g]
        if same:
            u = same[0]
            path.append(u)
            continue
        return dict(kappa=len(path), emit=g, path=path, full_used=True, status=0)


def verify_tree(model: OracleModel, route_slim, x, tok, parent, tau_acc, tau_full, T, forced=-1):
    """Tree walk on a model: every distribution is a fresh cache-free forward
    of x followed by the node's root path (slim route or all layers)."""
    def path_of(u):
        out = []
        while u >= 0:
            out.append(tok[u])
            u = parent[u]
        return list(x) + out[::-1]

    slim = lambda u: _softmax(model.forward_sequence(path_of(u), route_slim)[-1], T)
    full = lambda u: _softmax(model.forward_sequence(path_of(u))[-1], 1.0)
    return tree_walk(tok, parent, slim, full, tau_acc, tau_full, forced)
