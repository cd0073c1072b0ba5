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
