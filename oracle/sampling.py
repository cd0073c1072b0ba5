"""Sampling-mode verification rules (App. A) — TEST INFRASTRUCTURE ONLY.

The paper's main results sample (T > 0).  Its lossy speculative rule
(App. A): an escalated draft token x with drafter probability p(x) and
verifier probability q(x) is accepted with probability
min(1, q(x) / ((1 - alpha) p(x))) (Eq. A.2); a rejected token is replaced by
a sample of norm(max(0, q / beta - p)) (Eq. A.3); alpha = 0, beta = 1 is the
lossless rule, whose output is distributed exactly as q.  A slim-tier
rewrite samples the slim verifier q' (App. B.1: "rewrite x ~ q'").

Random draws are inputs: every draw is a uniform u in [0, 1) consumed by
``inverse_cdf``.  Readings: q and q' are the temperature-T softmax of the
logits; a residual with no mass (q / beta <= p everywhere) falls back to q;
p(x) = 0 accepts (the ratio is infinite).
"""
from __future__ import annotations

import math

import torch

F64 = torch.float64


def tempered(logits: torch.Tensor, T: float) -> torch.Tensor:
    """softmax(logits / T) over the last axis, fp64."""
    z = logits.to(F64) / T
    e = torch.exp(z - z.max())
    return e / e.sum()


def inverse_cdf(w: torch.Tensor, u: float) -> int:
    """The token drawn by uniform u from non-negative weights w (not
    necessarily normalised): the first index whose running sum exceeds
    u * sum(w), scanning in index order."""
    w = w.to(F64)
    target = u * float(w.sum())
    acc = 0.0
    last = 0
    for v in range(w.shape[0]):
        wv = float(w[v])
        if wv > 0.0:
            last = v
            acc += wv
            if acc > target:
                return v
    return last  # u * sum rounds up to the total: the last token with mass


def accept_prob(q_x: float, p_x: float, alpha: float) -> float:
    """Eq. A.2: min(1, q(x) / ((1 - alpha) p(x)))."""
    if p_x <= 0.0:
        return 1.0
    return min(1.0, q_x / ((1.0 - alpha) * p_x))


def residual(q: torch.Tensor, p: torch.Tensor, beta: float) -> torch.Tensor:
    """Eq. A.3 before normalisation: max(0, q / beta - p); q itself when that
    has no mass."""
    r = torch.clamp(q.to(F64) / beta - p.to(F64), min=0.0)
    return r if float(r.sum()) > 0.0 else q.to(F64)
