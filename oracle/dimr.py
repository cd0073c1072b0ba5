"""Routing-mask cost of DIMR (Sec. 3, Eqs. 9-12) — TEST INFRASTRUCTURE ONLY.

Plain fp64 statement of the KL-style verification cost the paper uses to
score a routing mask z (the slim verifier q'_z keeps the layers with
z_l = 1):

  per position t (Eq. 11, phi = ReLU), with p = q'_z and q the full
  verifier, l^p = log p_t, l^q = log q_t:
      z1(v) = log(1 - alpha) + l^p(v) - l^q(v)
      z2(v) = log(beta)      + l^p(v) - l^q(v)
      R_t   = sum_v p_t(v) ReLU(z1(v)) + sum_v q_t(v) ReLU(z2(v))
  over a window of tau positions (Eq. 12): C(z) = sum_t R_t.

Distributions are the temperature-T softmax of each model's logits.  The
window is a calibration token sequence, teacher-forced: position t's
distributions condition on tokens 0..t (the cache-free forward of
``OracleModel.forward_sequence``).  Only tests/ import this module.
"""
from __future__ import annotations

import math

import torch

from .model import OracleModel

F64 = torch.float64


def log_softmax(logits: torch.Tensor, T: float) -> torch.Tensor:
    """log softmax(logits / T) over the last axis, in fp64."""
    z = logits.to(F64) / T
    m = z.max(dim=-1, keepdim=True).values
    return z - m - torch.log(torch.exp(z - m).sum(dim=-1, keepdim=True))


def rkl_cost(q_logits: torch.Tensor, p_logits: torch.Tensor, T: float, alpha: float, beta: float) -> torch.Tensor:
    """R^KL_{alpha,beta}(q || p) of Eq. 11 for every row of [R, V] logits
    (q: the full verifier, p: the routed slim verifier).  Returns [R]."""
    if not (0.0 <= alpha < 1.0) or not beta > 0.0:
        raise ValueError("need 0 <= alpha < 1 and beta > 0")
    lq = log_softmax(q_logits, T)
    lp = log_softmax(p_logits, T)
    d = lp - lq
    z1 = math.log(1.0 - alpha) + d
    z2 = math.log(beta) + d
    return (torch.exp(lp) * torch.clamp(z1, min=0.0)).sum(dim=-1) + (torch.exp(lq) * torch.clamp(z2, min=0.0)).sum(dim=-1)


def mask_cost(model: OracleModel, route, tokens, T: float, alpha: float, beta: float) -> float:
    """C(z) of Eq. 12: the per-position costs of the routed model ``route``
    against the full model, summed over the teacher-forced positions of
    ``tokens``."""
    lq = model.forward_sequence(tokens)
    lp = model.forward_sequence(tokens, route)
    return float(rkl_cost(lq, lp, T, alpha, beta).sum())
