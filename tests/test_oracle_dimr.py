"""Pins of the DIMR routing cost (oracle/dimr.py) against values worked out by
hand from Eq. 11 (phi = ReLU) and against properties the definition fixes.

Hand cases (natural logs; p = slim q'_z, q = full verifier, T = 1):
* alpha = 0, beta = 1, p = (1/2, 1/2), q = (1/4, 3/4): only token 0 has
  p > q, so both terms pick up log(p/q) = ln 2 there:
  R = (1/2 + 1/4) ln 2.
* the same with p and q swapped: only token 1 has p > q:
  R = (3/4 + 1/2) ln(3/2)  (the cost is not symmetric).
* alpha = 1/2, beta = 2, p = (.6, .3, .1), q = (.2, .5, .3):
  log(p/q) = (ln 3, ln .6, -ln 3); the acceptance term is positive only for
  token 0 (ln .5 + ln 3 = ln 1.5), the replacement term for tokens 0 and 1
  (ln 2 + ln 3 = ln 6, ln 2 + ln .6 = ln 1.2):
  R = .6 ln 1.5 + .2 ln 6 + .5 ln 1.2.
"""
import math

import numpy as np
import pytest
import torch

from oracle.dimr import mask_cost, rkl_cost
from oracle.model import OracleModel
from workload import configs, gen


def lg(p):
    return torch.log(torch.tensor([p], dtype=torch.float64))


def test_two_token_worked_example():
    r = rkl_cost(lg([0.25, 0.75]), lg([0.5, 0.5]), 1.0, 0.0, 1.0)
    assert float(r[0]) == pytest.approx(0.75 * math.log(2.0), rel=1e-12)


def test_cost_is_not_symmetric():
    r = rkl_cost(lg([0.5, 0.5]), lg([0.25, 0.75]), 1.0, 0.0, 1.0)
    assert float(r[0]) == pytest.approx(1.25 * math.log(1.5), rel=1e-12)


def test_three_token_worked_example_with_alpha_and_beta():
    r = rkl_cost(lg([0.2, 0.5, 0.3]), lg([0.6, 0.3, 0.1]), 1.0, 0.5, 2.0)
    want = 0.6 * math.log(1.5) + 0.2 * math.log(6.0) + 0.5 * math.log(1.2)
    assert float(r[0]) == pytest.approx(want, rel=1e-12)


@pytest.mark.parametrize("alpha,beta", [(0.0, 1.0), (0.3, 0.5), (0.3, 1.7)])
def test_identical_distributions_cost_relu_log_beta(alpha, beta):
    g = torch.Generator().manual_seed(3)
    l = torch.randn(5, 97, generator=g, dtype=torch.float64) * 3
    r = rkl_cost(l, l.clone(), 1.7, alpha, beta)
    assert torch.allclose(r, torch.full((5,), max(0.0, math.log(beta)), dtype=torch.float64), atol=1e-12)


def test_row_shifts_and_temperature():
    g = torch.Generator().manual_seed(5)
    lq = torch.randn(4, 200, generator=g, dtype=torch.float64) * 4
    lp = lq + torch.randn(4, 200, generator=g, dtype=torch.float64)
    r = rkl_cost(lq, lp, 2.5, 0.1, 1.2)
    shifted = rkl_cost(lq + torch.randn(4, 1, generator=g, dtype=torch.float64) * 50,
                       lp - torch.randn(4, 1, generator=g, dtype=torch.float64) * 50, 2.5, 0.1, 1.2)
    assert torch.allclose(r, shifted, rtol=1e-10, atol=1e-12)
    assert torch.allclose(r, rkl_cost(lq / 2.5, lp / 2.5, 1.0, 0.1, 1.2), rtol=1e-12)
    # both terms are non-negative; the acceptance term cannot grow with alpha
    assert (r >= 0).all()
    a = [float(rkl_cost(lq, lp, 2.5, al, 1e-30).sum()) for al in (0.0, 0.2, 0.5, 0.9)]
    assert all(x >= y - 1e-12 for x, y in zip(a, a[1:]))


def test_mask_cost_of_the_full_route_is_relu_log_beta_per_position():
    cfg = configs.get("micro_f32")
    cfg["seed_c"] = 7
    md = cfg["model"]
    om = OracleModel(md, gen.model_weights(cfg))
    toks = gen.context_tokens(cfg, 0, 12)
    full = list(range(md["n_layers"]))
    assert mask_cost(om, full, toks, 1.0, 0.2, 1.5) == pytest.approx(12 * math.log(1.5), rel=1e-9)
    assert mask_cost(om, full, toks, 1.0, 0.2, 1.0) == pytest.approx(0.0, abs=1e-12)
    # a routed model differs from the full one: positive cost
    assert mask_cost(om, full[::2], toks, 1.0, 0.0, 1.0) > 0.0


def test_rejects_out_of_range_parameters():
    l = lg([0.5, 0.5])
    with pytest.raises(ValueError):
        rkl_cost(l, l, 1.0, 1.0, 1.0)
    with pytest.raises(ValueError):
        rkl_cost(l, l, 1.0, 0.0, 0.0)
