"""Pins of the sampling-mode rules (oracle/sampling.py, App. A).

* ``inverse_cdf`` over a fine grid of uniforms reproduces its weights
  (a draw is a quantile of the running sum).
* Lossless identity (alpha = 0, beta = 1): drafting x ~ p, keeping it with
  probability A.2 and otherwise drawing the A.3 residual yields exactly q
  (the speculative-sampling theorem) -- integrated over grids of the two
  uniforms, so a wrong acceptance ratio, residual or quantile rule breaks it.
* The lossy rule keeps more drafts as alpha grows, and beta > 1 shrinks the
  residual; q == p leaves no residual mass (the fallback to q).
* Through the Verifier on a micro model: a forced slim rewrite emits the
  quantile of q' from the cache-free forward of the slim route; forced
  escalation with u = 0 keeps every draft the verifier gives mass to.
"""
import numpy as np
import pytest
import torch

from oracle.decode import FORCED_FULL, FORCED_SLIM, Draft, TierParams, Verifier
from oracle.model import OracleModel
from oracle.sampling import accept_prob, inverse_cdf, residual, tempered
from workload import configs, gen

GRID = 4000


def grid():
    return (np.arange(GRID) + 0.5) / GRID


def test_inverse_cdf_reproduces_its_weights():
    w = torch.tensor([1.0, 0.0, 3.0, 2.0, 0.0, 2.0], dtype=torch.float64)
    counts = np.zeros(6)
    for u in grid():
        counts[inverse_cdf(w, float(u))] += 1
    assert counts[1] == 0 and counts[4] == 0
    assert np.allclose(counts / GRID, (w / w.sum()).numpy(), atol=1.0 / GRID)
    assert inverse_cdf(w, 0.0) == 0 and inverse_cdf(w, 0.9999999) == 5


def output_distribution(q, p, alpha, beta):
    """P(emitted token) of one escalated position with x ~ p, over the grids."""
    V = q.shape[0]
    out = np.zeros(V)
    r = residual(q, p, beta)
    res_tok = np.array([inverse_cdf(r, float(u)) for u in grid()])
    res_dist = np.bincount(res_tok, minlength=V) / GRID
    for x in range(V):
        if p[x] <= 0:
            continue
        a = accept_prob(float(q[x]), float(p[x]), alpha)
        keep = np.mean(grid() < a)
        out[x] += float(p[x]) * keep
        out += float(p[x]) * (1.0 - keep) * res_dist
    return out


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_lossless_rule_outputs_the_verifier_distribution(seed):
    g = torch.Generator().manual_seed(seed)
    q = torch.softmax(torch.randn(7, generator=g, dtype=torch.float64) * 2, 0)
    p = torch.softmax(torch.randn(7, generator=g, dtype=torch.float64) * 2, 0)
    got = output_distribution(q, p, 0.0, 1.0)
    assert np.allclose(got, q.numpy(), atol=3.0 / GRID)


def test_lossy_rule_is_not_q_and_keeps_more_drafts():
    q = torch.tensor([0.1, 0.6, 0.3], dtype=torch.float64)
    p = torch.tensor([0.5, 0.2, 0.3], dtype=torch.float64)
    lossy = output_distribution(q, p, 0.5, 1.0)
    assert abs(lossy[0] - 0.1) > 0.05          # token 0 is over-kept
    a = [accept_prob(0.1, 0.5, al) for al in (0.0, 0.3, 0.6, 0.9)]
    assert a == sorted(a) and a[0] == pytest.approx(0.2) and a[-1] == 1.0
    assert accept_prob(0.3, 0.0, 0.0) == 1.0


def test_residual_scaling_and_fallback():
    q = torch.tensor([0.1, 0.6, 0.3], dtype=torch.float64)
    p = torch.tensor([0.5, 0.2, 0.3], dtype=torch.float64)
    assert torch.allclose(residual(q, p, 1.0), torch.tensor([0.0, 0.4, 0.0], dtype=torch.float64))
    assert torch.allclose(residual(q, p, 1.5), torch.tensor([0.0, 0.2, 0.0], dtype=torch.float64))
    assert torch.equal(residual(q, q.clone(), 1.0), q)  # no mass left: fall back to q


def micro():
    cfg = configs.get("micro_f32")
    cfg["seed_c"] = 5
    md = cfg["model"]
    W = gen.model_weights(cfg)
    return cfg, md, OracleModel(md, W)


def test_forced_slim_rewrite_samples_the_slim_verifier():
    cfg, md, om = micro()
    toks = gen.context_tokens(cfg, 0, 10)
    ver = Verifier(om, cfg["route"])
    ver.prefill(toks)
    d = [int(t) for t in gen.context_tokens(cfg, 1, 3)]
    u = [[0.0, 0.37, 0.0]] * 3
    probs = {0: torch.full((3, md["vocab"]), 1.0 / md["vocab"], dtype=torch.float64)}
    dec = ver.step({0: Draft.chain(d)}, TierParams(forced=FORCED_SLIM, temperature=1.3),
                   sampling=dict(alpha=0.0, beta=1.0, probs=probs, u={0: u}))[0]
    # independent path: the cache-free slim forward on the prefix, then the quantile
    ls = om.forward_sequence(toks, cfg["route"])[-1]
    want = inverse_cdf(tempered(ls, 1.3), 0.37)
    assert dec["kappa"] == 0 and dec["emit"] == want


def test_forced_escalation_with_zero_uniform_keeps_every_draft():
    cfg, md, om = micro()
    toks = gen.context_tokens(cfg, 0, 9)
    ver = Verifier(om, cfg["route"])
    ver.prefill(toks)
    d = [int(t) for t in gen.context_tokens(cfg, 2, 4)]
    probs = {0: torch.full((4, md["vocab"]), 1.0 / md["vocab"], dtype=torch.float64)}
    dec = ver.step({0: Draft.chain(d)}, TierParams(forced=FORCED_FULL),
                   sampling=dict(alpha=0.0, beta=1.0, probs=probs, u={0: [[0.0, 0.5, 0.5]] * 4}))[0]
    assert dec["kappa"] == 4 and dec["emit"] == -1 and dec["full_ran"]
    assert ver.seqs[0].tokens[-4:] == d


def test_sampled_walk_first_token_is_distributed_as_q():
    """The walk itself (not only its rules): with escalated positions, the
    lossless rule and the first draft drawn from p_0, the first committed
    token (d_0 if kept, else the emitted sample) is distributed as q_0,
    integrated over grids of the acceptance and residual uniforms.  A walk
    that read the wrong uniform, the wrong p row or the wrong q row fails."""
    V, G = 5, 48
    g = torch.Generator().manual_seed(4)
    fl = torch.randn(2, V, generator=g, dtype=torch.float64) * 1.5       # full logits, rows 0 and 1
    p = torch.softmax(torch.randn(2, V, generator=g, dtype=torch.float64) * 1.5, -1)
    q0 = tempered(fl[0], 1.0)
    full = (fl, {"max": fl.max(dim=1).values.tolist()})
    slim = (torch.zeros(2, V, dtype=torch.float64), None)
    grid_g = (np.arange(G) + 0.5) / G
    dist = np.zeros(V)
    for d0 in range(V):
        for u0 in grid_g:
            for u2 in grid_g:
                u = [[float(u0), 0.5, float(u2)], [0.99, 0.5, 0.5]]   # the second draft is never kept
                dec = Verifier._walk_sampled(Draft.chain([d0, 0]), ["F", "F"], slim, full, 1.0, 0.0, 1.0, p, u)
                first = d0 if dec["kappa"] >= 1 else dec["emit"]
                dist[first] += float(p[0, d0]) / (G * G)
    assert np.allclose(dist, q0.numpy(), atol=3.0 / G)
