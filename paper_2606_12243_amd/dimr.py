"""Dynamic intra-model routing (Sec. 3): choose the slim verifier's routing
mask z by minimising the KL-style cost C(z) (Eq. 12) with random search and a
periodic Bayesian-optimisation proposal (Eq. 13).

``RoutingCost`` evaluates C(z) on the GPU: the full verifier's logits over a
teacher-forced calibration window are computed once; for each mask the
routed model's logits come from a probe forward of the slim route and
``via_dimr_cost`` reduces both over the vocabulary.  ``MaskSearch`` is the
host search; it only needs a cost function.
"""
from __future__ import annotations

import ctypes as C
import math

import numpy as np
import torch

from . import via


class RoutingCost:
    """C(z) of routing masks of one model over one calibration window.

    ``tokens``: the window (position t conditions on tokens 0..t; the cost
    sums its len(tokens) positions).  T, alpha, beta as in Eq. 11.
    """

    def __init__(self, model: via.Model, tokens, T=1.0, alpha=0.0, beta=1.0):
        self.m = model
        self.tokens = [int(t) for t in tokens]
        self.T, self.alpha, self.beta = float(T), float(alpha), float(beta)
        self.V = model.desc["vocab"]
        self.n = len(self.tokens)
        self.full_route = list(range(model.desc["n_layers"]))
        self.q_logits = self._logits(self.full_route, via.CACHE_FULL)
        self.cost_rows = torch.empty(self.n, dtype=torch.float32, device="cuda")
        self.evaluated = {}

    def _logits(self, route, cache):
        """Logits [n, V] of the model under ``route`` (the full cache runs all
        layers; the slim cache the route) over the window."""
        m = self.m
        if list(route) != m.route:  # needs no live KV handle of the model
            r, rp = via._i32(list(route))
            via.check(via.via_model_set_route(m.h, rp, len(r)))
            m.route = list(route)
        n = self.n
        blocks = (n + via.BLOCK - 1) // via.BLOCK + 2
        kv = via.KV(m, max_seqs=1, max_blocks_per_seq=blocks, blocks_full=blocks, blocks_slim=blocks,
                    max_rows=n, max_batch=1, max_drafts=1)
        try:
            sp = C.c_void_p(torch.cuda.current_stream().cuda_stream)
            via.check(via.via_kv_seq_reserve(kv.h, 0, 0))  # empty cache: the window is the whole sequence
            w = via.WindowBuf([0], [self.tokens], [[]], [[]], max_drafts=1)
            out = via.Out(1, n, 1, self.V, logits=True)
            p = via.tier_params(0.9, 0.5, 1.0)
            via.check(via.via_verify_probe(m.h, kv.h, cache, C.byref(w.c), C.byref(p), C.byref(out.c), sp))
            torch.cuda.current_stream().synchronize()
            return out.logits.view(n, self.V).clone()
        finally:
            kv.close()

    def __call__(self, route) -> float:
        key = tuple(sorted(int(l) for l in route))
        if key in self.evaluated:
            return self.evaluated[key]
        p_logits = self._logits(key, via.CACHE_SLIM)
        sp = C.c_void_p(torch.cuda.current_stream().cuda_stream)
        via.check(via.via_dimr_cost(self.q_logits.data_ptr(), p_logits.data_ptr(), self.n, self.V, self.V,
                                    self.T, self.alpha, self.beta, self.cost_rows.data_ptr(), sp))
        c = float(self.cost_rows.double().sum().item())
        self.evaluated[key] = c
        return c


class MaskSearch:
    """Search over masks keeping ``n_keep`` of ``n_layers`` layers (Eq. 13):
    every ``theta``-th step a Bayesian-optimisation proposal, otherwise a
    uniformly random unseen mask.  Stops after ``max_steps`` evaluations or
    when the best mask has not changed for ``patience`` steps.

    The Bayesian step fits a Gaussian-process surrogate to the evaluated
    (mask, cost) pairs -- kernel exp(-Hamming / ell) on the keep-indicator
    vectors, costs standardised -- and evaluates the candidate with the
    largest expected improvement (minimisation) among random unseen masks
    and the one-swap neighbours of the best mask.  ``fixed`` layers are
    always kept.
    """

    def __init__(self, n_layers, n_keep, cost_fn, seed=0, theta=4, max_steps=32, patience=10, fixed=(),
                 n_random_candidates=256):
        if not 1 <= n_keep <= n_layers or len(set(fixed)) > n_keep:
            raise ValueError("need 1 <= n_keep <= n_layers and at most n_keep fixed layers")
        self.L, self.k = n_layers, n_keep
        self.cost = cost_fn
        self.rng = np.random.default_rng(seed)
        self.theta, self.max_steps, self.patience = theta, max_steps, patience
        self.fixed = tuple(sorted(set(int(l) for l in fixed)))
        self.free = [l for l in range(n_layers) if l not in self.fixed]
        self.n_cand = n_random_candidates
        self.history = []  # (mask, cost, kind)

    def _random_mask(self):
        pick = self.rng.choice(len(self.free), self.k - len(self.fixed), replace=False)
        return tuple(sorted(self.fixed + tuple(self.free[i] for i in pick)))

    def _onehot(self, masks):
        X = np.zeros((len(masks), self.L))
        for i, m in enumerate(masks):
            X[i, list(m)] = 1.0
        return X

    def _neighbours(self, mask):
        keep = set(mask)
        out = []
        for a in mask:
            if a in self.fixed:
                continue
            for b in range(self.L):
                if b not in keep:
                    out.append(tuple(sorted((keep - {a}) | {b})))
        return out

    def _bayes_proposal(self, seen):
        masks = [h[0] for h in self.history]
        y = np.array([h[1] for h in self.history], np.float64)
        mu0, sd0 = y.mean(), y.std() or 1.0
        ys = (y - mu0) / sd0
        X = self._onehot(masks)
        ell = max(1.0, self.L / 4.0)

        def kern(A, B):
            ham = np.abs(A[:, None, :] - B[None, :, :]).sum(-1)
            return np.exp(-ham / ell)

        Kxx = kern(X, X) + 1e-6 * np.eye(len(X))
        Lc = np.linalg.cholesky(Kxx)
        alpha = np.linalg.solve(Lc.T, np.linalg.solve(Lc, ys))
        best = min(self.history, key=lambda h: h[1])[0]
        cands = {m for m in self._neighbours(best) if m not in seen}
        for _ in range(self.n_cand):
            m = self._random_mask()
            if m not in seen:
                cands.add(m)
        if not cands:
            return None
        cands = sorted(cands)
        Xc = self._onehot(cands)
        Ks = kern(Xc, X)
        mu = Ks @ alpha
        v = np.linalg.solve(Lc, Ks.T)
        var = np.clip(1.0 - (v * v).sum(0), 1e-12, None)
        sd = np.sqrt(var)
        fbest = ys.min()
        z = (fbest - mu) / sd
        cdf = 0.5 * (1.0 + np.vectorize(math.erf)(z / math.sqrt(2.0)))
        pdf = np.exp(-0.5 * z * z) / math.sqrt(2.0 * math.pi)
        ei = (fbest - mu) * cdf + sd * pdf
        return cands[int(np.argmax(ei))]

    def run(self):
        """Returns (best mask, its cost); ``history`` keeps every evaluation."""
        seen = set()
        best, best_c, since = None, math.inf, 0
        for step in range(self.max_steps):
            m = None
            if step > 0 and step % self.theta == 0 and len(self.history) >= 2:
                m, kind = self._bayes_proposal(seen), "bayes"
            if m is None:
                kind = "random"
                for _ in range(64):
                    m = self._random_mask()
                    if m not in seen:
                        break
                if m in seen:
                    break  # (nearly) exhausted search space
            seen.add(m)
            c = float(self.cost(m))
            self.history.append((m, c, kind))
            if c < best_c:
                best, best_c, since = m, c, 0
            else:
                since += 1
                if since >= self.patience:
                    break
        return best, best_c
