"""Sampling-rule decisions on the GPU (via_tier_decide_sampled, App. A)
against the oracle's sampled walk (oracle/decode.py, oracle/sampling.py).

Both sides decode the same sequences from the same chain drafts, drafter
distributions p and uniforms.  Per step the decision (status, kappa, the
accepted path, the emitted token, the new length) must match.  The two
sides compute q and q' from their own forwards (fp32 / bf16 kernels vs
fp64), which agree to the lock-step logit tolerance, so the uniforms are
chosen from the oracle's distributions with a margin that tolerance cannot
cross:
* an acceptance uniform stays further than the induced relative error
  from the A.2 probability;
* a sampling uniform is the midpoint of its token's interval of the
  running weight, when that interval is wider than the induced error of
  the running weight; otherwise the GPU's token is only checked to be one
  whose widened interval holds the uniform ("several results are
  correct").
Cases: forced escalation (every draft goes to the A.2/A.3 rules), forced
slim rewrite (a sample of q'), the ordinary tier thresholds with a greedy
drafter, the lossless and lossy rules, a residual with no mass (beta huge:
the fallback to q), a drafter probability of zero (always kept), a ragged
vocabulary (3001) past the kernel's 256-thread chunking.  After each step
the GPU commits the oracle's decision, so both keep the same state.
"""
import copy
import ctypes as C
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

from oracle.decode import (FORCED_FULL, FORCED_NONE, FORCED_SLIM, Draft, GreedyDrafter,  # noqa: E402
                           TierParams, Verifier)
from oracle.model import OracleModel  # noqa: E402
from oracle.sampling import accept_prob, inverse_cdf, residual, tempered  # noqa: E402
from paper_2606_12243_amd import via  # noqa: E402
from paper_2606_12243_amd.session import ModelDrafter, Session  # noqa: E402
from workload import configs, gen  # noqa: E402

TIER_CODE = {"A": 0, "S": 1, "F": 2}


def logit_tol(md):
    return 2e-2 if md["dtype"] == "bf16" else 1e-4


def running(w):
    """Interval ends F(v-1), F(v) of every token under weights w (fp64)."""
    c = torch.cumsum(w, 0) / w.sum()
    return torch.cat([torch.zeros(1, dtype=w.dtype), c[:-1]]), c


def pick_uniform(w, err, rng):
    """(u, exact, lo, hi): a uniform inside one token's interval, its
    midpoint when the interval's half-width exceeds err."""
    lo, hi = running(w)
    half = (hi - lo) / 2
    u0 = float(rng.random())
    v = int(torch.searchsorted(hi, torch.tensor([u0], dtype=hi.dtype), right=True).clamp(max=len(hi) - 1))
    if float(half[v]) <= err:
        v = int(torch.argmax(half))
    u = float(np.float32((lo[v] + hi[v]) / 2))
    return u, float(half[v]) > err + 1e-7, lo, hi


class SampledLockstep:
    def __init__(self, name, params, alpha, beta, greedy_drafts=False, seed=0, batch=3, k=4, drafter_route=None,
                 drafter_T=1.0, drafter_cfg=None):
        cfg = configs.get(name)
        cfg["seed_c"] = 21 + seed
        cfg["seed_d"] = 31 + seed
        self.cfg, self.md = cfg, cfg["model"]
        W = gen.model_weights(cfg)
        self.om = OracleModel(self.md, W)
        self.ver = Verifier(self.om, cfg["route"], block_size=16)
        self.gm = via.Model(self.md, W, cfg["route"])
        self.kv = via.KV(self.gm, max_seqs=batch, max_blocks_per_seq=16, blocks_full=64, blocks_slim=64,
                         max_rows=64, max_batch=batch, max_drafts=8)
        self.p = params
        self.sess = Session(self.gm, self.kv, via.tier_params(params.tau_acc, params.tau_full, params.temperature,
                                                             params.forced), logits=True)
        self.alpha, self.beta = alpha, beta
        self.rng = np.random.default_rng(1000 + seed)
        self.B, self.k = batch, k
        self.drafter = None
        if greedy_drafts:
            V = self.md["vocab"]
            self.drafter = GreedyDrafter(self.om, lambda b, step, j: gen.corruption(cfg["seed_d"], b, step, j,
                                                                                      0.3, V))
        # drafter model (GPU: ModelDrafter; oracle: cache-free forwards of its
        # route): the verifier's weights under a shallower route, or a model of
        # its own (drafter_cfg: own weights and dimensions, same vocabulary)
        self.dr, self.rel_p = None, 0.0
        if drafter_cfg is not None:
            dmd = drafter_cfg["model"]
            assert dmd["vocab"] == self.md["vocab"]
            dW = gen.model_weights(drafter_cfg)
            self.dr_om, self.dr_md = OracleModel(dmd, dW), dmd
            drafter_route = list(range(dmd["n_layers"])) if drafter_route is None else drafter_route
        else:
            dW, self.dr_om, self.dr_md = W, self.om, self.md
        if drafter_route is not None:
            self.dr_route, self.dr_T = list(drafter_route), float(drafter_T)
            self.dr_model = via.Model(self.dr_md, dW, self.dr_route)
            self.dr_kv = via.KV(self.dr_model, max_seqs=batch, max_blocks_per_seq=16, blocks_full=64,
                                blocks_slim=64, max_rows=64, max_batch=batch, max_drafts=8)
            self.dr = ModelDrafter(self.dr_model, self.dr_kv, self.dr_T)
            self.rel_p = math.exp(2 * logit_tol(self.dr_md) / self.dr_T) - 1
        self.oid = {}
        for b in range(batch):
            toks = gen.context_tokens(cfg, b, 9 + 5 * b)
            self.oid[b] = self.ver.prefill(toks)
            self.sess.prefill(b, toks)
            if self.drafter:
                self.drafter.attach(b)
            if self.dr:
                self.dr.attach(b, toks)
        self.stats = dict(exact=0, loose=0, kept=0, rejected=0, slim=0, fallback=0, steps=0)

    def close(self):
        if self.dr:
            self.dr_kv.close()
            self.dr_model.close()
        self.kv.close()
        self.gm.close()

    def model_drafts(self, order):
        """Drafts of the drafter model: the oracle picks each uniform
        (margin-safe midpoint of a token's interval under its own p) and its
        token; the GPU drafter draws with the same uniforms.  Compared: the
        tokens (exactly) and p (within the induced relative error)."""
        U = np.zeros((len(order), self.k), np.float32)
        drafts, probs = {}, {}
        for i, b in enumerate(order):
            pre = list(self.ver.seqs[self.oid[b]].tokens)
            d, rows = [], []
            for j in range(self.k):
                lg = self.dr_om.forward_sequence(pre + d, self.dr_route)[-1]
                p = tempered(lg, self.dr_T)
                u, exact, lo, hi = pick_uniform(p, 2 * self.rel_p, self.rng)
                assert exact, "no token interval is wide enough for an exact draw"
                U[i, j] = u
                d.append(inverse_cdf(p, u))
                rows.append(p)
            drafts[b], probs[b] = Draft.chain(d), torch.stack(rows)
        dg, P = self.dr.draft(order, self.k, U)
        for i, b in enumerate(order):
            assert dg[b] == drafts[b].tok, f"drafter tokens {dg[b]} vs oracle {drafts[b].tok}"
            pg = P[i].double().cpu()
            err = (pg - probs[b]).abs() - (self.rel_p * probs[b] + 1e-7)
            assert float(err.max()) <= 0, f"drafter p off by {float((pg - probs[b]).abs().max())}"
        self.stats["drafted"] = self.stats.get("drafted", 0) + len(order) * self.k
        return drafts, probs, P

    def drafts(self, step):
        V = self.md["vocab"]
        out = {}
        for b in range(self.B):
            if self.drafter:
                out[b] = self.drafter.chain(b, self.ver.seqs[self.oid[b]].tokens, self.k, step)
            else:
                out[b] = Draft.chain([int(t) for t in self.rng.integers(0, V, self.k)])
        return out

    def probs(self, drafts):
        V = self.md["vocab"]
        P = {}
        for b, d in drafts.items():
            z = torch.from_numpy(self.rng.standard_normal((len(d.tok), V))) * 1.5
            for j, x in enumerate(d.tok):  # give the drafted token a visible share
                z[j, x] += float(self.rng.uniform(0.0, 4.0))
            p = torch.softmax(z, -1).to(torch.float32)
            if len(d.tok) > 2:
                p[2, d.tok[2]] = 0.0  # p(x) = 0: the draft is always kept
                p[2] /= p[2].sum()
            P[b] = p.double()
        return P

    def step(self, step):
        T = self.p.temperature
        P_dev = None
        if self.dr:
            drafts, probs, P_dev = self.model_drafts(list(range(self.B)))
        else:
            drafts = self.drafts(step)
            probs = self.probs(drafts)
        order = sorted(drafts)
        oids = {b: self.oid[b] for b in order}
        D = max(len(drafts[b].tok) for b in order)
        rel = math.exp(2 * logit_tol(self.md) / T) - 1
        # the oracle's distributions for this step, from a copy of its state
        probe = copy.deepcopy(self.ver, memo={id(self.om): self.om})
        u_dummy = {oids[b]: [[0.5, 0.5, 0.5]] * len(drafts[b].tok) for b in order}
        pre = probe.step({oids[b]: drafts[b] for b in order}, self.p,
                         sampling=dict(alpha=self.alpha, beta=self.beta, probs={oids[b]: probs[b] for b in order},
                                       u=u_dummy))
        U = np.full((self.B, D, 3), 0.5, np.float32)
        checks = {}
        for i, b in enumerate(order):
            do = pre[oids[b]]
            d = drafts[b]
            for j, x in enumerate(d.tok):
                row = do["draft_row"][j]
                qs = tempered(do["slim_logits"][row], T)
                U[i, j, 1], ex1, lo1, hi1 = pick_uniform(qs, 2 * rel, self.rng)
                checks[(b, j, 1)] = (ex1, lo1, hi1, 2 * rel)
                if do["full_ran"]:
                    q = tempered(do["full_logits"][row], T)
                    a = accept_prob(float(q[x]), float(probs[b][j, x]), self.alpha)
                    m = (rel + self.rel_p) * a + 1e-6
                    can_keep, can_reject = a - m > 0, a + m < 1
                    keep = can_keep and (not can_reject or self.rng.random() < 0.6)
                    u0 = self.rng.uniform(0.0, a - m) if keep else self.rng.uniform(a + m, 1.0) if can_reject else 0.5
                    U[i, j, 0] = min(np.float32(u0), np.float32(0.99999))
                    r = residual(q, probs[b][j], self.beta)
                    if float(torch.clamp(q / self.beta - probs[b][j], min=0).sum()) <= 0:
                        err = 2 * rel
                        self.stats["fallback"] += 1
                    else:
                        err = 2 * (rel * float(q.sum()) / self.beta + self.rel_p) / float(r.sum())
                    U[i, j, 2], ex2, lo2, hi2 = pick_uniform(r, err, self.rng)
                    checks[(b, j, 2)] = (ex2, lo2, hi2, err)
        # the oracle's real step
        dec_o = self.ver.step({oids[b]: drafts[b] for b in order}, self.p,
                              sampling=dict(alpha=self.alpha, beta=self.beta,
                                            probs={oids[b]: probs[b] for b in order},
                                            u={oids[b]: U[i, :len(drafts[b].tok)].astype(np.float64).tolist()
                                               for i, b in enumerate(order)}))
        # the GPU step: same drafts, p, uniforms
        if P_dev is None:
            P = torch.full((self.B, D, self.md["vocab"]), 1.0 / self.md["vocab"], dtype=torch.float32)
            for i, b in enumerate(order):
                P[i, :len(drafts[b].tok)] = probs[b].float()
            P_dev = P.cuda()
        smp = via.Sampling(self.alpha, self.beta, P_dev, U)
        gd = {b: (drafts[b].tok, None) for b in order}
        w, h, run = self.sess.begin(gd, smp)
        tiers_g = self.sess.dec.tier.cpu().numpy()
        for i, b in enumerate(order):
            do = dec_o[oids[b]]
            n = len(drafts[b].tok)
            tg = tiers_g[i * w.max_drafts:i * w.max_drafts + n]
            if list(tg) != [TIER_CODE[t] for t in do["tiers"]]:
                # only where the oracle's draft logit sits on a threshold
                for j, t in enumerate(do["tiers"]):
                    if tg[j] != TIER_CODE[t]:
                        dl = do["slim_draft_logit"][j] - do["slim_stats"]["max"][do["draft_row"][j]]
                        near = min(abs(dl - T * math.log(self.p.tau_acc)), abs(dl - T * math.log(self.p.tau_full)))
                        assert near < 1e-3, f"tier of draft {j} differs at margin {near}"
                continue
            got = (int(h["status"][i]), int(h["kappa"][i]), int(h["new_len"][i]),
                   list(h["path"][i][:int(h["kappa"][i])]))
            want = (do["status"], do["kappa"], do["new_len"], list(do["path"]))
            assert got == want, f"step {step} seq {b}: GPU {got} oracle {want}"
            assert bool(run[i]) == do["full_ran"]
            self.stats["kept"] += do["kappa"]
            e_g, e_o = int(h["emit"][i]), do["emit"]
            if e_o < 0:
                assert e_g == -1
                continue
            j = do["kappa"]
            kind = 1 if do["tiers"][j] == "S" else 2
            self.stats["slim" if kind == 1 else "rejected"] += 1
            exact, lo, hi, err = checks[(b, j, kind)]
            u = float(U[i, j, kind])
            if exact:
                self.stats["exact"] += 1
                assert e_g == e_o, f"step {step} seq {b}: emitted {e_g}, oracle {e_o} (u={u})"
            else:
                self.stats["loose"] += 1
                assert float(lo[e_g]) - err <= u < float(hi[e_g]) + err, f"emitted {e_g} cannot hold u={u}"
        # keep both sides on the oracle's decision
        hh = dict(status=np.array([dec_o[oids[b]]["status"] for b in order], np.int32),
                  kappa=np.array([dec_o[oids[b]]["kappa"] for b in order], np.int32),
                  emit=np.array([dec_o[oids[b]]["emit"] for b in order], np.int32),
                  new_len=np.array([dec_o[oids[b]]["new_len"] for b in order], np.int32))
        path = np.full((len(order), w.max_drafts), -1, np.int32)
        for i, b in enumerate(order):
            pp = dec_o[oids[b]]["path"]
            path[i, :len(pp)] = pp
        hh["path"] = path
        n0 = {b: len(self.sess.tokens[b]) for b in order}
        self.sess.commit(w, gd, h=hh)
        for b in order:
            assert self.sess.tokens[b] == self.ver.seqs[oids[b]].tokens
        if self.dr:
            self.dr.sync({b: self.sess.tokens[b][n0[b]:] for b in order})
            for b in order:
                assert self.dr.sess.tokens[b] == self.sess.tokens[b]
        self.stats["steps"] += 1


CASES = [
    ("micro_f32", TierParams(0.9, 0.5, 1.0, FORCED_FULL), 0.0, 1.0, False),
    ("micro_f32", TierParams(0.9, 0.5, 0.8, FORCED_SLIM), 0.0, 1.0, False),
    ("micro_f32", TierParams(0.6, 0.05, 1.0, FORCED_NONE), 0.3, 1.5, True),
    ("micro_f32", TierParams(0.9, 0.5, 1.0, FORCED_FULL), 0.0, 1e30, False),
    ("micro_bf16", TierParams(0.9, 0.5, 1.0, FORCED_FULL), 0.2, 1.0, False),
    ("micro_bf16", TierParams(0.6, 0.05, 1.0, FORCED_NONE), 0.0, 1.0, True),
    ("small_bf16_hd128", TierParams(0.9, 0.5, 1.0, FORCED_FULL), 0.1, 1.2, False),
]


@pytest.mark.parametrize("name,params,alpha,beta,greedy", CASES)
def test_sampled_decisions_match_oracle(name, params, alpha, beta, greedy):
    print(f"[case] sampling {name} forced={params.forced} T={params.temperature} alpha={alpha} beta={beta}",
          flush=True)
    ls = SampledLockstep(name, params, alpha, beta, greedy_drafts=greedy, seed=len(name) + params.forced)
    try:
        for step in range(4):
            ls.step(step)
        print(f"[done] {ls.stats}", flush=True)
        st = ls.stats
        assert st["steps"] == 4
        if params.forced == FORCED_SLIM:
            assert st["slim"] > 0
        if params.forced == FORCED_FULL:
            assert st["rejected"] > 0 and st["kept"] > 0
        if beta > 1e20:
            assert st["fallback"] > 0
        if ls.md["dtype"] == "f32":
            assert st["exact"] > 0
    finally:
        ls.close()


@pytest.mark.parametrize("params,alpha,beta,drafter_T", [
    (TierParams(0.9, 0.5, 1.0, FORCED_FULL), 0.0, 1.0, 1.0),
    (TierParams(0.6, 0.05, 1.0, FORCED_NONE), 0.2, 1.0, 0.7),
])
def test_model_drafter_and_sampled_verification(params, alpha, beta, drafter_T):
    """Drafts and p from a drafter model (the micro model's layer 0, nested in
    the slim route [0, 2]) against the oracle's forwards of that route, then
    the sampled verification of those drafts, for several steps (the
    drafter's cache follows the committed tokens)."""
    print(f"[case] model drafter forced={params.forced} alpha={alpha} drafter T={drafter_T}", flush=True)
    ls = SampledLockstep("micro_f32", params, alpha, beta, seed=5 + params.forced, drafter_route=[0],
                         drafter_T=drafter_T)
    try:
        for step in range(4):
            ls.step(step)
        print(f"[done] {ls.stats}", flush=True)
        assert ls.stats["drafted"] == 4 * ls.B * ls.k and ls.stats["exact"] > 0
    finally:
        ls.close()


@pytest.mark.parametrize("alpha,beta", [(0.0, 1.0), (0.2, 1.0)])
def test_independent_drafter_model_and_sampled_verification(alpha, beta):
    """A drafter with weights and dimensions of its own (2 layers, d_model 64,
    one head, the verifier's vocabulary): its drafts and p against the
    oracle's forwards of that model, then the sampled verification of those
    drafts by the micro model, over four steps (the drafter's cache follows
    the committed tokens)."""
    params = TierParams(0.9, 0.5, 1.0, FORCED_NONE)
    print(f"[case] independent drafter alpha={alpha}", flush=True)
    ls = SampledLockstep("micro_f32", params, alpha, beta, seed=9, drafter_T=1.0,
                         drafter_cfg=configs.get("micro_f32_drafter"))
    try:
        for step in range(4):
            ls.step(step)
        print(f"[done] {ls.stats}", flush=True)
        assert ls.stats["drafted"] == 4 * ls.B * ls.k and ls.stats["exact"] > 0
    finally:
        ls.close()


def test_sample_rows_rejects_bad_arguments():
    cfg = configs.get("micro_f32")
    cfg["seed_c"] = 3
    md = cfg["model"]
    W = gen.model_weights(cfg)
    gm = via.Model(md, W, cfg["route"])
    kv = via.KV(gm, max_seqs=2, max_blocks_per_seq=8, blocks_full=16, blocks_slim=16, max_rows=16,
                max_batch=2, max_drafts=4)
    try:
        out = via.Out(2, 8, 4, md["vocab"], logits=True)
        tok = torch.zeros(2, dtype=torch.int32, device="cuda")
        sp = C.c_void_p(0)
        u = np.array([0.5, 0.5], np.float32)
        ok_r, ok_rp = via._i32([0, 3])
        call = lambda n, rows, uu, T=1.0, ld=md["vocab"]: via.via_sample_rows(  # noqa: E731
            kv.h, C.byref(out.c), 16, n, rows, T, uu.ctypes.data, tok.data_ptr(), None, ld, sp)
        assert call(3, ok_rp, u) == via.EINVAL                         # n > max_batch
        r2, rp2 = via._i32([0, 16])
        assert call(2, rp2, u) == via.EINVAL                           # row outside [0, out_rows)
        assert call(2, ok_rp, np.array([0.5, 1.0], np.float32)) == via.EINVAL
        assert call(2, ok_rp, u, T=0.0) == via.EINVAL
        assert via.via_sample_rows(kv.h, C.byref(out.c), 16, 2, ok_rp, 1.0, u.ctypes.data, tok.data_ptr(),
                                   out.logits.data_ptr(), md["vocab"] - 1, sp) == via.EINVAL  # probs_ld < vocab
        assert call(0, ok_rp, u) == via.OK
        torch.cuda.synchronize()
    finally:
        kv.close()
        gm.close()


def test_sampled_decide_rejects_bad_arguments():
    cfg = configs.get("micro_f32")
    cfg["seed_c"] = 3
    md = cfg["model"]
    W = gen.model_weights(cfg)
    gm = via.Model(md, W, cfg["route"])
    kv = via.KV(gm, max_seqs=1, max_blocks_per_seq=8, blocks_full=16, blocks_slim=16, max_rows=16,
                max_batch=1, max_drafts=4)
    try:
        V = md["vocab"]
        p = via.tier_params(0.9, 0.5, 1.0)
        sess = Session(gm, kv, p, logits=True)
        sess.prefill(0, gen.context_tokens(cfg, 0, 8))
        probs = torch.full((1, 3, V), 1.0 / V, device="cuda")
        good = np.full((1, 3, 3), 0.5, np.float32)
        w = sess.window({0: ([1, 2, 3], None)})
        via.check(via.via_verify_slim(gm.h, kv.h, C.byref(w.c), C.byref(p), C.byref(sess.out_slim.c), sess.sp()))
        sp = sess.sp()

        def call(smp, slim=sess.out_slim):
            return via.via_tier_decide_sampled(kv.h, C.byref(p), C.byref(slim.c), None, C.byref(smp.c),
                                               C.byref(sess.dec.c), sp)

        assert call(via.Sampling(1.0, 1.0, probs, good)) == via.EINVAL       # alpha = 1
        assert call(via.Sampling(0.0, 0.0, probs, good)) == via.EINVAL       # beta = 0
        assert call(via.Sampling(0.5, 0.4, probs, good)) == via.EINVAL       # beta < 1 - alpha (Eq. A.3)
        assert call(via.Sampling(0.5, float("inf"), probs, good)) == via.EINVAL
        bad = good.copy()
        bad[0, 1, 2] = 1.0
        assert call(via.Sampling(0.0, 1.0, probs, bad)) == via.EINVAL        # a uniform of 1
        no_logits = via.Out(1, 16, 4, V, logits=False)
        no_logits.c.row_max = sess.out_slim.c.row_max
        no_logits.c.row_argmax = sess.out_slim.c.row_argmax
        no_logits.c.row_sumexp = sess.out_slim.c.row_sumexp
        no_logits.c.draft_logit = sess.out_slim.c.draft_logit
        assert call(via.Sampling(0.0, 1.0, probs, good), slim=no_logits) == via.EINVAL
        assert via.via_tier_decide_sampled(kv.h, C.byref(p), C.byref(sess.out_slim.c), None, None,
                                           C.byref(sess.dec.c), sp) == via.EINVAL
        # the step is still open: decide it and commit
        via.check(call(via.Sampling(0.0, 1.0, probs, good)))
        torch.cuda.synchronize()
        h = sess._host(w)
        if h["status"][0] == 1:
            wl = sess.window({0: ([1, 2, 3], None)}, with_lag=True)
            r, rp = via._i32([1])
            via.check(via.via_verify_full(gm.h, kv.h, C.byref(wl.c), rp, C.byref(p), C.byref(sess.out_full.c), sp))
            via.check(via.via_tier_decide_sampled(kv.h, C.byref(p), C.byref(sess.out_slim.c),
                                                  C.byref(sess.out_full.c),
                                                  C.byref(via.Sampling(0.0, 1.0, probs, good).c),
                                                  C.byref(sess.dec.c), sp))
            torch.cuda.synchronize()
        via.check(via.via_kv_commit_rollback(kv.h, C.byref(sess.dec.c), sp))
        torch.cuda.synchronize()
        # tree windows are refused
        tw = sess.window({0: ([4, 5, 6], [-1, -1, 0])})
        via.check(via.via_verify_slim(gm.h, kv.h, C.byref(tw.c), C.byref(p), C.byref(sess.out_slim.c), sp))
        assert call(via.Sampling(0.0, 1.0, probs, good)) == via.EUNSUPPORTED
        via.check(via.via_tier_decide(kv.h, C.byref(p), C.byref(sess.out_slim.c), None, C.byref(sess.dec.c), sp))
        torch.cuda.synchronize()
    finally:
        kv.close()
        gm.close()
