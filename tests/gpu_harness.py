"""Lock-step parity runner: the HIP path (through the C ABI) and the oracle
decode the same sequences from the same drafts, step by step.

Each step both sides start from the same committed state.  Compared per
step: slim/full logits (fp32 dump; tolerance 2e-2 for bf16 models, 1e-4 for
fp32), row argmaxes, every draft's tier, which sequences escalate, the
accepted length, the emitted token, the new length, and both caches' valid
lengths and block tables.  A difference is allowed only where the oracle
itself is within 1e-3 of a decision boundary: a top-2 logit gap below 1e-3
(argmax / full-tier check) or a draft logit within 1e-3 of a threshold
(l'(d) - max l' vs T ln tau).  Exemptions are per sequence: a difference
in a sequence's decision is allowed only when that sequence itself has an
exempt position this step.  After such a difference the GPU is
re-synchronised to the oracle's decision (its commit takes the oracle's
kappa/emit) and the step is logged with the positions that allowed it.

At full sizes the oracle can follow a sample of the batch (``sample``): the
GPU still runs every sequence in the same launch, the sampled ones are
compared element by element, and the rest commit the GPU's own decisions.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from oracle.decode import (FORCED_NONE, Draft, GreedyDrafter, TierParams, Verifier)
from oracle.model import OracleModel, round_bf16
from paper_2606_12243_amd import via
from paper_2606_12243_amd.session import Session
from workload import gen

GAP_EXEMPT = 1e-3
TIER_CODE = {"A": 0, "S": 1, "F": 2}


def logit_tol(desc):
    return 2e-2 if desc["dtype"] == "bf16" else 1e-4


class Lockstep:
    def __init__(self, cfg, weights=None, max_rows=None, max_batch=None, max_drafts=None, max_blocks=None,
                 blocks=None, params=None, oracle_model=None, gpu_model=None, sample=None):
        self.cfg = cfg
        md = cfg["model"]
        self.md = md
        W = weights if weights is not None else gen.model_weights(cfg)
        self.om = oracle_model or OracleModel(md, W)
        self.p = params or TierParams(0.9, 0.5, cfg.get("temperature", 1.0))
        self.ver = Verifier(self.om, cfg["route"], block_size=16)
        V = md["vocab"]
        self.drafter = GreedyDrafter(self.om, lambda b, step, j: gen.corruption(
            cfg["seed_d"], b, step, j, cfg.get("corrupt", 0.3), V))
        B = max_batch or cfg.get("batch", 1)
        self.sample = None if sample is None else set(sample)
        self.own_gm = gpu_model is None
        self.gm = gpu_model or via.Model(md, W, cfg["route"])
        self.kv = via.KV(self.gm, max_seqs=B, max_blocks_per_seq=max_blocks or 64, blocks_full=blocks or 256,
                         blocks_slim=blocks or 256, max_rows=max_rows or 128, max_batch=B,
                         max_drafts=max_drafts or 16)
        self.sess = Session(self.gm, self.kv, via.tier_params(self.p.tau_acc, self.p.tau_full, self.p.temperature,
                                                             self.p.forced), logits=True)
        self.o_id = {}    # GPU sequence id -> oracle sequence index
        self.log = []
        # per step: which batch entries ran the full forward, with how many lag rows
        # (sampled sequences), and the committed kappa of each sampled sequence
        self.steps = []
        self.gpu_tiers = set()   # tiers the GPU gave any draft of the batch (sampled or not)
        self.seen_tiers = set()
        self.max_logit_err = 0.0

    def set_params(self, params):
        """Tier parameters of the following steps (both sides)."""
        self.p = params
        self.sess.p = via.tier_params(params.tau_acc, params.tau_full, params.temperature, params.forced)

    def close(self):
        self.kv.close()
        if self.own_gm:
            self.gm.close()

    def sampled(self, b):
        return self.sample is None or b in self.sample

    # ------------------------------------------------------------ setup
    def add_prompt(self, b, tokens):
        if self.sampled(b):
            self.o_id[b] = self.ver.prefill(tokens)
            self.drafter.attach(b)
        self.sess.prefill(b, tokens)

    def add_synthetic(self, b, tokens):
        """Sequence whose n-1 context slots hold seeded synthetic K/V (both sides)."""
        cfg, md = self.cfg, self.md
        n1 = len(tokens) - 1
        bf16 = md["dtype"] == "bf16"
        kv = {(c, s): gen.synthetic_kv(cfg, c, s, b, n1)
              for c, slots in ((gen.CACHE_FULL, md["n_layers"]), (gen.CACHE_SLIM, len(cfg["route"])))
              for s in range(slots)}

        def t64(a):
            if bf16:
                return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(torch.float64)
            return torch.from_numpy(a).to(torch.float64)

        if self.sampled(b):
            kvf = [(t64(kv[(gen.CACHE_FULL, s)][0]), t64(kv[(gen.CACHE_FULL, s)][1]))
                   for s in range(md["n_layers"])]
            kvs = [(t64(kv[(gen.CACHE_SLIM, s)][0]), t64(kv[(gen.CACHE_SLIM, s)][1]))
                   for s in range(len(cfg["route"]))]
            self.o_id[b] = self.ver.attach_context(tokens, kvf, kvs)
            if self.sample is None:
                self.drafter.attach(b, kvf)

        def dev(a):
            t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16) if bf16 else torch.from_numpy(a)
            return t

        self.sess.reserve(b, tokens, lambda c, s: (dev(kv[(c, s)][0]), dev(kv[(c, s)][1])))

    # ------------------------------------------------------------ checks
    def _cmp_logits(self, w, out, o_logits, b, what):
        R = w.max_rows
        V = self.md["vocab"]
        n = int(w.a["n_rows"][b])
        g = out.logits[b * R * V:(b * R + n) * V].view(n, V).double().cpu()
        err = float((g - o_logits).abs().max())
        self.max_logit_err = max(self.max_logit_err, err)
        assert err <= logit_tol(self.md), f"{what} logits of seq {b}: max |diff| {err}"
        am = out.row_argmax[b * R:b * R + n].cpu().numpy()
        return am

    def step(self, drafts: dict, step_idx: int):
        """drafts: {b: Draft}; runs both sides, compares, commits."""
        p = self.p
        order = sorted(drafts)
        lag_before = {b: self.ver.seqs[self.o_id[b]].n - 1 - self.ver.seqs[self.o_id[b]].full.valid
                      for b in order if self.sampled(b)}
        gpu_lag = {b: len(self.sess.lag(b)) for b in order}
        raw = self.ver.step({self.o_id[b]: drafts[b] for b in order if self.sampled(b)}, p)  # oracle decides, commits
        dec_o = {b: raw[self.o_id[b]] for b in order if self.sampled(b)}
        gd = {b: (drafts[b].tok, None if self._is_chain(drafts[b]) else drafts[b].parent) for b in order}
        s = self.sess
        w = s.window(gd, with_lag=True)
        via.check(via.via_verify_slim(s.m.h, s.kv.h, w.c, s.p, s.out_slim.c, s.sp()))
        via.check(via.via_tier_decide(s.kv.h, s.p, s.out_slim.c, None, s.dec.c, s.sp()))
        s.stream.synchronize()
        h1 = s._host(w)
        D = w.max_drafts
        tiers_all = s.dec.tier[:w.B * D].cpu().numpy().reshape(w.B, D)
        for i, b in enumerate(order):
            self.gpu_tiers.update("ASF"[t] for t in tiers_all[i, :len(drafts[b].tok)])
        exempt = {}   # batch entry -> the near-tie positions that allow it to differ
        T = p.temperature
        for i, b in enumerate(order):
            if b not in dec_o:
                continue
            do = dec_o[b]
            am = self._cmp_logits(w, s.out_slim, do["slim_logits"], i, "slim")
            st = do["slim_stats"]
            for r in range(len(am)):
                if am[r] != st["argmax"][r]:
                    assert st["gap"][r] < GAP_EXEMPT, f"slim argmax differs at gap {st['gap'][r]}"
                    exempt.setdefault(b, []).append(f"slim row {r} gap {st['gap'][r]:.2e}")
            D = w.max_drafts
            tier_g = s.dec.tier[i * D:i * D + len(drafts[b].tok)].cpu().numpy()
            for j, t in enumerate(do["tiers"]):
                self.seen_tiers.add(t)
                if tier_g[j] != TIER_CODE[t]:
                    dl = do["slim_draft_logit"][j] - st["max"][do["draft_row"][j]]
                    near = min(abs(dl - T * math.log(p.tau_acc)) if p.tau_acc > 0 else 1e9,
                               abs(dl - T * math.log(p.tau_full)) if p.tau_full > 0 else 1e9)
                    assert near < GAP_EXEMPT, f"tier of draft {j} differs ({tier_g[j]} vs {t}), margin {near}"
                    exempt.setdefault(b, []).append(f"draft {j} threshold margin {near:.2e}")
            if (h1["status"][i] == 1) != (do["first_status"] == 1):
                assert b in exempt, f"escalation differs for seq {b} without a near tie of its own"
        # full forward for the sequences the oracle escalated (keeps cache state in step)
        run = np.array([(1 if dec_o[b]["full_ran"] else 0) if b in dec_o else int(h1["status"][i] == 1)
                        for i, b in enumerate(order)], np.int32)
        if run.any():
            r, rp = via._i32(run)
            via.check(via.via_verify_full(s.m.h, s.kv.h, w.c, rp, s.p, s.out_full.c, s.sp()))
            via.check(via.via_tier_decide(s.kv.h, s.p, s.out_slim.c, s.out_full.c, s.dec.c, s.sp()))
            s.stream.synchronize()
            for i, b in enumerate(order):
                if not run[i] or b not in dec_o:
                    continue
                do = dec_o[b]
                am = self._cmp_logits(w, s.out_full, do["full_logits"], i, "full")
                st = do["full_stats"]
                for rr in range(len(am)):
                    if am[rr] != st["argmax"][rr]:
                        assert st["gap"][rr] < GAP_EXEMPT, f"full argmax differs at gap {st['gap'][rr]}"
                        exempt.setdefault(b, []).append(f"full row {rr} gap {st['gap'][rr]:.2e}")
        h = s._host(w)
        differ = []
        for i, b in enumerate(order):
            if b not in dec_o:
                continue
            do = dec_o[b]
            got = (int(h["status"][i]), int(h["kappa"][i]), int(h["emit"][i]), int(h["new_len"][i]))
            want = (do["status"], do["kappa"], do["emit"], do["new_len"])
            if got != want:
                assert b in exempt, f"step {step_idx} seq {b}: GPU {got} oracle {want} without a near tie of its own"
                differ.append(b)
        if differ:
            self.log.append(dict(step=step_idx, kind="resync", seqs={b: exempt[b] for b in differ}))
            D = w.max_drafts
            path = np.array(h["path"], np.int32).reshape(w.B, -1).copy()
            hh = {k: np.array(h[k], np.int32).copy() for k in ("status", "kappa", "emit", "new_len")}
            for i, b in enumerate(order):
                if b not in dec_o:
                    continue
                pp = dec_o[b]["path"]
                path[i, :] = -1
                path[i, :len(pp)] = pp
                for k in hh:
                    hh[k][i] = dec_o[b][k]
            hh["path"] = path
            s.commit(w, gd, hh)
        else:
            s.commit(w, gd)
        self.steps.append(dict(step=step_idx, run=run.tolist(),
                               full_start=s.kv.last_full_start() if run.any() else None,
                               gpu_lag={b: gpu_lag[b] for i, b in enumerate(order) if run[i]},
                               full_lag={b: lag_before[b] for i, b in enumerate(order) if b in dec_o and run[i]},
                               kappa={b: dec_o[b]["kappa"] for b in order if b in dec_o}))
        # committed tokens, valid lengths and block tables
        for b in order:
            if b not in dec_o:
                continue
            st = self.ver.seqs[self.o_id[b]]
            assert s.tokens[b] == st.tokens, f"seq {b} token streams differ"
            for cache, oc, which in ((via.CACHE_FULL, st.full, "full"), (via.CACHE_SLIM, st.slim, "slim")):
                valid, table = self.kv.seq_info(b, cache)
                assert valid == oc.valid, f"seq {b} {which} valid {valid} vs {oc.valid}"
                if self.sample is None:
                    assert table == self.ver.block_table(which, self.o_id[b]), f"seq {b} {which} block table differs"
                else:
                    # the GPU pool also serves the unsampled sequences: the table must cover the
                    # valid slots with distinct blocks (the exact ids are checked at small sizes)
                    assert len(table) == -(-valid // 16) and len(set(table)) == len(table), \
                        f"seq {b} {which} block table {len(table)} blocks for {valid} slots"
        return dec_o, h

    @staticmethod
    def _is_chain(d: Draft):
        return all(p == j - 1 for j, p in enumerate(d.parent))

    def run_chain(self, seqs, G, k):
        n0 = {b: len(self.ver.seqs[b].tokens) for b in seqs}
        step = 0
        while True:
            active = [b for b in seqs if len(self.ver.seqs[b].tokens) - n0[b] < G]
            if not active:
                break
            drafts = {b: self.drafter.chain(b, self.ver.seqs[b].tokens, k, step) for b in active}
            self.step(drafts, step)
            step += 1
        return step
