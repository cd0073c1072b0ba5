#!/usr/bin/env python
"""Benchmark of the VIA-SD verification step on one MI355X (gfx950).

A step is one pass of the whole verification hot path over a batch:
slim-verifier forward + fused head, tier decision (device->host read),
the full-verifier forward with its lag rows when any sequence escalates,
the second decision, and the KV commit/rollback.  Drafts come from a
synthetic drafter (the full verifier's greedy token with random
replacements) run beforehand: an untimed reference decode records every
step's drafts, then the KV state is reset and the recorded steps are
replayed; W replayed steps warm up, the next K are timed.

value = accepted (committed) tokens summed over the batch / timed seconds, at
the workload's logit temperature (calibrated for the 1B and the 8B chain and
tree workloads so that about half of the greedy drafts clear the accept
threshold; the long-context batch runs at its mixed-tier temperature).  The
JSON line adds the verify-step latency percentiles, the roofline of the
dominant kernel (HIP events carried by its dispatches during the timed
region), the whole step's algorithmic bytes against HBM peak, the same
workload at its mixed-tier temperature (all three tiers, escalations of part
of the batch with lag rows) and at T = 1 (every drafted position escalated to
the full verifier), and the oracle's rate on a bounded sample of the same
workload.

    python bench.py [--steps K] [--warmup W] [--config 8b_bf16_chain]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
METRIC = "accepted tokens/s + verify-step latency, 8B-shape bf16 k=8; % HBM/MFMA roofline"


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def build_session(cfg, W, pools=None, n_steps=64, logits=False):
    import torch
    from paper_2606_12243_amd import via
    from paper_2606_12243_amd.session import Session
    md = cfg["model"]
    B = cfg["batch"]
    ctx = cfg["ctx_lens"]
    k = cfg.get("k", 8)
    # rows per sequence: the window plus every committed token the full cache may
    # still lag by (the full verifier can stay idle for the whole run; the
    # drafter's probes and the next escalation feed those lag rows)
    grow = n_steps * ((k + 1) if cfg["draft"] != "tree" else len(cfg["tree_budget"]) + 1)
    rows_per_seq = (64 if cfg["draft"] == "tree" else k) + grow
    max_rows = B * rows_per_seq
    max_blocks = (max(ctx) + grow + rows_per_seq + 16) // 16 + 1
    blocks = B * max_blocks
    model = cfg.get("_model")
    kv = via.KV(model, max_seqs=B, max_blocks_per_seq=max_blocks, blocks_full=blocks, blocks_slim=blocks,
                max_rows=max_rows, max_batch=B, max_drafts=64, zero_pools=False, pools=pools)
    p = via.tier_params(0.9, 0.5, cfg["temperature"])
    return Session(model, kv, p, logits=logits)


def attach_context(cfg, sess, synthetic):
    from workload import gen
    import torch
    B = cfg["batch"]
    for b, n in enumerate(cfg["ctx_lens"]):
        toks = gen.context_tokens(cfg, b, n + 1)
        if synthetic:
            def kvv(cache, slot, b=b, n=n):
                K, V = gen.synthetic_kv(cfg, cache, slot, b, n)
                return (torch.from_numpy(K.view(np.int16)).view(torch.bfloat16),
                        torch.from_numpy(V.view(np.int16)).view(torch.bfloat16))
            sess.reserve(b, toks, kvv)
        else:
            sess.prefill(b, toks)


def step_bytes(cfg, kv_slim_tokens, full_seqs, run, full_start):
    """Algorithmic HBM bytes of one step: the routed layers' weights and the
    head for the slim forward plus the cached K/V it read (tokens summed over
    the batch); when the full verifier ran, the weights of the layers it ran,
    the head, and the K/V those layers read for the sequences it covered.
    ``full_seqs[b]`` = (cached + lag tokens, lag tokens) of the full cache
    before the step; ``full_start`` = the layer the full forward started at
    (the library reports it: after the layers the slim route shares with the
    full model when their states were kept, else 0), so the shared layers'
    weights and K/V are not counted when they were not read again."""
    from workload.configs import model_bytes
    md = cfg["model"]
    slim = model_bytes(md, cfg["route"])
    kvb = slim["kv_per_token_layer"]
    tot = slim["layers"] + slim["head"] + kvb * len(cfg["route"]) * kv_slim_tokens
    ran = [b for b in range(len(run)) if run[b]]
    if ran:
        layers = md["n_layers"] - max(0, full_start)
        tot += layers * slim["per_layer"] + slim["head"] + kvb * layers * sum(full_seqs[b][0] for b in ran)
    return tot


def sampling_inputs(cfg, drafts, step, alpha, beta):
    """Synthetic sampling-rule inputs of one step: the drafter's distribution
    p_j over the vocabulary (a softmax of N(0, 1.5^2) logits with the drafted
    token raised by 4, so p puts visible mass on its own draft) and the
    step's uniforms, both seeded by (seed_d, step)."""
    import torch
    from paper_2606_12243_amd import via
    V = cfg["model"]["vocab"]
    B = len(drafts)
    D = max(1, max(len(drafts[b][0]) for b in drafts))
    g = torch.Generator(device="cuda").manual_seed(cfg["seed_d"] * 1000 + step)
    z = torch.randn((B, D, V), generator=g, device="cuda") * 1.5
    for i, b in enumerate(drafts):
        tok = drafts[b][0]
        z[i, torch.arange(len(tok), device="cuda"), torch.tensor(tok, device="cuda")] += 4.0
    rng = np.random.default_rng([cfg["seed_d"], step])
    U = rng.random((B, D, 3)).astype(np.float32)
    return via.Sampling(alpha, beta, torch.softmax(z, -1), np.minimum(U, np.float32(0.99999)))


def run_workload(cfg, W, steps, warmup, temperature, timer_kind=None, sampling=None):
    """Reference decode with the synthetic drafter (records drafts and
    decisions), then a fresh handle on the same pools replays the recorded
    steps: `warmup` untimed, `steps` timed.  Returns the measurements.
    ``sampling`` = (alpha, beta) switches to the sampling rules with the
    synthetic inputs of ``sampling_inputs`` (recorded with the drafts)."""
    import torch
    from paper_2606_12243_amd import via
    from paper_2606_12243_amd.session import GreedyDrafter
    from workload import gen
    md = cfg["model"]
    V = md["vocab"]
    B = cfg["batch"]
    cfg = dict(cfg, temperature=temperature)
    synthetic = cfg.get("seed_kv") is not None
    n_steps = warmup + steps
    sess = build_session(cfg, W, n_steps=n_steps, logits=sampling is not None)
    t0 = time.time()
    attach_context(cfg, sess, synthetic)
    torch.cuda.synchronize()
    log(f"T={temperature:.4g}: context attached ({'synthetic K/V' if synthetic else 'prefill'}) "
        f"in {time.time() - t0:.1f}s")
    drafter = GreedyDrafter(sess, lambda b, step, j: gen.corruption(cfg["seed_d"], b, step, j, cfg["corrupt"], V))

    # ---- reference decode: record drafts and decisions
    recorded, t_draft = [], 0.0
    init_tokens = {b: list(sess.tokens[b]) for b in range(B)}
    for i in range(n_steps):
        ts = time.time()
        if cfg["draft"] == "tree":
            drafts = drafter.tree(list(range(B)), cfg["tree_budget"], cfg["tree_branch"], i)
        else:
            d = drafter.chain(list(range(B)), cfg["k"], i)
            drafts = {b: (d[b], None) for b in range(B)}
        smp = sampling_inputs(cfg, drafts, i, *sampling) if sampling is not None else None
        torch.cuda.synchronize()
        t_draft += time.time() - ts
        # cached tokens each forward of this step reads (for the step's algorithmic bytes)
        kv_slim = sum(sess.kv.seq_info(b, via.CACHE_SLIM)[0] for b in range(B))
        kv_full = [(sess.kv.seq_info(b, via.CACHE_FULL)[0] + len(sess.lag(b)), len(sess.lag(b))) for b in range(B)]
        h, run = sess.step(drafts, smp)
        recorded.append((drafts, h["new_len"].copy(), run.copy(), kv_slim, kv_full, smp, sess.kv.last_full_start()))
    log(f"T={temperature:.4g}: reference decode of {n_steps} steps, drafting {t_draft:.2f}s")

    # ---- reset: fresh handle on the same pools (context slots untouched)
    pools = (sess.kv.pool_full, sess.kv.pool_slim)
    sess.kv.close()

    def fresh():
        s2 = build_session(cfg, W, pools=pools, n_steps=n_steps, logits=sampling is not None)
        if synthetic:
            for b in range(B):
                s2.reserve(b, init_tokens[b], None)
        else:
            for b in range(B):
                s2.prefill(b, init_tokens[b])
        torch.cuda.synchronize()
        return s2

    def replay(timed_kind):
        """Warm-up steps, then the timed steps; with `timed_kind` the kernels of
        that kind carry timing events (a separate pass, so the timed pass runs
        without them).  Greedy steps run as one native via_step call each
        (window assembly, forwards, decisions and commit in the library); the
        sampling rules are driven call by call from the session."""
        import ctypes as C
        s2 = fresh()
        native = sampling is None
        if native:
            for b in range(B):
                t, tp = via._i32(init_tokens[b])
                via.check(via.via_kv_seq_set_tokens(s2.kv.h, b, tp, len(init_tokens[b])))
            bufs = [via.DraftsBuf(r[0]) for r in recorded]   # the drafts, resident before timing
            hp = s2.dec.h_packed.numpy()
            args = (s2.m.h, s2.kv.h, None, C.byref(s2.p), C.byref(s2.out_slim.c), C.byref(s2.out_full.c),
                    C.byref(s2.dec.c), s2.sp())

        def one(i):
            if native:
                via.check(via.via_step(args[0], args[1], C.byref(bufs[i].c), *args[3:]))
                return hp[3 * B:4 * B].copy(), hp[:B].copy()
            w, h, run = s2.begin(recorded[i][0], recorded[i][5])
            s2.commit(w, recorded[i][0])
            return h["new_len"].copy(), run

        mism = 0
        for i in range(warmup):
            new_len, run = one(i)
            mism += int((new_len != recorded[i][1]).any())
            # the replayed full forward starts where the recorded one did
            mism += int(bool(recorded[i][2].any()) and s2.kv.last_full_start() != recorded[i][6])
        torch.cuda.synchronize()
        if timed_kind is not None:
            s2.kv.timer_enable(1 << timed_kind)
            s2.kv.timer_read(timed_kind)
        lat, n_full_steps, outs = [], 0, []
        n_prev = np.array(recorded[warmup - 1][1] if warmup else [len(init_tokens[b]) for b in range(B)])
        torch.cuda.synchronize()
        t_start = time.perf_counter()
        for i in range(warmup, n_steps):
            ts = time.perf_counter()
            new_len, run = one(i)
            torch.cuda.synchronize()
            lat.append(time.perf_counter() - ts)
            outs.append((new_len, run))
        t_total = time.perf_counter() - t_start
        for i, (new_len, run) in zip(range(warmup, n_steps), outs):
            mism += int((new_len != recorded[i][1]).any())
            n_full_steps += int(np.asarray(run).any() if not native else recorded[i][2].any())
        accepted = int((np.asarray(outs[-1][0]) - n_prev).sum())
        timer = s2.kv.timer_read(timed_kind) if timed_kind is not None else (0, 0.0)
        s2.kv.timer_enable(0)
        s2.kv.close()
        return lat, accepted, n_full_steps, t_total, mism, timer

    lat, accepted, n_full_steps, t_total, mism, _ = replay(None)
    timer = replay(timer_kind)[5] if timer_kind is not None else (0, 0.0)
    bytes_tot = sum(step_bytes(cfg, r[3], r[4], r[2], r[6]) for r in recorded[warmup:])
    lat_ms = np.array(lat) * 1e3
    return dict(value=accepted / t_total, t_total=t_total, lat_ms=lat_ms, escalation=n_full_steps / max(1, steps),
                mismatch=mism, t_draft=t_draft, bytes=bytes_tot, timer=timer, recorded=recorded,
                init_tokens=init_tokens, accepted=accepted)


def run_drafter_variant(cfg, W, steps, warmup, temperature, route_d):
    """The serving loop with a drafter model: the verifier's weights under
    the nested route ``route_d`` (inside the slim route) draft k tokens per
    sequence from their temperature-T softmax, the verifier checks them under
    the lossless sampling rules (alpha = 0, beta = 1) with the drafter's p,
    and the drafter's cache takes the committed tokens.  Every phase is
    timed (synchronised); uniforms are seeded."""
    import torch
    from paper_2606_12243_amd import via
    from paper_2606_12243_amd.session import ModelDrafter
    from workload import gen
    md = cfg["model"]
    B, k = cfg["batch"], cfg["k"]
    cfg = dict(cfg, temperature=temperature)
    n_steps = warmup + steps
    sess = build_session(cfg, W, n_steps=n_steps, logits=True)
    attach_context(cfg, sess, cfg.get("seed_kv") is not None)
    dm = via.Model(md, W, list(route_d))
    max_blocks = (max(cfg["ctx_lens"]) + n_steps * (k + 1) + 32) // 16 + 1
    dkv = via.KV(dm, max_seqs=B, max_blocks_per_seq=max_blocks, blocks_full=B * max_blocks,
                 blocks_slim=B * max_blocks, max_rows=max(B * k, max(cfg["ctx_lens"])), max_batch=B,
                 max_drafts=k + 1, zero_pools=False)
    dr = ModelDrafter(dm, dkv, temperature)
    for b in range(B):
        dr.attach(b, list(sess.tokens[b]))
    torch.cuda.synchronize()
    rng = np.random.default_rng([cfg["seed_d"], 77])
    seqs = list(range(B))
    t_draft, t_verify, t_sync, accepted = [], [], [], 0
    for i in range(n_steps):
        Ud = rng.random((B, k)).astype(np.float32)
        Uv = np.minimum(rng.random((B, k, 3)).astype(np.float32), np.float32(0.99999))
        t0 = time.perf_counter()
        d, P = dr.draft(seqs, k, Ud)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        drafts = {b: (d[b], None) for b in seqs}
        n0 = [len(sess.tokens[b]) for b in seqs]
        sess.step(drafts, via.Sampling(0.0, 1.0, P, Uv))
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        dr.sync({b: sess.tokens[b][n0[b]:] for b in seqs})
        torch.cuda.synchronize()
        t3 = time.perf_counter()
        if i >= warmup:
            t_draft.append(t1 - t0)
            t_verify.append(t2 - t1)
            t_sync.append(t3 - t2)
            accepted += sum(len(sess.tokens[b]) - n0[b] for b in seqs)
    dkv.close()
    dm.close()
    sess.kv.close()
    tot = sum(t_draft) + sum(t_verify) + sum(t_sync)
    # algorithmic bytes of drafting: k probe forwards, each the route's
    # weights and the head (the cached K/V the probes read is small beside it)
    from workload.configs import model_bytes
    mb = model_bytes(md, list(route_d))
    draft_gbs = k * (mb["layers"] + mb["head"]) / float(np.mean(t_draft)) / 1e9
    return {"drafter_route": list(route_d), "temperature": temperature, "alpha": 0.0, "beta": 1.0,
            "value": round(accepted / tot, 2), "unit": "tokens/s (drafting included)", "steps": steps,
            "tokens_per_step": round(accepted / steps, 3),
            "ms_draft": round(1e3 * float(np.mean(t_draft)), 3), "ms_verify": round(1e3 * float(np.mean(t_verify)), 3),
            "ms_drafter_sync": round(1e3 * float(np.mean(t_sync)), 3),
            "draft_achieved_GBs": round(draft_gbs, 1), "draft_frac_of_hbm_peak": round(draft_gbs / HBM_PEAK_GBS, 4)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="8b_bf16_chain")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-full-tier", action="store_true",
                    help="skip the T = 1 variant (every position escalated to the full verifier)")
    ap.add_argument("--no-mixed", action="store_true",
                    help="skip the mixed-tier variant (its calibrated temperature: all three tiers)")
    ap.add_argument("--breakdown", action="store_true", help="extra replay timing every kernel kind")
    ap.add_argument("--no-sampling", action="store_true", help="skip the sampling-rules variant")
    ap.add_argument("--no-drafter", action="store_true", help="skip the drafter-model variant")
    ap.add_argument("--no-prefill-gemm", action="store_true", help="skip the prefill GEMM roofline")
    ap.add_argument("--prefill-only", action="store_true",
                    help="only the batched prefill of the workload's prompts (one warm-up call, one timed call), "
                         "as one JSON line; for kernel traces of a prefill")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 1 GiB device copy 5 times (the reference kernel for HBM counter scaling)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: the verification step of a batch "
                                   "is measured on a single MI355X (--gpus 1)", "n_gpus": args.gpus}))
        sys.exit(2)

    import torch
    if args.copy_probe:
        src = torch.empty(1 << 29, dtype=torch.int16, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": src.numel() * 2, "copy_probe_bytes_written": dst.numel() * 2}))
        return
    from paper_2606_12243_amd import via
    from workload import configs, gen

    cfg = configs.get(args.config)
    md = cfg["model"]
    cfg["ctx_lens"] = gen.context_lengths(cfg)
    synthetic = cfg.get("seed_kv") is not None
    t0 = time.time()
    W = gen.model_weights(cfg)
    log(f"weights generated in {time.time() - t0:.1f}s")
    t0 = time.time()
    cfg["_model"] = via.Model(md, W, cfg["route"])
    torch.cuda.synchronize()
    log(f"weights on device in {time.time() - t0:.1f}s")
    if args.prefill_only:
        print(json.dumps(prefill_forward_roofline(cfg, W, per_sequence=False)), flush=True)
        return
    kinds = {"qkv": via.KERNEL_QKV, "attn": via.KERNEL_ATTN, "o": via.KERNEL_O, "gateup": via.KERNEL_GATEUP,
             "down": via.KERNEL_DOWN, "head": via.KERNEL_HEAD, "decide": via.KERNEL_DECIDE}
    DOM = "gateup"
    T = float(cfg["temperature"])
    res = run_workload(cfg, W, args.steps, args.warmup, T, timer_kind=kinds[DOM])
    lat_ms = res["lat_ms"]
    n_launch, ms_dom = res["timer"]
    # algorithmic bytes of the dominant kernel per launch: gate/up weights of one layer
    F, d = md["d_ffn"], md["d_model"]
    esz = 2 if md["dtype"] == "bf16" else 4
    dom_bytes = 2 * F * d * esz
    avg_ms = ms_dom / max(1, n_launch)
    achieved = dom_bytes / (avg_ms * 1e-3) / 1e9 if n_launch else None
    roof = {"kernel": "gemm_gate_up: gate/up projection of one layer", "bound": "hbm",
            "achieved": round(achieved, 1) if achieved else None, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4) if achieved else None,
            "traffic": measured_traffic(args.config),
            "bytes_per_launch": dom_bytes, "avg_launch_us": round(avg_ms * 1e3, 2), "launches": n_launch}
    copy_gbs = measured_copy_gbs()
    step_gbs = res["bytes"] / res["t_total"] / 1e9
    step_roof = {"bytes": round(res["bytes"] / args.steps), "achieved_GBs": round(step_gbs, 1),
                 "frac": round(step_gbs / HBM_PEAK_GBS, 4),
                 "copy_kernel_GBs": round(copy_gbs, 1), "frac_of_copy_kernel": round(step_gbs / copy_gbs, 4)}
    roof["frac_of_copy_kernel"] = round(achieved / copy_gbs, 4) if achieved else None

    # the same workload at T = 1, where every drafted position goes to the full verifier
    full_tier = None
    if not args.no_full_tier and T != 1.0:
        r1 = run_workload(cfg, W, max(5, args.steps // 3), 2, 1.0)
        full_tier = {"temperature": 1.0, "value": round(r1["value"], 2), "unit": "tokens/s",
                     "ms_per_step": round(float(r1["lat_ms"].mean()), 3), "steps": len(r1["lat_ms"]),
                     "escalation_rate": round(r1["escalation"], 3), "replay_mismatch_steps": r1["mismatch"],
                     "step_roofline_frac": round(r1["bytes"] / r1["t_total"] / 1e9 / HBM_PEAK_GBS, 4)}

    # the same workload at the mixed-tier temperature: all three tiers occur,
    # escalations cover part of the batch and carry the lag rows of earlier steps
    from workload import calibrated
    mixed, rm = None, None
    Tm = calibrated.MIXED_TEMPERATURE.get(args.config)
    if not args.no_mixed and Tm is not None and Tm != T:
        rm = run_workload(cfg, W, max(5, args.steps // 2), 2, Tm)
        lm = rm["lat_ms"]
        mixed = {"temperature": Tm, "value": round(rm["value"], 2), "unit": "tokens/s",
                 "ms_per_step": round(float(lm.mean()), 3),
                 "latency_ms": {"p10": round(float(np.percentile(lm, 10)), 3),
                                "p50": round(float(np.percentile(lm, 50)), 3),
                                "p90": round(float(np.percentile(lm, 90)), 3)},
                 "steps": len(lm), "tokens_per_step": round(rm["accepted"] / len(lm), 3),
                 "escalation_rate": round(rm["escalation"], 3), "replay_mismatch_steps": rm["mismatch"],
                 "step_roofline_frac": round(rm["bytes"] / rm["t_total"] / 1e9 / HBM_PEAK_GBS, 4)}

    # the same workload under the sampling rules (App. A, lossless alpha = 0,
    # beta = 1): logits kept, the decision draws the owed samples
    sampled = None
    if not args.no_sampling and cfg["draft"] == "chain":  # the sampling rules take chain drafts
        rs = run_workload(cfg, W, max(5, args.steps // 3), 2, T, timer_kind=kinds["decide"], sampling=(0.0, 1.0))
        n, ms = rs["timer"]
        sampled = {"alpha": 0.0, "beta": 1.0, "temperature": T, "value": round(rs["value"], 2), "unit": "tokens/s",
                   "ms_per_step": round(float(rs["lat_ms"].mean()), 3), "steps": len(rs["lat_ms"]),
                   "escalation_rate": round(rs["escalation"], 3), "replay_mismatch_steps": rs["mismatch"],
                   "decide_launches": n, "decide_avg_us": round(ms * 1e3 / max(1, n), 2)}

    # the serving loop with a drafter model nested in the slim route (its
    # first layer), drafting included in the time
    drafter = None
    if not args.no_drafter and cfg["draft"] == "chain":
        drafter = run_drafter_variant(cfg, W, max(5, args.steps // 5), 2, T, cfg["route"][:1])

    breakdown = None
    if args.breakdown:
        breakdown = {}
        for nme, kd in kinds.items():
            rb = run_workload(cfg, W, min(args.steps, 10), 2, T, timer_kind=kd)
            n, ms = rb["timer"]
            breakdown[nme] = {"launches": n, "total_ms": round(ms, 3), "avg_us": round(ms * 1e3 / max(1, n), 2)}

    prefill = None
    if not args.no_prefill_gemm and md["dtype"] == "bf16":
        # prefill rows of the workload: every sequence's context, capped at 8192
        prefill = prefill_gemm_roofline(md, min(8192, int(sum(cfg["ctx_lens"]))))
        prefill["forward"] = prefill_forward_roofline(cfg, W)

    dimr = dimr_cost_roofline(md)
    dimr["at_1024_rows"] = {k: v for k, v in dimr_cost_roofline(md, rows=1024).items()
                            if k in ("us", "bytes_per_launch", "achieved", "frac")}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, W, res["recorded"], res["init_tokens"],
                           mixed=(Tm, rm["recorded"], rm["init_tokens"]) if rm is not None else None)

    out = {
        "metric": METRIC, "value": round(res["value"], 2), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(float(lat_ms.mean()), 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": md["dtype"], "data": "synthetic",
        "config": {"workload": args.config, "batch": cfg["batch"], "ctx": cfg["ctx"], "draft": cfg["draft"],
                   "k": cfg.get("k"), "route_layers": len(cfg["route"]), "n_layers": md["n_layers"],
                   "d_model": md["d_model"], "vocab": md["vocab"],
                   "context_kv": "synthetic N(0, (0.02 sqrt d)^2)" if synthetic else "prefill"},
        "latency_ms": {"p10": round(float(np.percentile(lat_ms, 10)), 3),
                       "p50": round(float(np.percentile(lat_ms, 50)), 3),
                       "p90": round(float(np.percentile(lat_ms, 90)), 3)},
        "temperature": T,
        "escalation_rate": round(res["escalation"], 3),
        "tokens_per_step": round(res["accepted"] / args.steps, 3),
        "replay_mismatch_steps": res["mismatch"],
        "drafting_s_untimed": round(res["t_draft"], 3),
        "roofline": roof,
        "step_roofline": step_roof,
        "mixed_tier_variant": mixed,
        "full_tier_variant": full_tier,
        "sampling_rules_variant": sampled,
        "drafter_model_variant": drafter,
        "prefill_gemm_roofline": prefill,
        "dimr_cost_roofline": dimr,
        "cpu_baseline": cpu,
    }
    if breakdown:
        out["kernels"] = breakdown
    print(json.dumps(out), flush=True)


def dimr_cost_roofline(md, rows=64, reps=10):
    """via_dimr_cost (the routing-mask cost over the vocabulary, one row per
    calibration position) on random fp32 logits of the model's vocabulary:
    algorithmic bytes = one read of both [rows, V] logit matrices; the kernel
    reads them twice (log-partition pass, cost pass)."""
    import ctypes as C
    import torch
    from paper_2606_12243_amd import via
    V = md["vocab"]
    g = torch.Generator(device="cuda").manual_seed(11)
    q = torch.randn(rows, V, device="cuda", generator=g) * 4
    p = q + torch.randn(rows, V, device="cuda", generator=g)
    out = torch.empty(rows, device="cuda")
    stream = torch.cuda.current_stream()
    sp = C.c_void_p(stream.cuda_stream)
    call = lambda: via.check(via.via_dimr_cost(q.data_ptr(), p.data_ptr(), rows, V, V, 1.0, 0.0, 1.0,
                                               out.data_ptr(), sp))
    call()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    alg = 2 * rows * V * 4
    return {"kernel": "dimr_cost_kernel: routing-mask cost, one row per calibration position", "bound": "hbm",
            "rows": rows, "vocab": V, "us": round(us, 2), "bytes_per_launch": alg,
            "achieved": round(alg / (us * 1e-6) / 1e9, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(alg / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}


def measured_copy_gbs(nbytes=1 << 30, reps=5):
    """A plain device-to-device copy of 1 GiB (bytes read + bytes written per
    second), the measured HBM ceiling the roofline fractions are also given
    against."""
    import torch
    src = torch.empty(nbytes // 2, dtype=torch.int16, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    return 2 * nbytes / (ms * 1e-3) / 1e9


def prefill_gemm_roofline(md, M, reps=10):
    """The prefill GEMM (the tile kernel of forwards of more than 512 rows) on
    plain bf16 operands at the model's four projection shapes with M prefill
    rows: algorithmic 2 M N K flops per launch / the average launch time (HIP
    events on the stream of the call) against the bf16 MFMA peak.  The four
    shapes run once untimed before the timed pass (steady clocks: a first
    pass right after the host-side set-up reads up to 15% low)."""
    import ctypes as C
    import torch
    from paper_2606_12243_amd import via
    d, F, V = md["d_model"], md["d_ffn"], md["vocab"]
    H, KVH, hd = md["n_heads"], md["n_kv_heads"], md["head_dim"]
    shapes = {"qkv": ((H + 2 * KVH) * hd, d), "o": (d, H * hd), "gate_up": (2 * F, d), "down": (d, F)}
    stream = torch.cuda.current_stream()
    sp = C.c_void_p(stream.cuda_stream)
    g = torch.Generator(device="cuda").manual_seed(7)

    def launch_ms(N, K):
        Mp = (M + 15) // 16 * 16
        x = (torch.randn(Mp * K, generator=g, device="cuda") * 0.5).to(torch.bfloat16)  # fragment layout
        w = torch.empty(via.via_packed_bytes(N, K, via.DTYPE_BF16) // 2, dtype=torch.bfloat16, device="cuda")
        w.copy_((torch.randn(w.numel(), generator=g, device="cuda") * 0.02).to(torch.bfloat16))
        c = torch.empty(M, N, dtype=torch.float32, device="cuda")
        run = lambda: via.check(via.via_gemm_bf16(x.data_ptr(), w.data_ptr(), c.data_ptr(), M, N, K, sp))
        run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            run()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    for N, K in shapes.values():  # untimed pass
        launch_ms(N, K)
    out, tot_flop, tot_ms = {}, 0.0, 0.0
    for name, (N, K) in shapes.items():
        ms = launch_ms(N, K)
        flop = 2.0 * M * N * K
        tf = flop / (ms * 1e-3) / 1e12
        out[name] = {"N": N, "K": K, "us": round(ms * 1e3, 1), "TFLOPs": round(tf, 1),
                     "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4)}
        tot_flop += flop
        tot_ms += ms
    ach = tot_flop / (tot_ms * 1e-3) / 1e12
    return {"kernel": "gemm_prefill: the four projections of one layer, plain bf16", "bound": "mfma",
            "achieved": round(ach, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(ach / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None, "M": M, "shapes": out}


def prefill_forward_roofline(cfg, W, n_seq=None, ctx=None, per_sequence=True):
    """Real prefills: the workload's sequences (their context lengths, capped
    at 2048 tokens) cached in both caches, full model then slim route, all
    sequences in one forward per cache (via_prefill_batch), and for
    comparison one via_prefill call per sequence.
    Algorithmic FLOPs = 2 * (parameters of the distinct layers run) * rows
    for the projections, counted once, plus the causal attention products
    (QK^T and PV, 4 * rows^2 / 2 * H * hd per layer).  The slim route's
    leading layers that are the full model's own (route[i] == i) compute the
    same values in both caches and count once.  The product computes the
    projections in 2 or 3 passes of bf16 terms (its fp32-activation
    contract), which is cost, not work."""
    import torch
    from paper_2606_12243_amd import via
    from paper_2606_12243_amd.session import Session
    from workload import gen
    md = cfg["model"]
    B = n_seq or cfg["batch"]
    n = min(2048, ctx or int(min(cfg["ctx_lens"]))) - 1
    max_blocks = (n + 64) // 16 + 2
    kv = via.KV(cfg["_model"], max_seqs=B, max_blocks_per_seq=max_blocks, blocks_full=B * max_blocks,
                blocks_slim=B * max_blocks, max_rows=B * n, max_batch=B, max_drafts=8, zero_pools=False)
    sess = Session(cfg["_model"], kv, via.tier_params(0.9, 0.5, 1.0))
    toks = {b: gen.context_tokens(cfg, b, n + 1) for b in range(B)}
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(batched):
        for warm in (True, False):
            torch.cuda.synchronize()
            e0.record()
            if batched:
                sess.prefill_batch(toks)
            else:
                for b in range(B):
                    sess.prefill(b, toks[b])
            e1.record()
            torch.cuda.synchronize()
            for b in range(B):
                sess.release(b)
        return e0.elapsed_time(e1)

    ms_seq = timed(False) if per_sequence else None
    ms = timed(True)
    kv.close()
    d, H, KVH, hd, F = md["d_model"], md["n_heads"], md["n_kv_heads"], md["head_dim"], md["d_ffn"]
    per_layer = d * (H + 2 * KVH) * hd + H * hd * d + 3 * F * d
    route = list(cfg["route"])
    n_shared = 0
    while n_shared < len(route) and route[n_shared] == n_shared:
        n_shared += 1
    layers = md["n_layers"] + len(route) - n_shared
    gemm_flop = 2.0 * per_layer * n * layers * B
    attn_flop = 2.0 * n * n * H * hd * layers * B   # causal half of 4 * n^2 * H * hd
    tf = (gemm_flop + attn_flop) / (ms * 1e-3) / 1e12
    return {"what": "via_prefill_batch of the workload's prompts (full model and slim route, all sequences in "
                    "one forward per cache; the slim route's shared leading layers run once)", "sequences": B,
            "distinct_layers": layers,
            "tokens_per_sequence": n, "ms": round(ms, 2), "algorithmic_TFLOP": round((gemm_flop + attn_flop) / 1e12, 2),
            "achieved": round(tf, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4),
            "one_sequence_per_call": None if ms_seq is None else {
                "ms": round(ms_seq, 2),
                "frac": round((gemm_flop + attn_flop) / (ms_seq * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)},
            "note": "projections run as 2 bf16-term passes of the prefill GEMM (fp32-activation "
                    "contract); the frac counts each product's 2MNK once"}


def measured_traffic(config):
    """HBM bytes per launch of the dominant kernel from the committed counter
    summary (FETCH_SIZE + WRITE_SIZE, scaled by the copy-probe factor), or
    None when the GEMM source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"gemm_gate_up_{config}_traffic.json")
    src = os.path.join(ROOT, "paper_2606_12243_amd", "csrc", "gemm.hip")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    with open(src, "rb") as f:
        digest = hashlib.sha256(f.read()).hexdigest()
    if rec.get("gemm_source_sha256") != digest:
        return None
    return rec.get("traffic_bytes_per_launch")


def _cpu_backend():
    """Threading and BLAS backends torch's CPU ops run on, as torch reports them."""
    import torch
    info = {}
    for line in torch.__config__.parallel_info().splitlines():
        if line.startswith("ATen parallel backend") or line.startswith("ATen/Parallel"):
            info["parallel"] = line.split(":", 1)[-1].strip()
    import re
    for key in ("BLAS_INFO", "LAPACK_INFO"):
        m = re.search(key + r"=([^,\s]+)", torch.__config__.show())
        if m:
            info[key.lower()] = m.group(1)
    return info


def oracle_steps(cfg, W, recorded, init_tokens, T, n_steps, om=None):
    """Replay the first recorded steps of sequence 0 through the oracle (fp64
    CPU): per-step seconds, committed tokens, and whether every step agreed
    with the GPU's committed length."""
    import torch
    from oracle.decode import Draft, TierParams, Verifier
    from oracle.model import OracleModel
    from workload import gen
    md = cfg["model"]
    om = om or OracleModel(md, W)
    ver = Verifier(om, cfg["route"])
    toks = init_tokens[0]
    if cfg.get("seed_kv") is not None:
        n = len(toks) - 1
        bits = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(torch.float64)
        kvf = [tuple(bits(x) for x in gen.synthetic_kv(cfg, 0, s, 0, n)) for s in range(md["n_layers"])]
        kvs = [tuple(bits(x) for x in gen.synthetic_kv(cfg, 1, s, 0, n)) for s in range(len(cfg["route"]))]
        ver.attach_context(toks, kvf, kvs)
    else:
        ver.prefill(toks)
    times, acc, agree, full = [], 0, True, 0
    for i in range(min(n_steps, len(recorded))):
        tok, par = recorded[i][0][0]
        d = Draft.chain(tok) if par is None else Draft(list(tok), list(par))
        n0 = ver.seqs[0].n
        t0 = time.perf_counter()
        dec = ver.step({0: d}, TierParams(0.9, 0.5, T))
        times.append(time.perf_counter() - t0)
        acc += dec[0]["new_len"] - n0
        full += int(dec[0]["full_ran"])
        agree = agree and dec[0]["new_len"] == int(recorded[i][1][0])
        if not agree:
            break
    return times, acc, agree, full, om


def cpu_baseline(cfg, W, recorded, init_tokens, mixed=None, n_steps=3):
    """The oracle, as it stands, on a bounded sample of the same workload:
    the first ``n_steps`` recorded steps of sequence 0 (slim forward,
    decision, full forward when it escalates, commit), replayed in fp64 on
    the host cores; ``mixed`` = (T, recorded, init_tokens) of the mixed-tier
    run adds the same figures there.  value = committed tokens / oracle
    seconds over the sample."""
    import torch
    T = float(cfg["temperature"])
    times, acc, agree, full, om = oracle_steps(cfg, W, recorded, init_tokens, T, n_steps)
    ms = np.array(times) * 1e3
    pct = lambda a: {"p10": round(float(np.percentile(a, 10)), 1), "p50": round(float(np.percentile(a, 50)), 1),
                     "p90": round(float(np.percentile(a, 90)), 1)}
    out = {"value": round(acc / sum(times), 4), "unit": "tokens/s", "cores": torch.get_num_threads(),
           "kind": "oracle",
           "sample": f"first {len(times)} verification steps of sequence 0 of {cfg['name']} at T = {T:.4g} "
                     f"(slim forward, decision, full forward in {full} of them, commit), fp64 numpy/torch on the "
                     f"host: {acc} tokens in {sum(times):.2f}s",
           "precision": "fp64", "step_ms": pct(ms), "steps": len(times), "agrees_with_gpu_steps": bool(agree),
           "affinity_cpus": len(os.sched_getaffinity(0)), "threads_used": torch.get_num_threads(),
           "backend": _cpu_backend()}
    if mixed is not None:
        Tm, rec_m, init_m = mixed
        tm, acc_m, agree_m, full_m, _ = oracle_steps(cfg, W, rec_m, init_m, Tm, n_steps, om)
        out["mixed_tier"] = {"temperature": Tm, "value": round(acc_m / sum(tm), 4), "unit": "tokens/s",
                             "step_ms": pct(np.array(tm) * 1e3), "steps": len(tm), "full_forward_steps": full_m,
                             "agrees_with_gpu_steps": bool(agree_m)}
    return out


if __name__ == "__main__":
    main()
