"""Calibrate the logit temperature of the bf16 workloads (calls only the oracle).

Writes workload/calibrated.py.  The 1B-shape workload scales its logits so
that about half of the drafted positions clear the accept threshold; the
8B-shape model (shared by the chain, tree and long-context workloads) gets
the same rule because at T = 1 none of its positions is accepted.

A second, "mixed" temperature serves the long-context batch (whose steps
must mix all three tiers and roll sequences back to differing lengths) and
the mixed-tier parity and benchmark variants of the 8B chain: the T that
maximises the smallest of the three tier fractions over drafted positions,
where a drafted position is the greedy draft with probability 1 - p and a
uniformly random token with probability p (p = the workload's corruption).
The random-token margins come from the same slim logit rows, at tokens drawn
by a calibration generator seeded per (window, position).

Statistic: teacher-forced windows along the greedy continuation of sequence
0 (drafts = the full verifier's greedy tokens, no corruption; forced full
tier, so every window commits all k drafts).  For draft j of a window with
slim logits l', let m_j = l'(d_j) - max l' <= 0.  The ratio confidence
c_j = exp(m_j / T) clears tau_acc iff T >= t_j = m_j / ln(tau_acc), so the
accepted fraction is the empirical distribution function of the t_j and
the temperature giving one half is the midpoint of its two central order
statistics -- the value a bisection on T converges to.

    python tests/golden/calibrate_temperature.py [1b_bf16] [8b_bf16_chain]
"""
from __future__ import annotations

import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle.decode import FORCED_FULL, GreedyDrafter, TierParams, Verifier  # noqa: E402
from oracle.model import OracleModel  # noqa: E402
from workload import configs, gen  # noqa: E402

TAU_ACC = configs.TAU_ACC
TAU_FULL = configs.TAU_FULL
RANDOM_PER_ROW = 64
# workloads that take the mixed-tier temperature, with their corruption rates
MIXED = {"8b_bf16_chain": {"8b_bf16_chain": 0.30, "8b_bf16_long": 0.35}}
# windows per model: the 8B-shape forwards cost seconds each in fp64
WINDOWS = {"1b_bf16": 16, "8b_bf16_chain": 4}
# workloads that take the 8B-shape model's temperature
SHARES = {"8b_bf16_chain": ["8b_bf16_chain", "8b_bf16_tree", "8b_bf16_long"]}


def log(*a):
    print("[calibrate]", *a, flush=True)


def margins(name: str, windows: int) -> np.ndarray:
    cfg = configs.get(name)
    md = cfg["model"]
    k = cfg["k"]
    t0 = time.time()
    W = gen.model_weights(cfg)
    om = OracleModel(md, W)
    ver = Verifier(om, cfg["route"])
    drafter = GreedyDrafter(om, lambda b, step, j: (False, 0))
    n = gen.context_lengths(cfg)[0]
    tokens = gen.context_tokens(cfg, 0, n + 1)
    if cfg.get("seed_kv") is not None:
        def t64(a):
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(torch.float64)
        kvf = [tuple(t64(x) for x in gen.synthetic_kv(cfg, gen.CACHE_FULL, s, 0, n)) for s in range(md["n_layers"])]
        kvs = [tuple(t64(x) for x in gen.synthetic_kv(cfg, gen.CACHE_SLIM, s, 0, n)) for s in range(len(cfg["route"]))]
        ver.attach_context(tokens, kvf, kvs)
        drafter.attach(0, kvf)
    else:
        ver.prefill(tokens)
        drafter.attach(0)
    log(f"{name}: context {n} ready in {time.time() - t0:.1f}s")
    out, rnd = [], []
    p = TierParams(TAU_ACC, configs.TAU_FULL, 1.0, FORCED_FULL)
    V = md["vocab"]
    for w in range(windows):
        d = drafter.chain(0, ver.seqs[0].tokens, k, w)
        dec = ver.step({0: d}, p)[0]
        st = dec["slim_stats"]
        lg = dec["slim_logits"]
        for j in range(k):
            r = dec["draft_row"][j]
            out.append(dec["slim_draft_logit"][j] - st["max"][r])
            toks = np.random.default_rng([int(cfg["seed_d"]), 99, w, j]).integers(0, V, RANDOM_PER_ROW)
            rnd.extend((lg[r, torch.from_numpy(toks)] - st["max"][r]).tolist())
        log(f"{name}: window {w + 1}/{windows} done ({time.time() - t0:.1f}s)")
    return np.array(out, np.float64), np.array(rnd, np.float64)


def tier_fractions(m: np.ndarray, T: float):
    """Fractions of margins m = l'(d) - max l' in tiers A, S, F at temperature T."""
    c = np.exp(m / T)
    a = float(np.mean(c >= TAU_ACC))
    f = float(np.mean(c < TAU_FULL))
    return a, 1.0 - a - f, f


def mixed_temperature(greedy: np.ndarray, rnd: np.ndarray, p: float):
    """T maximising min(accept, slim, full) over the corrupted-draft mixture
    (middle of the first best plateau of a fine log-spaced grid)."""
    grid = np.exp(np.linspace(math.log(0.25), math.log(128.0), 40001))
    best, lo, hi = -1.0, None, None
    for T in grid:
        g, r = tier_fractions(greedy, T), tier_fractions(rnd, T)
        mn = min((1 - p) * g[i] + p * r[i] for i in range(3))
        if mn > best + 1e-12:
            best, lo, hi = mn, T, T
        elif abs(mn - best) <= 1e-12 and hi is not None and np.isclose(T, hi * grid[1] / grid[0]):
            hi = T
    T = float(np.float32(math.sqrt(lo * hi)))
    g, r = tier_fractions(greedy, T), tier_fractions(rnd, T)
    return T, [round((1 - p) * g[i] + p * r[i], 4) for i in range(3)]


def half_accept_temperature(m: np.ndarray) -> float:
    t = np.sort(m / math.log(TAU_ACC))     # accept iff T >= t_j
    n = len(t)
    T = 0.5 * (t[n // 2 - 1] + t[n // 2])
    return float(np.float32(T))


def main():
    names = sys.argv[1:] or list(WINDOWS)
    path = os.path.join(ROOT, "workload", "calibrated.py")
    ns = {}
    if os.path.exists(path):
        exec(compile(open(path).read(), path, "exec"), ns)
    temps = dict(ns.get("TEMPERATURE", {}))
    mixed = dict(ns.get("MIXED_TEMPERATURE", {}))
    for name in names:
        m, rnd = margins(name, WINDOWS[name])
        T = half_accept_temperature(m)
        acc = float(np.mean(np.exp(m / T) >= TAU_ACC))
        full = float(np.mean(np.exp(m / T) < configs.TAU_FULL))
        log(f"{name}: {len(m)} positions, T = {T!r}: accept {acc:.3f}, full {full:.3f}; "
            f"at T = 1: accept {float(np.mean(np.exp(m) >= TAU_ACC)):.3f}")
        for target in SHARES.get(name, [name]):
            temps[target] = T
        for target, pc in MIXED.get(name, {}).items():
            Tm, fr = mixed_temperature(m, rnd, pc)
            mixed[target] = Tm
            log(f"{target}: mixed-tier T = {Tm!r} at corruption {pc}: accept/slim/full {fr}")
    # the long-context batch runs at its mixed-tier temperature (three tiers, ragged rollbacks)
    if "8b_bf16_long" in mixed:
        temps["8b_bf16_long"] = mixed["8b_bf16_long"]
    body = ['"""Temperatures fixed by tests/golden/calibrate_temperature.py (oracle only).',
            "",
            "TEMPERATURE: the 1B-shape and the 8B chain and tree workloads scale their",
            "logits so that about half of the drafted positions (teacher-forced greedy",
            "windows) clear the accept threshold; the long-context batch runs at its",
            "mixed-tier temperature.",
            "MIXED_TEMPERATURE: the temperature maximising the smallest of the three",
            "tier fractions over drafted positions (greedy drafts mixed with the",
            "workload's rate of uniformly random tokens).  Values are frozen as fp32",
            "literals.",
            '"""',
            "TEMPERATURE = {"]
    body += [f"    {n!r}: {t!r}," for n, t in sorted(temps.items())]
    body += ["}", "MIXED_TEMPERATURE = {"]
    body += [f"    {n!r}: {t!r}," for n, t in sorted(mixed.items())]
    body += ["}", ""]
    with open(path, "w") as f:
        f.write("\n".join(body))
    log(f"wrote {path}")


if __name__ == "__main__":
    main()
