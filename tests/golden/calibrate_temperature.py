"""Calibrate the logit temperature of the bf16 workloads (calls only the oracle).

Writes workload/calibrated.py.  The 1B-shape workload scales its logits so
that about half of the drafted positions clear the accept threshold; the
8B-shape model (shared by the chain, tree and long-context workloads) gets
the same rule because at T = 1 none of its positions is accepted.

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
    out = []
    p = TierParams(TAU_ACC, configs.TAU_FULL, 1.0, FORCED_FULL)
    for w in range(windows):
        d = drafter.chain(0, ver.seqs[0].tokens, k, w)
        dec = ver.step({0: d}, p)[0]
        st = dec["slim_stats"]
        for j in range(k):
            out.append(dec["slim_draft_logit"][j] - st["max"][dec["draft_row"][j]])
        log(f"{name}: window {w + 1}/{windows} done ({time.time() - t0:.1f}s)")
    return np.array(out, np.float64)


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
    for name in names:
        m = margins(name, WINDOWS[name])
        T = half_accept_temperature(m)
        acc = float(np.mean(np.exp(m / T) >= TAU_ACC))
        full = float(np.mean(np.exp(m / T) < configs.TAU_FULL))
        log(f"{name}: {len(m)} positions, T = {T!r}: accept {acc:.3f}, full {full:.3f}; "
            f"at T = 1: accept {float(np.mean(np.exp(m) >= TAU_ACC)):.3f}")
        for target in SHARES.get(name, [name]):
            temps[target] = T
    body = ['"""Temperatures fixed by tests/golden/calibrate_temperature.py (oracle only).',
            "",
            "Each bf16 workload scales its logits so that about half of the drafted",
            "positions (teacher-forced greedy windows) clear the accept threshold;",
            "the 8B-shape workloads share one model and one temperature.  Values are",
            'frozen as fp32 literals.',
            '"""',
            "TEMPERATURE = {"]
    body += [f"    {n!r}: {t!r}," for n, t in sorted(temps.items())]
    body += ["}", ""]
    with open(path, "w") as f:
        f.write("\n".join(body))
    log(f"wrote {path}")


if __name__ == "__main__":
    main()
