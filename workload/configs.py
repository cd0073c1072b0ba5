"""Synthetic workload configurations for the verification step.

Five named workloads (tiny fp32, 1B-shape bf16, 8B-shape bf16 chain / tree /
long-context batch) plus small shapes used by the parity tests.  A config is a
plain dict; nothing here computes any part of the method.

Architecture constants the paper leaves open (it names no architecture of its
own) are fixed here once: RMSNorm eps 1e-5 with unit gains, no biases,
rotate-half RoPE with theta 10000 at absolute positions, GQA head sharing
``kv = h * KVH // H``, SwiGLU FFN, untied LM head (shared between the full
verifier and the slim-verifier, Sec. 3.2 "shares embeddings and the output
head"), final RMSNorm before the head.

Tier thresholds are expressed on the ratio confidence c = q'(d)/max_u q'(u):
accept c >= tau_acc, slim tier tau_full <= c < tau_acc, full tier c < tau_full
(regions A/B/C of App. B.2 with tau_acc = 1 - alpha_1, tau_full = 1 - alpha_2).
"""
from __future__ import annotations

import copy

# 8B-shape slim route: first 8 + last 8 of 32 layers.
_ROUTE_8B = list(range(8)) + list(range(24, 32))

_MODEL_8B = dict(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                 d_ffn=14336, vocab=128256, dtype="bf16", rms_eps=1e-5, rope_theta=10000.0)

CONFIGS = {
    # Tiny fp32 verifier: exercises full and slim routing end to end.
    "tiny_fp32": dict(
        model=dict(n_layers=4, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, d_ffn=1024,
                   vocab=1024, dtype="f32", rms_eps=1e-5, rope_theta=10000.0),
        route=[0, 3], batch=1, ctx=(32, 32), draft="chain", k=4, corrupt=0.30,
        temperature=1.0, gen=64, block_size=16,
        seed_w=1001, seed_c=2001, seed_d=3001, seed_kv=None),
    # ~1B-shape bf16 verifier, slim = every other layer.
    "1b_bf16": dict(
        model=dict(n_layers=16, d_model=2048, n_heads=16, n_kv_heads=4, head_dim=128, d_ffn=5632,
                   vocab=32000, dtype="bf16", rms_eps=1e-5, rope_theta=10000.0),
        route=list(range(0, 16, 2)), batch=1, ctx=(1024, 1024), draft="chain", k=8, corrupt=0.25,
        # Calibrated so that about half of the drafted positions clear the
        # accept threshold (tests/golden/calibrate_temperature.py).
        temperature=None, gen=64, block_size=16,
        seed_w=1002, seed_c=2002, seed_d=3002, seed_kv=None),
    # 8B-shape bf16 verifier, batch 4, context 2048 in a paged cache.  The
    # 8B-shape workloads take the same temperature rule as the 1B shape (at
    # T = 1 no drafted position clears the accept threshold).
    "8b_bf16_chain": dict(
        model=dict(_MODEL_8B), route=list(_ROUTE_8B), batch=4, ctx=(2048, 2048), draft="chain",
        k=8, corrupt=0.30, temperature=None, gen=64, block_size=16,
        seed_w=1003, seed_c=2003, seed_d=3003, seed_kv=4003),
    # 8B-shape with a 60-node token tree (depth 6, branching <= 4).
    "8b_bf16_tree": dict(
        model=dict(_MODEL_8B), route=list(_ROUTE_8B), batch=1, ctx=(4096, 4096), draft="tree",
        tree_budget=[4, 12, 16, 14, 9, 5], tree_branch=4, corrupt=0.20, temperature=None, gen=64,
        block_size=16, seed_w=1003, seed_c=2004, seed_d=3004, seed_kv=4004),
    # 8B-shape long-context batched serving: 16 sequences, ragged contexts.
    "8b_bf16_long": dict(
        model=dict(_MODEL_8B), route=list(_ROUTE_8B), batch=16, ctx=(4096, 8192), draft="chain",
        k=6, corrupt=0.35, temperature=None, gen=64, block_size=16,
        seed_w=1003, seed_c=2005, seed_d=3005, seed_kv=4005),
}

# Thresholds on the ratio confidence (accept >= 0.9, slim in [0.5, 0.9), full < 0.5).
TAU_ACC = 0.9
TAU_FULL = 0.5

# Small shapes for parity tests: several GEMM tiles, ragged vocab tails,
# GQA groups of 1/2/4, head dims 64 and 128.
SMALL = {
    "micro_f32": dict(
        model=dict(n_layers=3, d_model=128, n_heads=2, n_kv_heads=1, head_dim=64, d_ffn=256,
                   vocab=500, dtype="f32", rms_eps=1e-5, rope_theta=10000.0),
        route=[0, 2], seed_w=11),
    "micro_bf16": dict(
        model=dict(n_layers=3, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ffn=512,
                   vocab=1000, dtype="bf16", rms_eps=1e-5, rope_theta=10000.0),
        route=[0, 2], seed_w=12),
    # a drafter with its own weights and dimensions for micro_f32 (same vocabulary)
    "micro_f32_drafter": dict(
        model=dict(n_layers=2, d_model=64, n_heads=1, n_kv_heads=1, head_dim=64, d_ffn=192,
                   vocab=500, dtype="f32", rms_eps=1e-5, rope_theta=10000.0),
        route=[0, 1], seed_w=14),
    "small_bf16_hd128": dict(
        model=dict(n_layers=4, d_model=512, n_heads=8, n_kv_heads=2, head_dim=128, d_ffn=1408,
                   vocab=3001, dtype="bf16", rms_eps=1e-5, rope_theta=10000.0),
        route=[0, 3], seed_w=13),
}


def get(name: str) -> dict:
    """Deep copy of a named config (five workloads or the small parity shapes)."""
    if name in CONFIGS:
        cfg = copy.deepcopy(CONFIGS[name])
    elif name in SMALL:
        cfg = copy.deepcopy(SMALL[name])
    else:
        raise KeyError(name)
    cfg["name"] = name
    if cfg.get("temperature", 1.0) is None:
        from . import calibrated
        cfg["temperature"] = calibrated.TEMPERATURE[name]
    return cfg


def model_bytes(m: dict, route=None) -> dict:
    """Algorithmic byte counts of one forward (weights of routed layers + head)."""
    esz = 4 if m["dtype"] == "f32" else 2
    d, H, KVH, hd, F, V = (m["d_model"], m["n_heads"], m["n_kv_heads"], m["head_dim"],
                           m["d_ffn"], m["vocab"])
    per_layer = (d * (H + 2 * KVH) * hd + H * hd * d + 2 * F * d + F * d + 2 * d) * esz
    layers = m["n_layers"] if route is None else len(route)
    return dict(per_layer=per_layer, layers=layers * per_layer, head=(V * d + d) * esz,
                kv_per_token_layer=2 * KVH * hd * esz)
