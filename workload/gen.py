"""Seeded synthetic inputs shared by the oracle and the GPU path.

Everything here is input data: weights, context tokens, context lengths,
synthetic context K/V values and the per-position draft corruption draws.
No part of the verification method is computed in this module.

Generators are counter-keyed: every tensor (and every chunk of
``CHUNK`` elements of it) has its own numpy ``SFC64`` stream seeded with
``SeedSequence(seed, spawn_key=(tensor_id, chunk))``, so values do not depend
on the number of worker threads and any chunk can be regenerated alone.
Weights are N(0, 0.02^2) drawn in float32; bf16 models store them as bf16
bit patterns (uint16) obtained by round-to-nearest-even of the float32 draw.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

CHUNK = 1 << 22
WEIGHT_STD = np.float32(0.02)

# tensor ids of the weight streams
TID_EMBED, TID_HEAD = 0, 1
TID_LAYER0, TID_PER_LAYER = 16, 8


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal_into(out: np.ndarray, seed: int, tid, std: np.float32, bf16: bool) -> None:
    """Fill ``out`` (flat) with std * N(0,1) float32 draws, chunk-keyed."""
    n = out.size
    nchunks = (n + CHUNK - 1) // CHUNK

    def work(c):
        lo, hi = c * CHUNK, min(n, (c + 1) * CHUNK)
        key = tid if isinstance(tid, tuple) else (tid,)
        g = np.random.Generator(np.random.SFC64(np.random.SeedSequence(seed, spawn_key=key + (c,))))
        buf = g.standard_normal(hi - lo, dtype=np.float32)
        np.multiply(buf, std, out=buf)
        if bf16:
            out[lo:hi] = f32_to_bf16_bits(buf)
        else:
            out[lo:hi] = buf

    if nchunks == 1:
        work(0)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(work, range(nchunks)))


def normal_tensor(shape, seed: int, tid, std=WEIGHT_STD, bf16=True) -> np.ndarray:
    out = np.empty(int(np.prod(shape)), dtype=np.uint16 if bf16 else np.float32)
    _normal_into(out, seed, tid, np.float32(std), bf16)
    return out.reshape(shape)


def weight_shapes(m: dict) -> dict:
    d, H, KVH, hd, F, V = (m["d_model"], m["n_heads"], m["n_kv_heads"], m["head_dim"],
                           m["d_ffn"], m["vocab"])
    return dict(embed=(V, d), lm_head=(V, d), final_norm=(d,), attn_norm=(d,),
                w_qkv=((H + 2 * KVH) * hd, d), w_o=(d, H * hd), ffn_norm=(d,),
                w_gate_up=(2 * F, d), w_down=(d, F))


def model_weights(cfg: dict) -> dict:
    """All weights of a config's verifier as numpy arrays.

    bf16 models: uint16 bf16 bit patterns.  f32 models: float32.
    Matrices are row-major ``[out_features, in_features]``; ``w_qkv`` stacks
    the Q rows (H*hd), then K rows (KVH*hd), then V rows (KVH*hd);
    ``w_gate_up`` stacks the gate rows (F) then the up rows (F).  Norm gains
    are 1.0.
    """
    m = cfg["model"]
    bf16 = m["dtype"] == "bf16"
    seed = cfg["seed_w"]
    sh = weight_shapes(m)
    one = np.uint16(0x3F80) if bf16 else np.float32(1.0)
    dt = np.uint16 if bf16 else np.float32
    W = dict(embed=normal_tensor(sh["embed"], seed, TID_EMBED, bf16=bf16),
             lm_head=normal_tensor(sh["lm_head"], seed, TID_HEAD, bf16=bf16),
             final_norm=np.full(sh["final_norm"], one, dtype=dt),
             attn_norm=[], w_qkv=[], w_o=[], ffn_norm=[], w_gate_up=[], w_down=[])
    for l in range(m["n_layers"]):
        base = TID_LAYER0 + TID_PER_LAYER * l
        W["attn_norm"].append(np.full(sh["attn_norm"], one, dtype=dt))
        W["ffn_norm"].append(np.full(sh["ffn_norm"], one, dtype=dt))
        W["w_qkv"].append(normal_tensor(sh["w_qkv"], seed, base + 0, bf16=bf16))
        W["w_o"].append(normal_tensor(sh["w_o"], seed, base + 1, bf16=bf16))
        W["w_gate_up"].append(normal_tensor(sh["w_gate_up"], seed, base + 2, bf16=bf16))
        W["w_down"].append(normal_tensor(sh["w_down"], seed, base + 3, bf16=bf16))
    return W


def context_lengths(cfg: dict) -> list:
    lo, hi = cfg["ctx"]
    if lo == hi:
        return [lo] * cfg["batch"]
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(cfg["seed_c"], spawn_key=(1 << 20,))))
    return [int(v) for v in g.integers(lo, hi + 1, size=cfg["batch"])]


def context_tokens(cfg: dict, b: int, n: int) -> list:
    """Uniform random prompt tokens in [0, vocab) for sequence ``b``."""
    V = cfg["model"]["vocab"]
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(cfg["seed_c"], spawn_key=(b,))))
    return [int(v) for v in g.integers(0, V, size=n)]


def kv_std(m: dict) -> float:
    """Scale of synthetic context K/V entries: the spread of y @ W for a
    unit-RMS row y and N(0, 0.02^2) weights, 0.02 * sqrt(d_model)."""
    return float(np.float32(0.02) * np.float32(np.sqrt(m["d_model"])))


CACHE_FULL, CACHE_SLIM = 0, 1


def synthetic_kv(cfg: dict, cache: int, layer_slot: int, b: int, n: int):
    """Synthetic context keys/values for ``n`` cached positions.

    Returns (K, V), each ``[n, n_kv_heads, head_dim]`` in the model's storage
    type (uint16 bf16 bits or float32).  Used in place of a prefill for the
    long-context 8B-shape workloads; the values stand for post-RoPE keys and
    values of an arbitrary context.
    """
    m = cfg["model"]
    bf16 = m["dtype"] == "bf16"
    shape = (n, m["n_kv_heads"], m["head_dim"])
    std = kv_std(m)
    # The slim route's leading layers are the full model's first layers
    # (route[i] == i), so a prefill caches the same keys and values for them
    # in both caches: those slim slots draw the full cache's stream.
    route = cfg["route"]
    if cache == CACHE_SLIM and all(route[i] == i for i in range(layer_slot + 1)):
        cache = CACHE_FULL
    K = normal_tensor(shape, cfg["seed_kv"], (cache, layer_slot, b, 0), std=std, bf16=bf16)
    V = normal_tensor(shape, cfg["seed_kv"], (cache, layer_slot, b, 1), std=std, bf16=bf16)
    return K, V


def corruption(seed_d: int, b: int, step: int, j: int, p: float, vocab: int):
    """Draw for draft position ``j`` of sequence ``b`` at decode step ``step``.

    Returns (replace, token): with probability ``p`` the drafted token is
    replaced by ``token``, uniform in [0, vocab).
    """
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed_d, spawn_key=(b, step, j))))
    u = g.random()
    tok = int(g.integers(0, vocab))
    return bool(u < p), tok
