"""Pins of the oracle's verifier forward against things other than itself.

* each op against an independent torch library routine (rms_norm, silu,
  scaled_dot_product_attention) or closed-form properties (RoPE);
* the whole cache-free forward against a second forward assembled from torch
  library routines with RoPE written as a complex rotation;
* the windowed (cached) forward against the cache-free one, and one token at
  a time;
* routing (Sec. 3.3, q'_z = Pi_z(q)): route = all layers reproduces q
  bit for bit; a route equals the model rebuilt without the bypassed layers.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from oracle.model import OracleModel, SeqCache, causal, forward_window, round_bf16
from workload import configs, gen

F64 = torch.float64


@pytest.fixture(scope="module")
def tiny():
    cfg = configs.get("tiny_fp32")
    return cfg, OracleModel(cfg["model"], gen.model_weights(cfg))


@pytest.fixture(scope="module")
def micro16():
    cfg = configs.get("micro_bf16")
    return cfg, OracleModel(cfg["model"], gen.model_weights(cfg))


def test_round_bf16_matches_fp32_to_bf16_conversion():
    g = torch.Generator().manual_seed(0)
    x32 = torch.randn(200000, generator=g, dtype=torch.float32) * torch.exp(
        torch.randn(200000, generator=g) * 4)
    # every fp32 value is exact in fp64, so rounding it directly to bf16 is a
    # single rounding, the same as torch's fp32 -> bf16 conversion (RNE)
    ref = x32.to(torch.bfloat16).to(F64)
    assert torch.equal(round_bf16(x32.to(F64)), ref)


def test_round_bf16_ties_to_even():
    # 1 + 2^-8 lies halfway between bf16 neighbours 1 and 1 + 2^-7: goes to 1 (even)
    # 1 + 3*2^-8 lies halfway between 1+2^-7 and 1+2^-6: goes to 1 + 2^-6 (even)
    x = torch.tensor([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 3.0, 0.0], dtype=F64)
    want = torch.tensor([1.0, 1 + 2 ** -6, -1.0, 3.0, 0.0], dtype=F64)
    assert torch.equal(round_bf16(x), want)


def test_rmsnorm_matches_library(tiny):
    _, m = tiny
    x = torch.randn(7, m.d, dtype=F64)
    g = torch.rand(m.d, dtype=F64) + 0.5
    ref = Fn.rms_norm(x, (m.d,), weight=g, eps=m.eps)
    assert torch.allclose(m.rmsnorm(x, g), ref, rtol=1e-13, atol=1e-13)


def test_silu_matches_library():
    z = torch.linspace(-30, 30, 1001, dtype=F64)
    assert torch.allclose(OracleModel.silu(z), Fn.silu(z), rtol=1e-14, atol=1e-14)


def test_rope_properties(tiny):
    _, m = tiny
    R = 5
    q = torch.randn(R, 1, m.hd, dtype=F64)
    k = torch.randn(R, 1, m.hd, dtype=F64)
    pos = torch.tensor([0, 3, 17, 100, 4095])
    # position 0 is the identity
    assert torch.equal(m.rope(q[:1], torch.tensor([0])), q[:1])
    # each (i, i + hd/2) pair is rotated: its norm is preserved
    r = m.rope(q, pos)
    half = m.hd // 2
    n0 = q[..., :half] ** 2 + q[..., half:] ** 2
    n1 = r[..., :half] ** 2 + r[..., half:] ** 2
    assert torch.allclose(n0, n1, rtol=1e-12)
    # scores depend only on the relative offset: <R(a)q, R(b)k> == <R(a+s)q, R(b+s)k>
    a, b, s = torch.tensor([40]), torch.tensor([7]), 999
    d1 = (m.rope(q[:1], a) * m.rope(k[:1], b)).sum()
    d2 = (m.rope(q[:1], a + s) * m.rope(k[:1], b + s)).sum()
    assert abs(float(d1 - d2)) < 1e-9
    # pair 0 turns by exactly pos radians (theta^0 = 1)
    e = torch.zeros(1, 1, m.hd, dtype=F64)
    e[0, 0, 0] = 1.0
    out = m.rope(e, torch.tensor([2]))
    assert abs(float(out[0, 0, 0]) - math.cos(2.0)) < 1e-15
    assert abs(float(out[0, 0, half]) - math.sin(2.0)) < 1e-15


def test_attention_matches_library(tiny):
    _, m = tiny
    H, KVH, hd = 4, 2, 16
    R, S = 3, 9
    q = torch.randn(R, H, hd, dtype=F64)
    K = torch.randn(S, KVH, hd, dtype=F64)
    V = torch.randn(S, KVH, hd, dtype=F64)
    vis = torch.rand(R, S) < 0.7
    vis[:, 0] = True
    out = m.attend(q, K, V, vis).reshape(R, H, hd)
    rep = H // KVH
    Kr = K.repeat_interleave(rep, dim=1).permute(1, 0, 2)
    Vr = V.repeat_interleave(rep, dim=1).permute(1, 0, 2)
    ref = Fn.scaled_dot_product_attention(q.permute(1, 0, 2), Kr, Vr, attn_mask=vis[None])
    assert torch.allclose(out.permute(1, 0, 2), ref, rtol=1e-12, atol=1e-12)


def _library_forward(m: OracleModel, tokens, route):
    """Second forward built from torch library routines; RoPE as a complex
    rotation of (x_i + i x_{i+hd/2})."""
    T = len(tokens)
    x = m.embed(tokens)
    half = m.hd // 2
    inv = 1.0 / (m.theta ** (torch.arange(half, dtype=F64) * 2 / m.hd))
    rot = torch.polar(torch.ones(T, half, dtype=F64), torch.arange(T, dtype=F64)[:, None] * inv)

    def rope(t):
        z = torch.complex(t[..., :half], t[..., half:]) * rot[:, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    H, KVH, hd = m.H, m.KVH, m.hd
    for l in route:
        y = Fn.rms_norm(x, (m.d,), weight=m.w("attn_norm", l), eps=m.eps)
        p = Fn.linear(y, m.w("w_qkv", l))
        q = rope(p[:, :H * hd].reshape(T, H, hd))
        k = rope(p[:, H * hd:(H + KVH) * hd].reshape(T, KVH, hd))
        v = p[:, (H + KVH) * hd:].reshape(T, KVH, hd)
        rep = H // KVH
        a = Fn.scaled_dot_product_attention(q.permute(1, 0, 2), k.repeat_interleave(rep, 1).permute(1, 0, 2),
                                            v.repeat_interleave(rep, 1).permute(1, 0, 2), is_causal=True)
        x = x + Fn.linear(a.permute(1, 0, 2).reshape(T, H * hd), m.w("w_o", l))
        y = Fn.rms_norm(x, (m.d,), weight=m.w("ffn_norm", l), eps=m.eps)
        gu = Fn.linear(y, m.w("w_gate_up", l))
        x = x + Fn.linear(Fn.silu(gu[:, :m.F]) * gu[:, m.F:], m.w("w_down", l))
    y = Fn.rms_norm(x, (m.d,), weight=m.w("final_norm"), eps=m.eps)
    return Fn.linear(y, m.w("lm_head"))


def test_forward_matches_library_forward(tiny):
    cfg, m = tiny
    toks = gen.context_tokens(cfg, 0, 24)
    for route in (range(m.L), cfg["route"]):
        a = m.forward_sequence(toks, route)
        b = _library_forward(m, toks, list(route))
        assert torch.allclose(a, b, rtol=0, atol=1e-11), float((a - b).abs().max())


def test_cached_equals_cache_free_and_stepwise(tiny):
    cfg, m = tiny
    toks = gen.context_tokens(cfg, 1, 21)
    for route in (list(range(m.L)), cfg["route"]):
        ref = m.forward_sequence(toks, route)
        # prefix of 13 cached, then a window of 8 causal rows
        c = SeqCache(len(route), m.KVH, m.hd)
        forward_window(m, route, c, toks[:13], range(13), causal(13))
        c.valid = 13
        win = forward_window(m, route, c, toks[13:], range(13, 21), causal(8))
        assert torch.allclose(win, ref[13:], rtol=0, atol=1e-11)
        # one token at a time
        c = SeqCache(len(route), m.KVH, m.hd)
        for t in range(len(toks)):
            lg = forward_window(m, route, c, [toks[t]], [t], [[True]])
            c.valid += 1
            assert torch.allclose(lg[0], ref[t], rtol=0, atol=1e-11)


def test_full_route_is_q_bitwise(micro16):
    cfg, m = micro16
    toks = gen.context_tokens(dict(cfg, seed_c=5), 0, 17)
    a = m.forward_sequence(toks)
    b = m.forward_sequence(toks, list(range(m.L)))
    assert torch.equal(a, b)


def test_route_equals_model_without_bypassed_layers(micro16):
    cfg, m = micro16
    route = cfg["route"]
    W = gen.model_weights(cfg)
    W2 = {k: ([v[l] for l in route] if isinstance(v, list) else v) for k, v in W.items()}
    desc = dict(cfg["model"], n_layers=len(route))
    m2 = OracleModel(desc, W2)
    toks = gen.context_tokens(dict(cfg, seed_c=6), 0, 15)
    assert torch.equal(m.forward_sequence(toks, route), m2.forward_sequence(toks))


def test_bf16_storage_points_hold_bf16_values(micro16):
    cfg, m = micro16
    assert m.storage_bf16
    toks = gen.context_tokens(dict(cfg, seed_c=7), 0, 9)
    c = SeqCache(m.L, m.KVH, m.hd)
    forward_window(m, range(m.L), c, toks, range(9), causal(9))
    for s in range(m.L):
        assert torch.equal(round_bf16(c.K[s][:9]), c.K[s][:9])
        assert torch.equal(round_bf16(c.V[s][:9]), c.V[s][:9])


def test_bf16_storage_changes_logits_little(micro16):
    cfg, _ = micro16
    W = gen.model_weights(cfg)
    a = OracleModel(cfg["model"], W, storage_bf16=True)
    b = OracleModel(cfg["model"], W, storage_bf16=False)
    toks = gen.context_tokens(dict(cfg, seed_c=8), 0, 12)
    d = (a.forward_sequence(toks) - b.forward_sequence(toks)).abs().max()
    assert 0 < float(d) < 5e-2


def test_weights_distribution():
    cfg = configs.get("micro_bf16")
    W = gen.model_weights(cfg)
    w = gen.bf16_bits_to_f32(W["w_qkv"][0]).astype(np.float64)
    assert abs(w.mean()) < 2e-3 and abs(w.std() - 0.02) < 1e-3
    assert (gen.bf16_bits_to_f32(W["attn_norm"][0]) == 1.0).all()
