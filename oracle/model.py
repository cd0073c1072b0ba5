"""Oracle verifier forward — TEST INFRASTRUCTURE ONLY.

A plain, slow, fp64 CPU implementation of the decoder-only verifier used by
the VIA-SD verification step, written from the definitions.  Only the test
suite, the smoke check and the benchmark's CPU-baseline leg may import this
package; the product path (the HIP library and its binding) never does, and
this package imports nothing from it.

What it follows:
  * The verifier q is a stack of L transformer layers; the slim-verifier
    q'_z = Pi_z(q) keeps the layers with z_l = 1 and bypasses the others
    (Sec. 3.3, routing mask z in {0,1}^L).  Bypassing a layer means the
    residual stream passes through it unchanged; the retained layers use the
    full model's own weights, and q' shares q's embedding, final norm and
    output head (Sec. 3.2).  ``route`` below is the sorted list of retained
    layer ids; the full verifier is ``route = range(L)``.
  * The layer itself is not specified by the paper; the architecture fixed
    by the workload (RMSNorm, rotate-half RoPE, GQA attention, SwiGLU, untied
    head) is written out here op by op, each from its textbook definition.

Precision: every quantity is fp64.  For bf16 models the "storage" mode
(default on) rounds to bf16 (nearest, ties to even) the one activation a
bf16 verifier stores in bf16: the key/value cache (K after RoPE, V), which
later rows read back.  Weights are bf16 values already; every other
activation (normalised rows, Q, attention output, SwiGLU product, residual
stream, logits) stays fp64.

Parity pins: see tests/test_oracle_model.py (library routines, RoPE
closed-form properties, cached == cache-free == token-by-token, routed ==
layer-deleted model).
"""
from __future__ import annotations

import math

import numpy as np
import torch

F64 = torch.float64


def round_bf16(x: torch.Tensor) -> torch.Tensor:
    """Nearest bf16 value (8 significant bits, ties to even) of fp64 ``x``.

    Computed directly from the fp64 value: x = m * 2**e with 0.5 <= |m| < 1,
    so m * 2**8 is the significand scaled to an integer range; rounding it
    half-to-even and scaling back gives the bf16 value (no double rounding
    through fp32).
    """
    m, e = torch.frexp(x)
    q = torch.round(torch.ldexp(m, torch.full_like(e, 8)))
    return torch.ldexp(q, e - 8)


def _to_torch(a):
    """numpy weight (uint16 bf16 bits or float32) -> torch tensor (bf16/f32)."""
    if isinstance(a, torch.Tensor):
        return a
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))


class OracleModel:
    """The verifier q and its routed sub-models, evaluated in fp64.

    ``weights``: dict as produced by ``workload.gen.model_weights`` (numpy
    arrays, row-major [out, in]).  ``storage_bf16``: round at the bf16
    storage points (default: on for bf16 models).
    """

    def __init__(self, desc: dict, weights: dict, storage_bf16=None, f64_cache_bytes=6 << 30):
        self.desc = dict(desc)
        self.L = desc["n_layers"]
        self.d = desc["d_model"]
        self.H = desc["n_heads"]
        self.KVH = desc["n_kv_heads"]
        self.hd = desc["head_dim"]
        self.F = desc["d_ffn"]
        self.V = desc["vocab"]
        self.eps = float(desc["rms_eps"])
        self.theta = float(desc["rope_theta"])
        bf16 = desc["dtype"] == "bf16"
        self.storage_bf16 = bf16 if storage_bf16 is None else bool(storage_bf16)
        self.W = {}
        for k, v in weights.items():
            self.W[k] = [_to_torch(t) for t in v] if isinstance(v, list) else _to_torch(v)
        n_param = sum((t.numel() for k, v in self.W.items() for t in (v if isinstance(v, list) else [v])))
        # Small models keep an fp64 copy of every weight; large ones upcast on use.
        self._keep = n_param * 8 <= f64_cache_bytes
        self._f64 = {}

    # ------------------------------------------------------------------ weights
    def w(self, name: str, layer=None) -> torch.Tensor:
        key = (name, layer)
        if key in self._f64:
            return self._f64[key]
        t = self.W[name] if layer is None else self.W[name][layer]
        t64 = t.to(F64)
        if self._keep:
            self._f64[key] = t64
        return t64

    def store(self, x: torch.Tensor) -> torch.Tensor:
        """Cache storage: round K/V to bf16 when that mode is on."""
        return round_bf16(x) if self.storage_bf16 else x

    # ---------------------------------------------------------------- ops
    def rmsnorm(self, x: torch.Tensor, g: torch.Tensor) -> torch.Tensor:
        """y = x / sqrt(mean(x^2) + eps) * g over the last axis."""
        ms = (x * x).sum(dim=-1, keepdim=True) / x.shape[-1]
        return x / torch.sqrt(ms + self.eps) * g

    def rope(self, x: torch.Tensor, pos: torch.Tensor) -> torch.Tensor:
        """Rotate-half rotary embedding: pair (i, i + hd/2) turned by
        pos * theta^(-2i/hd).  x: [R, heads, hd], pos: [R] (int)."""
        half = self.hd // 2
        i = torch.arange(half, dtype=F64)
        inv_freq = self.theta ** (-2.0 * i / self.hd)
        ang = pos.to(F64)[:, None] * inv_freq[None, :]
        c, s = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
        x1, x2 = x[..., :half], x[..., half:]
        return torch.cat([x1 * c - x2 * s, x2 * c + x1 * s], dim=-1)

    @staticmethod
    def silu(z: torch.Tensor) -> torch.Tensor:
        return z / (1.0 + torch.exp(-z))

    @staticmethod
    def softmax_rows(s: torch.Tensor) -> torch.Tensor:
        """exp(s - max) / sum(exp(s - max)) over the last axis; -inf entries
        are masked keys."""
        mx = s.max(dim=-1, keepdim=True).values
        e = torch.exp(s - mx)
        return e / e.sum(dim=-1, keepdim=True)

    def linear(self, x: torch.Tensor, name: str, layer=None, rows=None) -> torch.Tensor:
        """x @ W^T with W [out, in] (optionally only a row range of W)."""
        W = self.w(name, layer)
        if rows is not None:
            W = W[rows[0]:rows[1]]
        return x @ W.T

    # ------------------------------------------------------------ layers
    def qkv(self, y: torch.Tensor, l: int, pos: torch.Tensor):
        """Projections of normalised rows y [R, d] -> RoPE'd, stored Q/K/V."""
        R = y.shape[0]
        H, KVH, hd = self.H, self.KVH, self.hd
        p = self.linear(y, "w_qkv", l)
        q = p[:, : H * hd].reshape(R, H, hd)
        k = p[:, H * hd:(H + KVH) * hd].reshape(R, KVH, hd)
        v = p[:, (H + KVH) * hd:].reshape(R, KVH, hd)
        q = self.rope(q, pos)
        k = self.store(self.rope(k, pos))
        v = self.store(v)
        return q, k, v

    def attend(self, q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, vis: torch.Tensor):
        """Scaled dot-product attention with a visibility matrix.

        q [R, H, hd]; K, V [S, KVH, hd]; vis [R, S] bool.  Query head h reads
        KV head h * KVH // H.  Returns [R, H*hd].
        """
        R, H, hd = q.shape
        KVH = K.shape[1]
        kv_of = torch.tensor([h * KVH // H for h in range(H)])
        Kh = K[:, kv_of, :].permute(1, 0, 2)          # [H, S, hd]
        Vh = V[:, kv_of, :].permute(1, 0, 2)
        s = torch.matmul(q.permute(1, 0, 2), Kh.transpose(1, 2)) / math.sqrt(hd)   # [H, R, S]
        s = s.masked_fill(~vis[None, :, :], float("-inf"))
        p = self.softmax_rows(s)
        o = torch.matmul(p, Vh)                        # [H, R, hd]
        return o.permute(1, 0, 2).reshape(R, H * hd)

    def ffn(self, x: torch.Tensor, l: int) -> torch.Tensor:
        y = self.rmsnorm(x, self.w("ffn_norm", l))
        g = self.linear(y, "w_gate_up", l, rows=(0, self.F))
        u = self.linear(y, "w_gate_up", l, rows=(self.F, 2 * self.F))
        h = self.silu(g) * u
        return self.linear(h, "w_down", l)

    def head(self, x: torch.Tensor, chunk=16384) -> torch.Tensor:
        """Final RMSNorm then the output head: logits [R, V]."""
        y = self.rmsnorm(x, self.w("final_norm"))
        if self._keep:
            return self.linear(y, "lm_head")
        out = torch.empty((y.shape[0], self.V), dtype=F64)
        Wb = self.W["lm_head"]
        for lo in range(0, self.V, chunk):
            hi = min(self.V, lo + chunk)
            out[:, lo:hi] = y @ Wb[lo:hi].to(F64).T
        return out

    def embed(self, tokens) -> torch.Tensor:
        idx = torch.as_tensor(list(tokens), dtype=torch.long)
        return self.W["embed"][idx].to(F64)

    # --------------------------------------------------- cache-free forward
    def forward_sequence(self, tokens, route=None) -> torch.Tensor:
        """Textbook causal forward over a whole token sequence (no cache).

        Token t sits at position t and attends to positions 0..t.  Layers not
        in ``route`` are bypassed (identity on the residual stream).
        Returns logits [T, V].
        """
        route = list(range(self.L)) if route is None else list(route)
        T = len(tokens)
        pos = torch.arange(T)
        vis = torch.tril(torch.ones(T, T, dtype=torch.bool))
        x = self.embed(tokens)
        for l in route:
            y = self.rmsnorm(x, self.w("attn_norm", l))
            q, k, v = self.qkv(y, l, pos)
            a = self.attend(q, k, v, vis)
            x = x + self.linear(a, "w_o", l)
            x = x + self.ffn(x, l)
        return self.head(x)


class SeqCache:
    """One sequence's K/V for one route: slot-indexed arrays per route layer.

    ``valid`` slots [0, valid) hold committed positions; a forward writes its
    rows at slots valid, valid+1, ... without moving ``valid``.
    """

    def __init__(self, n_route: int, KVH: int, hd: int):
        self.K = [torch.zeros((0, KVH, hd), dtype=F64) for _ in range(n_route)]
        self.V = [torch.zeros((0, KVH, hd), dtype=F64) for _ in range(n_route)]
        self.valid = 0

    def _grow(self, s: int, n: int):
        cur = self.K[s].shape[0]
        if cur < n:
            pad = torch.zeros((n - cur,) + tuple(self.K[s].shape[1:]), dtype=F64)
            self.K[s] = torch.cat([self.K[s], pad])
            self.V[s] = torch.cat([self.V[s], pad.clone()])

    def write(self, s: int, slot0: int, k: torch.Tensor, v: torch.Tensor):
        self._grow(s, slot0 + k.shape[0])
        self.K[s][slot0:slot0 + k.shape[0]] = k
        self.V[s][slot0:slot0 + v.shape[0]] = v

    def set_context(self, s: int, k: torch.Tensor, v: torch.Tensor):
        """Install context K/V for slots [0, n) (synthetic-context workloads)."""
        self.K[s] = k.clone()
        self.V[s] = v.clone()

    def move(self, src: int, dst: int):
        """Copy the K/V of slot ``src`` to slot ``dst`` in every route layer."""
        for s in range(len(self.K)):
            self.K[s][dst] = self.K[s][src]
            self.V[s][dst] = self.V[s][src]


def forward_window(model: OracleModel, route, cache: SeqCache, tokens, positions, win_vis):
    """Forward a block of rows against a sequence's cache.

    Row r holds token ``tokens[r]`` at RoPE position ``positions[r]`` and is
    written to slot ``cache.valid + r``.  It attends to every committed slot
    [0, cache.valid) and to the block's rows r' with ``win_vis[r][r']`` true
    (a causal chain has win_vis lower-triangular; a token tree has the
    ancestors-and-self mask).  ``cache.valid`` is not changed.
    Returns logits [R, V].
    """
    route = list(route)
    R = len(tokens)
    base = cache.valid
    pos = torch.as_tensor(list(positions), dtype=torch.long)
    wv = torch.as_tensor(np.asarray(win_vis, dtype=bool))
    vis = torch.cat([torch.ones((R, base), dtype=torch.bool), wv], dim=1)
    x = model.embed(tokens)
    for s, l in enumerate(route):
        y = model.rmsnorm(x, model.w("attn_norm", l))
        q, k, v = model.qkv(y, l, pos)
        cache.write(s, base, k, v)
        K = cache.K[s][: base + R]
        V = cache.V[s][: base + R]
        a = model.attend(q, K, V, vis)
        x = x + model.linear(a, "w_o", l)
        x = x + model.ffn(x, l)
    return model.head(x)


def causal(R: int):
    return np.tril(np.ones((R, R), dtype=bool))
