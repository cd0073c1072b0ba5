"""ctypes binding of libvia.so (include/via.h), names as in the C ABI.

Argument marshalling only: every step of the verification path runs in the
library's HIP kernels.  torch supplies device memory (weights, KV pools,
workspace, outputs), pinned host buffers and the stream.  Importing this
module fails loudly if the built library is missing.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libvia.so")

OK, EINVAL, ENOMEM, EDEVICE, ESTATE, EUNSUPPORTED = 0, -1, -2, -3, -4, -5
DTYPE_F32, DTYPE_BF16 = 0, 1
CACHE_FULL, CACHE_SLIM = 0, 1
TIER_ACCEPT, TIER_SLIM, TIER_FULL = 0, 1, 2
FORCED_NONE, FORCED_ACCEPT, FORCED_SLIM, FORCED_FULL = -1, 0, 1, 2
BLOCK = 16
MAX_TREE_ROWS = 64
MAX_DRAFTS = 64


class ViaError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"via status {status}: {msg}")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_12243_amd.build`")
    return C.CDLL(LIB_PATH)


lib = _load()

P = C.c_void_p
I32 = C.c_int32
PI32 = C.POINTER(C.c_int32)


class ModelDesc(C.Structure):
    _fields_ = [("n_layers", I32), ("d_model", I32), ("n_heads", I32), ("n_kv_heads", I32),
                ("head_dim", I32), ("d_ffn", I32), ("vocab", I32), ("rms_eps", C.c_float),
                ("rope_theta", C.c_float), ("dtype", I32)]


class Weights(C.Structure):
    _fields_ = [("embed", P), ("lm_head", P), ("final_norm", P), ("attn_norm", C.POINTER(P)),
                ("w_qkv", C.POINTER(P)), ("w_o", C.POINTER(P)), ("ffn_norm", C.POINTER(P)),
                ("w_gate_up", C.POINTER(P)), ("w_down", C.POINTER(P))]


class TierParams(C.Structure):
    _fields_ = [("tau_acc", C.c_float), ("tau_full", C.c_float), ("temperature", C.c_float), ("forced", I32)]


class KvDesc(C.Structure):
    _fields_ = [("block_size", I32), ("max_seqs", I32), ("max_blocks_per_seq", I32), ("blocks_full", I32),
                ("blocks_slim", I32), ("pool_full", P), ("pool_slim", P), ("max_rows", I32),
                ("max_batch", I32), ("max_drafts", I32), ("workspace", P), ("workspace_bytes", C.c_size_t),
                ("pinned_staging", P), ("staging_bytes", C.c_size_t)]


class Window(C.Structure):
    # host pointers (int32 arrays; row_mask uint64), passed as addresses
    _fields_ = [("batch", I32), ("max_rows", I32), ("max_drafts", I32), ("max_lag", I32),
                ("seq_id", P), ("n_rows", P), ("row_tok", P), ("row_depth", P),
                ("row_mask", P), ("n_drafts", P), ("draft_tok", P),
                ("draft_row", P), ("draft_parent", P), ("n_lag", P), ("lag_tok", P)]


class VerifyOut(C.Structure):
    _fields_ = [("row_argmax", P), ("row_max", P), ("row_sumexp", P), ("row_gap", P),
                ("draft_logit", P), ("logits", P)]


class Decision(C.Structure):
    _fields_ = [("tier", P), ("conf", P), ("packed", P), ("h_packed", P)]


class SamplingC(C.Structure):
    _fields_ = [("alpha", C.c_float), ("beta", C.c_float), ("draft_probs", P), ("uniforms", P)]


def _sig(name, res, *args):
    f = getattr(lib, name)
    f.restype = res
    f.argtypes = list(args)
    return f


via_packed_bytes = _sig("via_packed_bytes", C.c_size_t, I32, I32, I32)
via_pack_weight = _sig("via_pack_weight", I32, P, P, I32, I32, I32, P)
via_pack_gate_up = _sig("via_pack_gate_up", I32, P, P, I32, I32, I32, P)
via_gemm_bf16 = _sig("via_gemm_bf16", I32, P, P, P, I32, I32, I32, P)
via_pool_bytes = _sig("via_pool_bytes", C.c_size_t, C.POINTER(ModelDesc), I32, I32, I32)
via_dimr_cost = _sig("via_dimr_cost", I32, P, P, I32, I32, I32, C.c_float, C.c_float, C.c_float, P, P)
via_workspace_bytes = _sig("via_workspace_bytes", C.c_size_t, C.POINTER(ModelDesc), I32, I32, I32, I32, I32)
via_staging_bytes = _sig("via_staging_bytes", C.c_size_t, C.POINTER(ModelDesc), I32, I32, I32, I32)
via_model_create = _sig("via_model_create", I32, C.POINTER(ModelDesc), C.POINTER(Weights), C.POINTER(P))
via_model_set_route = _sig("via_model_set_route", I32, P, PI32, I32)
via_model_destroy = _sig("via_model_destroy", I32, P)
via_kv_create = _sig("via_kv_create", I32, P, C.POINTER(KvDesc), C.POINTER(P))
via_kv_destroy = _sig("via_kv_destroy", I32, P)
via_kv_seq_reserve = _sig("via_kv_seq_reserve", I32, P, I32, I32)
via_prefill = _sig("via_prefill", I32, P, P, I32, PI32, I32, P)
via_prefill_batch = _sig("via_prefill_batch", I32, P, P, I32, PI32, PI32, PI32, P)
via_kv_seq_release = _sig("via_kv_seq_release", I32, P, I32)
via_kv_seq_info = _sig("via_kv_seq_info", I32, P, I32, I32, PI32, PI32, I32, PI32)
via_kv_last_full_start = _sig("via_kv_last_full_start", I32, P, PI32)
via_verify_slim = _sig("via_verify_slim", I32, P, P, C.POINTER(Window), C.POINTER(TierParams),
                       C.POINTER(VerifyOut), P)
via_verify_full = _sig("via_verify_full", I32, P, P, C.POINTER(Window), PI32, C.POINTER(TierParams),
                       C.POINTER(VerifyOut), P)
via_verify_probe = _sig("via_verify_probe", I32, P, P, I32, C.POINTER(Window), C.POINTER(TierParams),
                        C.POINTER(VerifyOut), P)
via_tier_decide = _sig("via_tier_decide", I32, P, C.POINTER(TierParams), C.POINTER(VerifyOut),
                       C.POINTER(VerifyOut), C.POINTER(Decision), P)
via_tier_decide_sampled = _sig("via_tier_decide_sampled", I32, P, C.POINTER(TierParams), C.POINTER(VerifyOut),
                               C.POINTER(VerifyOut), C.POINTER(SamplingC), C.POINTER(Decision), P)
via_sample_rows = _sig("via_sample_rows", I32, P, C.POINTER(VerifyOut), I32, I32, PI32, C.c_float, P, P, P, I32,
                       P)
via_sample_rows_static = _sig("via_sample_rows_static", I32, C.POINTER(VerifyOut), I32, I32, I32, PI32, C.c_float, P,
                              P, P, I32, P)
via_kv_commit_rollback = _sig("via_kv_commit_rollback", I32, P, C.POINTER(Decision), P)
via_kv_seq_set_tokens = _sig("via_kv_seq_set_tokens", I32, P, I32, PI32, I32)
via_kv_seq_tokens = _sig("via_kv_seq_tokens", I32, P, I32, PI32, I32, PI32)
via_kv_timer_enable = _sig("via_kv_timer_enable", I32, P, C.c_uint32)
via_kv_timer_read = _sig("via_kv_timer_read", I32, P, I32, PI32, C.POINTER(C.c_double))
via_last_error = _sig("via_last_error", C.c_char_p)
via_version = _sig("via_version", C.c_char_p)

EXPORTS = ["via_packed_bytes", "via_pack_weight", "via_pack_gate_up", "via_gemm_bf16", "via_dimr_cost", "via_pool_bytes", "via_workspace_bytes", "via_staging_bytes", "via_model_create",
           "via_model_set_route", "via_model_destroy", "via_kv_create", "via_kv_destroy",
           "via_kv_seq_reserve", "via_prefill", "via_prefill_batch", "via_kv_seq_release", "via_kv_seq_info",
           "via_kv_last_full_start",
           "via_verify_slim", "via_verify_full", "via_verify_probe", "via_tier_decide", "via_tier_decide_sampled", "via_sample_rows",
           "via_sample_rows_static", "via_kv_seq_set_tokens", "via_kv_seq_tokens", "via_step",
           "via_kv_commit_rollback", "via_kv_timer_enable", "via_kv_timer_read", "via_last_error",
           "via_version"]
KERNEL_QKV, KERNEL_ATTN, KERNEL_O, KERNEL_GATEUP, KERNEL_DOWN, KERNEL_HEAD, KERNEL_DECIDE = range(7)
KERNEL_NAMES = ["qkv", "attn", "o", "gateup", "down", "head", "decide"]


def check(status):
    if status != OK:
        raise ViaError(status, via_last_error().decode())
    return status


def _ptr(t: torch.Tensor):
    return C.c_void_p(t.data_ptr()) if t is not None else None


def _i32(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return a, a.ctypes.data_as(PI32)


def model_desc(m: dict) -> ModelDesc:
    return ModelDesc(m["n_layers"], m["d_model"], m["n_heads"], m["n_kv_heads"], m["head_dim"], m["d_ffn"],
                     m["vocab"], float(m["rms_eps"]), float(m["rope_theta"]),
                     DTYPE_BF16 if m["dtype"] == "bf16" else DTYPE_F32)


def stream_ptr(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


class Model:
    """Device weights + via_model handle.  ``weights`` as produced by the
    workload generator (numpy uint16 bf16 bits or float32)."""

    def __init__(self, desc: dict, weights: dict, route, device="cuda"):
        self.desc = dict(desc)
        self.cdesc = model_desc(desc)
        bf16 = desc["dtype"] == "bf16"

        def dev(a):
            if isinstance(a, torch.Tensor):
                return a.to(device).contiguous()
            t = torch.from_numpy(a.view(np.int16) if bf16 else a)
            t = t.view(torch.bfloat16) if bf16 else t
            return t.to(device).contiguous()

        dt = DTYPE_BF16 if bf16 else DTYPE_F32
        stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)

        def packed(a, gate_up=False):
            # row-major [rows, cols] -> device -> packed tiles (the layout the GEMMs stream);
            # the gate/up matrix has its gate and up rows interleaved by 8
            src = dev(a)
            rows, cols = src.shape
            nb = via_packed_bytes(rows, cols, dt)
            if nb == 0:
                raise ViaError(EUNSUPPORTED, f"cannot pack a [{rows}, {cols}] matrix")
            dst = torch.empty(nb // src.element_size(), dtype=src.dtype, device=device)
            if gate_up:
                check(via_pack_gate_up(src.data_ptr(), dst.data_ptr(), rows // 2, cols, dt, stream))
            else:
                check(via_pack_weight(src.data_ptr(), dst.data_ptr(), rows, cols, dt, stream))
            torch.cuda.current_stream().synchronize()
            return dst

        PACKED = ("lm_head", "w_qkv", "w_o", "w_down")
        self.t = {}
        for k, v in weights.items():
            if k == "w_gate_up":
                f = lambda x: packed(x, gate_up=True)
            else:
                f = packed if k in PACKED else dev
            self.t[k] = [f(x) for x in v] if isinstance(v, list) else f(v)
        L = desc["n_layers"]
        arr = lambda k: (P * L)(*[x.data_ptr() for x in self.t[k]])
        self._arrs = {k: arr(k) for k in ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")}
        w = Weights(self.t["embed"].data_ptr(), self.t["lm_head"].data_ptr(), self.t["final_norm"].data_ptr(),
                    self._arrs["attn_norm"], self._arrs["w_qkv"], self._arrs["w_o"], self._arrs["ffn_norm"],
                    self._arrs["w_gate_up"], self._arrs["w_down"])
        h = P()
        check(via_model_create(C.byref(self.cdesc), C.byref(w), C.byref(h)))
        self.h = h
        self.route = list(route)
        r, rp = _i32(self.route)
        check(via_model_set_route(self.h, rp, len(self.route)))

    def close(self):
        if self.h:
            check(via_model_destroy(self.h))
            self.h = None


class KV:
    """Paged full/slim KV pools, workspace and pinned staging of one handle."""

    def __init__(self, model: Model, max_seqs, max_blocks_per_seq, blocks_full, blocks_slim, max_rows,
                 max_batch, max_drafts, device="cuda", zero_pools=True, pools=None):
        self.model = model
        d = model.cdesc
        esz = 2 if model.desc["dtype"] == "bf16" else 4
        nb_full = via_pool_bytes(C.byref(d), model.desc["n_layers"], blocks_full, BLOCK)
        nb_slim = via_pool_bytes(C.byref(d), len(model.route), blocks_slim, BLOCK)
        mk = torch.zeros if zero_pools else torch.empty
        dt = torch.bfloat16 if esz == 2 else torch.float32
        if pools is not None:          # reuse pools (and their contents) of an earlier handle
            self.pool_full, self.pool_slim = pools
            assert self.pool_full.numel() * esz >= nb_full and self.pool_slim.numel() * esz >= nb_slim
        else:
            self.pool_full = mk(nb_full // esz, dtype=dt, device=device)
            self.pool_slim = mk(nb_slim // esz, dtype=dt, device=device)
        wsb = via_workspace_bytes(C.byref(d), max_rows, max_batch, max_blocks_per_seq, max_drafts, max_seqs)
        stb = via_staging_bytes(C.byref(d), max_rows, max_batch, max_blocks_per_seq, max_drafts)
        self.workspace = torch.empty(wsb, dtype=torch.uint8, device=device)
        self.staging = torch.empty(stb, dtype=torch.uint8, pin_memory=True)
        self.cd = KvDesc(BLOCK, max_seqs, max_blocks_per_seq, blocks_full, blocks_slim,
                         self.pool_full.data_ptr(), self.pool_slim.data_ptr(), max_rows, max_batch,
                         max_drafts, self.workspace.data_ptr(), wsb, self.staging.data_ptr(), stb)
        h = P()
        check(via_kv_create(model.h, C.byref(self.cd), C.byref(h)))
        self.h = h
        self.max_batch, self.max_drafts, self.max_rows = max_batch, max_drafts, max_rows

    def close(self):
        if self.h:
            check(via_kv_destroy(self.h))
            self.h = None

    def valid_len(self, seq, cache):
        valid, nb = C.c_int32(), C.c_int32()
        check(via_kv_seq_info(self.h, seq, cache, C.byref(valid), None, 0, C.byref(nb)))
        return valid.value

    def seq_info(self, seq, cache):
        valid, nb = C.c_int32(), C.c_int32()
        check(via_kv_seq_info(self.h, seq, cache, C.byref(valid), None, 0, C.byref(nb)))
        tab = np.zeros(max(1, nb.value), dtype=np.int32)
        check(via_kv_seq_info(self.h, seq, cache, C.byref(valid), tab.ctypes.data_as(PI32), len(tab),
                              C.byref(nb)))
        return valid.value, tab[:nb.value].tolist()

    def last_full_start(self):
        """Route index the last full forward started at (0, the shared-prefix length, or -1)."""
        v = C.c_int32()
        check(via_kv_last_full_start(self.h, C.byref(v)))
        return v.value

    def timer_enable(self, mask):
        check(via_kv_timer_enable(self.h, mask))

    def timer_read(self, kind):
        n, ms = C.c_int32(), C.c_double()
        check(via_kv_timer_read(self.h, kind, C.byref(n), C.byref(ms)))
        return n.value, ms.value

    def pool_view(self, cache):
        """Pool as [slots, KVH, blocks, 2, 16*hd]: K page [hd/8][16][8], V page [hd][16]."""
        m = self.model.desc
        slots = m["n_layers"] if cache == CACHE_FULL else len(self.model.route)
        nb = self.cd.blocks_full if cache == CACHE_FULL else self.cd.blocks_slim
        t = self.pool_full if cache == CACHE_FULL else self.pool_slim
        return t.view(slots, m["n_kv_heads"], nb, 2, BLOCK * m["head_dim"])


class WindowBuf:
    """Host arrays of a via_window (kept alive with the struct).  Every int32
    field lives in one buffer (the tree masks in a uint64 one), filled from
    Python lists and converted once: per-step cost matters, the window is
    built on the step's critical path."""

    def __init__(self, seq_ids, rows, drafts, draft_rows, parents=None, depths=None, masks=None,
                 lags=None, max_rows=None, max_drafts=None):
        B = len(seq_ids)
        self.B = B
        self.max_rows = R = max_rows or max(len(r) for r in rows)
        self.max_drafts = D = max_drafts or max(1, max(len(d) for d in drafts))
        self.max_lag = Lg = max(1, max((len(l) for l in lags), default=1)) if lags else 1
        tree = parents is not None
        spec = [("seq", B), ("n_rows", B), ("row_tok", B * R), ("n_drafts", B), ("draft_tok", B * D),
                ("draft_row", B * D)]
        if tree:
            spec += [("draft_parent", B * D), ("row_depth", B * R)]
        if lags is not None:
            spec += [("n_lag", B), ("lag_tok", B * Lg)]
        off, o = {}, 0
        for name, n in spec:
            off[name] = o
            o += n
        buf = [0] * o

        def put(name, lists, width):
            base = off[name]
            for b, l in enumerate(lists):
                buf[base + b * width: base + b * width + len(l)] = l

        buf[0:B] = seq_ids
        buf[off["n_rows"]:off["n_rows"] + B] = [len(r) for r in rows]
        put("row_tok", rows, R)
        buf[off["n_drafts"]:off["n_drafts"] + B] = [len(d) for d in drafts]
        put("draft_tok", drafts, D)
        put("draft_row", draft_rows, D)
        if tree:
            buf[off["draft_parent"]:off["draft_parent"] + B * D] = [-1] * (B * D)
            put("draft_parent", parents, D)
            put("row_depth", depths, R)
        if lags is not None:
            buf[off["n_lag"]:off["n_lag"] + B] = [len(l) for l in lags]
            put("lag_tok", lags, Lg)
        arr = np.array(buf, np.int32)
        self._buf = arr
        self.a = {name: arr[off[name]:off[name] + n] for name, n in spec}
        addr = arr.ctypes.data
        ptr = lambda k: addr + 4 * off[k] if k in off else None
        mask_ptr = None
        if tree:
            mk = [0] * (B * R)
            for b, l in enumerate(masks):
                mk[b * R: b * R + len(l)] = l
            self.a["row_mask"] = np.array(mk, np.uint64)
            mask_ptr = self.a["row_mask"].ctypes.data
        self.c = Window(B, R, D, Lg, ptr("seq"), ptr("n_rows"), ptr("row_tok"), ptr("row_depth"), mask_ptr,
                        ptr("n_drafts"), ptr("draft_tok"), ptr("draft_row"), ptr("draft_parent"), ptr("n_lag"),
                        ptr("lag_tok"))


class Out:
    """Device outputs of one verify forward."""

    def __init__(self, B, max_rows, max_drafts, vocab=None, logits=False, device="cuda"):
        n = B * max_rows
        self.row_argmax = torch.empty(n, dtype=torch.int32, device=device)
        self.row_max = torch.empty(n, dtype=torch.float32, device=device)
        self.row_sumexp = torch.empty(n, dtype=torch.float32, device=device)
        self.row_gap = torch.empty(n, dtype=torch.float32, device=device)
        self.draft_logit = torch.empty(B * max_drafts, dtype=torch.float32, device=device)
        self.logits = torch.empty(n * vocab, dtype=torch.float32, device=device) if logits else None
        self.c = VerifyOut(self.row_argmax.data_ptr(), self.row_max.data_ptr(), self.row_sumexp.data_ptr(),
                           self.row_gap.data_ptr(), self.draft_logit.data_ptr(),
                           self.logits.data_ptr() if logits else None)


class Dec:
    """Decision arrays (device) + pinned host mirror of the packed block."""

    def __init__(self, B, max_drafts, device="cuda"):
        self.B, self.D = B, max_drafts
        self.tier = torch.empty(B * max_drafts, dtype=torch.int8, device=device)
        self.conf = torch.empty(B * max_drafts, dtype=torch.float32, device=device)
        self.packed = torch.empty(4 * B + B * max_drafts, dtype=torch.int32, device=device)
        self.h_packed = torch.empty(4 * B + B * max_drafts, dtype=torch.int32, pin_memory=True)
        self.c = Decision(self.tier.data_ptr(), self.conf.data_ptr(), self.packed.data_ptr(),
                          self.h_packed.data_ptr())

    def host(self):
        h = self.h_packed.numpy()
        B = self.B
        return dict(status=h[:B].copy(), kappa=h[B:2 * B].copy(), emit=h[2 * B:3 * B].copy(),
                    new_len=h[3 * B:4 * B].copy(), path=h[4 * B:].reshape(B, self.D).copy())

    def set_host(self, status, kappa, emit, new_len, path):
        h = self.h_packed.numpy()
        B = self.B
        h[:B], h[B:2 * B], h[2 * B:3 * B], h[3 * B:4 * B] = status, kappa, emit, new_len
        h[4 * B:] = np.asarray(path, np.int32).reshape(-1)


class Drafts(C.Structure):
    _fields_ = [("batch", I32), ("max_drafts", I32), ("seq_id", P), ("n_drafts", P), ("draft_tok", P),
                ("draft_parent", P)]


class DraftsBuf:
    """Host arrays of a via_drafts (kept alive with the struct): {seq: (tokens,
    parents or None)} in batch order."""

    def __init__(self, drafts: dict):
        seqs = list(drafts)
        B = len(seqs)
        D = max(1, max(len(drafts[q][0]) for q in seqs))
        tree = any(drafts[q][1] is not None for q in seqs)
        a = np.zeros(2 * B + (2 if tree else 1) * B * D, np.int32)
        a[:B] = seqs
        a[B:2 * B] = [len(drafts[q][0]) for q in seqs]
        tok = a[2 * B:2 * B + B * D].reshape(B, D)
        for i, q in enumerate(seqs):
            tok[i, :len(drafts[q][0])] = drafts[q][0]
        par_ptr = None
        if tree:
            par = a[2 * B + B * D:].reshape(B, D)
            par[:] = -1
            for i, q in enumerate(seqs):
                pp = drafts[q][1] if drafts[q][1] is not None else [j - 1 for j in range(len(drafts[q][0]))]
                par[i, :len(pp)] = pp
            par_ptr = a.ctypes.data + 4 * (2 * B + B * D)
        self._a = a
        self.B, self.D = B, D
        self.c = Drafts(B, D, a.ctypes.data, a.ctypes.data + 4 * B, a.ctypes.data + 8 * B, par_ptr)


class Sampling:
    """Sampling-rule arguments of one step: alpha, beta, the drafter's
    distributions ``draft_probs`` (device fp32 [batch, max_drafts, vocab],
    kept referenced here) and the uniforms [batch, max_drafts, 3] (host)."""

    def __init__(self, alpha, beta, draft_probs, uniforms):
        self.probs = draft_probs.to(torch.float32).contiguous()
        self.u = np.ascontiguousarray(uniforms, np.float32)
        self.c = SamplingC(alpha, beta, self.probs.data_ptr(), self.u.ctypes.data)


def tier_params(tau_acc=0.9, tau_full=0.5, temperature=1.0, forced=FORCED_NONE):
    return TierParams(tau_acc, tau_full, temperature, forced)


via_step = _sig("via_step", I32, P, P, C.POINTER(Drafts), C.POINTER(TierParams), C.POINTER(VerifyOut),
                C.POINTER(VerifyOut), C.POINTER(Decision), P)
