"""Host-side step loop over the C ABI (Alg. 1 of the paper, App. B.1 form).

Per verification step: slim-verifier forward + fused head over the draft
window, tier decision, one small device->host read; if any sequence
escalates, the full-verifier forward (with the lag rows its cache misses)
and a second decision; then the KV commit.  The library keeps cache state
(valid lengths, block tables); this object keeps the committed tokens the
caller owns (pending token, lag rows) and builds windows.
"""
from __future__ import annotations

import ctypes as C

import numpy as np
import torch

from . import via


def tree_layout(tok, parent):
    """Fed rows of a token tree: root + every node with children, node order.

    Returns (row_nodes, draft_row, row_depth, row_mask)."""
    has_child = set(p for p in parent if p >= 0)
    row_nodes = [-1] + [j for j in range(len(tok)) if j in has_child]
    row_of = {u: r for r, u in enumerate(row_nodes)}
    depth = {}
    for j in range(len(tok)):
        depth[j] = 1 if parent[j] < 0 else depth[parent[j]] + 1
    draft_row = [row_of[p] for p in parent]
    row_depth = [0] + [depth[u] for u in row_nodes[1:]]
    masks = []
    for r, u in enumerate(row_nodes):
        m = 1 | (1 << r)
        while u >= 0:
            m |= 1 << row_of[u]
            u = parent[u]
        masks.append(m)
    return row_nodes, draft_row, row_depth, masks


class Session:
    def __init__(self, model: via.Model, kv: via.KV, params: via.TierParams, logits=False):
        self.m, self.kv, self.p = model, kv, params
        self.tokens = {}
        self.want_logits = logits
        # outputs are indexed by window row (lag rows produce none); a window has
        # at most 64 rows per sequence (chain: one per draft; tree: VIA_MAX_TREE_ROWS)
        B, R, D, V = kv.max_batch, min(kv.max_rows, 64), kv.max_drafts, model.desc["vocab"]
        self.out_slim = via.Out(B, R, D, V, logits)
        self.out_full = via.Out(B, R, D, V, logits)
        self.dec = via.Dec(B, D)
        self.stream = torch.cuda.current_stream()

    # ----------------------------------------------------------- sequences
    def sp(self):
        return C.c_void_p(self.stream.cuda_stream)

    def prefill(self, seq, tokens):
        """Cache tokens[0..n-2]; tokens[-1] becomes the pending token."""
        t, tp = via._i32(tokens[:-1])
        via.check(via.via_prefill(self.m.h, self.kv.h, seq, tp, len(tokens) - 1, self.sp()))
        self.tokens[seq] = list(tokens)

    def prefill_batch(self, prompts: dict):
        """prefill() for several sequences in shared forwards ({seq: tokens})."""
        seqs = list(prompts)
        ids, ip = via._i32(seqs)
        lens, lp = via._i32([len(prompts[q]) - 1 for q in seqs])
        flat, fp = via._i32([t for q in seqs for t in prompts[q][:-1]] or [0])
        via.check(via.via_prefill_batch(self.m.h, self.kv.h, len(seqs), ip, lp, fp, self.sp()))
        for q in seqs:
            self.tokens[q] = list(prompts[q])

    def reserve(self, seq, tokens, kv_values=None):
        """Attach with n-1 context slots whose K/V are supplied by the caller.

        kv_values(cache, layer_slot) -> (K, V) tensors [n-1, KVH, hd] in the
        model dtype (host or device); written into the paged pools."""
        n1 = len(tokens) - 1
        via.check(via.via_kv_seq_reserve(self.kv.h, seq, n1))
        self.tokens[seq] = list(tokens)
        if kv_values is not None:
            self.write_context(seq, n1, kv_values)

    def write_context(self, seq, n1, kv_values):
        md = self.m.desc
        KVH, hd = md["n_kv_heads"], md["head_dim"]
        for cache in (via.CACHE_FULL, via.CACHE_SLIM):
            _, table = self.kv.seq_info(seq, cache)
            pv = self.kv.pool_view(cache)
            nb = (n1 + via.BLOCK - 1) // via.BLOCK
            idx = torch.as_tensor(table[:nb], dtype=torch.long, device=pv.device)
            slots = pv.shape[0]
            for s in range(slots):
                K, V = kv_values(cache, s)
                K = torch.as_tensor(K).to(pv.device).view(pv.dtype) if K.dtype != pv.dtype else K.to(pv.device)
                V = torch.as_tensor(V).to(pv.device).view(pv.dtype) if V.dtype != pv.dtype else V.to(pv.device)
                pad = nb * via.BLOCK - n1
                if pad:
                    K = torch.cat([K, torch.zeros((pad, KVH, hd), dtype=K.dtype, device=K.device)])
                    V = torch.cat([V, torch.zeros((pad, KVH, hd), dtype=V.dtype, device=V.device)])
                # K page [hd/8][16 tokens][8], V page [hd][16 tokens]
                Kp = K.view(nb, via.BLOCK, KVH, hd // 8, 8).permute(2, 0, 3, 1, 4).reshape(KVH, nb, via.BLOCK * hd)
                Vp = V.view(nb, via.BLOCK, KVH, hd).permute(2, 0, 3, 1).reshape(KVH, nb, via.BLOCK * hd)
                pv[s, :, :, 0].index_copy_(1, idx, Kp.contiguous())
                pv[s, :, :, 1].index_copy_(1, idx, Vp.contiguous())

    def release(self, seq):
        via.check(via.via_kv_seq_release(self.kv.h, seq))
        self.tokens.pop(seq, None)

    def lag(self, seq):
        vf = self.kv.valid_len(seq, via.CACHE_FULL)
        n = len(self.tokens[seq])
        return self.tokens[seq][vf:n - 1]

    # --------------------------------------------------------------- windows
    def window(self, drafts: dict, with_lag=False):
        """drafts: {seq: (tokens, parents or None)} -> WindowBuf."""
        seqs = list(drafts)
        rows, dtoks, drows, parents, depths, masks, lags = [], [], [], [], [], [], []
        tree = any(drafts[s][1] is not None for s in seqs)
        for s in seqs:
            tok, par = drafts[s]
            pend = self.tokens[s][-1]
            if par is None and not tree:
                rows.append([pend] + list(tok[:-1]))
                dtoks.append(list(tok))
                drows.append(list(range(len(tok))))
            else:
                par = list(par) if par is not None else [j - 1 for j in range(len(tok))]
                rn, dr, rd, mk = tree_layout(tok, par)
                rows.append([pend] + [tok[u] for u in rn[1:]])
                dtoks.append(list(tok))
                drows.append(dr)
                parents.append(par)
                depths.append(rd)
                masks.append(mk)
            if with_lag:
                lags.append(self.lag(s))
        return via.WindowBuf(seqs, rows, dtoks, drows, parents if tree else None, depths if tree else None,
                             masks if tree else None, lags if with_lag else None,
                             max_rows=max(len(r) for r in rows), max_drafts=max(1, max(len(d) for d in dtoks)))

    # ------------------------------------------------------------------ step
    def _decide(self, full, sampling):
        fo = C.byref(self.out_full.c) if full else None
        if sampling is None:
            via.check(via.via_tier_decide(self.kv.h, C.byref(self.p), C.byref(self.out_slim.c), fo,
                                          C.byref(self.dec.c), self.sp()))
        else:
            via.check(via.via_tier_decide_sampled(self.kv.h, C.byref(self.p), C.byref(self.out_slim.c), fo,
                                                  C.byref(sampling.c), C.byref(self.dec.c), self.sp()))

    def begin(self, drafts: dict, sampling: via.Sampling = None):
        """Slim forward, decision, and the full forward where needed.
        Returns (window, host decision, full ran per batch entry).  The slim
        forward ignores lag rows; the window of the full forward (same rows)
        carries them and is built only when some sequence escalates.
        ``sampling`` (chain drafts, a session with logits) selects the
        sampling rules; its arrays follow the window's batch order."""
        if sampling is not None and not self.want_logits:
            raise ValueError("sampling rules need a session created with logits=True")
        w = self.window(drafts)
        self._w = w
        via.check(via.via_verify_slim(self.m.h, self.kv.h, C.byref(w.c), C.byref(self.p),
                                      C.byref(self.out_slim.c), self.sp()))
        self._decide(False, sampling)
        self.stream.synchronize()
        h = self._host(w)
        run = (h["status"] == 1).astype(np.int32)
        if run.any():
            r, rp = via._i32(run)
            wl = self.window(drafts, with_lag=True)
            via.check(via.via_verify_full(self.m.h, self.kv.h, C.byref(wl.c), rp, C.byref(self.p),
                                          C.byref(self.out_full.c), self.sp()))
            self._decide(True, sampling)
            self.stream.synchronize()
            h = self._host(w)
        self._h = h
        return w, h, run

    def _host(self, w):
        B, D = w.B, w.max_drafts
        if getattr(self, "_hp", None) is None:
            self._hp = self.dec.h_packed.numpy()  # view of the pinned read-back block
        a = self._hp[:4 * B + B * D].copy()
        return dict(status=a[:B], kappa=a[B:2 * B], emit=a[2 * B:3 * B], new_len=a[3 * B:4 * B],
                    path=a[4 * B:].reshape(B, D))

    def commit(self, w, drafts: dict, h=None):
        """Commit the open step; ``h`` (host decision) may replace the
        device's (lock-step parity re-sync)."""
        B, D = w.B, w.max_drafts
        if h is not None:
            hp = self.dec.h_packed.numpy()
            hp[:B], hp[B:2 * B], hp[2 * B:3 * B], hp[3 * B:4 * B] = h["status"], h["kappa"], h["emit"], h["new_len"]
            hp[4 * B:4 * B + B * D] = np.asarray(h["path"], np.int32).reshape(-1)
        elif getattr(self, "_w", None) is w and getattr(self, "_h", None) is not None:
            h = self._h  # the decision begin() read back for this window
        else:
            h = self._host(w)
        self._h = None
        via.check(via.via_kv_commit_rollback(self.kv.h, C.byref(self.dec.c), self.sp()))
        status, kappa, emit = (np.asarray(h[k]).tolist() for k in ("status", "kappa", "emit"))
        path = np.asarray(h["path"]).reshape(B, -1).tolist()
        for b, s in enumerate(w.a["seq"].tolist()):
            if status[b] != 0:
                continue
            tok = drafts[s][0]
            new = [tok[j] for j in path[b][:kappa[b]]]
            if emit[b] >= 0:
                new.append(emit[b])
            self.tokens[s].extend(new)
        return h

    def step(self, drafts: dict, sampling: via.Sampling = None):
        w, h, run = self.begin(drafts, sampling)
        self.commit(w, drafts)
        return h, run


class GreedyDrafter:
    """Synthetic drafter on the GPU: the full verifier's greedy token on the
    draft's own prefix (probe forwards, no change to the KV state), with
    positions replaced by the workload's corruption draws."""

    def __init__(self, sess: Session, corrupt_fn):
        self.s = sess
        self.corrupt = corrupt_fn
        kv = sess.kv
        self.out = via.Out(kv.max_batch, kv.max_rows, kv.max_drafts, sess.m.desc["vocab"], logits=False)

    def tree(self, seqs, budget, branch, step):
        """Token tree per sequence: per depth, earlier nodes expand first with
        up to ``branch`` children, the parent's top tokens under q (probe
        forward of the tree so far), each replaced at random."""
        s = self.s
        out = {}
        for q in seqs:
            toks, parents, frontier = [], [], [-1]
            for depth, nb in enumerate(budget, start=1):
                plan, left = [], nb
                for u in frontier:
                    if left <= 0:
                        break
                    plan.append((u, min(branch, left)))
                    left -= plan[-1][1]
                # probe rows: root + every node so far (all fed), ancestors mask
                rn = [-1] + list(range(len(toks)))
                row_of = {u: r for r, u in enumerate(rn)}
                dep = {}
                for j in range(len(toks)):
                    dep[j] = 1 if parents[j] < 0 else dep[parents[j]] + 1
                masks = []
                for r, u in enumerate(rn):
                    mk = 1 | (1 << r)
                    while u >= 0:
                        mk |= 1 << row_of[u]
                        u = parents[u]
                    masks.append(mk)
                rows = [s.tokens[q][-1]] + list(toks)
                w = via.WindowBuf([q], [rows], [[0]], [[0]], parents=[[-1]],
                                  depths=[[0] + [dep[j] for j in range(len(toks))]], masks=[masks],
                                  lags=[s.lag(q)], max_drafts=1)
                outt = via.Out(1, len(rows), 1, s.m.desc["vocab"], logits=True)
                via.check(via.via_verify_probe(s.m.h, s.kv.h, via.CACHE_FULL, C.byref(w.c), C.byref(s.p),
                                               C.byref(outt.c), s.sp()))
                lg = outt.logits.view(len(rows), -1)
                new_frontier = []
                for u, take in plan:
                    top = torch.topk(lg[row_of[u]], take).indices.cpu().tolist()
                    for t in top:
                        j = len(toks)
                        rep, tok = self.corrupt(q, step, j)
                        toks.append(tok if rep else int(t))
                        parents.append(u)
                        new_frontier.append(j)
                frontier = new_frontier
            out[q] = (toks, parents)
        return out

    def chain(self, seqs, k, step):
        s = self.s
        drafts = {q: [] for q in seqs}
        for j in range(k):
            rows = {q: [s.tokens[q][-1]] + drafts[q] for q in seqs}
            lags = [s.lag(q) for q in seqs]
            w = via.WindowBuf(seqs, [rows[q] for q in seqs], [[] for _ in seqs], [[] for _ in seqs],
                              lags=lags, max_drafts=1)
            via.check(via.via_verify_probe(s.m.h, s.kv.h, via.CACHE_FULL, C.byref(w.c), C.byref(s.p),
                                           C.byref(self.out.c), s.sp()))
            am = self.out.row_argmax.cpu().numpy()
            for b, q in enumerate(seqs):
                g = int(am[b * w.max_rows + len(rows[q]) - 1])
                rep, tok = self.corrupt(q, step, j)
                drafts[q].append(tok if rep else g)
        return drafts


class ModelDrafter:
    """Drafter model on the same kernels: its temperature-T softmax is the
    drafting distribution p of the sampling rules (App. A).  The model may
    share the verifier's weights under a shallower route (a nested mask
    inside the slim route) or be a separate small model with the same
    vocabulary.

    It keeps its own cache of the committed prefix (the model's route, slim
    cache of its own handle).  ``draft`` feeds the pending token and the
    drafts so far as probe rows (no change to the cache) and draws each next
    token from p with ``via_sample_rows``; ``sync`` appends the tokens a
    verify step committed (a forced-accept step of the drafter's handle).
    """

    def __init__(self, model: via.Model, kv: via.KV, temperature=1.0):
        self.sess = Session(model, kv, via.tier_params(0.9, 0.5, temperature, via.FORCED_ACCEPT), logits=True)
        self.T = float(temperature)
        self.V = model.desc["vocab"]
        self.tok = torch.empty(kv.max_batch, dtype=torch.int32, device="cuda")

    def attach(self, seq, tokens):
        self.sess.prefill(seq, tokens)

    def release(self, seq):
        self.sess.release(seq)

    def draft(self, seqs, k, uniforms=None):
        """k drafts per sequence: ({seq: tokens}, p) with p the drafting
        distributions as a device fp32 [len(seqs), k, V] tensor (the layout
        ``via.Sampling`` takes).  ``uniforms`` (host [len(seqs), k] in
        [0, 1)) selects the draws; None drafts greedily (lowest id among the
        maxima)."""
        s = self.sess
        B, V = len(seqs), self.V
        P = torch.empty((B, k, V), dtype=torch.float32, device="cuda")
        drafts = {q: [] for q in seqs}
        U = np.zeros((B, k), np.float32) if uniforms is None else np.ascontiguousarray(uniforms, np.float32)
        for j in range(k):
            rows = [[s.tokens[q][-1]] + drafts[q] for q in seqs]
            w = via.WindowBuf(seqs, rows, [[] for _ in seqs], [[] for _ in seqs], max_drafts=1)
            via.check(via.via_verify_probe(s.m.h, s.kv.h, via.CACHE_SLIM, C.byref(w.c), C.byref(s.p),
                                           C.byref(s.out_slim.c), s.sp()))
            R = w.max_rows
            r, rp = via._i32([b * R + len(rows[b]) - 1 for b in range(B)])
            u = np.ascontiguousarray(U[:, j])
            via.check(via.via_sample_rows(s.kv.h, C.byref(s.out_slim.c), B * R, B, rp, self.T, u.ctypes.data,
                                          self.tok.data_ptr(), P[:, j].data_ptr(), k * V, s.sp()))
            got = (s.out_slim.row_argmax[r.tolist()] if uniforms is None else self.tok[:B]).cpu().tolist()
            for b, q in enumerate(seqs):
                drafts[q].append(int(got[b]))
        return drafts, P

    def sync(self, new_tokens: dict):
        """Append the tokens each sequence committed ({seq: [tokens]}; empty
        lists are skipped)."""
        todo = {q: (list(t), None) for q, t in new_tokens.items() if len(t)}
        if todo:
            h, _ = self.sess.step(todo)
            assert (np.asarray(h["status"]) == 0).all()
