"""Error contract of the C ABI on the GPU (include/via.h): a call that fails
validation returns its status and leaves model and KV state unchanged; calls
out of order return VIA_ESTATE; a repeated step from the same state is
bitwise reproducible."""
import ctypes as C

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2606_12243_amd import via  # noqa: E402
from paper_2606_12243_amd.session import Session  # noqa: E402
from workload import configs, gen  # noqa: E402


def _setup(blocks=64, max_blocks=16, cfg_name="micro_bf16"):
    cfg = configs.get(cfg_name)
    cfg.update(seed_c=24, seed_d=34)
    md = cfg["model"]
    W = gen.model_weights(cfg)
    m = via.Model(md, W, cfg["route"])
    kv = via.KV(m, max_seqs=2, max_blocks_per_seq=max_blocks, blocks_full=blocks, blocks_slim=blocks,
                max_rows=32, max_batch=2, max_drafts=8)
    s = Session(m, kv, via.tier_params(0.9, 0.5, 1.0), logits=True)
    return cfg, m, kv, s


def _state(kv, seqs):
    return {(b, c): kv.seq_info(b, c) for b in seqs for c in (via.CACHE_FULL, via.CACHE_SLIM)}


def _status(fn, *args):
    return int(fn(*args))


def test_pool_exhaustion_leaves_state_unchanged():
    # 5 blocks per cache: a 49-token prompt takes 3 (48 slots), the window needs a 4th and 5th,
    # the second sequence's prompt takes the remaining ones
    cfg, m, kv, s = _setup(blocks=5, max_blocks=5)
    print("[case] pool exhaustion", flush=True)
    try:
        s.prefill(0, gen.context_tokens(cfg, 0, 49))
        s.prefill(1, gen.context_tokens(cfg, 1, 17))
        before = _state(kv, [0, 1])
        # 8 window rows for seq 0 need 4 blocks in all (48 + 8 slots): only 1 free block remains
        w = s.window({0: (list(range(10, 18)), None), 1: (list(range(20, 28)), None)}, with_lag=True)
        st = _status(via.via_verify_slim, m.h, kv.h, C.byref(w.c), C.byref(s.p), C.byref(s.out_slim.c), s.sp())
        assert st == via.ENOMEM, st
        assert _state(kv, [0, 1]) == before
        # a smaller window that fits still works afterwards (no step left open)
        w2 = s.window({1: (list(range(20, 24)), None)}, with_lag=True)
        via.check(via.via_verify_slim(m.h, kv.h, C.byref(w2.c), C.byref(s.p), C.byref(s.out_slim.c), s.sp()))
        via.check(via.via_tier_decide(kv.h, C.byref(s.p), C.byref(s.out_slim.c), None, C.byref(s.dec.c), s.sp()))
        s.stream.synchronize()
    finally:
        kv.close()
        m.close()


def test_calls_out_of_order():
    cfg, m, kv, s = _setup()
    print("[case] out of order", flush=True)
    try:
        s.prefill(0, gen.context_tokens(cfg, 0, 20))
        w = s.window({0: (list(range(10, 14)), None)}, with_lag=True)
        run, rp = via._i32(np.ones(1, np.int32))
        estate = via.ESTATE
        # full verify and commit need an open step
        assert _status(via.via_verify_full, m.h, kv.h, C.byref(w.c), rp, C.byref(s.p), C.byref(s.out_full.c),
                       s.sp()) == estate
        assert _status(via.via_kv_commit_rollback, kv.h, C.byref(s.dec.c), s.sp()) == estate
        via.check(via.via_verify_slim(m.h, kv.h, C.byref(w.c), C.byref(s.p), C.byref(s.out_slim.c), s.sp()))
        # a second slim pass and a probe while the step is open
        assert _status(via.via_verify_slim, m.h, kv.h, C.byref(w.c), C.byref(s.p), C.byref(s.out_slim.c),
                       s.sp()) == estate
        assert _status(via.via_verify_probe, m.h, kv.h, via.CACHE_FULL, C.byref(w.c), C.byref(s.p),
                       C.byref(s.out_slim.c), s.sp()) == estate
        # forced full tier: committing before the full verifier resolves it is refused
        pf = via.tier_params(0.9, 0.5, 1.0, via.FORCED_FULL)
        via.check(via.via_tier_decide(kv.h, C.byref(pf), C.byref(s.out_slim.c), None, C.byref(s.dec.c), s.sp()))
        s.stream.synchronize()
        before = _state(kv, [0])
        assert _status(via.via_kv_commit_rollback, kv.h, C.byref(s.dec.c), s.sp()) == estate
        assert _state(kv, [0]) == before
        # the intended order completes the step
        via.check(via.via_verify_full(m.h, kv.h, C.byref(w.c), rp, C.byref(pf), C.byref(s.out_full.c), s.sp()))
        via.check(via.via_tier_decide(kv.h, C.byref(pf), C.byref(s.out_slim.c), C.byref(s.out_full.c),
                                      C.byref(s.dec.c), s.sp()))
        s.stream.synchronize()
        via.check(via.via_kv_commit_rollback(kv.h, C.byref(s.dec.c), s.sp()))
        s.stream.synchronize()
        assert _status(via.via_kv_commit_rollback, kv.h, C.byref(s.dec.c), s.sp()) == estate
    finally:
        kv.close()
        m.close()


def test_repeated_step_is_bitwise_reproducible():
    outs = []
    for rep in range(2):
        cfg, m, kv, s = _setup()
        print(f"[case] determinism run {rep}", flush=True)
        try:
            s.prefill(0, gen.context_tokens(cfg, 0, 40))
            s.prefill(1, gen.context_tokens(cfg, 1, 23))
            drafts = {0: (list(range(30, 36)), None), 1: (list(range(40, 46)), None)}
            w, h, run = s.begin(drafts)
            R, V = w.max_rows, m.desc["vocab"]
            lg = s.out_slim.logits[:2 * R * V].clone().cpu()
            lf = s.out_full.logits[:2 * R * V].clone().cpu() if run.any() else None
            s.commit(w, drafts)
            s.stream.synchronize()
            outs.append((lg, lf, {k: np.array(v).copy() for k, v in h.items()}, dict(s.tokens)))
        finally:
            kv.close()
            m.close()
    (a, af, ha, ta), (b, bf, hb, tb) = outs
    assert torch.equal(a, b)
    assert (af is None and bf is None) or torch.equal(af, bf)
    for k in ha:
        assert np.array_equal(ha[k], hb[k]), k
    assert ta == tb
