"""GPU parity of the verification step against the oracle (through the C ABI).

Small shapes span several GEMM tiles, ragged vocab tails (500, 1000, 3001),
GQA groups 2 and 4, head dims 64 and 128, fp32 and bf16; the tiny fp32
workload decodes 64 tokens end to end.
"""
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

from oracle.decode import FORCED_FULL, TierParams  # noqa: E402
from workload import configs, gen  # noqa: E402

from gpu_harness import Lockstep  # noqa: E402


@pytest.mark.parametrize("name", ["micro_f32", "micro_bf16", "small_bf16_hd128"])
def test_small_decode_lockstep(name):
    cfg = configs.get(name)
    cfg.update(seed_c=21, seed_d=31, corrupt=0.3, temperature=1.0)
    print(f"[case] {name}", flush=True)
    ls = Lockstep(cfg, max_rows=96, max_batch=2, max_drafts=8, max_blocks=16, blocks=64)
    try:
        ls.add_prompt(0, gen.context_tokens(cfg, 0, 37))
        ls.add_prompt(1, gen.context_tokens(cfg, 1, 18))
        steps = ls.run_chain([0, 1], G=20, k=5)
        print(f"[done] {name} steps={steps} max_logit_err={ls.max_logit_err:.3g} tiers={sorted(ls.seen_tiers)} "
              f"resyncs={len(ls.log)}", flush=True)
    finally:
        ls.close()


@pytest.mark.parametrize("name", ["micro_f32", "micro_bf16"])
def test_degenerate_windows_lockstep(name):
    """Edge cases of the window, in lock-step with the oracle: a sequence whose
    prompt is one token (nothing cached: its first window attends only to
    itself), one-row windows (k = 1), window lengths that differ across the
    batch within a step (1, 3, 8), and a 32-draft window."""
    cfg = configs.get(name)
    cfg.update(seed_c=23, seed_d=37, corrupt=0.3, temperature=1.0)
    print(f"[case] {name} degenerate windows", flush=True)
    ls = Lockstep(cfg, max_rows=192, max_batch=3, max_drafts=32, max_blocks=16, blocks=96)
    try:
        ls.add_prompt(0, gen.context_tokens(cfg, 0, 1))
        ls.add_prompt(1, gen.context_tokens(cfg, 1, 9))
        ls.add_prompt(2, gen.context_tokens(cfg, 2, 30))
        ks = [(1, 3, 8), (8, 1, 3), (3, 8, 1), (1, 1, 1), (32, 2, 5), (2, 32, 1)]
        for step in range(len(ks)):
            drafts = {b: ls.drafter.chain(b, ls.ver.seqs[b].tokens, ks[step][b], step) for b in (0, 1, 2)}
            ls.step(drafts, step)
        print(f"[done] {name} max_logit_err={ls.max_logit_err:.3g} tiers={sorted(ls.seen_tiers)} "
              f"resyncs={len(ls.log)}", flush=True)
    finally:
        ls.close()


def test_largest_windows_lockstep():
    """Windows at the 64-draft limit, in lock-step with the oracle: a tree of
    64 drafts (two children of the root, then one child per node) that feeds
    63 rows through the tree-mask path, next to a 64-draft chain window in the
    same batch."""
    cfg = configs.get("micro_bf16")
    cfg.update(seed_c=29, seed_d=41, corrupt=0.3, temperature=1.0)
    print("[case] micro_bf16 largest windows", flush=True)
    ls = Lockstep(cfg, max_rows=320, max_batch=2, max_drafts=64, max_blocks=32, blocks=128)
    try:
        ls.add_prompt(0, gen.context_tokens(cfg, 0, 20))
        ls.add_prompt(1, gen.context_tokens(cfg, 1, 11))
        for step in range(4):
            t0, t1 = ls.ver.seqs[0].tokens, ls.ver.seqs[1].tokens
            tree = ls.drafter.tree(0, t0, [2] + [1] * 62, 2, step)
            assert len(tree.tok) == 64 and not Lockstep._is_chain(tree)
            ls.step({0: tree, 1: ls.drafter.chain(1, t1, 64, step)}, step)
        print(f"[done] largest windows max_logit_err={ls.max_logit_err:.3g} tiers={sorted(ls.seen_tiers)} "
              f"resyncs={len(ls.log)}", flush=True)
    finally:
        ls.close()


def test_tiny_fp32_workload_end_to_end():
    cfg = configs.get("tiny_fp32")
    print("[case] tiny_fp32 G=64", flush=True)
    ls = Lockstep(cfg, max_rows=64, max_batch=1, max_drafts=8, max_blocks=16, blocks=32)
    try:
        ls.add_prompt(0, gen.context_tokens(cfg, 0, cfg["ctx"][0]))
        steps = ls.run_chain([0], G=cfg["gen"], k=cfg["k"])
        assert ls.seen_tiers == {"A", "S", "F"}
        print(f"[done] tiny_fp32 steps={steps} max_logit_err={ls.max_logit_err:.3g} resyncs={len(ls.log)}",
              flush=True)
    finally:
        ls.close()


@pytest.mark.parametrize("name", ["micro_f32", "micro_bf16", "small_bf16_hd128"])
def test_lag_rows_start_after_shared_layers(name):
    """Full forwards of sequences whose full caches lag: the states of the lag
    slots after the layers the slim route shares with the full model are kept
    in the state ring, so the forward starts after those layers and still
    matches the oracle's all-layer forward, block tables included.  A lag
    that exactly fills the ring with the window still starts there; one more
    step of lag overflows it, and the forward runs every layer again."""
    from oracle.decode import FORCED_ACCEPT, FORCED_NONE

    cfg = configs.get(name)
    cfg.update(seed_c=26, seed_d=36, corrupt=0.3)
    route = list(cfg["route"])
    n_sh = next(i for i, l in enumerate(route + [-1]) if l != i)
    assert 0 < n_sh < len(route)
    k = 4
    print(f"[case] lag rows via the state ring {name}", flush=True)
    ls = Lockstep(cfg, max_rows=2 * (128 + k), max_batch=2, max_drafts=8, max_blocks=32, blocks=128)
    accept, full = TierParams(0.9, 0.5, 1.0, FORCED_ACCEPT), TierParams(0.9, 0.5, 1.0, FORCED_FULL)
    step = 0

    def run(params, n):
        nonlocal step
        ls.set_params(params)
        for _ in range(n):
            drafts = {b: ls.drafter.chain(b, ls.ver.seqs[b].tokens, k, step) for b in (0, 1)}
            ls.step(drafts, step)
            step += 1
        return ls.steps[-1]

    try:
        ls.add_prompt(0, gen.context_tokens(cfg, 0, 30))
        ls.add_prompt(1, gen.context_tokens(cfg, 1, 19))
        # (accepted steps before the escalation, lag rows it carries, expected start)
        for n_acc, lag, start in ((2, 2 * k, n_sh), (31, 31 * k, n_sh), (32, 32 * k, 0)):
            run(accept, n_acc)
            st = run(full, 1)
            assert st["run"] == [1, 1] and st["gpu_lag"] == {0: lag, 1: lag}, st
            assert st["full_start"] == start, (n_acc, st)
            print(f"[step] {step}: lag {lag} full forward from route index {st['full_start']}", flush=True)
        # natural tiers afterwards (the caches caught up)
        run(TierParams(0.9, 0.5, 1.0, FORCED_NONE), 4)
        print(f"[done] {name} steps={step} max_logit_err={ls.max_logit_err:.3g} resyncs={len(ls.log)}",
              flush=True)
    finally:
        ls.close()


def test_forced_full_matches_greedy_on_gpu():
    cfg = configs.get("micro_bf16")
    cfg.update(seed_c=22, seed_d=32, corrupt=0.3, temperature=1.0)
    ls = Lockstep(cfg, max_rows=64, max_batch=1, max_drafts=8, max_blocks=16, blocks=32,
                  params=TierParams(0.9, 0.5, 1.0, FORCED_FULL))
    try:
        ls.add_prompt(0, gen.context_tokens(cfg, 0, 25))
        ls.run_chain([0], G=16, k=4)
    finally:
        ls.close()


@pytest.mark.parametrize("name", ["micro_f32", "small_bf16_hd128"])
def test_synthetic_context_lockstep(name):
    """Context K/V written straight into the paged pools (the layout of
    include/via.h) instead of a prefill; ragged lengths across pages."""
    cfg = configs.get(name)
    cfg.update(seed_c=23, seed_d=33, seed_kv=43, corrupt=0.3, temperature=1.0)
    print(f"[case] synthetic {name}", flush=True)
    ls = Lockstep(cfg, max_rows=96, max_batch=2, max_drafts=8, max_blocks=32, blocks=96)
    try:
        ls.add_synthetic(0, gen.context_tokens(cfg, 0, 301))
        ls.add_synthetic(1, gen.context_tokens(cfg, 1, 47))
        steps = ls.run_chain([0, 1], G=16, k=6)
        print(f"[done] synthetic {name} steps={steps} max_logit_err={ls.max_logit_err:.3g} "
              f"tiers={sorted(ls.seen_tiers)} resyncs={len(ls.log)}", flush=True)
    finally:
        ls.close()


def test_nonfinite_full_logits_status2_no_commit():
    """Non-finite logits of the full verifier (the reading for a case the
    paper leaves open): the escalated sequence gets status 2, its tokens, valid
    lengths and block tables stay as before the step, and later steps go on
    normally.  Layer 1's down projection is +inf, a layer the slim route
    [0, 2] bypasses, so only the full forward turns non-finite."""
    import ctypes as C

    import numpy as np
    from oracle.decode import FORCED_ACCEPT, Draft, Verifier
    from oracle.model import OracleModel
    from paper_2606_12243_amd import via
    from paper_2606_12243_amd.session import Session

    cfg = configs.get("micro_bf16")
    cfg.update(seed_c=25, seed_d=35)
    md = cfg["model"]
    W = gen.model_weights(cfg)
    W["w_down"][1] = np.full_like(W["w_down"][1], 0x7F80)  # bf16 +inf
    print("[case] non-finite full logits", flush=True)
    om = OracleModel(md, W)
    ver = Verifier(om, cfg["route"])
    gm = via.Model(md, W, cfg["route"])
    kv = via.KV(gm, max_seqs=2, max_blocks_per_seq=16, blocks_full=64, blocks_slim=64, max_rows=64, max_batch=2,
                max_drafts=8)
    try:
        prompts = [gen.context_tokens(cfg, b, n) for b, n in ((0, 30), (1, 17))]
        s = Session(gm, kv, via.tier_params(0.9, 0.5, 1.0, via.FORCED_FULL), logits=True)
        for b, pr in enumerate(prompts):
            assert ver.prefill(pr) == b
            s.prefill(b, pr)
        drafts = {0: [5, 6, 7, 8], 1: [9, 10, 11, 12]}

        def state():
            return {(b, c): kv.seq_info(b, c) for b in (0, 1) for c in (via.CACHE_FULL, via.CACHE_SLIM)}

        before, toks = state(), {b: list(s.tokens[b]) for b in (0, 1)}
        dec = ver.step({b: Draft.chain(d) for b, d in drafts.items()}, TierParams(0.9, 0.5, 1.0, FORCED_FULL))
        w, h, run = s.begin({b: (d, None) for b, d in drafts.items()})
        assert run.tolist() == [1, 1]
        for i, b in enumerate((0, 1)):
            assert dec[b]["status"] == 2
            got = (int(h["status"][i]), int(h["kappa"][i]), int(h["emit"][i]), int(h["new_len"][i]))
            assert got == (2, 0, -1, len(toks[b])), got
            assert not torch.isfinite(s.out_full.row_max[i * w.max_rows]).item()
            assert torch.isfinite(s.out_slim.logits[:w.B * w.max_rows * md["vocab"]]).all().item()
        s.commit(w, {b: (d, None) for b, d in drafts.items()})
        assert state() == before and {b: s.tokens[b] for b in (0, 1)} == toks
        for b in (0, 1):
            for c, which in ((via.CACHE_FULL, "full"), (via.CACHE_SLIM, "slim")):
                assert kv.seq_info(b, c)[1] == ver.block_table(which, b)
        # the sequences go on: a forced-accept step commits every draft (the full cache lags)
        s.p = via.tier_params(0.9, 0.5, 1.0, via.FORCED_ACCEPT)
        dec = ver.step({b: Draft.chain(d) for b, d in drafts.items()}, TierParams(0.9, 0.5, 1.0, FORCED_ACCEPT))
        h, run = s.step({b: (d, None) for b, d in drafts.items()})
        assert not run.any() and h["status"].tolist() == [0, 0]
        for b in (0, 1):
            assert s.tokens[b] == ver.seqs[b].tokens == toks[b] + drafts[b]
            for c, which, oc in ((via.CACHE_FULL, "full", ver.seqs[b].full), (via.CACHE_SLIM, "slim", ver.seqs[b].slim)):
                valid, table = kv.seq_info(b, c)
                assert valid == oc.valid and table == ver.block_table(which, b)
    finally:
        kv.close()
        gm.close()


@pytest.mark.parametrize("tree", [False, True])
def test_native_step_matches_python_driven_step(tree):
    """via_step (window assembly from the library's committed tokens, slim
    forward, decision, escalation with lag rows, commit: one native call)
    against the same step driven call by call from Python, on two handles of
    one model: identical decisions, committed tokens, valid lengths and block
    tables every step (natural tiers at T = 1, so escalations and lag rows
    occur)."""
    import ctypes as C

    import numpy as np
    from paper_2606_12243_amd import via
    from paper_2606_12243_amd.session import GreedyDrafter, Session

    cfg = configs.get("micro_bf16")
    cfg.update(seed_c=26, seed_d=36)
    md = cfg["model"]
    print(f"[case] native step tree={tree}", flush=True)
    gm = via.Model(md, gen.model_weights(cfg), cfg["route"])
    kvs = [via.KV(gm, max_seqs=2, max_blocks_per_seq=16, blocks_full=64, blocks_slim=64, max_rows=128, max_batch=2,
                  max_drafts=16) for _ in range(2)]
    try:
        py, nat = (Session(gm, kv, via.tier_params(0.9, 0.5, 1.0), logits=False) for kv in kvs)
        for b, n in ((0, 27), (1, 12)):
            toks = gen.context_tokens(cfg, b, n)
            py.prefill(b, toks)
            nat.prefill(b, toks)
            t, tp = via._i32(toks)
            via.check(via.via_kv_seq_set_tokens(kvs[1].h, b, tp, len(toks)))
        drafter = GreedyDrafter(py, lambda b, step, j: gen.corruption(cfg["seed_d"], b, step, j, 0.3,
                                                                       md["vocab"]))
        escalated = False
        for step in range(10):
            if tree:
                drafts = drafter.tree([0, 1], [3, 4, 3], 2, step)
            else:
                d = drafter.chain([0, 1], 4, step)
                drafts = {b: (d[b], None) for b in (0, 1)}
            h, run = py.step(drafts)
            escalated |= bool(run.any())
            db = via.DraftsBuf(drafts)
            via.check(via.via_step(gm.h, kvs[1].h, C.byref(db.c), C.byref(nat.p), C.byref(nat.out_slim.c),
                                   C.byref(nat.out_full.c), C.byref(nat.dec.c), nat.sp()))
            B, D = db.B, db.D
            hp = nat.dec.h_packed.numpy()
            for k, i in (("status", 0), ("kappa", 1), ("emit", 2), ("new_len", 3)):
                assert hp[i * B:(i + 1) * B].tolist() == h[k].tolist(), (step, k)
            assert hp[4 * B:4 * B + B * D].tolist() == np.asarray(h["path"]).reshape(-1)[:B * D].tolist()
            for b in (0, 1):
                n = C.c_int32()
                out = np.zeros(512, np.int32)
                via.check(via.via_kv_seq_tokens(kvs[1].h, b, out.ctypes.data_as(via.PI32), 512, C.byref(n)))
                assert out[:n.value].tolist() == py.tokens[b], (step, b)
                for c in (via.CACHE_FULL, via.CACHE_SLIM):
                    assert kvs[0].seq_info(b, c) == kvs[1].seq_info(b, c), (step, b, c)
        assert escalated
    finally:
        for kv in kvs:
            kv.close()
        gm.close()
