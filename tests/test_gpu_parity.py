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
