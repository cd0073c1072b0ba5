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
