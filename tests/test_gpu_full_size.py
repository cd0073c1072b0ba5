"""GPU parity at the full sizes of the four bf16 workloads (1B shape; 8B shape
with chain drafts, tree drafts and long-context batched serving).

The GPU runs the whole batch in the launch configuration the benchmark times
(same batch, context lengths, draft shapes, row and block budgets); the
oracle follows a sample of the sequences, whose slim and full logits,
argmaxes, tiers, escalations, decisions, token streams and valid lengths are
compared element by element (tolerances and near-tie exemptions as in the
small lock-step tests).  Contexts are seeded synthetic K/V written straight
into both caches, so a multi-thousand-token prefill is not needed on the CPU.
Drafts come from the GPU greedy drafter; they are step inputs, handed to the
oracle unchanged.
"""
import pytest

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu, pytest.mark.slow]

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

from oracle.decode import Draft, TierParams  # noqa: E402
from oracle.model import OracleModel  # noqa: E402
from paper_2606_12243_amd import via  # noqa: E402
from paper_2606_12243_amd.session import GreedyDrafter as GpuDrafter  # noqa: E402
from workload import calibrated, configs, gen  # noqa: E402

from gpu_harness import Lockstep  # noqa: E402


@pytest.fixture(scope="module")
def models():
    """Weights, oracle model and GPU model, kept while consecutive cases share them."""
    cache = {}

    def get(cfg):
        key = (cfg["seed_w"], tuple(sorted(cfg["model"].items())), tuple(cfg["route"]))
        if key not in cache:
            for _, _, gm in cache.values():
                gm.close()
            cache.clear()
            W = gen.model_weights(cfg)
            cache[key] = (W, OracleModel(cfg["model"], W), via.Model(cfg["model"], W, cfg["route"]))
        return cache[key]

    yield get
    for _, _, gm in cache.values():
        gm.close()


# (workload, verify steps, sampled sequences, temperature).  At the half-accept
# temperatures (1B, 8B chain and tree) drafts split between the accept and
# slim tiers; T = 1 sends every position to the full verifier; at the
# mixed-tier temperature (the long-context batch's own, and "mixed" for the
# 8B chain) all three tiers occur, some steps escalate only part of the batch
# and the full forward of an escalated sequence carries the lag rows its cache
# missed on earlier steps; the tree workload (one sequence) at the chain's
# mixed-tier temperature has all three tiers inside one tree window, so a tree
# commit follows a full forward.  "ends": the shortest- and longest-context
# sequences.
CASES = [
    ("1b_bf16", 8, [0], None),
    ("8b_bf16_chain", 2, [3], None),
    ("8b_bf16_chain", 8, [0, 1, 2, 3], "mixed"),
    ("8b_bf16_chain", 2, [1], 1.0),
    ("8b_bf16_tree", 2, [0], None),
    ("8b_bf16_tree", 4, [0], "chain_mixed"),
    ("8b_bf16_tree", 2, [0], 1.0),
    ("8b_bf16_long", 3, "ends", None),
]


@pytest.mark.parametrize("name,steps,sample,temperature", CASES)
def test_full_size_sampled_parity(name, steps, sample, temperature, models):
    cfg = configs.get(name)
    md = cfg["model"]
    V = md["vocab"]
    if cfg.get("seed_kv") is None:
        cfg["seed_kv"] = 4000 + int(cfg["seed_w"]) % 1000
    ctx = gen.context_lengths(cfg)
    B = cfg["batch"]
    if sample == "ends":
        sample = sorted({min(range(B), key=lambda b: ctx[b]), max(range(B), key=lambda b: ctx[b])})
    if temperature == "mixed":
        temperature = calibrated.MIXED_TEMPERATURE[name]
    elif temperature == "chain_mixed":  # tree drafts where the chain's mix of tiers occurs
        temperature = calibrated.MIXED_TEMPERATURE["8b_bf16_chain"]
    tree = cfg["draft"] == "tree"
    k = cfg.get("k", 8)
    # the benchmark's row and block budgets (its default 35 replayed steps)
    grow = 35 * ((len(cfg["tree_budget"]) + 1) if tree else (k + 1))
    rows_per_seq = (64 if tree else k) + grow
    max_blocks = (max(ctx) + grow + rows_per_seq + 16) // 16 + 1
    T = float(cfg["temperature"] if temperature is None else temperature)
    mixed = T == calibrated.MIXED_TEMPERATURE.get(name)
    print(f"[case] {name} T={T:.4g} B={B} ctx={min(ctx)}..{max(ctx)} sample={sample} steps={steps}", flush=True)
    W, om, gm = models(cfg)
    ls = Lockstep(cfg, weights=W, oracle_model=om, gpu_model=gm, sample=sample, max_rows=B * rows_per_seq,
                  max_batch=B, max_drafts=64, max_blocks=max_blocks, blocks=B * max_blocks,
                  params=TierParams(0.9, 0.5, T))
    try:
        for b in range(B):
            ls.add_synthetic(b, gen.context_tokens(cfg, b, ctx[b] + 1))
        drafter = GpuDrafter(ls.sess, lambda b, step, j: gen.corruption(cfg["seed_d"], b, step, j,
                                                                         cfg["corrupt"], V))
        for step in range(steps):
            if tree:
                d = drafter.tree(list(range(B)), cfg["tree_budget"], cfg["tree_branch"], step)
                drafts = {b: Draft(list(d[b][0]), list(d[b][1])) for b in range(B)}
            else:
                d = drafter.chain(list(range(B)), k, step)
                drafts = {b: Draft.chain(list(d[b])) for b in range(B)}
            ls.step(drafts, step)
            print(f"[step] {name} {step}: max logit err {ls.max_logit_err:.3g} tiers {sorted(ls.seen_tiers)} "
                  f"resyncs {len(ls.log)} run {ls.steps[-1]['run']} lag {ls.steps[-1]['gpu_lag']} "
                  f"full start {ls.steps[-1]['full_start']} kappa {ls.steps[-1]['kappa']}", flush=True)
        if mixed:
            # the three tiers over the batch, a full forward over part of the batch, and
            # full forwards carrying lag rows (for a compared sequence when 2+ are followed
            # over 6+ steps)
            assert ls.gpu_tiers == {"A", "S", "F"}, ls.gpu_tiers
            assert any(0 < sum(st["run"]) < B for st in ls.steps), [st["run"] for st in ls.steps]
            assert any(lg > 0 for st in ls.steps for lg in st["gpu_lag"].values()), \
                [st["gpu_lag"] for st in ls.steps]
            if steps >= 6 and len(sample) >= 2:
                assert any(lg > 0 for st in ls.steps for lg in st["full_lag"].values()), \
                    [st["full_lag"] for st in ls.steps]
            # a full forward with lag rows that started after the layers the slim route shares
            # with the full model (the lag slots' states taken from the state ring)
            n_sh = next(i for i, l in enumerate(list(cfg["route"]) + [-1]) if l != i)
            assert any(st["full_start"] == n_sh and any(lg > 0 for lg in st["gpu_lag"].values())
                       for st in ls.steps), [(st["full_start"], st["gpu_lag"]) for st in ls.steps]
    finally:
        ls.close()
