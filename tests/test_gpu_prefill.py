"""The prefill GEMM: the compute-bound tile kernel that runs every projection
of a forward of more than 512 rows.

* via_gemm_bf16 (one activation term) against a float64 product of the same
  bf16 operands, within the rigorous bound of fp32 accumulation of exact bf16
  products, |err| <= K * 2^-24 * (|X| |W|^T); shapes cover one row, ragged
  M/N tails of the 256 x 256 tiles, K of one stage, and full prefill sizes.
* A prefill-sized forward (prompts of 600 and 514 tokens, so the prefill GEMM
  with its 2-term activations, and the SwiGLU epilogue of its gate/up tiles,
  builds the caches), followed by lock-step decoding against the oracle.
"""
import ctypes as C

import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2606_12243_amd import via  # noqa: E402
from workload import configs, gen  # noqa: E402

from gpu_harness import Lockstep  # noqa: E402


def to_fragments(x):
    """Row-major [M, K] -> the activation-fragment layout of include/via.h
    (rows padded to a multiple of 16 with zeros)."""
    M, K = x.shape
    Mp = (M + 15) // 16 * 16
    xp = torch.zeros(Mp, K, dtype=x.dtype)
    xp[:M] = x
    # element (m, k) -> group ((k/32) * Mp/16 + m/16) * 64 + ((k%32)/8) * 16 + m%16, offset k%8
    return xp.view(Mp // 16, 16, K // 32, 4, 8).permute(2, 0, 3, 1, 4).contiguous()


def gemm_bf16(x, w):
    M, K = x.shape
    N = w.shape[0]
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    xd = to_fragments(x).cuda()
    wd = w.cuda()
    wp = torch.empty(via.via_packed_bytes(N, K, via.DTYPE_BF16) // 2, dtype=torch.bfloat16, device="cuda")
    via.check(via.via_pack_weight(wd.data_ptr(), wp.data_ptr(), N, K, via.DTYPE_BF16, stream))
    c = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    via.check(via.via_gemm_bf16(xd.data_ptr(), wp.data_ptr(), c.data_ptr(), M, N, K, stream))
    torch.cuda.synchronize()
    return c.cpu()


@pytest.mark.parametrize("M,N,K", [(1, 64, 32), (300, 200, 96), (257, 513, 64), (2048, 1024, 4096),
                                   (8192, 512, 1024)])
def test_gemm_bf16_matches_fp64_reference(M, N, K):
    print(f"[case] gemm_bf16 M={M} N={N} K={K}", flush=True)
    g = torch.Generator().manual_seed(M * 7 + N * 3 + K)
    x = torch.randn(M, K, generator=g).to(torch.bfloat16)
    w = torch.randn(N, K, generator=g).to(torch.bfloat16)
    c = gemm_bf16(x, w).double()
    ref = x.double() @ w.double().T
    bound = K * 2.0 ** -24 * (x.double().abs() @ w.double().abs().T) + 1e-30
    assert torch.isfinite(c).all(), "every output element is written"
    ratio = ((c - ref).abs() / bound).max().item()
    print(f"[done] max |err| / bound = {ratio:.3g}", flush=True)
    assert ratio <= 1.0


def test_gemm_bf16_rejects_bad_shapes():
    stream = C.c_void_p(0)
    assert via.via_gemm_bf16(None, None, None, 1, 1, 32, stream) == via.EINVAL
    buf = torch.empty(64, dtype=torch.float32, device="cuda")
    p = buf.data_ptr()
    assert via.via_gemm_bf16(p, p, p, 1, 1, 48, stream) == via.EINVAL   # K not a multiple of 32
    assert via.via_gemm_bf16(p, p, p, 0, 1, 32, stream) == via.EINVAL


@pytest.mark.parametrize("name", ["micro_bf16", "small_bf16_hd128"])
def test_prefill_sized_forward_lockstep(name):
    cfg = configs.get(name)
    cfg.update(seed_c=24, seed_d=34, corrupt=0.3, temperature=1.0)
    print(f"[case] prefill-sized forward {name}", flush=True)
    ls = Lockstep(cfg, max_rows=640, max_batch=2, max_drafts=8, max_blocks=48, blocks=192)
    try:
        ls.add_prompt(0, gen.context_tokens(cfg, 0, 600))  # 599 rows per forward: ragged 256-row tiles
        ls.add_prompt(1, gen.context_tokens(cfg, 1, 514))  # 513 rows: just past the threshold
        steps = ls.run_chain([0, 1], G=16, k=6)
        print(f"[done] {name} steps={steps} max_logit_err={ls.max_logit_err:.3g} tiers={sorted(ls.seen_tiers)} "
              f"resyncs={len(ls.log)}", flush=True)
    finally:
        ls.close()


@pytest.mark.parametrize("name,max_rows", [("small_bf16_hd128", 1300), ("micro_bf16", 700)])
def test_batched_prefill_lockstep(name, max_rows):
    """via_prefill_batch: three prompts share the forwards (all of them in one
    1300-row forward, or with 700 rows per forward the second prompt split
    across two forwards and the third in the second), then lock-step decoding
    against the oracle's per-sequence prefill."""
    cfg = configs.get(name)
    cfg.update(seed_c=27, seed_d=37, corrupt=0.3, temperature=1.0)
    print(f"[case] batched prefill {name} max_rows={max_rows}", flush=True)
    ls = Lockstep(cfg, max_rows=max_rows, max_batch=3, max_drafts=8, max_blocks=64, blocks=256)
    try:
        prompts = {b: gen.context_tokens(cfg, b, n) for b, n in ((0, 520), (1, 611), (2, 170))}
        for b, toks in prompts.items():
            ls.o_id[b] = ls.ver.prefill(toks)
            ls.drafter.attach(b)
        ls.sess.prefill_batch(prompts)
        for b, toks in prompts.items():
            for c in (via.CACHE_FULL, via.CACHE_SLIM):
                assert ls.kv.seq_info(b, c)[0] == len(toks) - 1
        steps = ls.run_chain([0, 1, 2], G=10, k=5)
        print(f"[done] batched {name} steps={steps} max_logit_err={ls.max_logit_err:.3g} "
              f"tiers={sorted(ls.seen_tiers)} resyncs={len(ls.log)}", flush=True)
    finally:
        ls.close()


def test_batched_prefill_is_all_or_nothing():
    cfg = configs.get("micro_bf16")
    md = cfg["model"]
    gm = via.Model(md, gen.model_weights(cfg), cfg["route"])
    kv = via.KV(gm, max_seqs=3, max_blocks_per_seq=8, blocks_full=10, blocks_slim=10, max_rows=64, max_batch=3,
                max_drafts=4)
    try:
        stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
        toks, tp = via._i32(list(range(1, 200)))
        ids, ip = via._i32([0, 1])
        lens, lp = via._i32([100, 99])   # 7 + 7 blocks > 10 free
        assert via.via_prefill_batch(gm.h, kv.h, 2, ip, lp, tp, stream) == via.ENOMEM
        ids2, ip2 = via._i32([0, 0])
        lens2, lp2 = via._i32([5, 5])
        assert via.via_prefill_batch(gm.h, kv.h, 2, ip2, lp2, tp, stream) == via.EINVAL   # repeated id
        n, nb = C.c_int32(), C.c_int32()
        for q in (0, 1):
            assert via.via_kv_seq_info(kv.h, q, 0, C.byref(n), None, 0, C.byref(nb)) == via.EINVAL  # not attached
        lens3, lp3 = via._i32([40, 30])
        via.check(via.via_prefill_batch(gm.h, kv.h, 2, ip, lp3, tp, stream))
        torch.cuda.synchronize()
        assert kv.seq_info(0, 0)[0] == 40 and kv.seq_info(1, 1)[0] == 30
    finally:
        kv.close()
        gm.close()


def test_kv_create_rejects_misaligned_buffers():
    """The kernels read the workspace and the pools with 16-byte loads: a
    workspace off its 256-byte alignment or a pool off 16 bytes is refused
    before anything is allocated."""
    cfg = configs.get("micro_bf16")
    gm = via.Model(cfg["model"], gen.model_weights(cfg), cfg["route"])
    kv = via.KV(gm, max_seqs=2, max_blocks_per_seq=4, blocks_full=8, blocks_slim=8, max_rows=16, max_batch=2,
                max_drafts=4)
    try:
        for field, off in (("workspace", 64), ("pool_full", 8), ("pool_slim", 2)):
            d = via.KvDesc.from_buffer_copy(kv.cd)
            setattr(d, field, getattr(kv.cd, field) + off)
            h = C.c_void_p()
            assert via.via_kv_create(gm.h, C.byref(d), C.byref(h)) == via.EINVAL, field
            assert not h.value
    finally:
        kv.close()
        gm.close()
