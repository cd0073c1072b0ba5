"""The draw entry point that allocates nothing (via_sample_rows_static)
against via_sample_rows, its counterpart with a KV handle's workspace: the
same tokens and probabilities, bit for bit, on two calls in a row (the
second with fewer rows), and EINVAL beyond its row limit."""
import ctypes as C

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2606_12243_amd import via  # noqa: E402
from workload import configs, gen  # noqa: E402


def _out(logits, T):
    """A verify output whose logits and row statistics are given (fp32)."""
    rows, V = logits.shape
    o = via.Out(rows, 1, 1, V, logits=True)
    o.logits.copy_(logits.reshape(-1))
    mx = logits.max(dim=1).values
    o.row_max.copy_(mx)
    o.row_sumexp.copy_(torch.exp((logits - mx[:, None]) / T).sum(dim=1))
    return o


def test_static_draws_match_workspace_draws():
    cfg = configs.get("small_bf16_hd128")
    md = cfg["model"]
    V = md["vocab"]
    gm = via.Model(md, gen.model_weights(cfg), cfg["route"])
    kv = via.KV(gm, max_seqs=1, max_blocks_per_seq=4, blocks_full=4, blocks_slim=4, max_rows=16, max_batch=8,
                max_drafts=4)
    sp = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    try:
        g = torch.Generator(device="cuda").manual_seed(5)
        T = 0.7
        logits = torch.randn(12, V, generator=g, device="cuda") * 3.0
        out = _out(logits, T)
        rng = np.random.default_rng(9)
        for n, rows in ((7, [11, 0, 3, 3, 9, 5, 1]), (3, [2, 10, 4])):
            print(f"[case] static draws n={n} V={V}", flush=True)
            r, rp = via._i32(rows)
            u = rng.random(n).astype(np.float32)
            t_ws = torch.full((n,), -7, dtype=torch.int32, device="cuda")
            t_st = torch.full((n,), -7, dtype=torch.int32, device="cuda")
            p_ws = torch.full((n, V + 3), -1.0, device="cuda")
            p_st = torch.full((n, V + 3), -1.0, device="cuda")
            via.check(via.via_sample_rows(kv.h, C.byref(out.c), 12, n, rp, T, u.ctypes.data, t_ws.data_ptr(),
                                          p_ws.data_ptr(), V + 3, sp))
            via.check(via.via_sample_rows_static(C.byref(out.c), 12, V, n, rp, T, u.ctypes.data, t_st.data_ptr(),
                                                 p_st.data_ptr(), V + 3, sp))
            torch.cuda.synchronize()
            assert torch.equal(t_ws, t_st), (t_ws, t_st)
            assert torch.equal(p_ws, p_st)
            assert ((t_st >= 0) & (t_st < V)).all()
            # each draw is the inverse-CDF crossing of its uniform under the row's probabilities
            for i in range(n):
                q = p_st[i, :V].double().cpu()
                c = torch.cumsum(q, 0)
                tok = int(t_st[i])
                assert c[tok] >= float(u[i]) * float(c[-1]) - 1e-6
                assert tok == 0 or c[tok - 1] <= float(u[i]) * float(c[-1]) + 1e-6
        r, rp = via._i32(list(range(12)) * 6)
        u = np.full(72, 0.5, np.float32)
        tok = torch.empty(72, dtype=torch.int32, device="cuda")
        assert via.via_sample_rows_static(C.byref(out.c), 12, V, 65, rp, T, u.ctypes.data, tok.data_ptr(), None,
                                          V, sp) == via.EINVAL
        assert "65" in via.via_last_error().decode()
        assert via.via_sample_rows_static(C.byref(out.c), 12, V, 64, rp, T, u.ctypes.data, tok.data_ptr(), None,
                                          V, sp) == via.OK
        torch.cuda.synchronize()
    finally:
        kv.close()
        gm.close()
