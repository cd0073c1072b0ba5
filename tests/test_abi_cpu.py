"""The C-ABI library loads and exports every function include/via.h
declares; host-side validation that needs no GPU (no compute calls)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "via.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(via_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def via():
    from paper_2606_12243_amd import via as v
    return v


def test_library_exports_every_declared_symbol(via):
    names = header_functions()
    assert len(names) >= 19
    for n in names:
        assert hasattr(via.lib, n), n
    assert set(names) == set(via.EXPORTS)


def test_version(via):
    assert via.via_version().decode().startswith("via-gfx950")


def _desc(via, **kw):
    m = dict(n_layers=2, d_model=128, n_heads=2, n_kv_heads=1, head_dim=64, d_ffn=256, vocab=100,
             rms_eps=1e-5, rope_theta=1e4, dtype="bf16")
    m.update(kw)
    return via.model_desc(m)


def _weights(via, L=2):
    arr = (C.c_void_p * L)(*([8] * L))
    return via.Weights(8, 8, 8, arr, arr, arr, arr, arr, arr), arr


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), -5), (dict(n_heads=3, n_kv_heads=2), -5), (dict(d_model=100), -5),
    (dict(vocab=0), -1), (dict(dtype="f16"), None)])
def test_model_create_validation(via, kw, status):
    if kw.get("dtype") == "f16":
        d = _desc(via)
        d.dtype = 7
        status = -1
    else:
        d = _desc(via, **kw)
    w, keep = _weights(via)
    h = C.c_void_p()
    assert via.via_model_create(C.byref(d), C.byref(w), C.byref(h)) == status
    assert not h.value
    assert via.via_last_error()


def test_route_validation(via):
    d = _desc(via, n_layers=4)
    w, keep = _weights(via, 4)
    h = C.c_void_p()
    assert via.via_model_create(C.byref(d), C.byref(w), C.byref(h)) == 0
    for bad in ([], [0, 0], [2, 1], [0, 4], [-1]):
        a, p = via._i32(bad if bad else [0])
        assert via.via_model_set_route(h, p, len(bad)) == -1, bad
    a, p = via._i32([0, 3])
    assert via.via_model_set_route(h, p, 2) == 0
    assert via.via_model_destroy(h) == 0


def test_sizes(via):
    d = _desc(via)
    pb = via.via_pool_bytes(C.byref(d), 2, 10, 16)
    assert pb == 2 * 10 * 2 * 1 * 16 * 64 * 2
    ws = via.via_workspace_bytes(C.byref(d), 64, 2, 32, 8, 1)
    assert ws > 0 and ws % 256 == 0
    assert via.via_workspace_bytes(C.byref(d), 0, 2, 32, 8, 1) == 0
    assert via.via_workspace_bytes(C.byref(d), 64, 2, 32, 8, 0) == 0
    # each sequence id adds its ring of post-shared-layer states (VIA_STATE_ROWS fp32 rows of d_model)
    assert via.via_workspace_bytes(C.byref(d), 64, 2, 32, 8, 3) - ws == 2 * 128 * d.d_model * 4
    assert via.via_staging_bytes(C.byref(d), 64, 2, 32, 8) > 0
