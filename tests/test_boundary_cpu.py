"""The C-ABI library loads, exports every symbol include/cat.h declares, and
rejects invalid arguments with the documented status before touching the
GPU.  No compute call runs here (no GPU in this environment)."""
import ctypes
import os
import re

import pytest

import paper_2603_04359_amd as cat
from paper_2603_04359_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cat.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(cat_[a-z0-9_]+)\s*\(", src)))


def test_header_declarations_match_binding_list():
    assert _declared() == sorted(B.EXPORTED)


def test_library_exports_every_declared_symbol():
    L = cat.lib()
    for name in _declared():
        assert hasattr(L, name), name
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value


def test_version_and_error_strings():
    assert cat.cat_version().startswith("cat-mi355x")
    assert isinstance(cat.cat_last_error(), str)


# Fake, 16-byte aligned addresses: every call below fails validation before
# any pointer is dereferenced or any HIP call is made.
P = 1 << 20


def test_cov_invalid_args():
    L = cat.lib()
    assert L.cat_cov_accumulate(None, 1, 10, 64, 0, 1, P, P, 1 << 30, None) == B.CAT_ERR_INVALID_ARG
    assert "NULL" in cat.cat_last_error()
    assert L.cat_cov_accumulate(P, 7, 10, 64, 0, 1, P, P, 1 << 30, None) == B.CAT_ERR_INVALID_ARG
    assert L.cat_cov_accumulate(P, 1, 0, 64, 0, 1, P, P, 1 << 30, None) == B.CAT_ERR_INVALID_ARG
    assert L.cat_cov_accumulate(P, 1, 10, 64, 5, 1, P, P, 1 << 30, None) == B.CAT_ERR_INVALID_ARG
    assert L.cat_cov_accumulate(P, 1, 10, 64, 1, 24, P, P, 1 << 30, None) == B.CAT_ERR_INVALID_ARG
    assert L.cat_cov_accumulate(P, 1, 10, 64, 1, 1024, P, P, 1 << 30, None) == B.CAT_ERR_INVALID_ARG
    assert L.cat_cov_accumulate(P, 1, 10, 96, 1, 64, P, P, 1 << 30, None) == B.CAT_ERR_INVALID_ARG
    assert L.cat_cov_accumulate(P + 2, 1, 10, 64, 0, 1, P, P, 1 << 30, None) == B.CAT_ERR_INVALID_ARG
    assert "aligned" in cat.cat_last_error()


def test_transform_quant_invalid_args():
    L = cat.lib()
    ws = L.cat_transform_quant_workspace_bytes(8, 64, 16)
    ok = dict(X=P, xd=1, n=8, d=64, T=P, td=1, k=16, bits=4, codes=P, s=P, ws=P, wsb=ws)

    def call(**kw):
        a = dict(ok, **kw)
        return L.cat_transform_quant(a["X"], a["xd"], a["n"], a["d"], a["T"], a["td"], a["k"],
                                     a["bits"], a["codes"], a["s"], a["ws"], a["wsb"], None)
    assert call(X=None) == B.CAT_ERR_INVALID_ARG
    assert call(td=3) == B.CAT_ERR_INVALID_ARG
    assert call(n=0) == B.CAT_ERR_INVALID_ARG
    assert call(d=63) == B.CAT_ERR_INVALID_ARG
    assert call(k=12) == B.CAT_ERR_INVALID_ARG
    assert call(d=80, k=32) == B.CAT_ERR_INVALID_ARG
    assert call(bits=5) == B.CAT_ERR_UNSUPPORTED
    assert call(bits=3) == B.CAT_ERR_UNSUPPORTED
    assert call(ws=None) == B.CAT_ERR_WORKSPACE
    assert call(wsb=ws - 1) == B.CAT_ERR_WORKSPACE
    assert call(codes=P + 8) == B.CAT_ERR_INVALID_ARG


def test_transform_quant_status_invalid_args():
    # argument errors come back before the device is touched
    L = cat.lib()
    assert L.cat_transform_quant_status(None, 8, 64, 16, None) == B.CAT_ERR_INVALID_ARG
    assert L.cat_transform_quant_status(P, 0, 64, 16, None) == B.CAT_ERR_INVALID_ARG
    assert L.cat_transform_quant_status(P, 8, 0, 16, None) == B.CAT_ERR_INVALID_ARG
    assert L.cat_transform_quant_noalloc_status(0, 64, 16, None) == B.CAT_ERR_INVALID_ARG
    big = 1 << 20   # 2^20 tokens x 4096 channels: far beyond the scratch array
    assert L.cat_transform_quant_workspace_bytes(big, 4096, 128) > L.cat_transform_quant_noalloc_max_bytes()
    assert L.cat_transform_quant_noalloc_status(big, 4096, 128, None) == B.CAT_ERR_UNSUPPORTED
    assert "scratch" in cat.cat_last_error()


@pytest.mark.parametrize("fn", ["cat_w4a4_linear", "cat_int8_linear"])
def test_linear_invalid_args(fn):
    L = cat.lib()
    f = getattr(L, fn)
    assert f(None, P, P, P, 4, 64, 8, P, None, None) == B.CAT_ERR_INVALID_ARG
    assert f(P, P, P, P, 0, 64, 8, P, None, None) == B.CAT_ERR_INVALID_ARG
    assert f(P, P, P, P, 4, 48, 8, P, None, None) == B.CAT_ERR_INVALID_ARG
    assert f(P, P, P, P, 4, 2 * B.CAT_MAX_D_IN, 8, P, None, None) == B.CAT_ERR_UNSUPPORTED
    assert f(P, P, P, P, 4, 64, 8, P, P + 4, None) == B.CAT_ERR_INVALID_ARG


def test_sqnr_invalid_args():
    L = cat.lib()
    ws = L.cat_sqnr_workspace_bytes(1000)
    assert ws >= 16
    assert L.cat_sqnr(None, P, 1000, P, ws, P, None) == B.CAT_ERR_INVALID_ARG
    assert L.cat_sqnr(P, P, 0, P, ws, P, None) == B.CAT_ERR_INVALID_ARG
    assert L.cat_sqnr(P, P, 1000, P, 8, P, None) == B.CAT_ERR_WORKSPACE
    assert L.cat_sqnr(P, P, 1000, None, ws, P, None) == B.CAT_ERR_WORKSPACE


def test_workspace_sizes_grow_and_are_bounded():
    assert cat.cat_sqnr_workspace_bytes(1) == 16
    assert cat.cat_sqnr_workspace_bytes(10 ** 10) == 512 * 16
    assert cat.cat_transform_quant_workspace_bytes(1, 64, 16) >= 4
    assert cat.cat_transform_quant_workspace_bytes(8192, 4096, 128) >= 8192 * 4
    assert cat.cat_transform_quant_workspace_bytes(0, 64, 16) == 0


def test_host_calls_invalid_args():
    L = cat.lib()
    assert L.cat_build_transform(None, None, 8, 64, 16, 0, 1, None, None, None, 1) == \
        B.CAT_ERR_INVALID_ARG
    assert L.cat_build_transform(None, None, 8, 64, 16, 2, 1, P, None, None, 1) == \
        B.CAT_ERR_INVALID_ARG
    assert L.cat_build_transform(None, None, 8, 64, 12, 0, 1, P, None, None, 1) == \
        B.CAT_ERR_INVALID_ARG
    assert L.cat_build_transform(None, None, 8, 64, 16, 8, 1, P, None, None, 1) == \
        B.CAT_ERR_INVALID_ARG
    assert L.cat_quantize_weights(None, 4, 8, 4, P, P) == B.CAT_ERR_INVALID_ARG
    assert L.cat_quantize_weights(P, 4, 7, 4, P, P) == B.CAT_ERR_INVALID_ARG
    assert L.cat_quantize_weights(P, 4, 8, 5, P, P) == B.CAT_ERR_UNSUPPORTED


def test_binding_rejects_cpu_tensors():
    torch = pytest.importorskip("torch")
    x = torch.zeros(4, 64, dtype=torch.bfloat16)
    acc = torch.zeros(64, 64)
    with pytest.raises(ValueError):
        cat.cat_cov_accumulate(x, acc)


def test_asymmetric_entry_points_invalid_args():
    L = cat.lib()
    ws = L.cat_transform_quant_asym_workspace_bytes(8, 64, 16)
    f = L.cat_transform_quant_asym
    assert f(P, 1, 8, 64, P, 1, 16, P, P, None, P, ws, None) == B.CAT_ERR_INVALID_ARG
    assert f(P, 1, 8, 64, P, 1, 12, P, P, P, P, ws, None) == B.CAT_ERR_INVALID_ARG
    assert f(P, 1, 8, 64, P, 1, 16, P, P, P + 4, P, ws, None) == B.CAT_ERR_INVALID_ARG
    assert f(P, 1, 8, 64, P, 1, 16, P, P, P, P, ws - 1, None) == B.CAT_ERR_WORKSPACE
    g = L.cat_w4a4_linear_asym
    assert g(P, P, None, P, P, P, 4, 64, 8, P, None, None) == B.CAT_ERR_INVALID_ARG
    assert g(P, P, P, P, P, None, 4, 64, 8, P, None, None) == B.CAT_ERR_INVALID_ARG
    assert g(P, P, P, P, P, P + 4, 4, 64, 8, P, None, None) == B.CAT_ERR_INVALID_ARG
    assert g(P, P, P, P, P, P, 4, 48, 8, P, None, None) == B.CAT_ERR_INVALID_ARG
    assert L.cat_weight_code_sums(None, 4, 8, P) == B.CAT_ERR_INVALID_ARG
    assert L.cat_weight_code_sums(P, 4, 7, P) == B.CAT_ERR_INVALID_ARG


def test_sqnr_terms_invalid_args():
    L = cat.lib()
    f = L.cat_sqnr_terms
    assert f(None, 4, 4, P, 64, 16, P, 1, P, 8, 4, 1.0, P) == B.CAT_ERR_INVALID_ARG
    assert f(P, 4, 4, P, 64, 12, P, 1, P, 8, 4, 1.0, P) == B.CAT_ERR_INVALID_ARG
    assert f(P, 4, 9, P, 64, 16, P, 1, P, 8, 4, 1.0, P) == B.CAT_ERR_INVALID_ARG
    assert f(P, 4, 4, P, 64, 16, P, 7, P, 8, 4, 1.0, P) == B.CAT_ERR_INVALID_ARG


def test_full_hadamard_invalid_args():
    L = cat.lib()
    ws = L.cat_transform_quant_full_workspace_bytes(8, 1024, 128)
    assert ws == 8 * 1024 * 4
    f = L.cat_transform_quant_full
    assert f(None, 1, 8, 1024, P, 1, 128, P, P, P, ws, None) == B.CAT_ERR_INVALID_ARG
    assert f(P, 0, 8, 1024, P, 1, 128, P, P, P, ws, None) == B.CAT_ERR_UNSUPPORTED      # fp32 X
    assert f(P, 1, 8, 1024, P, 1, 64, P, P, P, ws, None) == B.CAT_ERR_UNSUPPORTED       # k = 64
    assert f(P, 1, 8, 384, P, 1, 128, P, P, P, ws, None) == B.CAT_ERR_UNSUPPORTED       # m = 3
    assert f(P, 1, 8, 1024, P, 1, 128, P, P, P, ws - 1, None) == B.CAT_ERR_WORKSPACE
    g = L.cat_full_hadamard_weights
    assert g(None, 4, 64, 8, P) == B.CAT_ERR_INVALID_ARG
    assert g(P, 4, 24, 8, P) == B.CAT_ERR_UNSUPPORTED                                   # m = 3


# ----------------------------------------------------------------------
# Buffer-size checks in the binding.  The C ABI receives bare pointers and
# cannot see how long a buffer is, so the binding compares every tensor's
# shape with the sizes the call implies and raises ValueError before the
# library is entered.  Here CPU tensors stand in for device tensors: the
# pointer helper is replaced by one that accepts them, and the library by
# a recorder, so a call that passes the checks is seen to reach the ABI and
# a call that fails them is seen not to.
class _Recorder:
    def __init__(self):
        self.calls = []

    def __getattr__(self, name):
        def call(*args):
            self.calls.append(name)
            return 0
        return call


@pytest.fixture
def fake_abi(monkeypatch):
    import torch
    rec = _Recorder()

    def ptr(t, name, dtypes=None, allow_none=False):
        if t is None:
            if allow_none:
                return None
            raise ValueError(f"{name} is required")
        if dtypes is not None and t.dtype not in dtypes:
            raise TypeError(name)
        return 16

    monkeypatch.setattr(B, "_dev_ptr", ptr)
    monkeypatch.setattr(B, "lib", lambda: rec)
    monkeypatch.setattr(B, "_stream_ptr", lambda s: None)
    return torch, rec


def test_binding_checks_gemm_buffer_sizes(fake_abi):
    torch, rec = fake_abi
    n, d_in, d_out = 8, 64, 16
    cx = torch.zeros((n, d_in // 2), dtype=torch.uint8)
    cw = torch.zeros((d_out, d_in // 2), dtype=torch.uint8)
    sx, sw = torch.zeros(n), torch.zeros(d_out)
    y = torch.zeros((n, d_out))
    acc = torch.zeros((n, d_out), dtype=torch.int32)
    B.cat_w4a4_linear(cx, sx, cw, sw, y, acc)
    assert rec.calls == ["cat_w4a4_linear"]
    bad = [dict(s_x=torch.zeros(n - 1)), dict(s_w=torch.zeros(d_out + 1)),
           dict(y_tilde=torch.zeros((n, d_out - 1))), dict(y_tilde=torch.zeros((n * d_out,))),
           dict(acc_out=torch.zeros((n - 1, d_out), dtype=torch.int32))]
    for b in bad:
        args = dict(codes_x=cx, s_x=sx, codes_w=cw, s_w=sw, y_tilde=y, acc_out=acc)
        args.update(b)
        with pytest.raises(ValueError):
            B.cat_w4a4_linear(**args)
    # int8 and asymmetric products share the checks
    c8x = torch.zeros((n, d_in), dtype=torch.int8)
    c8w = torch.zeros((d_out, d_in), dtype=torch.int8)
    with pytest.raises(ValueError):
        B.cat_int8_linear(c8x, sx, c8w, sw, torch.zeros((n + 1, d_out)))
    zm, rs = torch.zeros(n), torch.zeros(d_out, dtype=torch.int32)
    with pytest.raises(ValueError):
        B.cat_w4a4_linear_asym(cx, sx, torch.zeros(n - 1), cw, sw, rs, y)
    with pytest.raises(ValueError):
        B.cat_w4a4_linear_asym(cx, sx, zm, cw, sw, torch.zeros(d_out - 1, dtype=torch.int32), y)
    B.cat_w4a4_linear_asym(cx, sx, zm, cw, sw, rs, y)
    assert rec.calls == ["cat_w4a4_linear", "cat_w4a4_linear_asym"]


def test_binding_checks_transform_quant_buffer_sizes(fake_abi):
    torch, rec = fake_abi
    n, d, k = 8, 256, 32
    X = torch.zeros((n, d), dtype=torch.bfloat16)
    T = torch.zeros((d // k, k, k), dtype=torch.bfloat16)
    codes = torch.zeros((n, d // 2), dtype=torch.uint8)
    sx, ws = torch.zeros(n), torch.zeros(64, dtype=torch.uint8)
    B.cat_transform_quant(X, T, k, codes, sx, ws)
    with pytest.raises(ValueError):
        B.cat_transform_quant(X, T[:-1], k, codes, sx, ws)
    with pytest.raises(ValueError):
        B.cat_transform_quant(X, T, k, codes, torch.zeros(n - 1), ws)
    with pytest.raises(ValueError):
        B.cat_transform_quant(X, T, 48, codes, sx, ws)
    with pytest.raises(ValueError):
        B.cat_transform_quant_asym(X, T, k, codes, sx, torch.zeros(n + 1), ws)
    with pytest.raises(ValueError):
        B.cat_transform_quant_full(X, T[:, :, :16].contiguous(), k, codes, sx, ws)
    assert rec.calls == ["cat_transform_quant"]


def test_binding_checks_cov_and_sqnr_buffer_sizes(fake_abi):
    torch, rec = fake_abi
    n, d, k = 8, 256, 32
    X = torch.zeros((n, d), dtype=torch.bfloat16)
    ws = torch.zeros(64, dtype=torch.uint8)
    B.cat_cov_accumulate(X, torch.zeros((d, d)), B.CAT_COV_FULL, k, ws)
    B.cat_cov_accumulate(X, torch.zeros((d // k, k, k)), B.CAT_COV_BLOCK_DIAG, k, ws)
    # a block-diagonal accumulator passed in FULL mode would receive d*d floats
    with pytest.raises(ValueError):
        B.cat_cov_accumulate(X, torch.zeros((d // k, k, k)), B.CAT_COV_FULL, k, ws)
    with pytest.raises(ValueError):
        B.cat_cov_accumulate(X, torch.zeros((d, d)), B.CAT_COV_BLOCK_DIAG, k, ws)
    y = torch.zeros(100)
    B.cat_sqnr(y, y, ws, torch.zeros(3, dtype=torch.float64))
    with pytest.raises(ValueError):
        B.cat_sqnr(y, y, ws, torch.zeros(2, dtype=torch.float64))
    assert rec.calls == ["cat_cov_accumulate", "cat_cov_accumulate", "cat_sqnr"]
