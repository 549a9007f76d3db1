"""Thin ctypes binding of libcat.so (the C ABI declared in include/cat.h).

Argument marshalling only: every function here checks that tensors have
the dtype, device and contiguity the C call expects, passes raw pointers
and sizes, and turns a non-zero status into CatError.  All arithmetic of
the path runs in the library's HIP kernels (device calls) or its C++ host
code (transform construction).  PyTorch only provides device memory and
the current stream.  If the library is missing, every call raises: there
is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcat.so")

CAT_OK = 0
CAT_ERR_INVALID_ARG = -1
CAT_ERR_UNSUPPORTED = -2
CAT_ERR_WORKSPACE = -3
CAT_ERR_HIP = -4
CAT_ERR_INTERNAL = -5
CAT_ERR_TIMEOUT = -6

CAT_F32 = 0
CAT_BF16 = 1

CAT_COV_FULL = 0
CAT_COV_BLOCK_DIAG = 1

CAT_BUILD_HADAMARD = 1
CAT_BUILD_ALIGN = 2
CAT_BUILD_CAT = 3

CAT_MAX_D_IN = 131072
CAT_MAX_BLOCK = 512

# every symbol include/cat.h declares
EXPORTED = (
    "cat_cov_workspace_bytes", "cat_cov_accumulate", "cat_transform_quant_workspace_bytes",
    "cat_transform_quant_flag_offset", "cat_set_exchange_spin_limit", "cat_transform_quant", "cat_transform_quant_noalloc_max_bytes",
    "cat_transform_quant_noalloc", "cat_transform_quant_status", "cat_transform_quant_noalloc_status",
    "cat_w4a4_linear", "cat_int8_linear", "cat_transform_quant_asym_workspace_bytes",
    "cat_transform_quant_asym", "cat_w4a4_linear_asym",
    "cat_weight_code_sums", "cat_sqnr_terms", "cat_transform_quant_full_workspace_bytes",
    "cat_transform_quant_full", "cat_full_hadamard_weights", "cat_sqnr_workspace_bytes", "cat_sqnr", "cat_build_transform",
    "cat_quantize_weights", "cat_last_error", "cat_version",
)


class CatError(RuntimeError):
    def __init__(self, fn: str, code: int, msg: str):
        super().__init__(f"{fn} failed with status {code}: {msg}")
        self.fn = fn
        self.code = code


_lib = None
_c = ctypes
_i64 = ctypes.c_int64
_vp = ctypes.c_void_p
_int = ctypes.c_int
_sz = ctypes.c_size_t


def lib() -> ctypes.CDLL:
    """Load libcat.so (once).  Raises ImportError if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python paper_2603_04359_amd/build.py` (or __graft_entry__.build())")
    L = ctypes.CDLL(LIB_PATH)
    L.cat_cov_workspace_bytes.argtypes = [_int, _i64, _i64, _int, _i64]
    L.cat_cov_workspace_bytes.restype = _sz
    L.cat_cov_accumulate.argtypes = [_vp, _int, _i64, _i64, _int, _i64, _vp, _vp, _sz, _vp]
    L.cat_cov_accumulate.restype = _int
    L.cat_transform_quant_workspace_bytes.argtypes = [_i64, _i64, _i64]
    L.cat_transform_quant_workspace_bytes.restype = _sz
    L.cat_transform_quant_flag_offset.argtypes = [_i64, _i64, _i64]
    L.cat_transform_quant_flag_offset.restype = _sz
    L.cat_set_exchange_spin_limit.argtypes = [ctypes.c_uint32]
    L.cat_set_exchange_spin_limit.restype = None
    L.cat_transform_quant.argtypes = [_vp, _int, _i64, _i64, _vp, _int, _i64, _int, _vp, _vp,
                                      _vp, _sz, _vp]
    L.cat_transform_quant.restype = _int
    L.cat_transform_quant_noalloc_max_bytes.argtypes = []
    L.cat_transform_quant_noalloc_max_bytes.restype = _sz
    L.cat_transform_quant_noalloc.argtypes = [_vp, _int, _i64, _i64, _vp, _int, _i64, _int, _vp,
                                              _vp, _vp]
    L.cat_transform_quant_noalloc.restype = _int
    L.cat_transform_quant_status.argtypes = [_vp, _i64, _i64, _i64, _vp]
    L.cat_transform_quant_status.restype = _int
    L.cat_transform_quant_noalloc_status.argtypes = [_i64, _i64, _i64, _vp]
    L.cat_transform_quant_noalloc_status.restype = _int
    L.cat_w4a4_linear.argtypes = [_vp, _vp, _vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp]
    L.cat_w4a4_linear.restype = _int
    L.cat_int8_linear.argtypes = [_vp, _vp, _vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp]
    L.cat_int8_linear.restype = _int
    L.cat_transform_quant_asym_workspace_bytes.argtypes = [_i64, _i64, _i64]
    L.cat_transform_quant_asym_workspace_bytes.restype = _sz
    L.cat_transform_quant_asym.argtypes = [_vp, _int, _i64, _i64, _vp, _int, _i64, _vp, _vp, _vp,
                                           _vp, _sz, _vp]
    L.cat_transform_quant_asym.restype = _int
    L.cat_w4a4_linear_asym.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _vp, _vp,
                                       _vp]
    L.cat_w4a4_linear_asym.restype = _int
    L.cat_weight_code_sums.argtypes = [_vp, _i64, _i64, _vp]
    L.cat_weight_code_sums.restype = _int
    L.cat_sqnr_terms.argtypes = [_vp, _i64, _int, _vp, _i64, _i64, _vp, _int, _vp, _i64, _int,
                                 ctypes.c_double, _vp]
    L.cat_sqnr_terms.restype = _int
    L.cat_transform_quant_full_workspace_bytes.argtypes = [_i64, _i64, _i64]
    L.cat_transform_quant_full_workspace_bytes.restype = _sz
    L.cat_transform_quant_full.argtypes = [_vp, _int, _i64, _i64, _vp, _int, _i64, _vp, _vp, _vp,
                                           _sz, _vp]
    L.cat_transform_quant_full.restype = _int
    L.cat_full_hadamard_weights.argtypes = [_vp, _i64, _i64, _i64, _vp]
    L.cat_full_hadamard_weights.restype = _int
    L.cat_sqnr_workspace_bytes.argtypes = [_i64]
    L.cat_sqnr_workspace_bytes.restype = _sz
    L.cat_sqnr.argtypes = [_vp, _vp, _i64, _vp, _sz, _vp, _vp]
    L.cat_sqnr.restype = _int
    L.cat_build_transform.argtypes = [_vp, _vp, _i64, _i64, _i64, _int, _int, _vp, _vp, _vp, _int]
    L.cat_build_transform.restype = _int
    L.cat_quantize_weights.argtypes = [_vp, _i64, _i64, _int, _vp, _vp]
    L.cat_quantize_weights.restype = _int
    L.cat_last_error.argtypes = []
    L.cat_last_error.restype = ctypes.c_char_p
    L.cat_version.argtypes = []
    L.cat_version.restype = ctypes.c_char_p
    _lib = L
    return L


def cat_last_error() -> str:
    return lib().cat_last_error().decode()


def cat_version() -> str:
    return lib().cat_version().decode()


def _check(fn: str, rc: int):
    if rc != CAT_OK:
        raise CatError(fn, rc, cat_last_error())


# ------------------------------------------------------------ marshalling
def _torch():
    import torch
    return torch


def _dev_ptr(t, name, dtypes=None, allow_none=False):
    if t is None:
        if allow_none:
            return None
        raise ValueError(f"{name} is required")
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must live on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    return t.data_ptr()


def _shape(t, shape, name):
    """The C ABI takes bare pointers and cannot see buffer sizes, so every
    buffer's shape is checked here, before the call: a short buffer would
    otherwise be read or written past its end on the device."""
    if tuple(t.shape) != tuple(int(v) for v in shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _numel(t, count, name):
    if t.numel() != int(count):
        raise ValueError(f"{name} has {t.numel()} elements, expected {int(count)}")


def _t_blocks(T, d, k, name="T"):
    if k <= 0 or d % k:
        raise ValueError(f"d={d} is not a multiple of the block size k={k}")
    _numel(T, d * k, name)


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return CAT_BF16
    if t.dtype == torch.float32:
        return CAT_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream_ptr(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


# ------------------------------------------------------------ device calls
def cat_cov_workspace_bytes(x_dtype: int, n: int, d: int, mode: int = CAT_COV_FULL,
                            k: int = 1) -> int:
    return int(lib().cat_cov_workspace_bytes(x_dtype, n, d, mode, k))


def cat_cov_accumulate(X, acc, mode: int = CAT_COV_FULL, k: int = 1, workspace=None,
                       stream=None):
    """acc += X^T X (FULL: acc [d, d]; BLOCK_DIAG: acc [d/k, k, k]), fp32.
    `workspace`: a device tensor of at least cat_cov_workspace_bytes() bytes;
    when None, one is allocated for this call."""
    torch = _torch()
    px = _dev_ptr(X, "X", (torch.bfloat16, torch.float32))
    pa = _dev_ptr(acc, "acc", (torch.float32,))
    if X.dim() != 2:
        raise ValueError("X must be [n, d]")
    n, d = X.shape
    if mode == CAT_COV_FULL:
        _numel(acc, d * d, "acc")
    elif mode == CAT_COV_BLOCK_DIAG:
        if k <= 0 or d % k:
            raise ValueError(f"d={d} is not a multiple of the block size k={k}")
        _numel(acc, d * k, "acc ([d/k, k, k])")
    else:
        raise ValueError(f"unknown mode {mode}")
    code = _dtype_code(X)
    if workspace is None:
        need = cat_cov_workspace_bytes(code, n, d, mode, k)
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=X.device)
    pw = _dev_ptr(workspace, "workspace")
    wbytes = workspace.numel() * workspace.element_size()
    _check("cat_cov_accumulate",
           lib().cat_cov_accumulate(px, code, n, d, mode, k, pa, pw, wbytes,
                                    _stream_ptr(stream)))


def cat_transform_quant_workspace_bytes(n: int, d: int, k: int) -> int:
    return int(lib().cat_transform_quant_workspace_bytes(n, d, k))


def cat_transform_quant_flag_offset(n: int, d: int, k: int) -> int:
    """Byte offset of the exchange timeout word inside the workspace."""
    return int(lib().cat_transform_quant_flag_offset(n, d, k))


def cat_set_exchange_spin_limit(polls: int) -> None:
    """Testing hook: bound the single-pass exchange waits (0 = default)."""
    lib().cat_set_exchange_spin_limit(int(polls))


def cat_transform_quant(X, T, k: int, codes, s_x, workspace, bits: int = 4, stream=None):
    """codes and s_x [n] fp32 from X [n, d] and T [d/k, k, k].  codes:
    bits 4: uint8 [n, d/2] packed INT4; bits 6, 8: int8 [n, d]."""
    torch = _torch()
    px = _dev_ptr(X, "X", (torch.bfloat16, torch.float32))
    pt = _dev_ptr(T, "T", (torch.bfloat16, torch.float32))
    pc = _dev_ptr(codes, "codes", (torch.uint8,) if bits == 4 else (torch.int8,))
    ps = _dev_ptr(s_x, "s_x", (torch.float32,))
    pw = _dev_ptr(workspace, "workspace")
    if X.dim() != 2:
        raise ValueError("X must be [n, d]")
    n, d = X.shape
    if tuple(codes.shape) != (n, d // 2 if bits == 4 else d):
        raise ValueError(f"codes must be [{n}, {d // 2 if bits == 4 else d}] for bits={bits}")
    _t_blocks(T, d, k)
    _numel(s_x, n, "s_x")
    wbytes = workspace.numel() * workspace.element_size()
    _check("cat_transform_quant",
           lib().cat_transform_quant(px, _dtype_code(X), n, d, pt, _dtype_code(T), k, bits, pc, ps,
                                     pw, wbytes, _stream_ptr(stream)))


def _gemm_shapes(codes_x, s_x, codes_w, s_w, y_tilde, acc_out):
    """(n, row bytes, d_out) of a GEMM call after checking every buffer
    against them."""
    if codes_x.dim() != 2 or codes_w.dim() != 2:
        raise ValueError("codes_x and codes_w must be 2-D")
    n, row = codes_x.shape
    d_out = codes_w.shape[0]
    if codes_w.shape[1] != row:
        raise ValueError("codes_x and codes_w disagree on d_in")
    _numel(s_x, n, "s_x")
    _numel(s_w, d_out, "s_w")
    _shape(y_tilde, (n, d_out), "y_tilde")
    if acc_out is not None:
        _shape(acc_out, (n, d_out), "acc_out")
    return n, row, d_out


def cat_transform_quant_noalloc_max_bytes() -> int:
    return int(lib().cat_transform_quant_noalloc_max_bytes())


def cat_transform_quant_noalloc(X, T, k: int, codes, s_x, bits: int = 4, stream=None):
    """cat_transform_quant with the library's own per-device scratch instead
    of a caller workspace (no allocation on the call)."""
    torch = _torch()
    px = _dev_ptr(X, "X", (torch.bfloat16, torch.float32))
    pt = _dev_ptr(T, "T", (torch.bfloat16, torch.float32))
    pc = _dev_ptr(codes, "codes", (torch.uint8,) if bits == 4 else (torch.int8,))
    ps = _dev_ptr(s_x, "s_x", (torch.float32,))
    if X.dim() != 2:
        raise ValueError("X must be [n, d]")
    n, d = X.shape
    if tuple(codes.shape) != (n, d // 2 if bits == 4 else d):
        raise ValueError(f"codes must be [{n}, {d // 2 if bits == 4 else d}] for bits={bits}")
    _t_blocks(T, d, k)
    _numel(s_x, n, "s_x")
    _check("cat_transform_quant_noalloc",
           lib().cat_transform_quant_noalloc(px, _dtype_code(X), n, d, pt, _dtype_code(T), k, bits,
                                             pc, ps, _stream_ptr(stream)))


def cat_transform_quant_status(workspace, n: int, d: int, k: int, stream=None):
    """Waits for the stream, then reads and clears the exchange timeout word
    of a workspace used by calls of shape (n, d, k); raises CatError
    (code CAT_ERR_TIMEOUT) when a wait ran out."""
    torch = _torch()
    pw = _dev_ptr(workspace, "workspace", (torch.uint8,))
    if workspace.numel() < cat_transform_quant_flag_offset(n, d, k) + 4:
        raise ValueError("workspace is smaller than a workspace of this shape")
    _check("cat_transform_quant_status",
           lib().cat_transform_quant_status(pw, n, d, k, _stream_ptr(stream)))


def cat_transform_quant_noalloc_status(n: int, d: int, k: int, stream=None):
    """cat_transform_quant_status for the library's per-device scratch of
    cat_transform_quant_noalloc."""
    _check("cat_transform_quant_noalloc_status",
           lib().cat_transform_quant_noalloc_status(n, d, k, _stream_ptr(stream)))


def cat_w4a4_linear(codes_x, s_x, codes_w, s_w, y_tilde, acc_out=None, stream=None):
    """y_tilde [n, d_out] fp32 (and optionally acc_out int32) from packed codes."""
    torch = _torch()
    pcx = _dev_ptr(codes_x, "codes_x", (torch.uint8,))
    psx = _dev_ptr(s_x, "s_x", (torch.float32,))
    pcw = _dev_ptr(codes_w, "codes_w", (torch.uint8,))
    psw = _dev_ptr(s_w, "s_w", (torch.float32,))
    py = _dev_ptr(y_tilde, "y_tilde", (torch.float32,))
    pacc = _dev_ptr(acc_out, "acc_out", (torch.int32,), allow_none=True)
    n, half, d_out = _gemm_shapes(codes_x, s_x, codes_w, s_w, y_tilde, acc_out)
    _check("cat_w4a4_linear",
           lib().cat_w4a4_linear(pcx, psx, pcw, psw, n, 2 * half, d_out, py, pacc,
                                 _stream_ptr(stream)))


def cat_int8_linear(codes_x, s_x, codes_w, s_w, y_tilde, acc_out=None, stream=None):
    """y_tilde [n, d_out] fp32 (and optionally acc_out int32) from int8
    codes, one per element (the 6- and 8-bit widths)."""
    torch = _torch()
    pcx = _dev_ptr(codes_x, "codes_x", (torch.int8,))
    psx = _dev_ptr(s_x, "s_x", (torch.float32,))
    pcw = _dev_ptr(codes_w, "codes_w", (torch.int8,))
    psw = _dev_ptr(s_w, "s_w", (torch.float32,))
    py = _dev_ptr(y_tilde, "y_tilde", (torch.float32,))
    pacc = _dev_ptr(acc_out, "acc_out", (torch.int32,), allow_none=True)
    n, d_in, d_out = _gemm_shapes(codes_x, s_x, codes_w, s_w, y_tilde, acc_out)
    _check("cat_int8_linear",
           lib().cat_int8_linear(pcx, psx, pcw, psw, n, d_in, d_out, py, pacc,
                                 _stream_ptr(stream)))


def cat_transform_quant_asym_workspace_bytes(n: int, d: int, k: int) -> int:
    return int(lib().cat_transform_quant_asym_workspace_bytes(n, d, k))


def cat_transform_quant_asym(X, T, k: int, codes, s_x, zmin_x, workspace, stream=None):
    """Asymmetric INT4: codes uint8 [n, d/2] (q - 8 packed), s_x and
    zmin_x [n] fp32, from X [n, d] and T [d/k, k, k]."""
    torch = _torch()
    px = _dev_ptr(X, "X", (torch.bfloat16, torch.float32))
    pt = _dev_ptr(T, "T", (torch.bfloat16, torch.float32))
    pc = _dev_ptr(codes, "codes", (torch.uint8,))
    ps = _dev_ptr(s_x, "s_x", (torch.float32,))
    pm = _dev_ptr(zmin_x, "zmin_x", (torch.float32,))
    pw = _dev_ptr(workspace, "workspace")
    if X.dim() != 2:
        raise ValueError("X must be [n, d]")
    n, d = X.shape
    if tuple(codes.shape) != (n, d // 2):
        raise ValueError(f"codes must be [{n}, {d // 2}]")
    _t_blocks(T, d, k)
    _numel(s_x, n, "s_x")
    _numel(zmin_x, n, "zmin_x")
    wbytes = workspace.numel() * workspace.element_size()
    _check("cat_transform_quant_asym",
           lib().cat_transform_quant_asym(px, _dtype_code(X), n, d, pt, _dtype_code(T), k, pc, ps,
                                          pm, pw, wbytes, _stream_ptr(stream)))


def cat_w4a4_linear_asym(codes_x, s_x, zmin_x, codes_w, s_w, rsum_w, y_tilde, acc_out=None,
                         stream=None):
    """y_tilde [n, d_out] fp32 from asymmetric activation codes and
    symmetric weight codes with their row sums rsum_w int32 [d_out]."""
    torch = _torch()
    pcx = _dev_ptr(codes_x, "codes_x", (torch.uint8,))
    psx = _dev_ptr(s_x, "s_x", (torch.float32,))
    pmx = _dev_ptr(zmin_x, "zmin_x", (torch.float32,))
    pcw = _dev_ptr(codes_w, "codes_w", (torch.uint8,))
    psw = _dev_ptr(s_w, "s_w", (torch.float32,))
    prs = _dev_ptr(rsum_w, "rsum_w", (torch.int32,))
    py = _dev_ptr(y_tilde, "y_tilde", (torch.float32,))
    pacc = _dev_ptr(acc_out, "acc_out", (torch.int32,), allow_none=True)
    n, half, d_out = _gemm_shapes(codes_x, s_x, codes_w, s_w, y_tilde, acc_out)
    _numel(zmin_x, n, "zmin_x")
    _numel(rsum_w, d_out, "rsum_w")
    _check("cat_w4a4_linear_asym",
           lib().cat_w4a4_linear_asym(pcx, psx, pmx, pcw, psw, prs, n, 2 * half, d_out, py, pacc,
                                      _stream_ptr(stream)))


def cat_weight_code_sums(codes_w):
    """Host: int32 [d_out] row sums of packed INT4 weight codes [d_out, d_in/2]."""
    c, pc = _host(codes_w, np.uint8, "codes_w")
    d_out, half = c.shape
    out = np.empty(d_out, dtype=np.int32)
    _check("cat_weight_code_sums", lib().cat_weight_code_sums(pc, d_out, 2 * half, out.ctypes.data))
    return out


def cat_sqnr_terms(s_x, bits_x: int, sigma_sum_blocks, T, t_dtype: int, W_prime, bits_w: int,
                   sum_y2: float):
    """Host Theorem 2.4 terms: returns dict C_x, C_w, A, sqnr_pred, sqnr_pred_db."""
    sx, psx = _host(s_x, np.float32, "s_x")
    S, pS = _host(sigma_sum_blocks, np.float64, "sigma_sum_blocks")
    Tn, pT = _host(T, np.uint16 if t_dtype == CAT_BF16 else np.float32, "T")
    Wp, pW = _host(W_prime, np.float64, "W_prime")
    if S.ndim != 3 or S.shape[1] != S.shape[2]:
        raise ValueError("sigma_sum_blocks must be [d_in/k, k, k]")
    nb, k, _ = S.shape
    d_out, d_in = Wp.shape
    if nb * k != d_in or Tn.size != d_in * k:
        raise ValueError("sigma_sum_blocks, T and W_prime disagree on d_in or k")
    out = np.empty(5, dtype=np.float64)
    _check("cat_sqnr_terms", lib().cat_sqnr_terms(psx, sx.shape[0], bits_x, pS, d_in, k, pT,
                                                  t_dtype, pW, d_out, bits_w, float(sum_y2),
                                                  out.ctypes.data))
    return dict(zip(("C_x", "C_w", "A", "sqnr_pred", "sqnr_pred_db"), out.tolist()))


def cat_transform_quant_full_workspace_bytes(n: int, d: int, k: int) -> int:
    return int(lib().cat_transform_quant_full_workspace_bytes(n, d, k))


def cat_transform_quant_full(X, T, k: int, codes, s_x, workspace, stream=None):
    """Full-dimension Hadamard transform + INT4: codes uint8 [n, d/2] and
    s_x [n] fp32 from X [n, d] bf16 and the blocks T [d/k, k, k] bf16."""
    torch = _torch()
    px = _dev_ptr(X, "X", (torch.bfloat16,))
    pt = _dev_ptr(T, "T", (torch.bfloat16,))
    pc = _dev_ptr(codes, "codes", (torch.uint8,))
    ps = _dev_ptr(s_x, "s_x", (torch.float32,))
    pw = _dev_ptr(workspace, "workspace")
    if X.dim() != 2:
        raise ValueError("X must be [n, d]")
    n, d = X.shape
    if tuple(codes.shape) != (n, d // 2):
        raise ValueError(f"codes must be [{n}, {d // 2}]")
    _t_blocks(T, d, k)
    _numel(s_x, n, "s_x")
    wbytes = workspace.numel() * workspace.element_size()
    _check("cat_transform_quant_full",
           lib().cat_transform_quant_full(px, CAT_BF16, n, d, pt, CAT_BF16, k, pc, ps, pw, wbytes,
                                          _stream_ptr(stream)))


def cat_full_hadamard_weights(W_prime, k: int):
    """Host: W_full = W' (H_m (x) I_k)^T / sqrt(m), fp64."""
    Wp, pw = _host(W_prime, np.float64, "W_prime")
    d_out, d_in = Wp.shape
    out = np.empty_like(Wp)
    _check("cat_full_hadamard_weights",
           lib().cat_full_hadamard_weights(pw, d_out, d_in, k, out.ctypes.data))
    return out


def cat_sqnr_workspace_bytes(count: int) -> int:
    return int(lib().cat_sqnr_workspace_bytes(count))


def cat_sqnr(y, y_tilde, workspace, out, stream=None):
    """out [3] fp64 = (sum y^2, sum (y - y~)^2, dB)."""
    torch = _torch()
    py = _dev_ptr(y, "y", (torch.float32,))
    pt = _dev_ptr(y_tilde, "y_tilde", (torch.float32,))
    pw = _dev_ptr(workspace, "workspace")
    po = _dev_ptr(out, "out", (torch.float64,))
    if y.numel() != y_tilde.numel():
        raise ValueError("y and y_tilde differ in size")
    _numel(out, 3, "out")
    wbytes = workspace.numel() * workspace.element_size()
    _check("cat_sqnr", lib().cat_sqnr(py, pt, y.numel(), pw, wbytes, po, _stream_ptr(stream)))


# -------------------------------------------------------------- host calls
def _host(a, dtype, name):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data


def cat_build_transform(sigma_x_blocks, W, k: int, flags: int = CAT_BUILD_CAT,
                        t_dtype: int = CAT_BF16, want_exact: bool = False,
                        want_w_prime: bool = True, n_threads: int = 0):
    """Host transform construction.  Returns (T, T_exact or None, W_prime or None);
    T is uint16 bf16 bits (t_dtype = CAT_BF16) or fp32, shape [d_in/k, k, k]."""
    W, pw = _host(W, np.float32, "W")
    d_out, d_in = W.shape
    if sigma_x_blocks is not None:
        sx, psx = _host(sigma_x_blocks, np.float64, "sigma_x_blocks")
        if sx.shape != (d_in // k, k, k):
            raise ValueError("sigma_x_blocks must be [d_in/k, k, k]")
    else:
        sx, psx = None, None
    T = np.empty((d_in // k, k, k), dtype=np.uint16 if t_dtype == CAT_BF16 else np.float32)
    Te = np.empty((d_in // k, k, k), dtype=np.float64) if want_exact else None
    Wp = np.empty((d_out, d_in), dtype=np.float64) if want_w_prime else None
    _check("cat_build_transform",
           lib().cat_build_transform(psx, pw, d_out, d_in, k, flags, t_dtype, T.ctypes.data,
                                     Te.ctypes.data if Te is not None else None,
                                     Wp.ctypes.data if Wp is not None else None, n_threads))
    return T, Te, Wp


def cat_quantize_weights(W_prime, bits: int = 4):
    """Host per-output-channel quantization: returns (codes, s_w fp32);
    codes uint8 [d_out, d_in/2] packed INT4 (bits 4) or int8 [d_out, d_in]
    (bits 6, 8)."""
    Wp, pwp = _host(W_prime, np.float64, "W_prime")
    d_out, d_in = Wp.shape
    codes = (np.empty((d_out, d_in // 2), dtype=np.uint8) if bits == 4
             else np.empty((d_out, d_in), dtype=np.int8))
    s_w = np.empty(d_out, dtype=np.float32)
    _check("cat_quantize_weights",
           lib().cat_quantize_weights(pwp, d_out, d_in, bits, codes.ctypes.data, s_w.ctypes.data))
    return codes, s_w
