"""The CAT-quantized linear layer as a sequence of library calls.

  calibrate_blocks  the d/k diagonal k x k blocks of Sigma_x = E[x x^T]
                    (Sec. 4; Sec. 6 "Calibration"), accumulated on the GPU
                    by cat_cov_accumulate in batches of at most 8192 tokens
  build_layer       host transform construction (cat_build_transform,
                    Sec. 4 eq. 7 and eq. 10) and per-channel weight codes
                    (cat_quantize_weights), uploaded to the device
  LayerRunner       one batch through cat_transform_quant, the integer GEMM
                    and cat_sqnr (Sec. 3 eq. 5; Sec. 2 eq. 1) on buffers it
                    allocates once
  reference_output  the unquantized output y = X W^T, formed in fp64 on the
                    device and stored as fp32: the signal the SQNR compares
                    against (an input of the SQNR step, not part of the path)

Plumbing only: every operation on the path is one of the C-ABI entry
points; torch supplies device memory.  The single host-side arithmetic step
is the division of the second-moment sums by the calibration token count,
which the transform builder takes as its input convention.
"""
from __future__ import annotations

import numpy as np

from . import binding as B


def _torch():
    import torch
    return torch


def to_device(a: np.ndarray, dtype: str, device="cuda"):
    """Host array -> device tensor in the storage type of a layer: 'bf16'
    takes fp32 values already representable in bf16 (the cast is exact),
    'f32' copies fp32."""
    torch = _torch()
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def calibrate_blocks(X_cal, k: int, chunk: int = 8192) -> np.ndarray:
    """Sigma_x diagonal blocks [d/k, k, k] in fp64, from a device tensor
    X_cal [n_cal, d] (bf16 or fp32): block sums on the GPU, then / n_cal."""
    torch = _torch()
    n_cal, d = X_cal.shape
    acc = torch.zeros((d // k, k, k), dtype=torch.float32, device=X_cal.device)
    for a in range(0, n_cal, chunk):
        B.cat_cov_accumulate(X_cal[a:a + chunk], acc, B.CAT_COV_BLOCK_DIAG, k)
    torch.cuda.synchronize()
    return acc.double().cpu().numpy() / n_cal


def build_layer(sigma_blocks: np.ndarray, W: np.ndarray, k: int, t_dtype: int,
                flags: int = B.CAT_BUILD_CAT, bits=(4,), device="cuda") -> dict:
    """Transform blocks T (host and device), W' = W T^-1 and the weight
    codes and scales of every width in `bits` (host and device)."""
    torch = _torch()
    T_host, T_exact, Wp = B.cat_build_transform(sigma_blocks, W, k, flags, t_dtype,
                                                want_exact=True)
    if t_dtype == B.CAT_BF16:
        T_dev = torch.from_numpy(T_host.view(np.int16)).to(device).view(torch.bfloat16)
    else:
        T_dev = torch.from_numpy(T_host).to(device)
    out = {"k": k, "t_dtype": t_dtype, "T_host": T_host, "T_exact": T_exact, "T": T_dev,
           "W_prime": Wp, "weights": {}}
    for b in bits:
        cw, sw = B.cat_quantize_weights(Wp, b)
        out["weights"][b] = {"codes_host": cw, "s_host": sw,
                             "codes": torch.from_numpy(cw.view(np.int8) if b != 4 else cw).to(device),
                             "s": torch.from_numpy(sw).to(device)}
    return out


def reference_output(X_dev, W: np.ndarray):
    """y = X W^T with fp64 products and sums on the device (X exact in fp64,
    W fp32 -> fp64), rounded once to fp32 [n, d_out]."""
    torch = _torch()
    Wd = torch.from_numpy(np.ascontiguousarray(W, dtype=np.float32)).to(X_dev.device).double()
    y = torch.matmul(X_dev.double(), Wd.t().contiguous()).float()
    del Wd
    return y


class LayerRunner:
    """Device buffers for one batch of n tokens of a built layer, and the
    path over them: transform+quant, GEMM, SQNR."""

    def __init__(self, layer: dict, n: int, d_in: int, d_out: int, device="cuda"):
        torch = _torch()
        self.layer, self.n, self.d_in, self.d_out = layer, n, d_in, d_out
        k = layer["k"]
        self.codes4 = torch.empty((n, d_in // 2), dtype=torch.uint8, device=device)
        self.s_x = torch.empty(n, dtype=torch.float32, device=device)
        self.ws_q = torch.empty(max(16, B.cat_transform_quant_asym_workspace_bytes(n, d_in, k)),
                                dtype=torch.uint8, device=device)
        self.y_t = torch.empty((n, d_out), dtype=torch.float32, device=device)
        self.ws_s = torch.empty(B.cat_sqnr_workspace_bytes(n * d_out), dtype=torch.uint8,
                                device=device)
        self.out = torch.empty(3, dtype=torch.float64, device=device)
        self._codes8 = None

    def codes(self, bits: int):
        if bits == 4:
            return self.codes4
        if self._codes8 is None:
            torch = _torch()
            self._codes8 = torch.empty((self.n, self.d_in), dtype=torch.int8,
                                       device=self.codes4.device)
        return self._codes8

    def transform_quant(self, X, bits: int = 4):
        B.cat_transform_quant(X, self.layer["T"], self.layer["k"], self.codes(bits), self.s_x,
                              self.ws_q, bits=bits)

    def linear(self, bits: int = 4):
        w = self.layer["weights"][bits]
        if bits == 4:
            B.cat_w4a4_linear(self.codes4, self.s_x, w["codes"], w["s"], self.y_t)
        else:
            B.cat_int8_linear(self.codes(bits), self.s_x, w["codes"], w["s"], self.y_t)

    def sqnr(self, y):
        B.cat_sqnr(y, self.y_t, self.ws_s, self.out)

    def run(self, X, y, bits: int = 4) -> np.ndarray:
        """The whole batch; returns (sum y^2, sum (y - y~)^2, dB) on the host."""
        self.transform_quant(X, bits)
        self.linear(bits)
        self.sqnr(y)
        _torch().cuda.synchronize()
        return self.out.cpu().numpy()
