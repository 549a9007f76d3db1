"""Parity of the full-dimension Hadamard transform T = H_d blockdiag(M_b)
(Sec. 4, T = H M with H over all channels) with the CPU oracle: block
transform, cross-block Hadamard (Sylvester, or Paley's order 28 (x)
Sylvester), per-token INT4 quantization, and the whole chain's SQNR."""
import numpy as np
import pytest

import paper_2603_04359_amd as cat
import workloads as wl
from oracle import cat_oracle as o
from paper_2603_04359_amd import binding as B

from gpu_common import dev, host, say, torch_mod

pytestmark = pytest.mark.gpu


def _tq_full(X, T, k):
    torch = torch_mod()
    n, d = X.shape
    codes = torch.empty((n, d // 2), dtype=torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(cat.cat_transform_quant_full_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    cat.cat_transform_quant_full(dev(X, "bf16"), dev(T, "bf16"), k, codes, s_x, ws)
    return o.unpack_int4(host(codes)), host(s_x)


def _check_full(q, s, X, T, k, label):
    q_or, s_or = o.transform_quant_full(X, T, 4)
    mism = q != q_or
    nm = int(mism.sum())
    if nm:
        Z = o.full_hadamard_mix(o.transform_rows(X, T), k)
        amax = np.abs(Z).max(axis=1, keepdims=True)
        with np.errstate(divide="ignore", invalid="ignore"):
            u = np.abs(Z * (7.0 / amax))[mism]
        tie = (np.abs(q[mism].astype(int) - q_or[mism].astype(int)) == 1) & \
              (np.abs(u - np.floor(u) - 0.5) <= 2.0 ** -20 * np.maximum(1.0, u))
        assert tie.all(), f"{label}: {int((~tie).sum())} non-tie mismatches of {q.size}"
        assert nm <= max(1, int(1e-6 * q.size)), f"{label}: {nm} ties"
    assert np.all((s == 0) == (s_or == 0))
    nz = s_or != 0
    assert np.max(np.abs(s[nz].astype(np.float64) - s_or[nz]) / s_or[nz], initial=0) <= 1e-6
    say(f"  {label}: codes {q.size}, tie mismatches {nm}")


@pytest.mark.parametrize("d,k,n", [(1024, 128, 257), (4096, 128, 130), (3584, 128, 70),
                                   (7168, 256, 33), (14336, 128, 17), (14336, 256, 40),
                                   (256, 128, 5), (4096, 128, 8192)])
def test_transform_quant_full_matches_oracle(d, k, n):
    say(f"tq full Hadamard d={d} k={k} (m={d // k}) n={n}")
    rng = np.random.default_rng(d + k + n)
    X = o.round_storage((rng.standard_normal((n, d)) * np.exp(rng.standard_normal(d))
                         ).astype(np.float32), "bf16")
    X[n // 2] = 0.0
    T = o.round_storage(rng.standard_normal((d // k, k, k)) / np.sqrt(k), "bf16")
    q, s = _tq_full(X, T, k)
    _check_full(q, s, X, T, k, f"d={d} k={k}")
    assert s[n // 2] == 0 and not q[n // 2].any()


def test_end_to_end_full_hadamard_sqnr():
    """A 3584 -> 512 bf16 layer (m = 28: the Paley factor) through the whole
    chain with the full-dimension CAT transform; SQNR within 0.05 dB of the
    oracle's chain."""
    torch = torch_mod()
    cfg = wl.get_config("attn4096", d_in=3584, d_out=512, n_cal=4096, n=256)
    lay = wl.make_layer(cfg, seed=8)
    Xc, X, W, k, d = lay["X_cal"], lay["X"], lay["W"], cfg.k, cfg.d_in
    acc = torch.zeros((d // k, k, k), dtype=torch.float32, device="cuda")
    cat.cat_cov_accumulate(dev(Xc, "bf16"), acc, B.CAT_COV_BLOCK_DIAG, k)
    T, _, Wp = cat.cat_build_transform(host(acc).astype(np.float64) / Xc.shape[0], W, k,
                                       B.CAT_BUILD_CAT, B.CAT_BF16)
    Tf = (T.astype(np.uint32) << 16).view(np.float32)
    Wfull = cat.cat_full_hadamard_weights(Wp, k)
    cw, sw = cat.cat_quantize_weights(Wfull, 4)
    n = X.shape[0]
    codes = torch.empty((n, d // 2), dtype=torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(cat.cat_transform_quant_full_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    cat.cat_transform_quant_full(dev(X, "bf16"), dev(Tf, "bf16"), k, codes, s_x, ws)
    yt = torch.empty((n, cfg.d_out), dtype=torch.float32, device="cuda")
    cat.cat_w4a4_linear(codes, s_x, dev(cw, "u8"), dev(sw, "f32"), yt)
    y = o.reference_output(X, W).astype(np.float32)
    sws = torch.empty(cat.cat_sqnr_workspace_bytes(y.size), dtype=torch.uint8, device="cuda")
    out = torch.empty(3, dtype=torch.float64, device="cuda")
    cat.cat_sqnr(dev(y, "f32"), yt, sws, out)
    gpu_db = float(host(out)[2])
    To = o.round_storage(o.cat_transform(o.second_moment(Xc), W, k), "bf16")
    qx, sx = o.transform_quant_full(X.astype(np.float64), To, 4)
    qw, swo = o.quantize_weights(o.transform_weights_full(W, To), 4)
    _, yto = o.w4a4_linear(qx, sx, qw, swo)
    or_db = o.sqnr(y, yto)[2]
    say(f"  full-Hadamard CAT SQNR gpu {gpu_db:.4f} dB, oracle {or_db:.4f} dB")
    assert abs(gpu_db - or_db) <= 0.05
