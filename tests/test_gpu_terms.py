"""The Theorem 2.4 decomposition (Sec. 2) of a real-size layer from device
results: per-token scales from transform+quant, block second-moment sums of
the batch from the Sigma_x kernel and sum y^2 from the SQNR kernel, against
the oracle's concentration, alignment and prediction from the transformed
rows themselves."""
import numpy as np
import pytest

import paper_2603_04359_amd as cat
import workloads as wl
from oracle import cat_oracle as o
from paper_2603_04359_amd import binding as B

from gpu_common import dev, host, say, torch_mod

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("bits", [4, 8])
def test_theorem_2_4_terms_from_device_results(bits):
    torch = torch_mod()
    cfg = wl.get_config("attn4096", d_in=1024, d_out=512, n_cal=4096, n=2048)
    lay = wl.make_layer(cfg, seed=12)
    X, W, k, d, n = lay["X"], lay["W"], cfg.k, cfg.d_in, cfg.n
    say(f"Theorem 2.4 terms bits={bits} d={d} n={n}")
    T = o.round_storage(o.cat_transform(o.second_moment(lay["X_cal"]), W, k), "bf16")
    Tbits = (T.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    Wp = o.transform_weights(W, T)
    dX = dev(X, "bf16")
    # per-token scales (device)
    wide = bits != 4
    codes = torch.empty((n, d if wide else d // 2), dtype=torch.int8 if wide else torch.uint8,
                        device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(cat.cat_transform_quant_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    cat.cat_transform_quant(dX, dev(T, "bf16"), k, codes, s_x, ws, bits=bits)
    # block second-moment sums of the batch (device)
    acc = torch.zeros((d // k, k, k), dtype=torch.float32, device="cuda")
    cat.cat_cov_accumulate(dX, acc, B.CAT_COV_BLOCK_DIAG, k)
    # sum y^2 and the measured SQNR of the quantized layer (device)
    cw, sw = cat.cat_quantize_weights(Wp, bits)
    yt = torch.empty((n, cfg.d_out), dtype=torch.float32, device="cuda")
    if wide:
        cat.cat_int8_linear(codes, s_x, dev(cw, "i8"), dev(sw, "f32"), yt)
    else:
        cat.cat_w4a4_linear(codes, s_x, dev(cw, "u8"), dev(sw, "f32"), yt)
    y = o.reference_output(X, W).astype(np.float32)
    sws = torch.empty(cat.cat_sqnr_workspace_bytes(y.size), dtype=torch.uint8, device="cuda")
    out = torch.empty(3, dtype=torch.float64, device="cuda")
    cat.cat_sqnr(dev(y, "f32"), yt, sws, out)
    res = host(out)
    r = cat.cat_sqnr_terms(host(s_x), bits, host(acc).astype(np.float64), Tbits, B.CAT_BF16, Wp,
                           bits, float(res[0]))
    Z = o.transform_rows(X, T)
    cx, cw_, a = o.concentration_act(Z), o.concentration_weight(Wp), o.alignment(Z, Wp)
    pred = o.to_db(o.theorem_2_4(Z, Wp, bits, bits))
    say(f"  C(x') {r['C_x']:.6g} ({cx:.6g}), C(W') {r['C_w']:.6g}, A {r['A']:.6g} ({a:.6g}); "
        f"predicted {r['sqnr_pred_db']:.3f} dB ({pred:.3f}), measured {res[2]:.3f} dB")
    assert r["C_x"] == pytest.approx(cx, rel=1e-5)
    assert r["C_w"] == pytest.approx(cw_, rel=1e-12)
    assert r["A"] == pytest.approx(a, rel=1e-5)
    assert abs(r["sqnr_pred_db"] - pred) <= 0.01
    # the decomposition is an approximation of the measured SQNR
    assert abs(r["sqnr_pred_db"] - res[2]) <= 3.0
