"""Parity of asymmetric per-token activation quantization (the paper's own
activation set-up, Sec. 6; range max - min, Sec. 2 after Lemma 2.2) with
the CPU oracle: transform+quant with the row minimum, the product with its
code-sum correction, and the whole chain's SQNR."""
import numpy as np
import pytest

import paper_2603_04359_amd as cat
import workloads as wl
from oracle import cat_oracle as o
from paper_2603_04359_amd import binding as B

from gpu_common import check_tile_rows, dev, host, say, torch_mod

pytestmark = pytest.mark.gpu


def _tq_asym(X, T, k, x_dtype, t_dtype):
    torch = torch_mod()
    n, d = X.shape
    codes = torch.empty((n, d // 2), dtype=torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    zmin = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(cat.cat_transform_quant_asym_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    cat.cat_transform_quant_asym(dev(X, x_dtype), dev(T, t_dtype), k, codes, s_x, zmin, ws)
    return o.unpack_int4(host(codes)).astype(np.int16) + 8, host(s_x), host(zmin)


def _check_asym(q, s, m, X, T, label):
    """Codes equal the oracle's except at rounding ties (off by one, the
    exact multiplier u* = (z - min) 15 / r within 2^-20 max(1, u*) of a
    half-integer), at most 1e-6 * 15/7 of them (the symmetric INT4 bar scaled
    by the grid's intervals, 15 against 7 per sign); scales and minima
    within 1e-6 of the row range."""
    q_or, s_or, m_or = o.transform_quant_asym(X, T, 4)
    mism = q != q_or
    nm = int(mism.sum())
    if nm:
        Z = o.transform_rows(X, T)
        zmin = Z.min(axis=1, keepdims=True)
        r = Z.max(axis=1, keepdims=True) - zmin
        with np.errstate(divide="ignore", invalid="ignore"):
            u = (Z - zmin) * (15.0 / r)
        um = u[mism]
        tie = (np.abs(q[mism].astype(int) - q_or[mism].astype(int)) == 1) & \
              (np.abs(um - np.floor(um) - 0.5) <= 2.0 ** -20 * np.maximum(1.0, um))
        assert tie.all(), f"{label}: {int((~tie).sum())} non-tie mismatches"
        assert nm <= max(1, int(1e-6 * 15 / 7 * q.size)), f"{label}: {nm} ties"
    r_or = (s_or.astype(np.float64) * 15.0)
    assert np.all((s == 0) == (s_or == 0)), label
    assert np.all(np.abs(s.astype(np.float64) - s_or) <= 1e-6 * np.maximum(s_or, 1e-30)), label
    assert np.all(np.abs(m.astype(np.float64) - m_or) <= 1e-6 * np.maximum(np.abs(m_or), r_or)
                  + 1e-30), label
    say(f"  {label}: codes {q.size}, tie mismatches {nm}")


# bf16 group kernels (k <= 256, d a multiple of 256), ring kernels (k = 512,
# and k = 128 at d = 640) and vector-ALU kernels (fp32)
@pytest.mark.parametrize("d,k,n,x_dtype,t_dtype", [
    (4096, 128, 300, "bf16", "bf16"), (1024, 256, 129, "bf16", "bf16"),
    (1024, 512, 65, "bf16", "bf16"), (512, 64, 70, "bf16", "bf16"), (256, 32, 33, "f32", "f32"),
    (14336, 256, 130, "bf16", "bf16"), (768, 32, 65, "bf16", "bf16"), (640, 128, 97, "bf16", "bf16"),
    (8192, 128, 130, "bf16", "bf16"), (2048, 128, 257, "bf16", "bf16"), (4096, 128, 3, "bf16", "bf16"),
])
def test_transform_quant_asym_matches_oracle(d, k, n, x_dtype, t_dtype):
    say(f"tq asym d={d} k={k} n={n} {x_dtype}/{t_dtype}")
    rng = np.random.default_rng(d + k + n)
    Xf = (rng.standard_normal((n, d)) * np.exp(rng.standard_normal(d)) +
          rng.standard_normal(d)).astype(np.float32)
    Xf[1] = 0.0                                   # zero row
    Xf[2] = np.abs(Xf[2]) + 0.5                   # all positive
    X = o.round_storage(Xf, x_dtype)
    T = o.round_storage(rng.standard_normal((d // k, k, k)) / np.sqrt(k), t_dtype)
    q, s, m = _tq_asym(X, T, k, x_dtype, t_dtype)
    _check_asym(q, s, m, X, T, f"asym d={d} k={k}")
    assert s[1] == 0 and m[1] == 0 and not q[1].any()


@pytest.mark.parametrize("d,n", [(4096, 192), (4096, 3135), (4096, 3584), (8192, 1537),
                                 (2048, 6145)])
def test_transform_quant_asym_single_pass_tiles_per_workgroup(d, n):
    # the asymmetric single pass at token counts that give each workgroup 1,
    # 7 and 8 tiles of 64 tokens, on both sides of the exchange lag of 6
    # steps, with unequal token-tile rows and a zero row in the last tile
    say(f"tq asym single pass d={d} k=128 n={n} (tiles per workgroup)")
    rng = np.random.default_rng(3 * n + d)
    Xf = (rng.standard_normal((n, d)) * np.exp(0.5 * rng.standard_normal(d)) +
          rng.standard_normal(d)).astype(np.float32)
    Xf[n - 1] = 0.0
    X = o.round_storage(Xf, "bf16")
    T = o.round_storage(rng.standard_normal((d // 128, 128, 128)) / np.sqrt(128), "bf16")
    q, s, m = _tq_asym(X, T, 128, "bf16", "bf16")
    _check_asym(q, s, m, X, T, f"asym single pass d={d} n={n}")
    assert s[n - 1] == 0 and m[n - 1] == 0 and not q[n - 1].any()


@pytest.mark.parametrize("d", [512, 4096])
def test_transform_quant_asym_identity_constant_rows_exact(d):
    # T = I: z = x exactly on both sides, so codes, scales and minima are
    # identical; a constant row is reconstructed exactly by its minimum
    # (d = 4096: the single-pass kernel, d = 512: two passes)
    say(f"tq asym identity bf16 k=128 d={d}")
    X = wl.random_bf16_matrix(200, d, seed=7, scale=2.0).astype(np.float64)
    X[3] = 1.5
    T = np.stack([np.eye(128)] * (d // 128))
    q, s, m = _tq_asym(X, T, 128, "bf16", "bf16")
    q_or, s_or, m_or = o.transform_quant_asym(X, T, 4)
    assert np.array_equal(q, q_or)
    assert np.array_equal(s, s_or) and np.array_equal(m, m_or)
    assert s[3] == 0 and m[3] == 1.5 and not q[3].any()


def _asym_gemm(n, d_in, d_out, seed, with_acc=True):
    torch = torch_mod()
    rng = np.random.default_rng(seed)
    qx = rng.integers(0, 16, size=(n, d_in)).astype(np.int16)
    qw = wl.random_codes(d_out, d_in, seed + 1)
    sx = rng.uniform(0.01, 1.0, n).astype(np.float32)
    mx = rng.uniform(-3.0, 1.0, n).astype(np.float32)
    sw = rng.uniform(0.01, 1.0, d_out).astype(np.float32)
    sx[0] = 0.0                                   # a constant row: only its minimum
    qx[0] = 0
    acc_or, y_or = o.linear_asym(qx, sx, mx, qw, sw)
    pw = o.pack_int4(qw)
    rs = cat.cat_weight_code_sums(pw)
    y = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    acc = torch.empty((n, d_out), dtype=torch.int32, device="cuda") if with_acc else None
    cat.cat_w4a4_linear_asym(dev(o.pack_int4(qx - 8), "u8"), dev(sx, "f32"), dev(mx, "f32"),
                             dev(pw, "u8"), dev(sw, "f32"), dev(rs, "i32"), y, acc)
    return (host(acc) if with_acc else None), host(y), acc_or, y_or


@pytest.mark.parametrize("n,d_in,d_out", [
    (1, 32, 1), (130, 256, 200), (257, 4096, 384), (64, 160, 96), (512, 256, 512),
])
def test_w4a4_linear_asym_matches_oracle(n, d_in, d_out):
    say(f"w4a4 asym n={n} d_in={d_in} d_out={d_out}")
    acc, y, acc_or, y_or = _asym_gemm(n, d_in, d_out, seed=n + d_out)
    assert np.array_equal(acc, acc_or)
    assert np.array_equal(y, y_or)
    _, y2, _, _ = _asym_gemm(n, d_in, d_out, seed=n + d_out, with_acc=False)
    assert np.array_equal(y2, y_or)


@pytest.mark.parametrize("n,d_in,d_out,rows", [(4097, 256, 4100, 256), (1900, 4160, 3000, 128),
                                              (2048, 4096, 4096, 128)])
def test_w4a4_linear_asym_both_tile_heights(n, d_in, d_out, rows):
    say(f"w4a4 asym tile rows {rows}: n={n} d_in={d_in} d_out={d_out}")
    check_tile_rows(n, d_out, rows)
    acc, y, acc_or, y_or = _asym_gemm(n, d_in, d_out, seed=n + d_in)
    assert np.array_equal(acc, acc_or)
    assert np.array_equal(y, y_or)
    _, y2, _, _ = _asym_gemm(n, d_in, d_out, seed=n + d_in, with_acc=False)
    assert np.array_equal(y2, y_or)


def test_end_to_end_asym_vs_sym_sqnr():
    """A bf16 layer with ReLU-like (non-negative) activations through the
    whole chain, symmetric and asymmetric: each SQNR within 0.05 dB of the
    oracle's; the asymmetric range wins on such data (Sec. 2.1)."""
    torch = torch_mod()
    cfg = wl.get_config("attn4096", d_in=1024, d_out=512, n_cal=4096, n=256)
    lay = wl.make_layer(cfg, seed=6)
    Xc = o.round_storage(np.abs(lay["X_cal"]), "bf16")
    X = o.round_storage(np.abs(lay["X"]), "bf16")
    W, k, d = lay["W"], cfg.k, cfg.d_in
    acc = torch.zeros((d // k, k, k), dtype=torch.float32, device="cuda")
    cat.cat_cov_accumulate(dev(Xc, "bf16"), acc, B.CAT_COV_BLOCK_DIAG, k)
    T, _, Wp = cat.cat_build_transform(host(acc).astype(np.float64) / Xc.shape[0], W, k,
                                       B.CAT_BUILD_CAT, B.CAT_BF16)
    Tf = (T.astype(np.uint32) << 16).view(np.float32)
    cw, sw = cat.cat_quantize_weights(Wp, 4)
    rs = cat.cat_weight_code_sums(cw)
    n = X.shape[0]
    codes = torch.empty((n, d // 2), dtype=torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    zmin = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(cat.cat_transform_quant_asym_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    y = o.reference_output(X, W).astype(np.float32)
    dy = dev(y, "f32")
    sws = torch.empty(cat.cat_sqnr_workspace_bytes(y.size), dtype=torch.uint8, device="cuda")
    out = torch.empty(3, dtype=torch.float64, device="cuda")
    yt = torch.empty((n, cfg.d_out), dtype=torch.float32, device="cuda")
    dX, dT, dcw, dsw = dev(X, "bf16"), dev(Tf, "bf16"), dev(cw, "u8"), dev(sw, "f32")
    cat.cat_transform_quant_asym(dX, dT, k, codes, s_x, zmin, ws)
    cat.cat_w4a4_linear_asym(codes, s_x, zmin, dcw, dsw, dev(rs, "i32"), yt)
    cat.cat_sqnr(dy, yt, sws, out)
    asym_db = float(host(out)[2])
    cat.cat_transform_quant(dX, dT, k, codes, s_x, ws)
    cat.cat_w4a4_linear(codes, s_x, dcw, dsw, yt)
    cat.cat_sqnr(dy, yt, sws, out)
    sym_db = float(host(out)[2])
    To = o.round_storage(o.cat_transform(o.second_moment(Xc), W, k), "bf16")
    Wpo = o.transform_weights(W, To)
    or_asym = o.sqnr(y, o.quantized_forward_asym(X, To, Wpo, 4)["y_tilde"])[2]
    or_sym = o.sqnr(y, o.quantized_forward(X, To, Wpo, 4)["y_tilde"])[2]
    say(f"  asym gpu {asym_db:.4f} oracle {or_asym:.4f}; sym gpu {sym_db:.4f} oracle {or_sym:.4f}")
    assert abs(asym_db - or_asym) <= 0.05
    assert abs(sym_db - or_sym) <= 0.05
    assert asym_db > sym_db


@pytest.mark.parametrize("d", [1024, 4096])
def test_asym_pair_graph_replays_match_eager(d):
    # the asymmetric pair captured once and replayed with new activations,
    # against eager calls: d = 1024 runs the key clear and two passes,
    # d = 4096 the single pass (a device tag per replay)
    torch = torch_mod()
    n, d_out, k = 300, 384, 128
    say(f"asymmetric pair under graph capture d={d}: 3 replays vs eager")
    rng = np.random.default_rng(71)
    T = o.round_storage(rng.standard_normal((d // k, k, k)) / np.sqrt(k), "bf16")
    dT = dev(T, "bf16")
    qw = wl.random_codes(d_out, d, seed=72)
    pw = o.pack_int4(qw)
    dqw, drs = dev(pw, "u8"), dev(cat.cat_weight_code_sums(pw), "i32")
    dsw = dev(rng.uniform(0.01, 1.0, d_out).astype(np.float32), "f32")
    Xs = [o.round_storage((rng.standard_normal((n, d)) + 1.0).astype(np.float32), "bf16")
          for _ in range(3)]

    def buffers():
        return dict(codes=torch.empty((n, d // 2), dtype=torch.uint8, device="cuda"),
                    s_x=torch.empty(n, dtype=torch.float32, device="cuda"),
                    zmin=torch.empty(n, dtype=torch.float32, device="cuda"),
                    yt=torch.empty((n, d_out), dtype=torch.float32, device="cuda"),
                    ws=torch.empty(cat.cat_transform_quant_asym_workspace_bytes(n, d, k),
                                   dtype=torch.uint8, device="cuda"))

    def pair(dX, b):
        cat.cat_transform_quant_asym(dX, dT, k, b["codes"], b["s_x"], b["zmin"], b["ws"])
        cat.cat_w4a4_linear_asym(b["codes"], b["s_x"], b["zmin"], dqw, dsw, drs, b["yt"])

    dX = dev(Xs[0], "bf16")
    g_b, e_b = buffers(), buffers()
    pair(dX, g_b)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=torch.cuda.Stream()):
        pair(dX, g_b)
    for i, X in enumerate(Xs):
        dX.copy_(dev(X, "bf16"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        pair(dX, e_b)
        torch.cuda.synchronize()
        for key in ("codes", "s_x", "zmin", "yt"):
            assert torch.equal(g_b[key], e_b[key]), f"replay {i}: {key}"


def test_asym_mlp_up_full_size():
    # 8192 x 4096 activations (transform+quant over every token) and the
    # 4096 -> 14336 product checked on a 64 x 64 sample of rows and columns
    torch = torch_mod()
    n, d, d_out, k = 8192, 4096, 14336, 128
    say(f"asym full size {n} x {d} -> {d_out}")
    cfg = wl.get_config("mlp_up", n=n, n_cal=16)
    X = wl.make_layer(cfg, seed=3, with_cal=False, with_weights=False)["X"].astype(np.float64)
    rng = np.random.default_rng(81)
    T = o.round_storage(rng.standard_normal((d // k, k, k)) / np.sqrt(k), "bf16")
    q, s, m = _tq_asym(X, T, k, "bf16", "bf16")
    _check_asym(q, s, m, X, T, "mlp_up asym")
    qw = wl.random_codes(d_out, d, seed=82)
    sw = rng.uniform(0.01, 1.0, d_out).astype(np.float32)
    pw = o.pack_int4(qw)
    y = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    acc = torch.empty((n, d_out), dtype=torch.int32, device="cuda")
    cat.cat_w4a4_linear_asym(dev(o.pack_int4(q - 8), "u8"), dev(s, "f32"), dev(m, "f32"),
                             dev(pw, "u8"), dev(sw, "f32"), dev(cat.cat_weight_code_sums(pw), "i32"),
                             y, acc)
    rows = np.unique(np.concatenate([rng.choice(n, 62, replace=False), [0, n - 1]]))
    cols = np.unique(np.concatenate([rng.choice(d_out, 62, replace=False), [0, d_out - 1]]))
    acc_or, y_or = o.linear_asym(q[rows], s[rows], m[rows], qw[cols], sw[cols])
    ri, ci = torch.from_numpy(rows).cuda(), torch.from_numpy(cols).cuda()
    assert np.array_equal(host(acc[ri][:, ci]), acc_or)
    assert np.array_equal(host(y[ri][:, ci]), y_or)
