"""Parity of the 6- and 8-bit widths (the W6A6 / W8A8 layers the paper
compares CAT W4A4 against, Sec. 4 "CAT Block Approximation" and the Fig. 6 caption) with the CPU oracle: transform+quant
writing one int8 per code on every kernel path, the int8-code GEMM, and the
whole chain's SQNR."""
import numpy as np
import pytest

import paper_2603_04359_amd as cat
import workloads as wl
from oracle import cat_oracle as o
from paper_2603_04359_amd import binding as B

from gpu_common import check_codes, check_tile_rows, dev, host, rel_fro, say, torch_mod

pytestmark = pytest.mark.gpu


def _tq_wide(X, T, k, x_dtype, t_dtype, bits):
    torch = torch_mod()
    n, d = X.shape
    codes = torch.empty((n, d), dtype=torch.int8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(cat.cat_transform_quant_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    cat.cat_transform_quant(dev(X, x_dtype), dev(T, t_dtype), k, codes, s_x, ws, bits=bits)
    return host(codes), host(s_x)


def _scales_close(s_gpu, s_or, label):
    assert np.all((s_gpu == 0) == (s_or == 0)), label
    nz = s_or != 0
    rel = np.abs(s_gpu[nz].astype(np.float64) - s_or[nz]) / s_or[nz]
    assert rel.max(initial=0) <= 1e-6, f"{label}: s_x rel err {rel.max()}"


def _rand_T(d, k, seed, dtype):
    rng = np.random.default_rng(seed)
    return o.round_storage(rng.standard_normal((d // k, k, k)) / np.sqrt(k), dtype)


# (d, k, n, x_dtype, t_dtype): the single-pass kernel (d = 2048, 4096,
# 8192, k = 128, bf16), the two-pass group kernels (k <= 256 with d a multiple of 256),
# the ring kernels (k = 512; k = 128 at d = 640), the small-block MFMA
# kernel (k = 64 at d = 384) and the vector-ALU kernels (fp32, k = 16)
PATHS = [(4096, 128, 300, "bf16", "bf16"), (8192, 128, 130, "bf16", "bf16"),
         (2048, 128, 97, "bf16", "bf16"), (1024, 128, 257, "bf16", "bf16"),
         (1024, 256, 129, "bf16", "bf16"), (1024, 512, 65, "bf16", "bf16"),
         (512, 64, 200, "bf16", "bf16"), (512, 32, 131, "bf16", "bf16"),
         (640, 128, 77, "bf16", "bf16"), (384, 64, 90, "bf16", "bf16"),
         (256, 32, 70, "f32", "f32"), (256, 16, 33, "bf16", "bf16")]


@pytest.mark.parametrize("bits", [6, 8])
@pytest.mark.parametrize("d,k,n,x_dtype,t_dtype", PATHS)
def test_transform_quant_wide_codes(d, k, n, x_dtype, t_dtype, bits):
    say(f"tq bits={bits} d={d} k={k} n={n} {x_dtype}/{t_dtype}")
    rng = np.random.default_rng(d + k + n + bits)
    Xf = (rng.standard_normal((n, d)) * np.exp(rng.standard_normal(d))).astype(np.float32)
    X = o.round_storage(Xf, x_dtype)
    X[n // 2] = 0.0                               # a zero token row
    T = _rand_T(d, k, seed=k + bits, dtype=t_dtype)
    codes, s = _tq_wide(X, T, k, x_dtype, t_dtype, bits)
    _, _, s_or = check_codes(codes, X, T, bits=bits, label=f"bits={bits} d={d} k={k}")
    _scales_close(s, s_or, f"bits={bits} d={d} k={k}")
    assert s[n // 2] == 0 and not codes[n // 2].any()
    assert np.abs(codes.view(np.int8)).max() == o.qmax_of(bits)


def _int8_case(n, d_in, d_out, qmax, seed, with_acc=True):
    torch = torch_mod()
    qx = wl.random_codes(n, d_in, seed, qmax=qmax)
    qw = wl.random_codes(d_out, d_in, seed + 1, qmax=qmax)
    rng = np.random.default_rng(seed + 2)
    sx = rng.uniform(0.01, 1.0, n).astype(np.float32)
    sw = rng.uniform(0.01, 1.0, d_out).astype(np.float32)
    qx[0] = 0
    sx[0] = 0
    acc_or, y_or = o.w4a4_linear(qx, sx, qw, sw)
    y = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    acc = torch.empty((n, d_out), dtype=torch.int32, device="cuda") if with_acc else None
    cat.cat_int8_linear(dev(qx, "i8"), dev(sx, "f32"), dev(qw, "i8"), dev(sw, "f32"), y, acc)
    return (host(acc) if with_acc else None), host(y), acc_or, y_or


@pytest.mark.parametrize("qmax", [127, 31])
@pytest.mark.parametrize("n,d_in,d_out", [
    (1, 32, 1), (130, 256, 200), (257, 4096, 384), (64, 160, 96), (300, 1024, 1000),
    (512, 96, 512),
])
def test_int8_linear_matches_oracle(n, d_in, d_out, qmax):
    say(f"int8 linear qmax={qmax} n={n} d_in={d_in} d_out={d_out}")
    acc, y, acc_or, y_or = _int8_case(n, d_in, d_out, qmax, seed=n + d_in + qmax)
    assert np.array_equal(acc, acc_or)                 # int32 bit-exact
    assert rel_fro(y, y_or) <= 1e-3
    assert np.array_equal(y, y_or)                     # same fp32 epilogue order
    assert not y[0].any()
    _, y2, _, _ = _int8_case(n, d_in, d_out, qmax, seed=n + d_in + qmax, with_acc=False)
    assert np.array_equal(y2, y_or)                    # full tiles' store path


@pytest.mark.parametrize("n,d_in,d_out,rows", [(4097, 160, 4100, 256), (2048, 1088, 4096, 128),
                                              (1900, 1056, 3000, 128)])
def test_int8_linear_both_tile_heights(n, d_in, d_out, rows):
    say(f"int8 linear tile rows {rows}: n={n} d_in={d_in} d_out={d_out}")
    check_tile_rows(n, d_out, rows)
    acc, y, acc_or, y_or = _int8_case(n, d_in, d_out, 127, seed=n + d_out)
    assert np.array_equal(acc, acc_or)
    assert np.array_equal(y, y_or)
    _, y2, _, _ = _int8_case(n, d_in, d_out, 127, seed=n + d_out, with_acc=False)
    assert np.array_equal(y2, y_or)


def test_int8_linear_extreme_codes_at_max_d_in():
    # 127^2 * 131072 = 2.11e9: the largest sum, still below 2^31
    torch = torch_mod()
    d_in = B.CAT_MAX_D_IN
    say(f"int8 linear extreme codes d_in={d_in}")
    qx = np.full((2, d_in), 127, np.int8)
    qx[1] = -127
    qw = np.full((3, d_in), 127, np.int8)
    qw[1] = -127
    qw[2, ::2] = -127
    sx = np.ones(2, np.float32)
    sw = np.ones(3, np.float32)
    acc_or, y_or = o.w4a4_linear(qx, sx, qw, sw)
    y = torch.empty((2, 3), dtype=torch.float32, device="cuda")
    acc = torch.empty((2, 3), dtype=torch.int32, device="cuda")
    cat.cat_int8_linear(dev(qx, "i8"), dev(sx, "f32"), dev(qw, "i8"), dev(sw, "f32"), y, acc)
    assert np.array_equal(host(acc), acc_or)
    assert host(acc)[0, 0] == 127 * 127 * d_in
    assert np.array_equal(host(y), y_or)


def test_int8_linear_mlp_up_full_size_sampled():
    # 8192 x 4096 -> 14336 with 8-bit codes; a 64 x 64 sample of rows and
    # columns over every panel, including the last ones
    torch = torch_mod()
    n, d_in, d_out = 8192, 4096, 14336
    say(f"int8 linear mlp_up full size {n} x {d_in} -> {d_out}")
    qx = wl.random_codes(n, d_in, seed=91, qmax=127)
    qw = wl.random_codes(d_out, d_in, seed=92, qmax=127)
    rng = np.random.default_rng(93)
    sx = rng.uniform(0.01, 1.0, n).astype(np.float32)
    sw = rng.uniform(0.01, 1.0, d_out).astype(np.float32)
    dqx, dsx, dqw, dsw = dev(qx, "i8"), dev(sx, "f32"), dev(qw, "i8"), dev(sw, "f32")
    y_fast = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    cat.cat_int8_linear(dqx, dsx, dqw, dsw, y_fast)
    y = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    acc = torch.empty((n, d_out), dtype=torch.int32, device="cuda")
    cat.cat_int8_linear(dqx, dsx, dqw, dsw, y, acc)
    assert torch.equal(y_fast, y)
    rows = np.unique(np.concatenate([rng.choice(n, 62, replace=False), [0, n - 1]]))
    cols = np.unique(np.concatenate([rng.choice(d_out, 62, replace=False), [0, d_out - 1]]))
    acc_or, y_or = o.w4a4_linear(qx[rows], sx[rows], qw[cols], sw[cols])
    ri, ci = torch.from_numpy(rows).cuda(), torch.from_numpy(cols).cuda()
    assert np.array_equal(host(acc[ri][:, ci]), acc_or)
    assert np.array_equal(host(y[ri][:, ci]), y_or)


def _chain_sqnr(cfg, lay, bits, x_dtype):
    """GPU chain: block Sigma_x -> host CAT transform -> transform+quant ->
    weight codes -> integer GEMM -> SQNR; and the oracle's chain from the
    same generator arrays."""
    torch = torch_mod()
    Xc, X, W = lay["X_cal"], lay["X"], lay["W"]
    k, d = cfg.k, cfg.d_in
    acc = torch.zeros((d // k, k, k), dtype=torch.float32, device="cuda")
    cat.cat_cov_accumulate(dev(Xc, x_dtype), acc, B.CAT_COV_BLOCK_DIAG, k)
    sx_blocks = host(acc).astype(np.float64) / Xc.shape[0]
    t_code = B.CAT_F32 if x_dtype == "f32" else B.CAT_BF16
    T, _, Wp = cat.cat_build_transform(sx_blocks, W, k, B.CAT_BUILD_CAT, t_code)
    if t_code == B.CAT_BF16:                      # bf16 bits -> their fp32 values
        T = (T.astype(np.uint32) << 16).view(np.float32)
    cw, sw = cat.cat_quantize_weights(Wp, bits)
    n = X.shape[0]
    wide = bits != 4
    codes = torch.empty((n, d if wide else d // 2), dtype=torch.int8 if wide else torch.uint8,
                        device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(cat.cat_transform_quant_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    cat.cat_transform_quant(dev(X, x_dtype), dev(T, x_dtype), k, codes, s_x, ws, bits=bits)
    yt = torch.empty((n, cfg.d_out), dtype=torch.float32, device="cuda")
    if wide:
        cat.cat_int8_linear(codes, s_x, dev(cw, "i8"), dev(sw, "f32"), yt)
    else:
        cat.cat_w4a4_linear(codes, s_x, dev(cw, "u8"), dev(sw, "f32"), yt)
    y = o.reference_output(X, W).astype(np.float32)
    sws = torch.empty(cat.cat_sqnr_workspace_bytes(y.size), dtype=torch.uint8, device="cuda")
    out = torch.empty(3, dtype=torch.float64, device="cuda")
    cat.cat_sqnr(dev(y, "f32"), yt, sws, out)
    gpu_db = float(host(out)[2])
    To = o.round_storage(o.cat_transform(o.second_moment(Xc), W, k), x_dtype)
    fw = o.quantized_forward(X.astype(np.float64), To, o.transform_weights(W, To), bits)
    or_db = o.sqnr(y, fw["y_tilde"])[2]
    return gpu_db, or_db


def test_end_to_end_tiny_layer_w4a4_w6a6_w8a8():
    """The tiny fp32 layer through the whole chain at 4, 6 and 8 bits: each
    SQNR within 0.05 dB of the oracle's, and each extra two bits worth
    roughly 12 dB (Theorem 2.4: SQNR scales with N(b)^2)."""
    cfg = wl.get_config("tiny")
    lay = wl.make_layer(cfg, seed=0)
    dbs = {}
    for bits in (4, 6, 8):
        gpu_db, or_db = _chain_sqnr(cfg, lay, bits, "f32")
        say(f"  tiny CAT W{bits}A{bits}: SQNR gpu {gpu_db:.4f} dB, oracle {or_db:.4f} dB")
        assert abs(gpu_db - or_db) <= 0.05
        dbs[bits] = gpu_db
    assert 9.0 < dbs[6] - dbs[4] < 15.0
    assert 9.0 < dbs[8] - dbs[6] < 15.0


def test_end_to_end_bf16_layer_w4a4_w6a6_w8a8():
    """An attention-projection-shaped bf16 layer (1024 -> 512, block 128,
    LogNormal channel scales with outliers) through the whole chain at 4, 6
    and 8 bits, each SQNR within 0.05 dB of the oracle's."""
    cfg = wl.get_config("attn4096", d_in=1024, d_out=512, n_cal=4096, n=256)
    lay = wl.make_layer(cfg, seed=4)
    prev = None
    for bits in (4, 6, 8):
        gpu_db, or_db = _chain_sqnr(cfg, lay, bits, "bf16")
        say(f"  attn-shaped CAT W{bits}A{bits}: SQNR gpu {gpu_db:.4f} dB, oracle {or_db:.4f} dB")
        assert abs(gpu_db - or_db) <= 0.05
        if prev is not None:
            assert gpu_db > prev + 6.0
        prev = gpu_db


def test_w8a8_pair_graph_replays_match_eager():
    # 8-bit transform+quant at the single-pass shape (its own exchange tag
    # under capture) and the int8 GEMM, captured once and replayed with new
    # activations; every replay equals the eager calls bit for bit
    torch = torch_mod()
    n, d, d_out, k = 256, 4096, 512, 128
    say("W8A8 pair under graph capture: 3 replays vs eager")
    T = _rand_T(d, k, seed=61, dtype="bf16")
    dT = dev(T, "bf16")
    qw = wl.random_codes(d_out, d, seed=62, qmax=127)
    dqw = dev(qw, "i8")
    dsw = dev(np.random.default_rng(63).uniform(0.01, 1.0, d_out).astype(np.float32), "f32")
    rng = np.random.default_rng(64)
    Xs = [o.round_storage(rng.standard_normal((n, d)).astype(np.float32), "bf16")
          for _ in range(3)]

    def buffers():
        return dict(codes=torch.empty((n, d), dtype=torch.int8, device="cuda"),
                    s_x=torch.empty(n, dtype=torch.float32, device="cuda"),
                    yt=torch.empty((n, d_out), dtype=torch.float32, device="cuda"),
                    ws=torch.empty(cat.cat_transform_quant_workspace_bytes(n, d, k),
                                   dtype=torch.uint8, device="cuda"))

    def pair(dX, b):
        cat.cat_transform_quant(dX, dT, k, b["codes"], b["s_x"], b["ws"], bits=8)
        cat.cat_int8_linear(b["codes"], b["s_x"], dqw, dsw, b["yt"])

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
        for key in ("codes", "s_x", "yt"):
            assert torch.equal(g_b[key], e_b[key]), f"replay {i}: {key}"
