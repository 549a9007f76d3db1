"""Parity of the four HIP kernels (through the C ABI) with the CPU oracle,
at sizes the oracle finishes in seconds that span several tiles and ragged
tails, plus the edge cases each kernel has."""
import numpy as np
import pytest

import paper_2603_04359_amd as cat
import workloads as wl
from oracle import cat_oracle as o
from paper_2603_04359_amd import binding as B

from gpu_common import check_codes, check_tile_rows, dev, host, rel_fro, say, torch_mod

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------------ SQNR
@pytest.mark.parametrize("count", [1, 3, 1000, 4097, 4 * 256 * 2048 * 2 + 5])
def test_sqnr_matches_oracle(count):
    torch = torch_mod()
    say(f"sqnr count={count}")
    y, yt = wl.random_pair(count, seed=count % 1000)
    S, E, dB = o.sqnr(y, yt)
    ws = torch.empty(cat.cat_sqnr_workspace_bytes(count), dtype=torch.uint8, device="cuda")
    out = torch.empty(3, dtype=torch.float64, device="cuda")
    dy, dyt = dev(y, "f32"), dev(yt, "f32")
    cat.cat_sqnr(dy, dyt, ws, out)
    r = host(out)
    assert r[0] == pytest.approx(S, rel=1e-12)
    assert r[1] == pytest.approx(E, rel=1e-12)
    assert abs(r[2] - dB) < 1e-6
    # fixed reduction order: bit-reproducible
    out2 = torch.empty_like(out)
    cat.cat_sqnr(dy, dyt, ws, out2)
    assert np.array_equal(host(out2), r)


def test_sqnr_zero_error_is_infinite():
    torch = torch_mod()
    y, _ = wl.random_pair(777, seed=1)
    dy = dev(y, "f32")
    ws = torch.empty(cat.cat_sqnr_workspace_bytes(777), dtype=torch.uint8, device="cuda")
    out = torch.empty(3, dtype=torch.float64, device="cuda")
    cat.cat_sqnr(dy, dy.clone(), ws, out)
    r = host(out)
    assert r[1] == 0.0 and r[2] == np.inf


# ------------------------------------------------------------------ GEMM
def _gemm_case(n, d_in, d_out, seed, zero_rows=(), with_acc=True):
    torch = torch_mod()
    qx = wl.random_codes(n, d_in, seed)
    qw = wl.random_codes(d_out, d_in, seed + 1)
    rng = np.random.default_rng(seed + 2)
    sx = rng.uniform(0.01, 1.0, n).astype(np.float32)
    sw = rng.uniform(0.01, 1.0, d_out).astype(np.float32)
    for r in zero_rows:
        qx[r] = 0
        sx[r] = 0
    acc_or, y_or = o.w4a4_linear(qx, sx, qw, sw)
    y = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    acc = torch.empty((n, d_out), dtype=torch.int32, device="cuda") if with_acc else None
    cat.cat_w4a4_linear(dev(o.pack_int4(qx), "u8"), dev(sx, "f32"), dev(o.pack_int4(qw), "u8"),
                        dev(sw, "f32"), y, acc)
    return (host(acc) if with_acc else None), host(y), acc_or, y_or


@pytest.mark.parametrize("n,d_in,d_out", [
    (1, 32, 1), (130, 256, 200), (257, 4096, 384), (64, 160, 96), (300, 1024, 1000),
])
def test_w4a4_linear_matches_oracle(n, d_in, d_out):
    say(f"w4a4 n={n} d_in={d_in} d_out={d_out}")
    acc, y, acc_or, y_or = _gemm_case(n, d_in, d_out, seed=n + d_in, zero_rows=(0,))
    assert np.array_equal(acc, acc_or)                 # int32 bit-exact
    assert rel_fro(y, y_or) <= 1e-3                    # the stated bar
    assert np.array_equal(y, y_or)                     # same fp32 epilogue order
    assert not y[0].any()


@pytest.mark.parametrize("n,d_in,d_out", [
    (512, 256, 512), (256, 4096, 768), (300, 1024, 1000), (1, 32, 1), (257, 160, 300),
    (768, 96, 256),
])
def test_w4a4_linear_without_acc_out_matches_oracle(n, d_in, d_out):
    # without acc_out, full 256 x 256 tiles take a separate store path
    say(f"w4a4 no acc_out n={n} d_in={d_in} d_out={d_out}")
    _, y, _, y_or = _gemm_case(n, d_in, d_out, seed=3 * n + d_out, zero_rows=(0,), with_acc=False)
    assert np.array_equal(y, y_or)
    assert not y[0].any()


# (n, d_in, d_out, acc_out, token rows per tile on a 256-CU device)
TILE_HEIGHT_CASES = [
    (4097, 160, 4100, True, 256),     # 289 tiles of 256 rows: ragged rows, outputs and K
    (4352, 1056, 3840, False, 256),   # 255 tiles of 256 rows: one CU idle, stays at 256
    (1900, 4160, 3000, True, 128),    # 96 tiles of 256 rows become 180 of 128, ragged
    (2048, 4096, 4096, False, 128),   # the attention-projection shape, full tiles
    (129, 96, 8000, False, 128),      # a last 128-row panel holding one row
]


@pytest.mark.parametrize("n,d_in,d_out,with_acc,rows", TILE_HEIGHT_CASES)
def test_w4a4_linear_both_tile_heights(n, d_in, d_out, with_acc, rows):
    # the launcher takes 128-row tiles when 256-row ones leave CUs idle
    say(f"w4a4 tile rows {rows}: n={n} d_in={d_in} d_out={d_out} acc={with_acc}")
    check_tile_rows(n, d_out, rows)
    acc, y, acc_or, y_or = _gemm_case(n, d_in, d_out, seed=n + d_in + d_out, zero_rows=(0, n - 1),
                                      with_acc=with_acc)
    if with_acc:
        assert np.array_equal(acc, acc_or)
    assert np.array_equal(y, y_or)
    assert not y[0].any() and not y[n - 1].any()


@pytest.mark.parametrize("d_in", [96, 224])
def test_w4a4_linear_many_short_tiles_per_workgroup(d_in):
    # 8192 x 8192 outputs = 1024 tiles, four per workgroup, each only one or
    # two K steps deep: the scale slots and the operand stream roll over
    # from tile to tile every step or two
    torch = torch_mod()
    n = d_out = 8192
    say(f"w4a4 short tiles n={n} d_in={d_in} d_out={d_out}")
    qx = wl.random_codes(n, d_in, seed=d_in)
    qw = wl.random_codes(d_out, d_in, seed=d_in + 1)
    rng = np.random.default_rng(d_in + 2)
    sx = rng.uniform(0.01, 1.0, n).astype(np.float32)
    sw = rng.uniform(0.01, 1.0, d_out).astype(np.float32)
    acc_or, y_or = o.w4a4_linear(qx, sx, qw, sw)
    args = (dev(o.pack_int4(qx), "u8"), dev(sx, "f32"), dev(o.pack_int4(qw), "u8"), dev(sw, "f32"))
    y = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    acc = torch.empty((n, d_out), dtype=torch.int32, device="cuda")
    cat.cat_w4a4_linear(*args, y, acc)
    assert np.array_equal(host(acc), acc_or)
    assert np.array_equal(host(y), y_or)
    y2 = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    cat.cat_w4a4_linear(*args, y2)
    assert torch.equal(y2, y)


@pytest.mark.parametrize("n,d_in,d_out,with_acc,int8", [
    (512, 1024, 512, False, False), (300, 800, 510, True, False), (512, 1024, 512, False, True),
])
def test_linear_scales_across_the_fp32_range(n, d_in, d_out, with_acc, int8):
    # scales log-uniform over 1e-30 .. 1e30 (and some zero): y~ =
    # fl(fl(acc) s_x) s_w runs into subnormal and infinite values, which
    # the epilogue must round as IEEE fp32 does (no flush to zero), bit for
    # bit with the oracle; full tiles without acc_out take the straight-line
    # epilogue, the others the checked one
    say(f"linear extreme scales n={n} d_in={d_in} d_out={d_out} acc={with_acc} int8={int8}")
    torch = torch_mod()
    rng = np.random.default_rng(n + d_out + int8)
    sx = np.exp(rng.uniform(np.log(1e-30), np.log(1e30), n)).astype(np.float32)
    sw = np.exp(rng.uniform(np.log(1e-30), np.log(1e30), d_out)).astype(np.float32)
    sx[rng.random(n) < 0.05] = 0.0
    qmax = 127 if int8 else 7
    qx = wl.random_codes(n, d_in, n + 1, qmax=qmax)
    qw = wl.random_codes(d_out, d_in, n + 2, qmax=qmax)
    with np.errstate(over="ignore"):
        acc_or, y_or = o.w4a4_linear(qx, sx, qw, sw)
    assert np.isinf(y_or).any() and ((y_or != 0) & (np.abs(y_or) < np.finfo(np.float32).tiny)).any()
    y = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    acc = torch.empty((n, d_out), dtype=torch.int32, device="cuda") if with_acc else None
    if int8:
        cat.cat_int8_linear(dev(qx, "i8"), dev(sx, "f32"), dev(qw, "i8"), dev(sw, "f32"), y, acc)
    else:
        cat.cat_w4a4_linear(dev(o.pack_int4(qx), "u8"), dev(sx, "f32"), dev(o.pack_int4(qw), "u8"),
                            dev(sw, "f32"), y, acc)
    assert np.array_equal(host(y), y_or)
    if with_acc:
        assert np.array_equal(host(acc), acc_or)


def test_w4a4_linear_extreme_codes_at_max_d_in():
    torch = torch_mod()
    d_in = B.CAT_MAX_D_IN
    say(f"w4a4 extreme codes d_in={d_in}")
    qx = np.full((2, d_in), 7, np.int8)
    qx[1] = -7
    qw = np.full((3, d_in), 7, np.int8)
    qw[1] = -7
    qw[2, ::2] = -7
    sx = np.ones(2, np.float32)
    sw = np.ones(3, np.float32)
    acc_or, y_or = o.w4a4_linear(qx, sx, qw, sw)
    y = torch.empty((2, 3), dtype=torch.float32, device="cuda")
    acc = torch.empty((2, 3), dtype=torch.int32, device="cuda")
    cat.cat_w4a4_linear(dev(o.pack_int4(qx), "u8"), dev(sx, "f32"), dev(o.pack_int4(qw), "u8"),
                        dev(sw, "f32"), y, acc)
    assert np.array_equal(host(acc), acc_or)
    assert host(acc)[0, 0] == 49 * d_in


def test_w4a4_linear_mlp_up_full_size_sampled():
    # 8192 x 4096 -> 14336, the shape and launch the benchmark times; the
    # oracle checks a 64 x 64 sample of rows and columns spread over every
    # row panel and column panel, including the last ones
    torch = torch_mod()
    n, d_in, d_out = 8192, 4096, 14336
    say(f"w4a4 mlp_up full size {n} x {d_in} -> {d_out}")
    qx = wl.random_codes(n, d_in, seed=81)
    qw = wl.random_codes(d_out, d_in, seed=82)
    rng = np.random.default_rng(83)
    sx = rng.uniform(0.01, 1.0, n).astype(np.float32)
    sw = rng.uniform(0.01, 1.0, d_out).astype(np.float32)
    dqx, dsx, dqw, dsw = dev(o.pack_int4(qx), "u8"), dev(sx, "f32"), dev(o.pack_int4(qw), "u8"), \
        dev(sw, "f32")
    # the benchmark's call passes no acc_out (full tiles take the straight-line
    # store path); the second call also writes the int32 accumulators
    y_fast = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    cat.cat_w4a4_linear(dqx, dsx, dqw, dsw, y_fast)
    y = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    acc = torch.empty((n, d_out), dtype=torch.int32, device="cuda")
    cat.cat_w4a4_linear(dqx, dsx, dqw, dsw, y, acc)
    assert torch.equal(y_fast, y)
    rows = np.unique(np.concatenate([rng.choice(n, 62, replace=False), [0, n - 1]]))
    cols = np.unique(np.concatenate([rng.choice(d_out, 62, replace=False), [0, d_out - 1]]))
    acc_or, y_or = o.w4a4_linear(qx[rows], sx[rows], qw[cols], sw[cols])
    acc_g = host(acc[torch.from_numpy(rows).cuda()][:, torch.from_numpy(cols).cuda()])
    y_g = host(y[torch.from_numpy(rows).cuda()][:, torch.from_numpy(cols).cuda()])
    assert np.array_equal(acc_g, acc_or)
    assert np.array_equal(y_g, y_or)


# ------------------------------------------------------ transform + quant
def _tq_gpu(X, T, k, x_dtype, t_dtype):
    torch = torch_mod()
    n, d = X.shape
    dX = dev(X, x_dtype)
    dT = dev(T, t_dtype)
    codes = torch.empty((n, d // 2), dtype=torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(cat.cat_transform_quant_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    cat.cat_transform_quant(dX, dT, k, codes, s_x, ws)
    return host(codes), host(s_x)


def _tq_gpu_from_device(dX, T, k):
    torch = torch_mod()
    n, d = dX.shape
    dT = dev(T, "bf16")
    codes = torch.empty((n, d // 2), dtype=torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(cat.cat_transform_quant_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    cat.cat_transform_quant(dX, dT, k, codes, s_x, ws)
    return host(codes), host(s_x)


def _check_scales(s_gpu, s_or, label):
    assert np.all((s_gpu == 0) == (s_or == 0)), label
    nz = s_or != 0
    rel = np.abs(s_gpu[nz].astype(np.float64) - s_or[nz]) / s_or[nz]
    assert rel.max(initial=0) <= 1e-6, f"{label}: s_x rel err {rel.max()}"
    say(f"  {label}: s_x max rel {rel.max(initial=0):.2e}, exact {np.mean(s_gpu == s_or):.4f}")


def test_transform_quant_identity_is_exact_rtn():
    # T = I: z = x exactly on both sides, so there is no tie ambiguity and
    # every code and scale must be identical.
    say("tq identity bf16 k=128")
    X = wl.random_bf16_matrix(300, 512, seed=3, scale=2.0).astype(np.float64)
    T = np.stack([np.eye(128)] * 4)
    codes, s = _tq_gpu(X, T, 128, "bf16", "bf16")
    q_or, s_or = o.transform_quant(X, T, 4)
    assert np.array_equal(o.unpack_int4(codes), q_or)
    assert np.array_equal(s, s_or)


def _cat_T(X_cal, W, k, dtype):
    S = o.second_moment(X_cal)
    return o.round_storage(o.cat_transform(S, W, k), dtype)


@pytest.mark.parametrize("k", [32, 64, 128, 256, 512])
def test_transform_quant_cat_bf16(k):
    say(f"tq CAT bf16 k={k}")
    cfg = wl.get_config("attn4096", d_in=1024, d_out=512, k=k, n_cal=4096, n=257)
    lay = wl.make_layer(cfg, seed=k)
    X = lay["X"].astype(np.float64)
    X[5] = 0.0                                   # a zero token row
    T = _cat_T(lay["X_cal"], lay["W"], k, "bf16")
    codes, s = _tq_gpu(X, T, k, "bf16", "bf16")
    _, _, s_or = check_codes(codes, X, T, label=f"k={k}")
    _check_scales(s, s_or, f"k={k}")
    assert s[5] == 0 and not codes[5].any()


def test_transform_quant_tiny_fp32_config():
    say("tq tiny fp32 k=32")
    cfg = wl.get_config("tiny")
    lay = wl.make_layer(cfg, seed=0)
    X = lay["X"].astype(np.float64)
    T = _cat_T(lay["X_cal"], lay["W"], cfg.k, "f32")
    codes, s = _tq_gpu(X, T, cfg.k, "f32", "f32")
    _, _, s_or = check_codes(codes, X, T, label="tiny")
    _check_scales(s, s_or, "tiny")


@pytest.mark.parametrize("x_dtype,t_dtype,k,n", [
    ("bf16", "f32", 64, 129), ("f32", "bf16", 64, 129), ("bf16", "bf16", 16, 70),
    ("bf16", "bf16", 1, 33), ("f32", "f32", 8, 1), ("bf16", "bf16", 128, 1),
])
def test_transform_quant_other_paths(x_dtype, t_dtype, k, n):
    say(f"tq {x_dtype}/{t_dtype} k={k} n={n}")
    d = 256
    rng = np.random.default_rng(k + n)
    Xf = (rng.standard_normal((n, d)) * np.exp(rng.standard_normal(d))).astype(np.float32)
    X = o.round_storage(Xf, x_dtype)
    W = rng.standard_normal((96, d))
    T = _cat_T(Xf[:, :] if n > 8 else rng.standard_normal((512, d)), W, k, t_dtype)
    codes, s = _tq_gpu(X, T, k, x_dtype, t_dtype)
    _, _, s_or = check_codes(codes, X, T, label=f"{x_dtype}/{t_dtype} k={k}")
    _check_scales(s, s_or, f"{x_dtype}/{t_dtype} k={k}")


@pytest.mark.parametrize("x_dtype,t_dtype,k,bits", [
    ("f32", "bf16", 64, 8), ("bf16", "f32", 256, 4), ("bf16", "f32", 512, 6),
    ("f32", "f32", 512, 8), ("f32", "f32", 16, 4),
])
def test_transform_quant_fp32_operands_cancelling_sums(x_dtype, t_dtype, k, bits):
    # the vector-ALU path (an fp32 operand): blocks with k up to 512 and
    # rows whose block sums cancel heavily (each even row made nearly
    # orthogonal to the first row of every T_b), where an fp32 running sum
    # can move a code across a rounding boundary or the row maximum by more
    # than 1e-6; the kernel's sums must keep codes to the tie rule and s_x
    # within 1e-6, and exact on almost every token
    say(f"tq {x_dtype}/{t_dtype} k={k} bits={bits} cancelling sums")
    rng = np.random.default_rng(k + bits)
    n, d = 160, 2 * k if k >= 256 else 8 * k
    Xf = (rng.standard_normal((n, d)) * np.exp(0.7 * rng.standard_normal(d))).astype(np.float32)
    T = o.round_storage(rng.standard_normal((d // k, k, k)) / np.sqrt(k), t_dtype)
    for t in range(0, n, 2):
        for b in range(d // k):
            sl = slice(b * k, (b + 1) * k)
            x, w = Xf[t, sl].astype(np.float64), T[b][0].astype(np.float64)
            Xf[t, sl] = (x - (x @ w) / (w @ w) * w + 1e-4 * rng.standard_normal(k)).astype(np.float32)
    X = o.round_storage(Xf, x_dtype)
    torch = torch_mod()
    codes = torch.empty((n, d // 2 if bits == 4 else d),
                        dtype=torch.uint8 if bits == 4 else torch.int8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(16, cat.cat_transform_quant_workspace_bytes(n, d, k)), dtype=torch.uint8,
                     device="cuda")
    cat.cat_transform_quant(dev(X, x_dtype), dev(T, t_dtype), k, codes, s_x, ws, bits=bits)
    s = host(s_x)
    _, _, s_or = check_codes(host(codes), X, T, bits=bits, label=f"cancelling k={k} bits={bits}")
    _check_scales(s, s_or, f"cancelling k={k} bits={bits}")
    assert np.mean(s == s_or) >= 0.99


# ------------------------------------------ single-pass transform+quant
# k = 128 with d a multiple of 4096 runs the single-pass kernel, which
# exchanges per-block row maxima between workgroups through the workspace.

def _rand_T(d, k, seed):
    rng = np.random.default_rng(seed)
    return o.round_storage(rng.standard_normal((d // k, k, k)) / np.sqrt(k), "bf16")


def _wide_X(n, d, seed):
    # mlp_up-structured activations, tiled or cut to width d
    X = _mlp_up_X(n, seed)
    return np.tile(X, (1, (d + 4095) // 4096))[:, :d].copy() if d != 4096 else X


def _mlp_up_X(n, seed):
    cfg = wl.get_config("mlp_up", n=n, n_cal=16)
    return wl.make_layer(cfg, seed=seed, with_cal=False, with_weights=False)["X"].astype(np.float64)


@pytest.mark.parametrize("n", [1, 300, 2049])
def test_transform_quant_single_pass(n):
    say(f"tq single pass d=4096 k=128 n={n}")
    X = _mlp_up_X(n, seed=n)
    if n > 1:
        X[n // 2] = 0.0                           # a zero token row
    T = _rand_T(4096, 128, seed=1)
    codes, s = _tq_gpu(X, T, 128, "bf16", "bf16")
    _, _, s_or = check_codes(codes, X, T, label=f"single pass n={n}")
    _check_scales(s, s_or, f"single pass n={n}")
    if n > 1:
        assert s[n // 2] == 0 and not codes[n // 2].any()


@pytest.mark.parametrize("d,n", [(128, 777), (1024, 65), (2048, 1000), (8192, 300), (8192, 4097)])
def test_transform_quant_k128_other_widths(d, n):
    # k = 128 at widths other than the single-pass one (two passes), from
    # one 128-channel block to the stress layer's 8192
    say(f"tq k=128 d={d} n={n}")
    rng = np.random.default_rng(d + n)
    X = o.round_storage(rng.standard_normal((n, d)) * np.exp(rng.standard_normal(d)), "bf16")
    X[n // 3] = 0.0
    T = _rand_T(d, 128, seed=d)
    codes, s = _tq_gpu(X, T, 128, "bf16", "bf16")
    _, _, s_or = check_codes(codes, X, T, label=f"k=128 d={d} n={n}")
    _check_scales(s, s_or, f"k=128 d={d} n={n}")
    assert s[n // 3] == 0 and not codes[n // 3].any()


@pytest.mark.parametrize("d,k,n", [
    (14336, 256, 300), (8192, 256, 97), (768, 32, 65), (256, 32, 1), (2048, 64, 130),
    (640, 128, 300), (384, 64, 129), (2048, 512, 1000), (4096, 512, 33),
])
def test_transform_quant_two_pass_shapes(d, k, n):
    # bf16 two-pass paths: 256-channel group kernels (k <= 256, d a multiple
    # of 256; the mlp_down width with a ragged last tile), the ring and
    # small-block kernels they leave to (d = 640, 384), and k = 512 ring
    # workgroups paired on one XCD
    say(f"tq two-pass d={d} k={k} n={n}")
    rng = np.random.default_rng(3 * d + k + n)
    X = o.round_storage(rng.standard_normal((n, d)) * np.exp(rng.standard_normal(d)), "bf16")
    if n > 2:
        X[n // 2] = 0.0
    T = _rand_T(d, k, seed=d + k)
    codes, s = _tq_gpu(X, T, k, "bf16", "bf16")
    _, _, s_or = check_codes(codes, X, T, label=f"two-pass d={d} k={k} n={n}")
    _check_scales(s, s_or, f"two-pass d={d} k={k} n={n}")
    if n > 2:
        assert s[n // 2] == 0 and not codes[n // 2].any()


@pytest.mark.parametrize("d,n", [(4096, 192), (4096, 512), (4096, 2561), (4096, 3135), (4096, 3584),
                                 (8192, 1537), (2048, 6145)])
def test_transform_quant_single_pass_tiles_per_workgroup(d, n):
    # token counts that give each workgroup 1 to 7 tiles of 64 tokens, on
    # both sides of the exchange lag of 6 steps: calls that are all ramp,
    # and token-tile rows of unequal length (the first row one tile longer)
    say(f"tq single pass d={d} k=128 n={n} (tiles per workgroup)")
    X = _wide_X(n, d, seed=5 * n + d)
    X[n - 1] = 0.0                                # a zero token row in the last tile
    T = _rand_T(d, 128, seed=d + 7)
    codes, s = _tq_gpu(X, T, 128, "bf16", "bf16")
    _, _, s_or = check_codes(codes, X, T, label=f"single pass d={d} n={n}")
    _check_scales(s, s_or, f"single pass d={d} n={n}")
    assert s[n - 1] == 0 and not codes[n - 1].any()


@pytest.mark.parametrize("d,n", [(8192, 1), (8192, 65), (8192, 2049), (2048, 1), (2048, 300),
                                 (2048, 4097)])
def test_transform_quant_single_pass_other_widths(d, n):
    # the single-pass kernel with 64 and 16 blocks per token-tile row (one
    # and four owned tokens per workgroup and tile)
    say(f"tq single pass d={d} k=128 n={n}")
    X = _wide_X(n, d, seed=n + d)
    if n > 2:
        X[n // 2] = 0.0
    T = _rand_T(d, 128, seed=d)
    codes, s = _tq_gpu(X, T, 128, "bf16", "bf16")
    _, _, s_or = check_codes(codes, X, T, label=f"single pass d={d} n={n}")
    _check_scales(s, s_or, f"single pass d={d} n={n}")
    if n > 2:
        assert s[n // 2] == 0 and not codes[n // 2].any()


def test_transform_quant_single_pass_stress_full_size():
    # 16384 tokens x 8192 channels, the stress layer's k = 128 shape
    say("tq single pass stress 16384 x 8192")
    cfg = wl.get_config("stress", n=16384, n_cal=16, k=128)
    X = wl.make_layer(cfg, seed=0, with_cal=False, with_weights=False)["X"].astype(np.float64)
    T = _rand_T(8192, 128, seed=7)
    codes, s = _tq_gpu(X, T, 128, "bf16", "bf16")
    _, _, s_or = check_codes(codes, X, T, label="stress full")
    _check_scales(s, s_or, "stress full")


def test_transform_quant_single_pass_mlp_up_full_size():
    # 8192 tokens x 4096 channels, the shape and launch the benchmark times
    say("tq single pass mlp_up 8192 x 4096")
    X = _mlp_up_X(8192, seed=0)
    T = _rand_T(4096, 128, seed=2)
    codes, s = _tq_gpu(X, T, 128, "bf16", "bf16")
    _, _, s_or = check_codes(codes, X, T, label="mlp_up full")
    _check_scales(s, s_or, "mlp_up full")


def test_transform_quant_workspace_reuse_across_paths():
    # One workspace through single-pass, two-pass and single-pass calls on
    # different data: words left by earlier calls must never pass for the
    # current call's.
    say("tq workspace reuse: single pass / two pass / single pass at two widths")
    torch = torch_mod()
    n = 300
    wsb = max(cat.cat_transform_quant_workspace_bytes(n, 4096, 128),
              cat.cat_transform_quant_workspace_bytes(n, 1024, 128))
    ws = torch.zeros(wsb, dtype=torch.uint8, device="cuda")
    T4 = _rand_T(4096, 128, seed=3)
    T1 = _rand_T(1024, 128, seed=4)
    T8 = _rand_T(8192, 128, seed=5)
    wsb = max(wsb, cat.cat_transform_quant_workspace_bytes(n, 8192, 128))
    ws = torch.zeros(wsb, dtype=torch.uint8, device="cuda")
    cases = [(_mlp_up_X(n, seed=10), T4), (_mlp_up_X(n, seed=11)[:, :1024].copy(), T1),
             (_wide_X(n, 8192, seed=13), T8), (_mlp_up_X(n, seed=12) * 2.0 ** -6, T4),
             (_mlp_up_X(n, seed=10), T4)]
    first = None
    for i, (X, T) in enumerate(cases):
        d = X.shape[1]
        codes = torch.empty((n, d // 2), dtype=torch.uint8, device="cuda")
        s_x = torch.empty(n, dtype=torch.float32, device="cuda")
        # the single-pass kernel's bounded waits record a timeout in the word
        # at cat_transform_quant_flag_offset of the call's shape (wider calls
        # put exchange words where a narrower call's flag sits, so each call
        # clears and checks its own)
        fo = cat.cat_transform_quant_flag_offset(n, d, 128)
        ws[fo:fo + 4].zero_()
        cat.cat_transform_quant(dev(X, "bf16"), dev(T, "bf16"), 128, codes, s_x, ws)
        c, s = host(codes), host(s_x)
        assert int(host(ws[fo:fo + 4].view(torch.int32))[0]) == 0, f"timeout flag, call {i}"
        _, _, s_or = check_codes(c, X, T, label=f"reuse call {i}")
        _check_scales(s, s_or, f"reuse call {i}")
        if i == 0:
            first = (c, s)
    assert np.array_equal(first[0], c) and np.array_equal(first[1], s)


@pytest.mark.parametrize("d", [4096, 8192, 2048])
def test_transform_quant_graph_replays_see_fresh_inputs(d):
    # A captured single-pass call replayed with new activations each time:
    # every replay must publish under a tag of its own (made on the device),
    # and eager calls on the same workspace in between (host tags) must not
    # mix with it.  The workspace starts with whatever memory holds.
    say(f"tq graph capture d={d}: 4 replays with new X, eager calls between")
    torch = torch_mod()
    n, k = 300, 128
    T = _rand_T(d, k, seed=21)
    dT = dev(T, "bf16")
    Xs = [_wide_X(n, d, seed=30 + i) for i in range(4)]
    Xs[2] = Xs[2] * 2.0 ** -6
    dX = dev(Xs[0], "bf16")
    wsb = cat.cat_transform_quant_workspace_bytes(n, d, k)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    fo = cat.cat_transform_quant_flag_offset(n, d, k)
    ws[fo:fo + 4].zero_()             # only the timeout word, to read it afterwards
    codes = torch.empty((n, d // 2), dtype=torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    cat.cat_transform_quant(dX, dT, k, codes, s_x, ws)      # eager warm-up
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.graph(g, stream=side):
        cat.cat_transform_quant(dX, dT, k, codes, s_x, ws)
    codes_e = torch.empty_like(codes)
    s_x_e = torch.empty_like(s_x)
    for i, X in enumerate(Xs):
        dX.copy_(dev(X, "bf16"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        c, sx = host(codes), host(s_x)
        _, _, s_or = check_codes(c, X, T, label=f"replay {i}")
        _check_scales(sx, s_or, f"replay {i}")
        cat.cat_transform_quant(dX, dT, k, codes_e, s_x_e, ws)   # eager, same workspace
        torch.cuda.synchronize()
        assert np.array_equal(host(codes_e), c) and np.array_equal(host(s_x_e), sx)
    assert int(host(ws[fo:fo + 4].view(torch.int32))[0]) == 0


# ------------------------------------------------------- second moment
def _cov_gpu(X, dtype, mode, k, acc0=None, splits=None):
    torch = torch_mod()
    n, d = X.shape
    shape = (d, d) if mode == B.CAT_COV_FULL else (d // k, k, k)
    acc = torch.zeros(shape, dtype=torch.float32, device="cuda") if acc0 is None else acc0
    dX = dev(X, dtype)
    bounds = [0] + list(splits or []) + [n]
    for a, b in zip(bounds[:-1], bounds[1:]):
        cat.cat_cov_accumulate(dX[a:b], acc, mode, k)
    return host(acc)


def _blocks(S, k):
    d = S.shape[0]
    return np.stack([S[b * k:(b + 1) * k, b * k:(b + 1) * k] for b in range(d // k)])


def _assert_symmetric(acc):
    # a diagonal tile is computed as a full square, whose two triangles may
    # round their sums differently: equal to within a few ulp
    asym = np.max(np.abs(acc - acc.T))
    assert asym <= 4e-7 * max(1.0, float(np.max(np.abs(acc))))


@pytest.mark.parametrize("d,n,dtype", [(256, 5000, "bf16"), (320, 1000, "bf16"),
                                       (256, 2048, "f32"), (96, 300, "bf16"),
                                       (1024, 3001, "bf16"), (768, 40, "bf16"),
                                       (256, 1, "bf16"), (512, 17, "bf16")])
def test_cov_full_matches_oracle(d, n, dtype):
    say(f"cov full d={d} n={n} {dtype}")
    cfg = wl.get_config("attn4096", d_in=d, d_out=d, n_cal=n, n=1)
    X = wl.make_layer(cfg, seed=d + n, with_eval=False, with_weights=False)["X_cal"]
    X = o.round_storage(X, dtype)
    acc = _cov_gpu(X, dtype, B.CAT_COV_FULL, 1)
    ref = o.second_moment_sum(X)
    err = rel_fro(acc, ref)
    say(f"  rel fro {err:.2e}")
    assert err <= 1e-5
    _assert_symmetric(acc)


def test_cov_full_size_mlp_up_batch():
    """The 4096-channel full matrix over one 8192-token mlp_up batch (the
    shape the benchmark times), accumulated onto a non-zero symmetric start."""
    say("cov full 4096 x 4096, 8192 tokens")
    torch = torch_mod()
    cfg = wl.get_config("mlp_up", n_cal=8192, n=1)
    X = wl.make_layer(cfg, seed=5, with_eval=False, with_weights=False)["X_cal"]
    start = wl.random_spd(256, seed=3)
    S0 = np.kron(np.eye(16), start).astype(np.float32)
    acc0 = torch.from_numpy(S0).cuda()
    acc = _cov_gpu(X, "bf16", B.CAT_COV_FULL, 1, acc0=acc0)
    ref = S0.astype(np.float64) + o.second_moment_sum(X)
    err = rel_fro(acc, ref)
    say(f"  rel fro {err:.2e}")
    assert err <= 1e-5
    _assert_symmetric(acc)


@pytest.mark.parametrize("k,dtype", [(64, "bf16"), (128, "bf16"), (256, "bf16"), (32, "bf16"),
                                     (32, "f32"), (512, "bf16")])
def test_cov_block_diag_matches_oracle(k, dtype):
    say(f"cov block k={k} {dtype}")
    d, n = (1024 if k == 512 else 512), 4500
    cfg = wl.get_config("attn4096", d_in=d, d_out=d, n_cal=n, n=1)
    X = o.round_storage(wl.make_layer(cfg, seed=k, with_eval=False, with_weights=False)["X_cal"],
                        dtype)
    acc = _cov_gpu(X, dtype, B.CAT_COV_BLOCK_DIAG, k)
    ref = _blocks(o.second_moment_sum(X), k)
    err = rel_fro(acc, ref)
    say(f"  rel fro {err:.2e}")
    assert err <= 1e-5


@pytest.mark.parametrize("d,k,n", [(320, 64, 3001), (384, 128, 700), (768, 64, 33),
                                   (256, 128, 1), (512, 32, 8193)])
def test_cov_block_diag_shapes(d, k, n):
    """Blocks of 32-128 channels: whole 256-channel groups (d % 256 == 0) run
    packed through the 256-tile kernel, other widths through the 128/64-tile
    kernel; ragged token counts, one token, and a batch over 8192 tokens
    (two launches)."""
    say(f"cov block d={d} k={k} n={n}")
    cfg = wl.get_config("attn4096", d_in=d, d_out=d, n_cal=n, n=1)
    X = o.round_storage(wl.make_layer(cfg, seed=d + k + n, with_eval=False,
                                      with_weights=False)["X_cal"], "bf16")
    acc = _cov_gpu(X, "bf16", B.CAT_COV_BLOCK_DIAG, k)
    ref = _blocks(o.second_moment_sum(X), k)
    err = rel_fro(acc, ref)
    say(f"  rel fro {err:.2e}")
    assert err <= 1e-5


@pytest.mark.parametrize("name,k", [("mlp_up", 128), ("stress", 64)])
def test_cov_block_diag_full_size_batch(name, k):
    """Calibration blocks at layer width over one 8192-token batch, onto a
    non-zero start (the packed 256-channel groups)."""
    torch = torch_mod()
    cfg = wl.get_config(name, n_cal=8192, n=1)
    d = cfg.d_in
    say(f"cov block full size {name} d={d} k={k}")
    X = wl.make_layer(cfg, seed=7, with_eval=False, with_weights=False)["X_cal"]
    start = wl.random_spd(k, seed=4).astype(np.float32)
    S0 = np.broadcast_to(start, (d // k, k, k)).copy()
    acc0 = torch.from_numpy(S0).cuda()
    acc = _cov_gpu(X, "bf16", B.CAT_COV_BLOCK_DIAG, k, acc0=acc0)
    ref = S0.astype(np.float64) + np.stack(
        [o.second_moment_sum(X[:, b * k:(b + 1) * k]) for b in range(d // k)])
    err = rel_fro(acc, ref)
    say(f"  rel fro {err:.2e}")
    assert err <= 1e-5


@pytest.mark.parametrize("mode,k,d,n,dtype,seed", [
    (B.CAT_COV_BLOCK_DIAG, 1, 512, 3000, "bf16", 122),
    (B.CAT_COV_BLOCK_DIAG, 16, 512, 5000, "bf16", 92),
    (B.CAT_COV_FULL, 1, 200, 5000, "f32", 7),
])
def test_cov_heavy_tailed_columns(mode, k, d, n, dtype, seed):
    # Student-t (two degrees of freedom) columns on the vector-ALU path
    # (blocks under 64 channels, fp32 X): sums of squares whose terms span
    # many orders of magnitude.  fp32 running sums left the k = 1 case of
    # seed 122 at 1.14e-5; the kernel's fp64 partials keep it near 1e-7
    say(f"cov heavy tails mode={mode} k={k} d={d} n={n} {dtype}")
    rng = np.random.default_rng(seed)
    X = o.round_storage((rng.standard_t(2, (n, d)) * np.exp(0.7 * rng.standard_normal(d))
                         ).astype(np.float32), dtype)
    acc = _cov_gpu(X, dtype, mode, k)
    S = o.second_moment_sum(X)
    ref = S if mode == B.CAT_COV_FULL else _blocks(S, k)
    err = rel_fro(acc, ref)
    say(f"  rel Frobenius {err:.2e}")
    assert err <= 1e-5
    assert err <= 1e-6


def test_cov_split_batches_equal_one_shot():
    say("cov split batches")
    cfg = wl.get_config("attn4096", d_in=256, d_out=256, n_cal=3000, n=1)
    X = o.round_storage(wl.make_layer(cfg, seed=11, with_eval=False,
                                      with_weights=False)["X_cal"], "bf16")
    one = _cov_gpu(X, "bf16", B.CAT_COV_FULL, 1)
    split = _cov_gpu(X, "bf16", B.CAT_COV_FULL, 1, splits=[1, 700, 2001])
    assert rel_fro(split, one) <= 1e-6
    assert rel_fro(split, o.second_moment_sum(X)) <= 1e-5


# ------------------------------------------------------------ end to end
@pytest.mark.parametrize("transform", ["I", "H", "CAT"])
def test_end_to_end_tiny_layer_sqnr(transform):
    """C1 (tiny, fp32): GPU Sigma_x -> host transform -> GPU transform+quant
    -> GPU W4A4 GEMM -> GPU SQNR, against the oracle's own chain from the
    same generator arrays; SQNR within 0.05 dB."""
    torch = torch_mod()
    say(f"end-to-end tiny T={transform}")
    cfg = wl.get_config("tiny")
    lay = wl.make_layer(cfg, seed=0)
    Xc, X, W = lay["X_cal"], lay["X"], lay["W"]
    k, d = cfg.k, cfg.d_in
    flags = {"I": 0, "H": B.CAT_BUILD_HADAMARD, "CAT": B.CAT_BUILD_CAT}[transform]
    # GPU calibration (block-diagonal second moment)
    acc = torch.zeros((d // k, k, k), dtype=torch.float32, device="cuda")
    cat.cat_cov_accumulate(dev(Xc, "f32"), acc, B.CAT_COV_BLOCK_DIAG, k)
    sx_blocks = host(acc).astype(np.float64) / cfg.n_cal
    T, _, Wp = cat.cat_build_transform(sx_blocks, W, k, flags, B.CAT_F32)
    cw, sw = cat.cat_quantize_weights(Wp, 4)
    n = X.shape[0]
    codes = torch.empty((n, d // 2), dtype=torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(cat.cat_transform_quant_workspace_bytes(n, d, k), dtype=torch.uint8,
                     device="cuda")
    cat.cat_transform_quant(dev(X, "f32"), dev(T, "f32"), k, codes, s_x, ws)
    yt = torch.empty((n, cfg.d_out), dtype=torch.float32, device="cuda")
    cat.cat_w4a4_linear(codes, s_x, dev(cw, "u8"), dev(sw, "f32"), yt)
    y = o.reference_output(X, W).astype(np.float32)
    sws = torch.empty(cat.cat_sqnr_workspace_bytes(y.size), dtype=torch.uint8, device="cuda")
    out = torch.empty(3, dtype=torch.float64, device="cuda")
    cat.cat_sqnr(dev(y, "f32"), yt, sws, out)
    gpu_db = float(host(out)[2])
    # oracle chain
    if transform == "I":
        To = np.stack([np.eye(k)] * (d // k))
    elif transform == "H":
        To = o.cat_transform(None, W, k, use_alignment=False)
    else:
        To = o.cat_transform(o.second_moment(Xc), W, k)
    To = o.round_storage(To, "f32")
    fw = o.quantized_forward(X.astype(np.float64), To, o.transform_weights(W, To), 4)
    or_db = o.sqnr(y, fw["y_tilde"])[2]
    say(f"  SQNR gpu {gpu_db:.4f} dB, oracle {or_db:.4f} dB")
    assert abs(gpu_db - or_db) <= 0.05


# ------------------------------------------- device addresses above 2^31
def _view_with_bit31(torch, nbytes):
    """A uint8 device view of `nbytes` whose address has bit 31 of its low
    32-bit word set (the kernels take wave-uniform 64-bit base addresses
    apart into 32-bit halves; this catches a sign-extended low half)."""
    buf = torch.empty((1 << 31) + nbytes + 4096, dtype=torch.uint8, device="cuda")
    base = buf.data_ptr()
    off = 0 if base & 0x80000000 else (0x80000000 - (base & 0xFFFFFFFF)) % (1 << 32)
    off = (off + 15) // 16 * 16
    v = buf[off:off + nbytes]
    assert v.data_ptr() & 0x80000000 and v.data_ptr() % 16 == 0
    return buf, v


def test_inputs_at_addresses_with_bit31_set():
    say("cov / transform_quant / w4a4 on inputs at addresses with bit 31 set")
    torch = torch_mod()
    n, d, k = 300, 512, 128
    cfg = wl.get_config("attn4096", d_in=d, d_out=d, n_cal=n, n=1)
    X = o.round_storage(wl.make_layer(cfg, seed=31, with_eval=False, with_weights=False)["X_cal"],
                        "bf16")
    xbits = torch.from_numpy(wl.to_bf16_bits(X).view(np.uint8).reshape(-1).copy())
    keep, xv = _view_with_bit31(torch, xbits.numel())
    xv.copy_(xbits.cuda())
    dX = xv.view(torch.bfloat16).view(n, d)
    acc = torch.zeros((d, d), dtype=torch.float32, device="cuda")
    cat.cat_cov_accumulate(dX, acc, B.CAT_COV_FULL, 1)
    assert rel_fro(host(acc), o.second_moment_sum(X)) <= 1e-5
    T = _cat_T(X, wl.random_bf16_matrix(d, d, seed=2, scale=0.05), k, "bf16")
    codes, _ = _tq_gpu_from_device(dX, T, k)
    _, _, _ = check_codes(codes, X, T, label="bit31 tq")
    qw = wl.random_codes(256, d, seed=4)
    pw = o.pack_int4(qw)
    keep2, wv = _view_with_bit31(torch, pw.size)
    wv.copy_(torch.from_numpy(pw.reshape(-1).copy()).cuda())
    cw = wv.view(256, d // 2)
    sw = torch.rand(256, device="cuda") + 0.5
    cx = torch.from_numpy(codes).cuda()
    sx = torch.rand(n, device="cuda") + 0.5
    y = torch.empty((n, 256), dtype=torch.float32, device="cuda")
    acc_i = torch.empty((n, 256), dtype=torch.int32, device="cuda")
    cat.cat_w4a4_linear(cx, sx, cw, sw, y, acc_i)
    ref_acc, _ = o.w4a4_linear(o.unpack_int4(codes), host(sx), qw, host(sw))
    assert np.array_equal(host(acc_i), ref_acc.astype(np.int32))
    del keep, keep2


def test_single_pass_transform_quant_at_addresses_with_bit31_set():
    say("tq single pass on inputs at addresses with bit 31 set")
    torch = torch_mod()
    n, d, k = 300, 4096, 128
    X = o.round_storage(_mlp_up_X(n, seed=31), "bf16")
    xbits = torch.from_numpy(wl.to_bf16_bits(X).view(np.uint8).reshape(-1).copy())
    keep, xv = _view_with_bit31(torch, xbits.numel())
    xv.copy_(xbits.cuda())
    dX = xv.view(torch.bfloat16).view(n, d)
    T = _rand_T(d, k, seed=5)
    codes, s = _tq_gpu_from_device(dX, T, k)
    _, _, s_or = check_codes(codes, X, T, label="bit31 single pass")
    _check_scales(s, s_or, "bit31 single pass")
    del keep


def test_whole_step_graph_replays_match_eager():
    # transform_quant (single-pass shape), GEMM, SQNR and a full Sigma_x
    # accumulation captured once and replayed with new activations; every
    # replay must equal the same calls run eagerly, bit for bit (all four
    # kernels are deterministic)
    say("whole step under graph capture: 3 replays vs eager")
    torch = torch_mod()
    n, d_in, d_out, k = 512, 4096, 1024, 128
    T = _rand_T(d_in, k, seed=41)
    dT = dev(T, "bf16")
    qw = wl.random_codes(d_out, d_in, seed=42)
    rng = np.random.default_rng(43)
    dqw = dev(o.pack_int4(qw), "u8")
    dsw = dev(rng.uniform(0.01, 1.0, d_out).astype(np.float32), "f32")
    Xs = [_mlp_up_X(n, seed=50 + i) for i in range(3)]
    dy = dev(rng.standard_normal((n, d_out)).astype(np.float32), "f32")

    def buffers():
        return dict(
            codes=torch.empty((n, d_in // 2), dtype=torch.uint8, device="cuda"),
            s_x=torch.empty(n, dtype=torch.float32, device="cuda"),
            yt=torch.empty((n, d_out), dtype=torch.float32, device="cuda"),
            out=torch.empty(3, dtype=torch.float64, device="cuda"),
            acc=torch.zeros((d_in, d_in), dtype=torch.float32, device="cuda"),
            tq_ws=torch.empty(cat.cat_transform_quant_workspace_bytes(n, d_in, k),
                              dtype=torch.uint8, device="cuda"),
            sq_ws=torch.empty(cat.cat_sqnr_workspace_bytes(n * d_out), dtype=torch.uint8,
                              device="cuda"),
            cov_ws=torch.empty(max(16, cat.cat_cov_workspace_bytes(B.CAT_BF16, n, d_in,
                                                                   B.CAT_COV_FULL, 1)),
                               dtype=torch.uint8, device="cuda"))

    def step(dX, b):
        cat.cat_transform_quant(dX, dT, k, b["codes"], b["s_x"], b["tq_ws"])
        cat.cat_w4a4_linear(b["codes"], b["s_x"], dqw, dsw, b["yt"])
        cat.cat_sqnr(dy, b["yt"], b["sq_ws"], b["out"])
        cat.cat_cov_accumulate(dX, b["acc"], B.CAT_COV_FULL, 1, workspace=b["cov_ws"])

    dX = dev(Xs[0], "bf16")
    g_b, e_b = buffers(), buffers()
    step(dX, g_b)                      # warm-up
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.graph(graph, stream=side):
        step(dX, g_b)
    for i, X in enumerate(Xs):
        dX.copy_(dev(X, "bf16"))
        g_b["acc"].zero_()
        e_b["acc"].zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        step(dX, e_b)
        torch.cuda.synchronize()
        for key in ("codes", "s_x", "yt", "out", "acc"):
            assert torch.equal(g_b[key], e_b[key]), f"replay {i}: {key}"


@pytest.mark.parametrize("name,k", [("attn4096", 128), ("mlp_down", 256), ("stress", 128),
                                    ("stress", 512)])
def test_full_size_layer_shapes_sampled(name, k):
    # Every kernel at a layer's full dimensions and token counts, with the
    # layer's own activation structure; checked on samples the oracle
    # computes one by one (tokens, a 64 x 64 output block, a 64 x 64 block
    # of the second moment) and, for SQNR, on all entries in fp64 chunks.
    torch = torch_mod()
    cfg = wl.get_config(name, k=k)
    n, d_in, d_out = cfg.n, cfg.d_in, cfg.d_out
    say(f"full size {name}: {n} x {d_in} -> {d_out}, k={k}, n_cal={cfg.n_cal}")
    L = wl.make_layer(cfg, seed=7, with_weights=False)
    X_cal, X = L["X_cal"], L["X"]
    rng = np.random.default_rng(sum(map(ord, name)) + k)
    rows = np.unique(np.concatenate([rng.choice(n, 62, replace=False), [0, n - 1]]))

    # transform + quantize over all n tokens; sampled tokens against the oracle
    T = _rand_T(d_in, k, seed=k)
    dX = dev(X, "bf16")
    codes = torch.empty((n, d_in // 2), dtype=torch.uint8, device="cuda")
    s_x = torch.empty(n, dtype=torch.float32, device="cuda")
    ws = torch.empty(cat.cat_transform_quant_workspace_bytes(n, d_in, k), dtype=torch.uint8,
                     device="cuda")
    cat.cat_transform_quant(dX, dev(T, "bf16"), k, codes, s_x, ws)
    dr = torch.from_numpy(rows).cuda()
    c_rows, s_rows = host(codes[dr]), host(s_x[dr])
    _, _, s_or = check_codes(c_rows, X[rows].astype(np.float64), T, label=f"{name} tq rows")
    _check_scales(s_rows, s_or, f"{name} tq rows")

    # GEMM on those codes against random weight codes; sampled block exact
    qw = wl.random_codes(d_out, d_in, seed=k + 1)
    sw = rng.uniform(0.01, 1.0, d_out).astype(np.float32)
    dqw, dsw = dev(o.pack_int4(qw), "u8"), dev(sw, "f32")
    y = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    acc = torch.empty((n, d_out), dtype=torch.int32, device="cuda")
    cat.cat_w4a4_linear(codes, s_x, dqw, dsw, y, acc)
    cols = np.unique(np.concatenate([rng.choice(d_out, 62, replace=False), [0, d_out - 1]]))
    dc = torch.from_numpy(cols).cuda()
    acc_or, y_or = o.w4a4_linear(o.unpack_int4(c_rows), s_rows, qw[cols], sw[cols])
    assert np.array_equal(host(acc[dr][:, dc]), acc_or)
    assert np.array_equal(host(y[dr][:, dc]), y_or)
    y_fast = torch.empty_like(y)
    cat.cat_w4a4_linear(codes, s_x, dqw, dsw, y_fast)
    assert torch.equal(y_fast, y)
    del acc, y_fast

    # SQNR over all n x d_out entries; the oracle sums fp64 chunks
    g = torch.Generator(device="cuda")
    g.manual_seed(k)
    y_ref = y + 0.1 * torch.randn(y.shape, device="cuda", generator=g)
    out = torch.empty(3, dtype=torch.float64, device="cuda")
    sws = torch.empty(cat.cat_sqnr_workspace_bytes(y.numel()), dtype=torch.uint8, device="cuda")
    cat.cat_sqnr(y_ref, y, sws, out)
    S = E = 0.0
    for a in range(0, n, 2048):
        Sa, Ea, _ = o.sqnr(host(y_ref[a:a + 2048]), host(y[a:a + 2048]))
        S, E = S + Sa, E + Ea
    r = host(out)
    assert r[0] == pytest.approx(S, rel=1e-9) and r[1] == pytest.approx(E, rel=1e-9)
    assert abs(r[2] - 10.0 * np.log10(S / E)) < 1e-6
    del y, y_ref

    # full second moment over the n_cal calibration tokens; a sampled block
    # and exact symmetry
    dXc = dev(X_cal, "bf16")
    sacc = torch.zeros((d_in, d_in), dtype=torch.float32, device="cuda")
    cat.cat_cov_accumulate(dXc, sacc, B.CAT_COV_FULL, 1)
    I = np.sort(rng.choice(d_in, 64, replace=False))
    J = np.sort(rng.choice(d_in, 64, replace=False))
    ref = o.second_moment_sum(np.hstack([X_cal[:, I], X_cal[:, J]]))[:64, 64:]
    got = host(sacc[torch.from_numpy(I).cuda()][:, torch.from_numpy(J).cuda()])
    assert rel_fro(got, ref) <= 1e-5
    assert torch.equal(sacc, sacc.t())
