"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-types an oracle formula: each compares the oracle with a
library routine, a closed form from elsewhere, an invariant, a brute-force
search on tiny inputs or a value printed in the paper (tests/golden/).
"""
import json
import os

import numpy as np
import pytest
import scipy.linalg as sla

import workloads as wl
from oracle import cat_oracle as o

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_spd(rng, n, shift=0.1):
    a = rng.standard_normal((n, n))
    return a @ a.T + shift * np.eye(n)


def _act(rng, n, d, heavy=True):
    X = rng.standard_normal((n, d))
    if heavy:
        X *= np.exp(rng.standard_normal(d))[None, :]
    return X


# ------------------------------------------------------------- Sigma_x
def test_second_moment_matches_numpy_cov_identity():
    # E[x x^T] = Cov(x) + mu mu^T, with numpy's biased covariance.
    rng = np.random.default_rng(0)
    X = rng.standard_normal((777, 13)) + rng.standard_normal(13)[None, :]
    ref = np.cov(X, rowvar=False, bias=True) + np.outer(X.mean(0), X.mean(0))
    np.testing.assert_allclose(o.second_moment(X), ref, rtol=1e-12, atol=1e-12)


def test_second_moment_batch_split_equals_one_shot():
    rng = np.random.default_rng(1)
    X = rng.standard_normal((1000, 17))
    parts = sum(o.second_moment_sum(X[a:b]) for a, b in
                [(0, 1), (1, 333), (333, 1000)])
    np.testing.assert_allclose(parts, o.second_moment_sum(X), rtol=1e-13,
                               atol=1e-12)


def test_second_moment_of_scaled_basis_vectors_is_diagonal():
    c = np.array([3.0, -2.0, 0.5, 7.0])
    X = np.diag(c)                  # row i = c_i e_i
    S = o.second_moment_sum(X)
    assert np.array_equal(S, np.diag(c * c))


def test_second_moment_is_symmetric_psd():
    rng = np.random.default_rng(2)
    S = o.second_moment(rng.standard_normal((50, 20)))
    assert np.array_equal(S, S.T)
    assert np.linalg.eigvalsh(S).min() > -1e-12


# ----------------------------------------------------- geometric mean
def test_geometric_mean_2x2_closed_form():
    # Bhatia, Positive Definite Matrices, Prop. 4.1.12:
    # A # B = sqrt(ab) / sqrt(det(A/a + B/b)) (A/a + B/b), a = sqrt det A, ...
    rng = np.random.default_rng(3)
    for _ in range(20):
        A, B = _rand_spd(rng, 2), _rand_spd(rng, 2)
        a, b = np.sqrt(np.linalg.det(A)), np.sqrt(np.linalg.det(B))
        C = A / a + B / b
        ref = np.sqrt(a * b) / np.sqrt(np.linalg.det(C)) * C
        np.testing.assert_allclose(o.geometric_mean(A, B), ref, rtol=1e-11,
                                   atol=1e-12)


def test_geometric_mean_solves_riccati_and_is_symmetric():
    # A # B is the unique SPD X with X A^-1 X = B, and A # B = B # A.
    rng = np.random.default_rng(4)
    A, B = _rand_spd(rng, 9), _rand_spd(rng, 9)
    G = o.geometric_mean(A, B)
    assert np.linalg.eigvalsh(G).min() > 0
    np.testing.assert_allclose(G @ np.linalg.solve(A, G), B, rtol=1e-9,
                               atol=1e-9 * np.abs(B).max())
    np.testing.assert_allclose(G, o.geometric_mean(B, A), rtol=1e-9,
                               atol=1e-10 * np.abs(G).max())


def test_geometric_mean_commuting_case():
    a = np.array([1.0, 4.0, 0.25, 9.0])
    b = np.array([4.0, 1.0, 16.0, 1.0])
    G = o.geometric_mean(np.diag(a), np.diag(b))
    np.testing.assert_allclose(G, np.diag(np.sqrt(a * b)), atol=1e-14)


# ------------------------------------------------ optimal alignment
def test_optimal_alignment_beats_every_perturbation():
    # eq. 7: M_hat is the argmax of A(M x, W M^-1).
    rng = np.random.default_rng(5)
    X = _act(rng, 4000, 6)
    W = rng.standard_normal((10, 6))
    Sx, Sw = o.second_moment(X), W.T @ W
    M = o.optimal_alignment(Sx, Sw)
    best = o.alignment_from_moments(M @ Sx @ M.T, np.linalg.inv(M).T @ Sw @ np.linalg.inv(M))
    for _ in range(500):
        P = M + 0.05 * rng.standard_normal(M.shape) * np.abs(M).max()
        Pi = np.linalg.inv(P)
        a = o.alignment_from_moments(P @ Sx @ P.T, Pi.T @ Sw @ Pi)
        assert a <= best * (1 + 1e-12)


def test_optimal_alignment_reaches_svd_maximum():
    # The maximum alignment equals sum s^2 / (sum s)^2 for the singular
    # values s of W Sigma_x^(1/2) (eq. 9, corrected reading); computed here
    # with scipy's sqrtm and svd, independently of the oracle.
    rng = np.random.default_rng(6)
    X = _act(rng, 3000, 8)
    W = rng.standard_normal((12, 8)) * np.exp(rng.standard_normal(8))[None, :]
    Sx, Sw = o.second_moment(X), W.T @ W
    s = np.linalg.svd(W @ np.real(sla.sqrtm(Sx)), compute_uv=False)
    ref = np.sum(s ** 2) / np.sum(s) ** 2
    M = o.optimal_alignment(Sx, Sw)
    Mi = np.linalg.inv(M)
    got = o.alignment(X @ M.T, W @ Mi)
    assert got == pytest.approx(ref, rel=1e-10)
    assert o.max_alignment(Sx, Sw) == pytest.approx(ref, rel=1e-10)
    assert got >= o.alignment(X, W)


def test_optimal_alignment_with_rank_deficient_sigma_w():
    # fewer outputs (5) than channels (8): Sigma_w has rank 5.  G = M_hat^2 =
    # Sigma_w # Sigma_x^-1 still solves its Riccati equation G Sigma_x G =
    # Sigma_w (X B^-1 X = A for X = A # B), and M_hat Sigma_x M_hat has the
    # square roots of the spectrum of Sigma_x^(1/2) Sigma_w Sigma_x^(1/2)
    # (eq. 8), computed with scipy's sqrtm, independently of the oracle.
    # Three of those are zero; the eigenvalue floor of the inner square root
    # (EIG_FLOOR times the largest eigenvalue) sets them to
    # sqrt(EIG_FLOOR) times the largest.
    rng = np.random.default_rng(17)
    X = _act(rng, 3000, 8)
    W = rng.standard_normal((5, 8))
    Sx, Sw = o.second_moment(X), W.T @ W
    M = o.optimal_alignment(Sx, Sw)
    G = M @ M
    np.testing.assert_allclose(G @ Sx @ G, Sw, atol=1e-9 * np.abs(Sw).max())
    sxh = np.real(sla.sqrtm(Sx))
    ev = np.sort(np.sqrt(np.clip(np.linalg.eigvalsh(sxh @ Sw @ sxh), 0.0, None)))
    got = np.sort(np.linalg.eigvalsh(M @ Sx @ M))
    np.testing.assert_allclose(got[3:], ev[3:], rtol=1e-8)
    np.testing.assert_allclose(got[:3], np.sqrt(o.EIG_FLOOR) * ev[-1], rtol=1e-6)


def test_optimal_alignment_balance_identity():
    # eq. 8, first equality: M Sx M = M^-1 Sw M^-1; its spectrum is sqrt of
    # the spectrum of Sx^(1/2) Sw Sx^(1/2).
    rng = np.random.default_rng(7)
    X = _act(rng, 2000, 7)
    W = rng.standard_normal((9, 7))
    Sx, Sw = o.second_moment(X), W.T @ W
    M = o.optimal_alignment(Sx, Sw)
    Mi = np.linalg.inv(M)
    L, R = M @ Sx @ M, Mi @ Sw @ Mi
    np.testing.assert_allclose(L, R, rtol=1e-9, atol=1e-10 * np.abs(L).max())
    sxh = np.real(sla.sqrtm(Sx))
    ev = np.sqrt(np.linalg.eigvalsh(sxh @ Sw @ sxh))
    np.testing.assert_allclose(np.sort(np.linalg.eigvalsh(L)), np.sort(ev),
                               rtol=1e-8)


def test_k1_special_case_closed_form():
    # k = 1: M = diag(m) with m_i = (sum_j W_ji^2 / E[x_i^2])^(1/4), the
    # scalar geometric mean (Sec. 4, last paragraph, corrected reading).
    rng = np.random.default_rng(8)
    X = _act(rng, 1000, 16)
    W = rng.standard_normal((24, 16))
    T = o.cat_transform(o.second_moment(X), W, 1, use_hadamard=False)
    m = (np.sum(W ** 2, axis=0) / np.mean(X ** 2, axis=0)) ** 0.25
    np.testing.assert_allclose(T[:, 0, 0], m, rtol=1e-12)


# ------------------------------------------------------ Hadamard / blocks
@pytest.mark.parametrize("k", [1, 2, 8, 32, 128])
def test_hadamard_matches_scipy(k):
    H = o.hadamard(k)
    np.testing.assert_allclose(H, sla.hadamard(k) / np.sqrt(k), atol=0)
    np.testing.assert_allclose(H @ H.T, np.eye(k), atol=1e-14)


def test_block_cat_reaches_block_optimum_closed_form():
    # For block-diagonal M the best alignment is
    # Tr(Sw Sx) / (sum_b ||W_b Sx_b^(1/2)||_*)^2 (nuclear norms); derived
    # from eq. 7 applied per block plus Cauchy-Schwarz across blocks.
    rng = np.random.default_rng(9)
    d, k = 32, 8
    X = _act(rng, 5000, d)
    W = rng.standard_normal((40, d))
    Sx, Sw = o.second_moment(X), W.T @ W
    T = o.cat_transform(Sx, W, k, use_hadamard=True)
    Tfull = sla.block_diag(*T)
    got = o.alignment(X @ Tfull.T, W @ np.linalg.inv(Tfull))
    nuc = sum(np.linalg.svd(W[:, b * k:(b + 1) * k] @
                            np.real(sla.sqrtm(Sx[b * k:(b + 1) * k, b * k:(b + 1) * k])),
                            compute_uv=False).sum() for b in range(d // k))
    ref = np.trace(Sw @ Sx) / nuc ** 2
    assert got == pytest.approx(ref, rel=1e-9)
    # the Hadamard factor leaves the alignment unchanged (eq. 4)
    T0 = sla.block_diag(*o.cat_transform(Sx, W, k, use_hadamard=False))
    assert o.alignment(X @ T0.T, W @ np.linalg.inv(T0)) == pytest.approx(got, rel=1e-10)


def test_alignment_rotation_invariance():
    rng = np.random.default_rng(10)
    X, W = _act(rng, 500, 16), rng.standard_normal((20, 16))
    R, _ = np.linalg.qr(rng.standard_normal((16, 16)))
    assert o.alignment(X @ R.T, W @ R.T) == pytest.approx(o.alignment(X, W), rel=1e-12)


def test_transform_weights_preserves_function():
    rng = np.random.default_rng(11)
    d, k = 64, 16
    X = _act(rng, 300, d)
    W = rng.standard_normal((24, d))
    T = o.round_storage(o.cat_transform(o.second_moment(X), W, k), "bf16")
    Wp = o.transform_weights(W, T)
    Z = o.transform_rows(X, T)
    np.testing.assert_allclose(Z @ Wp.T, X @ W.T, rtol=1e-10,
                               atol=1e-10 * np.abs(X @ W.T).max())


# ------------------------------------------------------------ quantizer
def _golden_rtn():
    rows = []
    for line in open(os.path.join(GOLDEN, "rtn_examples.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        z, q, s = (p.split() for p in line.split(";"))
        rows.append((np.array(z, np.float32), np.array(q, np.int8), float(s[0])))
    return rows


def test_quantizer_hand_examples():
    for z, q, s in _golden_rtn():
        codes, scale = o.quantize_rows(z[None, :], 4)
        assert codes[0].tolist() == q.tolist(), (z, codes)
        assert float(scale[0]) == s


@pytest.mark.parametrize("bits", [4, 6, 8])
def test_quantizer_is_nearest_grid_point_brute_force(bits):
    # Every code is the nearest of the 2 qmax + 1 grid levels to
    # z * (qmax/amax) (brute-force argmin), ties aside; qmax = 7, 31, 127.
    qm = {4: 7, 6: 31, 8: 127}[bits]
    rng = np.random.default_rng(12)
    Z = (rng.standard_normal((64, 48)) * np.exp(rng.standard_normal(48))).astype(np.float32)
    codes, scale = o.quantize_rows(Z, bits)
    levels = np.arange(-qm, qm + 1)
    amax = np.abs(Z.astype(np.float64)).max(1)
    u = Z.astype(np.float64) * (qm / amax)[:, None]
    dist = np.abs(u[..., None] - levels[None, None, :])
    best = levels[np.argmin(dist, axis=-1)]
    near_tie = np.abs(np.abs(u - np.floor(u)) - 0.5) < 1e-5
    assert np.all((codes == best) | near_tie)
    # dequantization error within half a step
    err = np.abs(Z - codes * scale[:, None])
    assert np.all(err <= 0.5 * scale[:, None] * (1 + 1e-5))


@pytest.mark.parametrize("bits,qm", [(4, 7), (6, 31), (8, 127)])
def test_quantizer_extremes_and_range(bits, qm):
    rng = np.random.default_rng(13)
    Z = rng.standard_normal((32, 40)).astype(np.float32)
    codes, scale = o.quantize_rows(Z, bits)
    assert codes.min() >= -qm and codes.max() <= qm
    i = np.argmax(np.abs(Z), axis=1)
    assert np.all(np.abs(codes[np.arange(32), i]) == qm)
    z0, s0 = o.quantize_rows(np.zeros((2, 8), np.float32), bits)
    assert not z0.any() and not s0.any()


@pytest.mark.parametrize("bits", [4, 6, 8])
def test_quantizer_power_of_two_scale_invariance(bits):
    rng = np.random.default_rng(14)
    Z = rng.standard_normal((16, 32)).astype(np.float32)
    c0, s0 = o.quantize_rows(Z, bits)
    for m in (-7, -1, 3, 20):
        c, s = o.quantize_rows(Z * np.float32(2.0 ** m), bits)
        assert np.array_equal(c, c0)
        assert np.array_equal(s, (s0 * np.float32(2.0 ** m)).astype(np.float32))


@pytest.mark.parametrize("bits,qm", [(4, 7), (6, 31), (8, 127)])
def test_transform_quant_identity_is_plain_rtn(bits, qm):
    # T = I: codes are the nearest grid points of x itself (brute force).
    X = wl.random_bf16_matrix(40, 64, seed=15, scale=3.0).astype(np.float64)
    T = np.stack([np.eye(16)] * 4)
    codes, scale = o.transform_quant(X, T, bits)
    amax = np.abs(X).max(1)
    u = X * (qm / amax)[:, None]
    levels = np.arange(-qm, qm + 1)
    best = levels[np.argmin(np.abs(u[..., None] - levels), axis=-1)]
    near_tie = np.abs(np.abs(u - np.floor(u)) - 0.5) < 1e-5
    assert np.all((codes == best) | near_tie)
    np.testing.assert_allclose(scale, amax / qm, rtol=1e-7)


def test_transform_quant_orthogonal_T_preserves_unquantized_output():
    rng = np.random.default_rng(16)
    d, k = 64, 32
    X = rng.standard_normal((20, d))
    W = rng.standard_normal((8, d))
    T = np.stack([o.hadamard(k)] * (d // k))
    Wp = o.transform_weights(W, T)
    np.testing.assert_allclose(Wp, W @ sla.block_diag(*T).T, atol=1e-13)
    np.testing.assert_allclose(o.transform_rows(X, T) @ Wp.T, X @ W.T,
                               atol=1e-12 * np.abs(X @ W.T).max())


# -------------------------------------------------------------- packing
def test_pack_int4_hand_bytes():
    for line in open(os.path.join(GOLDEN, "int4_packing.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        a, b, h = line.split()
        packed = o.pack_int4(np.array([[int(a), int(b)]]))
        assert packed[0, 0] == int(h, 16), line
        assert o.unpack_int4(packed)[0].tolist() == [int(a), int(b)]


def test_pack_roundtrip_all_pairs():
    v = np.arange(-7, 8)
    pairs = np.array([[a, b] for a in v for b in v])
    assert np.array_equal(o.unpack_int4(o.pack_int4(pairs)), pairs)


# ---------------------------------------------------------------- GEMM
def test_w4a4_linear_brute_force_loops():
    qx = wl.random_codes(3, 10, seed=17)
    qw = wl.random_codes(4, 10, seed=18)
    sx = np.array([0.5, 0.25, 3.0], np.float32)
    sw = np.array([1.0, 0.125, 2.0, 0.75], np.float32)
    acc, y = o.w4a4_linear(qx, sx, qw, sw)
    for t in range(3):
        for j in range(4):
            ref = 0
            for i in range(10):
                ref += int(qx[t, i]) * int(qw[j, i])
            assert acc[t, j] == ref
            # power-of-two scales: the dequantized value is exact
            assert float(y[t, j]) == ref * float(sx[t]) * float(sw[j])


def test_linear_int8_codes_brute_force_loops():
    # 8-bit codes over a 4096-long reduction: sums reach 127^2 * 4096 > 2^24,
    # so acc is exact in int32 while its fp32 conversion rounds (to nearest
    # even, the conversion the dequantization starts from).
    qx = wl.random_codes(2, 4096, seed=23, qmax=127)
    qw = wl.random_codes(3, 4096, seed=24, qmax=127)
    qx[0] = 127
    qw[0] = 127
    sx = np.array([0.375, 1.5], np.float32)
    sw = np.array([0.5, 2.0, 0.0625], np.float32)
    acc, y = o.w4a4_linear(qx, sx, qw, sw)
    for t in range(2):
        for j in range(3):
            ref = sum(int(a) * int(b) for a, b in zip(qx[t], qw[j]))
            assert acc[t, j] == ref
            want = np.float32(np.float32(np.float32(ref) * sx[t]) * sw[j])
            assert y[t, j] == want
    assert acc[0, 0] == 127 * 127 * 4096 and acc[0, 0] > 2 ** 24


def test_w4a4_linear_equals_fake_quant_and_is_permutation_invariant():
    qx = wl.random_codes(16, 64, seed=19)
    qw = wl.random_codes(24, 64, seed=20)
    rng = np.random.default_rng(21)
    sx = rng.uniform(0.1, 2, 16).astype(np.float32)
    sw = rng.uniform(0.1, 2, 24).astype(np.float32)
    acc, y = o.w4a4_linear(qx, sx, qw, sw)
    fake = (sx[:, None] * qx.astype(np.float64)) @ (sw[:, None] * qw.astype(np.float64)).T
    np.testing.assert_allclose(y, fake, rtol=2e-7, atol=1e-6)
    p = rng.permutation(64)
    acc_p, _ = o.w4a4_linear(qx[:, p], sx, qw[:, p], sw)
    assert np.array_equal(acc, acc_p)


# ---------------------------------------------------------------- SQNR
def test_sqnr_hand_values():
    S, E, dB = o.sqnr([3.0, 4.0], [3.0, 4.5])
    assert (S, E) == (25.0, 0.25)
    assert dB == pytest.approx(20.0)
    S, E, dB = o.sqnr([1.0, -1.0], [1.0, -1.0])
    assert E == 0.0 and dB == np.inf


def _quantize_layer(X, W, bx, bw):
    qx, sx = o.quantize_rows(X.astype(np.float32), bx)
    qw, sw = o.quantize_rows(W.astype(np.float32), bw)
    return (qx * sx[:, None].astype(np.float64)), (qw * sw[:, None].astype(np.float64))


@pytest.mark.parametrize("bits", [4, 6, 8])
def test_sqnr_gaussian_matches_theorem_closed_form(bits):
    # On Gaussian data the uniform-noise model behind Lemmas 2.2/2.3 holds,
    # so brute-force SQNR must match Theorem 2.4 within 0.1 dB.
    rng = np.random.default_rng(22 + bits)
    d = 256
    X = rng.standard_normal((4096, d))
    W = rng.standard_normal((256, d)) / np.sqrt(d)
    Xq, Wq = _quantize_layer(X, W, bits, bits)
    y = X @ W.T
    _, _, joint = o.sqnr(y, Xq @ Wq.T)
    pred = o.to_db(o.theorem_2_4(X, W, bits, bits))
    assert joint == pytest.approx(pred, abs=0.1)
    # Lemma 2.1: joint ~ act-only || weight-only
    _, _, act = o.sqnr(y, Xq @ W.T)
    _, _, wgt = o.sqnr(y, X @ Wq.T)
    comp = o.to_db(o.parallel(10 ** (act / 10), 10 ** (wgt / 10)))
    assert joint == pytest.approx(comp, abs=0.1)
    # Lemmas 2.2 and 2.3 on their own
    assert act == pytest.approx(o.to_db(o.sqnr_act_only(X, W, bits)), abs=0.1)
    assert wgt == pytest.approx(o.to_db(o.sqnr_weight_only(X, W, bits)), abs=0.1)


def test_sqnr_gain_per_bit_matches_paper():
    g = json.load(open(os.path.join(GOLDEN, "paper_values.json")))
    rng = np.random.default_rng(30)
    X = rng.standard_normal((4096, 256))
    W = rng.standard_normal((256, 256)) / 16.0
    y = X @ W.T
    db = {}
    for b in (6, 7, 10):
        Xq, Wq = _quantize_layer(X, W, b, b)
        db[b] = o.sqnr(y, Xq @ Wq.T)[2]
    # about 6 dB per joint bit (factor 4) once the grid is fine
    assert db[7] - db[6] == pytest.approx(g["sqnr_gain_per_joint_bit"]["db"], abs=0.5)
    # weight-only SQNR: +4 weight bits shift it by about 24 dB
    w = {}
    for b in (4, 8):
        _, Wq = _quantize_layer(X, W, 8, b)
        w[b] = o.sqnr(y, X @ Wq.T)[2]
    assert w[8] - w[4] == pytest.approx(g["sqnr_gain_plus4_weight_bits_db"]["db"], abs=1.5)


def test_minimum_concentration_matches_paper():
    g = json.load(open(os.path.join(GOLDEN, "paper_values.json")))
    x = np.zeros((1, 32))
    x[0, 5] = -3.7
    sym = o.concentration_act(x)
    assert sym == g["min_concentration_symmetric"]["value"]
    assert o.to_db(sym) == pytest.approx(g["min_concentration_symmetric"]["db"], abs=0.05)
    assert o.concentration_weight(x) == g["min_concentration_symmetric"]["value"]
    xa = np.zeros((1, 32))
    xa[0, 1], xa[0, 9] = 2.5, -2.5
    asym = o.concentration_act(xa, asymmetric=True)
    assert asym == g["min_concentration_asymmetric"]["value"]
    assert o.to_db(asym) == pytest.approx(g["min_concentration_asymmetric"]["db"], abs=0.05)
    # nothing goes below the minimum
    rng = np.random.default_rng(31)
    Z = rng.standard_normal((200, 32)) ** 5
    for row in Z:
        assert o.concentration_act(row[None, :]) >= 0.25
        assert o.concentration_act(row[None, :], asymmetric=True) >= 0.5 - 1e-12


def test_concentration_and_alignment_are_scale_invariant():
    rng = np.random.default_rng(32)
    X, W = _act(rng, 300, 16), rng.standard_normal((12, 16))
    assert o.concentration_act(7.5 * X) == pytest.approx(o.concentration_act(X), rel=1e-12)
    assert o.concentration_weight(0.3 * W) == pytest.approx(o.concentration_weight(W), rel=1e-12)
    assert o.alignment(3 * X, 0.1 * W) == pytest.approx(o.alignment(X, W), rel=1e-12)


def test_cat_improves_sqnr_on_outlier_layer():
    # Qualitative claim (Sec. 4, Fig. 6): the CAT transform beats Hadamard,
    # which beats no transform, on an outlier-heavy layer.  Report-level
    # ordering only; no absolute value is printed in the paper.
    cfg = wl.get_config("tiny")
    lay = wl.make_layer(cfg, seed=0)
    X, Xc, W = lay["X"].astype(np.float64), lay["X_cal"], lay["W"].astype(np.float64)
    Sx = o.second_moment(Xc)
    y = o.reference_output(X, W)
    res = {}
    for name, T in [("I", np.stack([np.eye(cfg.k)] * (cfg.d_in // cfg.k))),
                    ("H", o.cat_transform(Sx, W, cfg.k, use_alignment=False)),
                    ("CAT", o.cat_transform(Sx, W, cfg.k))]:
        T = o.round_storage(T, "f32")
        fw = o.quantized_forward(X, T, o.transform_weights(W, T), 4)
        res[name] = o.sqnr(y, fw["y_tilde"])[2]
    assert res["CAT"] > res["H"] + 3.0 > res["I"] + 3.0


# ------------------------------------------------- asymmetric activations
@pytest.mark.parametrize("bits", [4, 8])
def test_asym_quantizer_is_nearest_affine_grid_point_brute_force(bits):
    # Every code is the nearest of the 2^b levels min + s l (l = 0 .. 2^b - 1)
    # to z (brute-force argmin), ties aside; error within half a step.
    L = (1 << bits) - 1
    rng = np.random.default_rng(31 + bits)
    Z = (rng.standard_normal((64, 48)) * np.exp(rng.standard_normal(48)) +
         rng.standard_normal((64, 1)) * 3).astype(np.float32)
    q, s, m = o.quantize_rows_asym(Z, bits)
    Zd = Z.astype(np.float64)
    r = Zd.max(1) - Zd.min(1)
    u = (Zd - Zd.min(1)[:, None]) * (L / r)[:, None]
    levels = np.arange(L + 1)
    best = levels[np.argmin(np.abs(u[..., None] - levels), axis=-1)]
    near_tie = np.abs(np.abs(u - np.floor(u)) - 0.5) < 1e-5
    assert np.all((q == best) | near_tie)
    assert q.min() >= 0 and q.max() <= L
    err = np.abs(Zd - (q * s[:, None].astype(np.float64) + m[:, None]))
    assert np.all(err <= 0.5 * s[:, None] * (1 + 1e-5) + 1e-6 * np.abs(Zd))


def test_asym_quantizer_extremes_and_constant_rows():
    rng = np.random.default_rng(33)
    Z = rng.standard_normal((32, 40)).astype(np.float32)
    Z[3] = 2.5                                    # constant row
    Z[4] = 0.0                                    # zero row
    Z[5] = np.abs(Z[5]) + 1.0                     # all positive: no zero inside
    q, s, m = o.quantize_rows_asym(Z, 4)
    rows = [i for i in range(32) if i not in (3, 4)]
    assert np.all(q[rows, np.argmin(Z[rows], axis=1)] == 0)
    assert np.all(q[rows, np.argmax(Z[rows], axis=1)] == 15)
    for i in (3, 4):
        assert s[i] == 0 and not q[i].any() and m[i] == Z[i, 0]
    assert m[5] == Z[5].min() and m[5] > 0


def test_asym_sqnr_matches_lemma_2_2_closed_form():
    # Lemma 2.2 with the asymmetric range and its 2^b - 1 intervals:
    # SQNR(W x~) ~= 12 (2^b - 1)^2 C_asym(x) A(x, W), on shifted Gaussian
    # data (where the asymmetric range is the smaller one).
    rng = np.random.default_rng(34)
    X = rng.standard_normal((4096, 256)) + 1.5
    W = rng.standard_normal((128, 256))
    for bits in (4, 6):
        q, s, m = o.quantize_rows_asym(X.astype(np.float32), bits)
        Xq = q * s[:, None].astype(np.float64) + m[:, None]
        Y = X @ W.T
        E = (X - Xq) @ W.T
        brute = 10 * np.log10(np.sum(Y * Y) / np.sum(E * E))
        pred = 10 * np.log10(12 * ((1 << bits) - 1) ** 2 *
                             o.concentration_act(X, asymmetric=True) * o.alignment(X, W))
        assert brute == pytest.approx(pred, abs=0.15), (bits, brute, pred)
        # and it beats the symmetric quantizer on this shifted data
        qs, ss = o.quantize_rows(X.astype(np.float32), bits)
        Es = (X - qs * ss[:, None]) @ W.T
        assert brute > 10 * np.log10(np.sum(Y * Y) / np.sum(Es * Es)) + 2.0


def test_linear_asym_brute_force_loops_and_fake_quant():
    rng = np.random.default_rng(35)
    qx = rng.integers(0, 16, size=(3, 40)).astype(np.int16)
    qw = wl.random_codes(4, 40, seed=36)
    sx = np.array([0.5, 0.25, 0.0], np.float32)
    mx = np.array([-1.25, 0.5, 3.0], np.float32)
    sw = np.array([1.0, 0.125, 2.0, 0.75], np.float32)
    acc, y = o.linear_asym(qx, sx, mx, qw, sw)
    for t in range(3):
        for j in range(4):
            ref = sum(int(a) * int(b) for a, b in zip(qx[t], qw[j]))
            assert acc[t, j] == ref
            R = int(qw[j].astype(np.int64).sum())
            # power-of-two scales and short sums: every fp32 step is exact
            assert float(y[t, j]) == (ref * float(sx[t]) + float(mx[t]) * R) * float(sw[j])
    # dequantize-then-multiply in fp64 gives the same product
    X = qx * sx[:, None].astype(np.float64) + mx[:, None]
    Wq = qw * sw[:, None].astype(np.float64)
    np.testing.assert_allclose(y, X @ Wq.T, rtol=1e-6, atol=1e-6)


# ------------------------------------------- full-dimension Hadamard
@pytest.mark.parametrize("m", [1, 2, 8, 32, 28, 56, 112])
def test_hadamard_orders_are_hadamard(m):
    H = o.hadamard_order(m)
    assert set(np.unique(H)) <= {-1, 1}
    assert np.array_equal(H @ H.T, m * np.eye(m, dtype=np.int64))
    if not (m & (m - 1)):
        assert np.array_equal(H, sla.hadamard(m))


def test_full_mix_of_hadamard_blocks_is_the_kronecker_hadamard():
    # with M = I every block is H_k / sqrt(k); block transform then mix is
    # x -> kron(H_m, H_k) x / sqrt(d)
    rng = np.random.default_rng(51)
    for m, k in ((4, 8), (28, 4)):
        d = m * k
        X = rng.standard_normal((6, d))
        Tb = np.stack([o.hadamard(k)] * m)
        Z = o.full_hadamard_mix(o.transform_rows(X, Tb), k)
        K = np.kron(o.hadamard_order(m), o.hadamard_order(k)) / np.sqrt(d)
        np.testing.assert_allclose(Z, X @ K.T, atol=1e-12)
        np.testing.assert_allclose(K @ K.T, np.eye(d), atol=1e-12)


def test_full_transform_preserves_function():
    rng = np.random.default_rng(52)
    d, k = 28 * 8, 8
    X = rng.standard_normal((10, d))
    W = rng.standard_normal((12, d))
    S = X.T @ X / 10 + np.eye(d)
    T = o.cat_transform(S, W, k)
    Wpp = o.transform_weights_full(W, T)
    Z = o.full_hadamard_mix(o.transform_rows(X, T), k)
    np.testing.assert_allclose(Z @ Wpp.T, X @ W.T, atol=1e-9 * np.abs(X @ W.T).max())


# ------------------------------------------------- bf16 storage rounding
# bf16 keeps 8 significant bits, so the spacing just above 1.0 is 2^-7 and
# 1 + 2^-8 sits exactly halfway between two neighbours.
@pytest.mark.parametrize("x,expected", [
    (1.0, 1.0),                                   # exact
    (1 + 2.0 ** -8, 1.0),                         # tie, 1.0 has the even last bit
    (1 + 3 * 2.0 ** -8, 1 + 2.0 ** -6),           # tie, rounds up to the even neighbour
    (1 + 2.0 ** -8 + 2.0 ** -20, 1 + 2.0 ** -7),  # just above the tie
    (1 + 2.0 ** -8 - 2.0 ** -20, 1.0),            # just below the tie
    (-(1 + 3 * 2.0 ** -8), -(1 + 2.0 ** -6)),     # sign is symmetric
    (-(1 + 2.0 ** -8), -1.0),
    (2 - 2.0 ** -8, 2.0),                         # tie across a binade: up to 2.0 (even)
    (2 - 3 * 2.0 ** -8, 2 - 2.0 ** -6),           # tie inside [1, 2): down to the even neighbour
    (3 * 2.0 ** 100 + 2.0 ** 93, 3 * 2.0 ** 100),  # tie at a large exponent (even below)
    (2.0 ** -149, 0.0),                           # smallest fp32 subnormal flushes to +0
    (2.0 ** -134, 0.0),                           # subnormal tie, 0 is even
    (1.5 * 2.0 ** -133, 2.0 ** -132),             # subnormal tie, rounds up to the even one
    (2.0 ** -133, 2.0 ** -133),                   # exact subnormal
])
def test_round_bf16_hand_values_and_ties(x, expected):
    # every input is exact in fp32; the expected values are worked out by
    # hand from the 8-bit significand and ties-to-even
    assert np.float64(np.float32(x)) == x
    got = o.round_bf16(np.array([x]))[0]
    assert got == expected and np.signbit(got) == np.signbit(expected)


def test_round_bf16_is_nearest_with_even_ties_brute_force():
    # Independent of the bit manipulation: for each fp32 value take its two
    # bf16 neighbours (truncation and the next representable value above in
    # magnitude), choose the nearer by exact fp64 distance, and on a tie the
    # one whose significand is even.  Half of the inputs are exact ties.
    rng = np.random.default_rng(81)
    bits = rng.integers(0x00800000, 0x7F000000, size=20000, dtype=np.uint32)
    bits[::2] = (bits[::2] & 0xFFFF0000) | 0x8000           # ties
    bits[1::4] |= 0x80000000                                # negatives
    x32 = bits.view(np.float32)
    got = o.round_bf16(x32)
    mag = np.abs(x32.astype(np.float64))
    lo_bits = (np.abs(x32).view(np.uint32) & 0xFFFF0000)
    lo = lo_bits.view(np.float32).astype(np.float64)
    hi = (lo_bits + 0x10000).view(np.float32).astype(np.float64)
    d_lo, d_hi = mag - lo, hi - mag
    lo_even = ((lo_bits >> 16) & 1) == 0
    pick_lo = (d_lo < d_hi) | ((d_lo == d_hi) & lo_even)
    ref = np.where(pick_lo, lo, hi) * np.sign(x32.astype(np.float64))
    assert np.array_equal(got, ref)
    assert (d_lo == d_hi).sum() >= 10000


def test_round_bf16_matches_torch_conversion():
    # torch's float32 -> bfloat16 cast rounds to nearest, ties to even
    import torch
    rng = np.random.default_rng(82)
    x = (rng.standard_normal(50000) * np.exp(rng.uniform(-30, 30, 50000))).astype(np.float32)
    x[:2000] = (x[:2000].view(np.uint32) & 0xFFFF0000 | 0x8000).view(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(o.round_bf16(x), ref)


# ------------------------------------------------------ eigenvalue floor
def test_eigenvalue_floor_closed_forms():
    # Eigenvalues below 1e-12 lambda_max are raised to that value before a
    # power is taken, so the powers stay finite on singular blocks.
    np.testing.assert_allclose(o.spd_power(np.diag([1.0, 1e-20]), -0.5),
                               np.diag([1.0, 1e6]), rtol=1e-12, atol=0)
    np.testing.assert_allclose(o.spd_power(np.diag([1.0, 0.0]), 0.5),
                               np.diag([1.0, 1e-6]), rtol=1e-12, atol=0)
    # a rotated singular matrix: Q diag(4, 1e-30) Q^T to the power -1/2 is
    # Q diag(1/2, (4e-12)^-1/2) Q^T
    c, s = np.cos(0.3), np.sin(0.3)
    Q = np.array([[c, -s], [s, c]])
    S = Q @ np.diag([4.0, 1e-30]) @ Q.T
    ref = Q @ np.diag([0.5, (4e-12) ** -0.5]) @ Q.T
    np.testing.assert_allclose(o.spd_power(S, -0.5), ref, rtol=1e-9, atol=1e-9 * 5e5)
    # eigenvalues above the floor are left alone
    np.testing.assert_allclose(o.spd_power(np.diag([1.0, 1e-11]), -0.5),
                               np.diag([1.0, 1e-11 ** -0.5]), rtol=1e-12)
    with pytest.raises(ValueError):
        o.spd_power(np.zeros((2, 2)), 0.5)


def test_eigenvalue_floor_keeps_the_transform_finite_on_a_dead_channel():
    # A channel that is zero on every calibration token makes its Sigma_x
    # block singular.  With the floor, the block's M has the floored
    # eigenvalue's closed form on that channel: for a diagonal block,
    # m_i = (sum_j W_ji^2 / max(E[x_i^2], 1e-12 lambda_max))^(1/4).
    k = 4
    Sx = np.diag([2.0, 0.5, 0.0, 1.0])
    w = np.array([[1.0, 2.0, 3.0, 0.5]])
    # rank-one Sigma_w: the block transform stays finite
    T = o.cat_transform(Sx, w.astype(np.float32), k, use_hadamard=False)[0]
    assert np.all(np.isfinite(T))
    # diagonal Sigma_w commutes with Sigma_x, so M is diagonal with the
    # closed form above; lambda_max = 2 sets the floor 2e-12 on channel 2
    cw = (w.astype(np.float32).astype(np.float64) ** 2)[0]
    ex = np.maximum(np.diag(Sx), 1e-12 * 2.0)
    Tdiag = o.optimal_alignment(Sx, np.diag(cw))
    np.testing.assert_allclose(np.diag(Tdiag), (cw / ex) ** 0.25, rtol=1e-9)
    np.testing.assert_allclose(Tdiag - np.diag(np.diag(Tdiag)), 0.0, atol=1e-12)


# ---------------------------------------------- alignment from moments
def test_alignment_from_moments_equals_sample_alignment():
    # Tr(W^T W X^T X) = ||X W^T||_F^2, so the moment form with Sigma_x =
    # X^T X / n and Sigma_w = W^T W equals the sample form of Lemma 2.2
    rng = np.random.default_rng(83)
    X, W = _act(rng, 400, 24), rng.standard_normal((10, 24))
    a_mom = o.alignment_from_moments(o.second_moment(X), W.T @ W)
    assert a_mom == pytest.approx(o.alignment(X, W), rel=1e-12)


def test_alignment_from_moments_closed_forms():
    rng = np.random.default_rng(84)
    d = 16
    Sw = _rand_spd(rng, d)
    # isotropic inputs: A = Tr(Sigma_w) / (Tr(Sigma_w) d) = 1 / d
    assert o.alignment_from_moments(np.eye(d), Sw) == pytest.approx(1.0 / d, rel=1e-14)
    # one input direction v and one weight row w: A = cos^2(v, w)
    v, w = rng.standard_normal(d), rng.standard_normal(d)
    cos2 = np.dot(v, w) ** 2 / (np.dot(v, v) * np.dot(w, w))
    assert o.alignment_from_moments(np.outer(v, v), np.outer(w, w)) == pytest.approx(cos2,
                                                                                      rel=1e-12)
    # orthogonal directions give zero alignment
    u = np.zeros(d); u[0] = 1.0
    t = np.zeros(d); t[1] = 1.0
    assert o.alignment_from_moments(np.outer(u, u), np.outer(t, t)) == 0.0
