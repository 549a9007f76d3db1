"""The library's host-side transform construction and weight quantizer
against the CPU oracle (independent implementations of Sec. 4, eq. 7 and
eq. 10, and of the Sec. 6 weight quantizer)."""
import numpy as np
import pytest

import paper_2603_04359_amd as cat
import workloads as wl
from oracle import cat_oracle as o
from paper_2603_04359_amd import binding as B


def _diag_blocks(S, k):
    d = S.shape[0]
    return np.stack([S[b * k:(b + 1) * k, b * k:(b + 1) * k] for b in range(d // k)])


def _bf16_boundary_distance(v):
    """Relative distance of fp64 values to the nearest bf16 rounding
    boundary (midpoint between two bf16 neighbours), computed in fp64."""
    f = np.abs(np.asarray(v, np.float64))
    e = np.floor(np.log2(np.where(f > 0, f, 1.0)))
    ulp = 2.0 ** (e - 7)
    frac = f / ulp - np.floor(f / ulp)
    return np.abs(frac - 0.5) * ulp / np.where(f > 0, f, 1.0)


def _layer(d_in, d_out, k, n_cal, seed):
    rng = np.random.default_rng(seed)
    scale = np.exp(rng.standard_normal(d_in))
    scale[rng.choice(d_in, 3, replace=False)] *= 30
    X = (rng.standard_normal((n_cal, d_in)) * scale).astype(np.float32)
    W = (rng.standard_normal((d_out, d_in)) / np.sqrt(d_in)).astype(np.float32)
    return X, W


@pytest.mark.parametrize("d_in,d_out,k,t_dtype", [
    (64, 48, 16, "bf16"), (256, 256, 32, "f32"), (256, 200, 64, "bf16"), (512, 384, 128, "bf16"),
])
def test_build_transform_matches_oracle(d_in, d_out, k, t_dtype):
    X, W = _layer(d_in, d_out, k, 4096, seed=d_in + k)
    S = o.second_moment(X)
    T_or = o.cat_transform(S, W, k)
    td = B.CAT_BF16 if t_dtype == "bf16" else B.CAT_F32
    T, Te, Wp = cat.cat_build_transform(_diag_blocks(S, k), W, k, B.CAT_BUILD_CAT, td,
                                        want_exact=True, n_threads=4)
    # fp64 transform before rounding (cond of the blocks is moderate here)
    err = np.abs(Te - T_or).max() / np.abs(T_or).max()
    assert err < 1e-9, err
    # rounded transform: identical except where the fp64 value sits on a
    # rounding boundary (relative distance below the solvers' disagreement)
    T_or_r = o.round_storage(T_or, t_dtype)
    T_lib = (wl.bf16_bits_to_f32(T) if t_dtype == "bf16" else T).astype(np.float64)
    diff = T_lib != T_or_r
    if t_dtype == "bf16":
        assert np.all(_bf16_boundary_distance(T_or[diff]) < 1e-8)
    else:
        assert np.all(np.abs(Te[diff] - T_or[diff]) <= 1e-9 * np.abs(T_or[diff]))
    assert diff.mean() < 1e-3
    # W' = W T^-1 with the rounded T (oracle on its own rounded T)
    if not diff.any():
        Wp_or = o.transform_weights(W, T_or_r)
        assert np.abs(Wp - Wp_or).max() <= 1e-9 * np.abs(Wp_or).max()
    # function preservation W' T x = W x with the library's own outputs
    Z = o.transform_rows(X[:64].astype(np.float64), T_lib)
    ref = X[:64].astype(np.float64) @ W.astype(np.float64).T
    assert np.abs(Z @ Wp.T - ref).max() <= 1e-9 * np.abs(ref).max()


def test_build_transform_identity_and_hadamard_flags():
    _, W = _layer(128, 64, 32, 16, seed=3)
    T, _, Wp = cat.cat_build_transform(None, W, 32, 0, B.CAT_F32)
    assert np.array_equal(T, np.stack([np.eye(32, dtype=np.float32)] * 4))
    assert np.array_equal(Wp, W.astype(np.float64))
    T, _, Wp = cat.cat_build_transform(None, W, 32, B.CAT_BUILD_HADAMARD, B.CAT_F32)
    H = o.hadamard(32).astype(np.float32)
    assert np.array_equal(T, np.stack([H] * 4))


def test_build_transform_k1_closed_form():
    X, W = _layer(32, 40, 1, 2048, seed=5)
    S = o.second_moment(X)
    T, Te, _ = cat.cat_build_transform(_diag_blocks(S, 1), W, 1, B.CAT_BUILD_ALIGN, B.CAT_F32,
                                       want_exact=True)
    m = (np.sum(W.astype(np.float64) ** 2, 0) / np.diag(S)) ** 0.25
    np.testing.assert_allclose(Te[:, 0, 0], m, rtol=1e-12)


def test_build_transform_ill_conditioned_block():
    # nearly rank-deficient calibration block: the eigenvalue floor keeps the
    # result finite and invertible
    rng = np.random.default_rng(7)
    k = 16
    A = rng.standard_normal((k, 3))
    S = A @ A.T + 1e-9 * np.eye(k)
    W = rng.standard_normal((32, k)).astype(np.float32)
    T, Te, Wp = cat.cat_build_transform(S[None], W, k, B.CAT_BUILD_CAT, B.CAT_F32, want_exact=True)
    assert np.all(np.isfinite(Te)) and np.all(np.isfinite(Wp))
    T_or = o.cat_transform(S, W, k)
    # the two eigensolvers agree to about eps * cond(S) (cond ~ 3e10 here)
    cond = np.linalg.cond(S)
    assert np.abs(Te - T_or).max() / np.abs(T_or).max() < 1e-15 * cond


@pytest.mark.parametrize("bits", [4, 6, 8])
def test_quantize_weights_matches_oracle_bit_exact(bits):
    rng = np.random.default_rng(9)
    Wp = rng.standard_normal((70, 96)) * np.exp(rng.standard_normal(70))[:, None]
    Wp[3] = 0.0
    Wp[5, 7] = 1e3
    codes, s_w = cat.cat_quantize_weights(Wp, bits)
    q_or, s_or = o.quantize_weights(Wp, bits)
    assert np.array_equal(codes, o.pack_int4(q_or) if bits == 4 else q_or)
    assert np.array_equal(s_w, s_or)
    assert s_w[3] == 0 and not codes[3].any()


def test_weight_code_sums_match_unpacked_codes():
    qw = wl.random_codes(37, 96, seed=41)
    qw[0] = -8 + 1                                 # all -7
    qw[1] = 7
    rs = cat.cat_weight_code_sums(o.pack_int4(qw))
    assert rs.dtype == np.int32
    assert np.array_equal(rs, qw.astype(np.int64).sum(axis=1))


@pytest.mark.parametrize("t_dtype", ["f32", "bf16"])
def test_sqnr_terms_match_oracle_decomposition(t_dtype):
    # Theorem 2.4's terms from a batch's block second-moment sums, the
    # per-token scales and sum y^2, against the oracle's concentration,
    # alignment and prediction computed from the transformed rows directly
    cfg = wl.get_config("tiny")
    lay = wl.make_layer(cfg, seed=3)
    X, W, k = lay["X"].astype(np.float64), lay["W"].astype(np.float64), cfg.k
    T = o.round_storage(o.cat_transform(o.second_moment(lay["X_cal"]), W, k), t_dtype)
    Wp = o.transform_weights(W, T)
    Z = o.transform_rows(X, T)
    _, s_x = o.transform_quant(X, T, 4)
    S = np.stack([X[:, b * k:(b + 1) * k].T @ X[:, b * k:(b + 1) * k] for b in range(cfg.d_in // k)])
    Y = X @ W.T
    if t_dtype == "bf16":
        Tc = (T.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        tcode = cat.CAT_BF16
    else:
        Tc, tcode = T.astype(np.float32), cat.CAT_F32
    r = cat.cat_sqnr_terms(s_x, 4, S, Tc, tcode, Wp, 4, float(np.sum(Y * Y)))
    assert r["C_x"] == pytest.approx(o.concentration_act(Z), rel=1e-6)
    assert r["C_w"] == pytest.approx(o.concentration_weight(Wp), rel=1e-12)
    assert r["A"] == pytest.approx(o.alignment(Z, Wp), rel=1e-9)
    assert r["sqnr_pred"] == pytest.approx(o.theorem_2_4(Z, Wp, 4, 4), rel=1e-6)
    assert r["sqnr_pred_db"] == pytest.approx(10 * np.log10(r["sqnr_pred"]))


@pytest.mark.parametrize("m,k", [(8, 16), (28, 8), (56, 4), (112, 2)])
def test_full_hadamard_weights_match_oracle(m, k):
    rng = np.random.default_rng(m + k)
    Wp = rng.standard_normal((9, m * k))
    Tb = np.stack([np.eye(k)] * m)
    ref = o.transform_weights_full(Wp, Tb)          # W' itself when T_b = I
    got = cat.cat_full_hadamard_weights(Wp, k)
    np.testing.assert_allclose(got, ref, atol=1e-12 * np.abs(ref).max())


def test_build_transform_rounds_exact_bf16_ties_to_even():
    # k = 1 makes each block the scalar m_i = (sum_j W_ji^2 / E[x_i^2])^(1/4)
    # (eq. 7).  With E[x_i^2] = 1 and one weight row W_0i = m_i^2, every
    # intermediate is exact, so T_i = m_i; the m_i below sit exactly on
    # bf16 rounding boundaries (spacing 2^-7 on [1, 2)) and on either side.
    m = np.array([1 + 2.0 ** -8,              # tie: down to 1.0 (even)
                  1 + 3 * 2.0 ** -8,          # tie: up to 1 + 2^-6 (even)
                  1 + 2.0 ** -7,              # exact
                  1.5,                        # exact
                  1 + 5 * 2.0 ** -8,          # tie: down to 1 + 2^-6 (even)
                  1 + 7 * 2.0 ** -8])         # tie: up to 1 + 2^-5
    # neighbours of 1 + (2j+1) 2^-8 are 1 + j 2^-7 and 1 + (j+1) 2^-7;
    # the even one has the even multiple of 2^-7
    expected = []
    for v in m:
        j = np.floor((v - 1.0) / 2.0 ** -7)
        lo, hi = 1.0 + j * 2.0 ** -7, 1.0 + (j + 1) * 2.0 ** -7
        if v - lo < hi - v:
            expected.append(lo)
        elif v - lo > hi - v:
            expected.append(hi)
        else:
            expected.append(lo if j % 2 == 0 else hi)
    expected = np.array(expected)
    np.testing.assert_array_equal(expected, [1.0, 1 + 2.0 ** -6, 1 + 2.0 ** -7, 1.5,
                                             1 + 2.0 ** -6, 1 + 2.0 ** -5])
    d = m.size
    W = (m ** 2).astype(np.float32)[None, :]
    assert np.array_equal(W[0].astype(np.float64), m ** 2)
    sx = np.ones((d, 1, 1))
    T, Te, _ = cat.cat_build_transform(sx, W, 1, B.CAT_BUILD_ALIGN, B.CAT_BF16, want_exact=True)
    np.testing.assert_array_equal(Te.reshape(-1), m)
    np.testing.assert_array_equal(wl.bf16_bits_to_f32(T).reshape(-1).astype(np.float64), expected)
    # the oracle's T and its storage rounding land on the same values
    T_or = o.cat_transform(np.eye(d), W, 1, use_hadamard=False)
    np.testing.assert_array_equal(T_or.reshape(-1), m)
    np.testing.assert_array_equal(o.round_storage(T_or, "bf16").reshape(-1), expected)
