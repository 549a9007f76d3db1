"""CPU oracle for the block Concentration-Alignment Transform (CAT) W4A4
linear-layer path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call
this module: only the tests, the smoke check and the benchmark's CPU
baseline leg do.  It shares no code with the HIP library (no kernels, no
headers, no helpers, no tables); the two meet only through the seeded
input generators in ``workloads``.

Plain, slow, obviously correct: numpy in fp64 wherever the paper fixes no
precision, and fp32 emulation exactly where a result is defined by fp32
rounding (the quantizer and the dequantization epilogue).

Paper: "Dissecting Quantization Error: A Concentration-Alignment
Perspective" (Federici, van Breugel, Whatmough, Nagel).

Function -> passage -> what pins it (tests/test_oracle_*.py):
  round_bf16         storage precision of T and X (no passage)
                                                -> hand-worked values with
                     exact ties both ways, brute-force nearest-neighbour
                     search, torch's float32 -> bfloat16 cast
  spd_power floor    (reading below; the paper is silent)
                                                -> closed forms on singular
                     and rotated-singular matrices, dead-channel closed
                     form of M through the floor
  second_moment      Sec. 4 (autocorrelation E[x x^T] used by eq. 7),
                     Sec. 6 "Calibration"       -> numpy.cov identity,
                     batch-split invariance, basis-vector case, PSD
  geometric_mean     Sec. 4, eq. 7 definition of A # B
                                                -> 2x2 closed form
                     (Bhatia, Positive Definite Matrices, Prop. 4.1.12),
                     Riccati equation, commuting case, symmetry
  optimal_alignment  Sec. 4, eq. 7              -> optimality under random
                     perturbation, k=1 closed form, balance identity
                     (eq. 8, first equality), maximum alignment via SVD
                     (eq. 9 in its corrected reading)
  hadamard           Sec. 3 (Hadamard), Sec. 4 (T = H M) -> scipy.linalg
                     .hadamard, orthogonality
  cat_transform      Sec. 4 "CAT Block Approximation", eq. 10
                                                -> block optimum closed form,
                     rotation invariance of alignment (eq. 4)
  transform_weights  Sec. 3, eq. 5 (W T^-1)     -> function preservation
  quantize_rows      Sec. 2 Lemma 2.2 (range r(x)), App. A.2.1 (step s),
                     Sec. 6 "Quantization set-up" (per token / per channel)
                                                -> RTN error bound, max maps
                     to +-qmax, power-of-two scale invariance, ties to even
  transform_quant    Sec. 3 eq. 5 (Q(T x)), Sec. 4 eq. 10
                                                -> T = I gives plain RTN,
                     orthogonal T preserves W x
  quantize_rows_asym Sec. 2 after Lemma 2.2 (asymmetric range), Sec. 6
                     (activations per token, asymmetric)
                                                -> nearest affine grid point
                     (brute force), min/max map to 0 and 2^b - 1,
                     constant rows exact, Lemma 2.2 closed form with
                     2^b - 1 intervals on Gaussian data
  linear_asym        Sec. 3, eq. 5 with asymmetric activations
                                                -> brute-force loops,
                     dequantize-then-multiply product
  hadamard_order, paley2_hadamard, full_hadamard_mix, transform_quant_full
                     Sec. 4 (T = H M, H full-dimension), Sec. 3 (Hadamard rotations)
                                                -> H H^T = m I and +-1
                     entries (orders 1 .. 112, incl. 28 = Paley II q = 13),
                     Sylvester = scipy.linalg.hadamard, mix of H_k blocks =
                     kron(H_m, H_k) / sqrt(d), function preservation
  pack_int4          storage layout (no passage) -> hand-computed bytes
  w4a4_linear        Sec. 3, eq. 5 (Q(W T^-1) Q(T x))
                                                -> brute-force loops,
                     fake-quant product, K-permutation invariance
  sqnr               Sec. 2, eq. 1               -> hand-computed values,
                     uniform-noise closed form on Gaussian data
  alignment_from_moments
                     Sec. 2 Lemma 2.2 (A written with second moments)
                                                -> equals the sample
                     alignment, isotropic 1/d and rank-one cos^2 closed forms
  concentration_*, alignment, theorem_2_4, parallel
                     Sec. 2 Lemmas 2.1-2.3, Theorem 2.4; Sec. 2.1
                                                -> paper's printed minimum
                     concentration 1/4 (golden fixture), rotation invariance,
                     brute-force SQNR on Gaussian data
Every function is pinned; none is "parity unpinned".

Readings where the paper is silent, ambiguous or garbled (same list as in
the design notes):
  * Asymmetric activations: 2^b levels from the row minimum, s = fl(r /
    (2^b - 1)) with r = fl(max - min); codes clamp(rint(fl(fl(z - min) *
    fl((2^b - 1) / r))), 0, 2^b - 1); dequantized as s q + min (no integer
    zero point: the minimum is kept in fp32).  A constant row gets s = 0.
    The product's fp32 order: fl(fl(fl(acc) s_x) + fl(min fl(R))) s_w.
  * Full-dimension Hadamard (the variant of T = H M with H over all d
    channels): H_d = H_m (x) H_k with m = d / k; H_m Sylvester for m a
    power of two, else H_28 (Paley II, q = 13) (x) Sylvester_(m/28).  So
    T = (H_m (x) I_k) / sqrt(m) blockdiag(H_k M_b / sqrt(k)), and the
    weights take the same cross-block mix.
  * Quantization widths 6 and 8 bits store one int8 per code; their tie
    bar is the INT4 one scaled by qmax / 7.
  * Symmetric integer grid: codes in [-qmax, qmax], qmax = 2^(b-1)-1, so
    the grid has N(b) = 2^b - 2 intervals (the paper's N(b) is "the number
    of quantization intervals"; its 2^b - 1 counts a 2^b-level grid).
  * Round to nearest, ties to even.
  * Quantization arithmetic in fp32: amax = max|z|; s = fl(amax/qmax);
    inv = fl(qmax/amax); q = clamp(rint(fl(z*inv)), -qmax, qmax).
    A row with amax = 0 gets s = 0 and all-zero codes.
  * Dynamic per-token range over the whole transformed row (not per block).
  * Sigma_x is the non-centred E[x x^T].
  * The Hadamard factor of T = H M_block is block-local (H_k, Sylvester
    order, normalised), so T stays block-diagonal.
  * M_b is used exactly as the geometric mean gives it (no rescaling).
  * Eigenvalues below 1e-12 * lambda_max are floored to that value.
  * T is rounded to its storage precision before W' = W T^-1 is formed.
  * eq. 9 as printed is inconsistent; the maximum alignment is
    sum(sigma_i^2) / (sum sigma_i)^2 with sigma_i the singular values of
    W Sigma_x^(1/2).
  * The k = 1 special case printed at the end of Sec. 4 is the inverse
    square of what eq. 7 gives; eq. 7 gives m_i = (sum_j W_ji^2 / E[x_i^2])^(1/4).
"""
from __future__ import annotations

import numpy as np

EIG_FLOOR = 1e-12


# --------------------------------------------------------------- helpers
def _f32(a):
    return np.asarray(a, dtype=np.float32)


def round_bf16(a) -> np.ndarray:
    """Round to the nearest bf16 value (ties to even), returned as fp64.
    Written independently of any other rounding helper: split the fp32
    pattern and round the low half."""
    x = np.ascontiguousarray(np.asarray(a, dtype=np.float64).astype(np.float32))
    bits = x.view(np.uint32).astype(np.uint64)
    low = bits & 0xFFFF
    high = bits >> 16
    round_up = (low > 0x8000) | ((low == 0x8000) & ((high & 1) == 1))
    high = high + round_up.astype(np.uint64)
    out = (high << 16).astype(np.uint32).view(np.float32)
    return out.astype(np.float64)


def round_storage(a, dtype: str) -> np.ndarray:
    """Round to the storage precision of a transform or activation
    ("bf16" or "f32"), returned as fp64."""
    if dtype == "bf16":
        return round_bf16(a)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float64).astype(np.float32).astype(np.float64)
    raise ValueError(dtype)


# ---------------------------------------------------------- a1: Sigma_x
def second_moment_sum(X) -> np.ndarray:
    """Unnormalised second moment sum_t x_t x_t^T = X^T X, fp64.
    Sec. 4: Sigma_x = E[x x^T] (non-centred), estimated from a calibration
    set (Sec. 6, "Calibration")."""
    X = np.asarray(X, dtype=np.float64)
    return X.T @ X


def second_moment(X) -> np.ndarray:
    """Sigma_x = E[x x^T] over the rows of X (Sec. 4, eq. 7 notation)."""
    X = np.asarray(X, dtype=np.float64)
    return second_moment_sum(X) / X.shape[0]


# ------------------------------------------ host: transform construction
def _eigh_floor(S):
    S = 0.5 * (S + S.T)
    w, V = np.linalg.eigh(S)
    floor = EIG_FLOOR * max(w.max(), 0.0)
    if floor <= 0.0:
        raise ValueError("matrix is not positive definite")
    return np.maximum(w, floor), V


def spd_power(S, p: float) -> np.ndarray:
    """Principal power S^p of a symmetric positive definite matrix."""
    w, V = _eigh_floor(np.asarray(S, dtype=np.float64))
    return (V * w ** p) @ V.T


def geometric_mean(A, B) -> np.ndarray:
    """Matrix geometric mean A # B = A^(1/2) (A^(-1/2) B A^(-1/2))^(1/2) A^(1/2)
    (Sec. 4, definition under eq. 7), written out literally."""
    Ah = spd_power(A, 0.5)
    Aih = spd_power(A, -0.5)
    inner = Aih @ B @ Aih
    inner = 0.5 * (inner + inner.T)
    out = Ah @ spd_power(inner, 0.5) @ Ah
    return 0.5 * (out + out.T)


def optimal_alignment(sigma_x, sigma_w) -> np.ndarray:
    """M_hat = (Sigma_w # Sigma_x^(-1))^(1/2), the maximiser of
    A(M x, W M^-1) (Sec. 4, eq. 7).  Sigma_w = W^T W.
    The mean is symmetric (A # B = B # A), and it is evaluated as
    Sigma_x^(-1) # Sigma_w, whose congruence inverts only the positive
    definite Sigma_x^(-1).  Sigma_w has rank below k when the layer has
    fewer outputs than the block has channels, and the literal A # B would
    then invert it."""
    sx_inv = spd_power(sigma_x, -1.0)
    sx_inv = 0.5 * (sx_inv + sx_inv.T)
    return spd_power(geometric_mean(sx_inv, sigma_w), 0.5)


def hadamard(k: int) -> np.ndarray:
    """Normalised Sylvester Hadamard matrix H_k / sqrt(k) (k a power of two).
    Sec. 3 (Hadamard rotations) and Sec. 4 (T = H M)."""
    if k < 1 or (k & (k - 1)):
        raise ValueError("k must be a power of two")
    H = np.ones((1, 1))
    while H.shape[0] < k:
        H = np.block([[H, H], [H, -H]])
    return H / np.sqrt(k)


def paley2_hadamard(q: int) -> np.ndarray:
    """Unnormalised Hadamard matrix of order 2 (q + 1) by Paley's second
    construction, q a prime with q = 1 (mod 4): the symmetric conference
    matrix C = [[0, 1^T], [1, Q]] (Q_ij = Legendre symbol of i - j mod q)
    gives H = C (x) [[1, 1], [1, -1]] + I (x) [[1, -1], [-1, -1]]."""
    if q % 4 != 1 or any(q % p == 0 for p in range(2, int(q ** 0.5) + 1)):
        raise ValueError("q must be a prime = 1 mod 4")
    squares = {(x * x) % q for x in range(1, q)}
    chi = np.array([0] + [1 if a in squares else -1 for a in range(1, q)])
    Q = np.array([[chi[(i - j) % q] for j in range(q)] for i in range(q)])
    C = np.zeros((q + 1, q + 1), dtype=np.int64)
    C[0, 1:] = 1
    C[1:, 0] = 1
    C[1:, 1:] = Q
    return np.kron(C, np.array([[1, 1], [1, -1]])) + \
        np.kron(np.eye(q + 1, dtype=np.int64), np.array([[1, -1], [-1, -1]]))


def hadamard_order(m: int) -> np.ndarray:
    """Unnormalised Hadamard matrix of order m for the full-dimension
    transform: Sylvester when m is a power of two, else H_28 (Paley II,
    q = 13) (x) Sylvester_(m/28) (the widths 28 2^a, e.g. 14336 / 128 =
    112).  The row index is b = b1 m / 28 + b2 for the Kronecker factor."""
    if m >= 1 and not (m & (m - 1)):
        return np.rint(hadamard(m) * np.sqrt(m)).astype(np.int64)
    if m % 28 == 0 and not ((m // 28) & (m // 28 - 1)):
        return np.kron(paley2_hadamard(13), hadamard_order(m // 28))
    raise ValueError(f"no Hadamard order {m} here")


def full_hadamard_mix(Z, k: int) -> np.ndarray:
    """Cross-block part of T = H_d M_block with H_d = H_m (x) H_k
    (Sec. 4, T = H M with a full-dimension H; Sec. 3, Hadamard
    rotations): z'_(b, j) = sum_b' H_m[b, b'] z_(b', j) / sqrt(m), fp64."""
    Z = np.asarray(Z, dtype=np.float64)
    n, d = Z.shape
    m = d // k
    H = hadamard_order(m).astype(np.float64) / np.sqrt(m)
    return np.einsum("ab,nbj->naj", H, Z.reshape(n, m, k)).reshape(n, d)


def transform_quant_full(X, T_blocks, bits: int = 4):
    """Q(H_d M x): the block transform T_b = H_k M_b, the cross-block
    Hadamard, one rounding to fp32, then the per-token quantizer."""
    k = T_blocks.shape[1]
    Z32 = full_hadamard_mix(transform_rows(X, T_blocks), k).astype(np.float32)
    return quantize_rows(Z32, bits)


def transform_weights_full(W, T_blocks) -> np.ndarray:
    """W'' = W T_full^-1 = (W blockdiag(T_b)^-1) (H_m (x) I_k)^T / sqrt(m),
    so that W'' T_full x = W x."""
    Wp = transform_weights(W, T_blocks)
    k = T_blocks.shape[1]
    # row times (H_m (x) I_k)^T / sqrt(m) is the same mix applied to the row
    return full_hadamard_mix(Wp, k)


def cat_transform(sigma_x, W, k: int, use_hadamard: bool = True,
                  use_alignment: bool = True) -> np.ndarray:
    """Block CAT transform (Sec. 4, "CAT Block Approximation", eq. 10):
    T_b = H_k M_b for each of the d/k diagonal blocks, with
    M_b = (Sigma_w,b # Sigma_x,b^-1)^(1/2) optimised on its own block and
    Sigma_w,b = W[:, b]^T W[:, b].  Returns [d/k, k, k] fp64 so that the
    transformed activation block is z_b = T_b x_b.

    use_alignment=False gives the block-Hadamard baseline (M_b = I);
    use_hadamard=False gives the alignment-only transform."""
    if use_alignment:
        sigma_x = np.asarray(sigma_x, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    d = W.shape[1]
    if d % k:
        raise ValueError("d must be a multiple of k")
    H = hadamard(k) if use_hadamard else np.eye(k)
    blocks = np.empty((d // k, k, k))
    for b in range(d // k):
        sl = slice(b * k, (b + 1) * k)
        if use_alignment:
            Wb = W[:, sl]
            M = optimal_alignment(sigma_x[sl, sl], Wb.T @ Wb)
        else:
            M = np.eye(k)
        blocks[b] = H @ M
    return blocks


def transform_weights(W, T_blocks) -> np.ndarray:
    """W' = W T^-1 for block-diagonal T (Sec. 3, eq. 5), per block by an
    fp64 linear solve: W'_b T_b = W_b."""
    W = np.asarray(W, dtype=np.float64)
    nb, k, _ = T_blocks.shape
    out = np.empty_like(W)
    for b in range(nb):
        sl = slice(b * k, (b + 1) * k)
        # W'_b T_b = W_b  <=>  T_b^T W'_b^T = W_b^T
        out[:, sl] = np.linalg.solve(T_blocks[b].T, W[:, sl].T).T
    return out


# ---------------------------------------------------------- a2: quantizer
def qmax_of(bits: int) -> int:
    return (1 << (bits - 1)) - 1


def quantize_rows(Z32, bits: int = 4):
    """Symmetric dynamic per-row quantizer in fp32 (Lemma 2.2: symmetric
    range r = 2 max|x_i|; App. A.2.1: uniform step; Sec. 6: per token for
    activations, per output channel for weights).
    Returns (codes int8 [rows, cols], scale fp32 [rows])."""
    Z = _f32(Z32)
    if Z.ndim != 2:
        raise ValueError("expected a 2-D array")
    qmax = np.float32(qmax_of(bits))
    amax = np.max(np.abs(Z), axis=1) if Z.shape[1] else np.zeros(Z.shape[0], np.float32)
    amax = amax.astype(np.float32)
    nz = amax > 0
    scale = np.zeros_like(amax)
    inv = np.zeros_like(amax)
    scale[nz] = (amax[nz] / qmax).astype(np.float32)
    inv[nz] = (qmax / amax[nz]).astype(np.float32)
    u = (Z * inv[:, None]).astype(np.float32)
    q = np.clip(np.rint(u), -qmax, qmax).astype(np.int8)
    return q, scale


def transform_rows(X, T_blocks) -> np.ndarray:
    """z_b = T_b x_b for every block of every row, computed in fp64 from the
    exact stored values (Sec. 4, eq. 10 applied to activations)."""
    X = np.asarray(X, dtype=np.float64)
    nb, k, _ = T_blocks.shape
    if X.shape[1] != nb * k:
        raise ValueError("X width does not match the transform")
    Z = np.empty_like(X)
    for b in range(nb):
        sl = slice(b * k, (b + 1) * k)
        Z[:, sl] = X[:, sl] @ T_blocks[b].T
    return Z


def transform_quant(X, T_blocks, bits: int = 4):
    """Q(T x) per token: block transform in fp64, rounded once to fp32,
    then the fp32 symmetric per-token quantizer over the whole row
    (Sec. 3, eq. 5; Sec. 4, eq. 10; Sec. 6 "Quantization set-up").
    Returns (codes int8 [n, d], s_x fp32 [n])."""
    Z32 = transform_rows(X, T_blocks).astype(np.float32)
    return quantize_rows(Z32, bits)


def quantize_weights(W_prime, bits: int = 4):
    """Per-output-channel symmetric RTN of fp32(W') (Sec. 6)."""
    return quantize_rows(np.asarray(W_prime, dtype=np.float64).astype(np.float32), bits)


# ------------------------------------------- asymmetric activations
def quantize_rows_asym(Z32, bits: int = 4):
    """Asymmetric dynamic per-row quantizer in fp32 (Sec. 2 after Lemma
    2.2: range r = max_i x_i - min_i x_i; Sec. 6: activations per token,
    asymmetric).  Affine grid of 2^b levels from the row minimum:
      r = fl(max - min), s = fl(r / (2^b - 1)), inv = fl((2^b - 1) / r),
      q = clamp(rint(fl(fl(z - min) * inv)), 0, 2^b - 1),
    dequantized as s q + min.  A row with r = 0 gets s = 0, q = 0 and is
    reconstructed exactly by its minimum.
    Returns (codes int16 [rows, cols] in [0, 2^b - 1], scale fp32 [rows],
    minimum fp32 [rows])."""
    Z = _f32(Z32)
    if Z.ndim != 2:
        raise ValueError("expected a 2-D array")
    lv = np.float32((1 << bits) - 1)
    zmax = np.max(Z, axis=1).astype(np.float32)
    zmin = np.min(Z, axis=1).astype(np.float32)
    r = (zmax - zmin).astype(np.float32)
    nz = r > 0
    scale = np.zeros_like(r)
    inv = np.zeros_like(r)
    scale[nz] = (r[nz] / lv).astype(np.float32)
    inv[nz] = (lv / r[nz]).astype(np.float32)
    u = ((Z - zmin[:, None]).astype(np.float32) * inv[:, None]).astype(np.float32)
    q = np.clip(np.rint(u), 0, lv).astype(np.int16)
    return q, scale, zmin


def transform_quant_asym(X, T_blocks, bits: int = 4):
    """Q_asym(T x) per token: the block transform as in transform_quant,
    then the asymmetric per-token quantizer over the whole row."""
    Z32 = transform_rows(X, T_blocks).astype(np.float32)
    return quantize_rows_asym(Z32, bits)


def linear_asym(codes_x, s_x, min_x, codes_w, s_w):
    """Q_asym(x)-by-Q(W) product (Sec. 3, eq. 5 with asymmetric
    activations): sum_j (s q_j + m) w~_j = s sum_j q_j qw_j + m sum_j qw_j,
    both integer sums exact, then in fp32
      y_tilde = fl(fl(fl(acc) s_x[t]) + fl(m_t fl(R_o))) s_w[o],
    acc = sum_j q_tj qw_oj and R_o = sum_j qw_oj.
    Returns (acc int32 [n, d_out], y_tilde fp32 [n, d_out])."""
    qx = np.asarray(codes_x, dtype=np.float64)
    qw = np.asarray(codes_w, dtype=np.float64)
    acc = qx @ qw.T
    R = qw.sum(axis=1)
    for a in (acc, R):
        if not np.array_equal(a.astype(np.int64).astype(np.float64), a):
            raise AssertionError("integer sum not exact")
    sx, mx, sw = _f32(s_x), _f32(min_x), _f32(s_w)
    t1 = (acc.astype(np.float32) * sx[:, None]).astype(np.float32)
    t2 = (mx[:, None] * R.astype(np.float32)[None, :]).astype(np.float32)
    y = ((t1 + t2).astype(np.float32) * sw[None, :]).astype(np.float32)
    return acc.astype(np.int64).astype(np.int32), y


def quantized_forward_asym(X, T_blocks, W_prime, bits: int = 4):
    """The whole layer with asymmetric per-token activations and
    symmetric per-channel weights (the paper's set-up, Sec. 6)."""
    qx, sx, mx = transform_quant_asym(X, T_blocks, bits)
    qw, sw = quantize_weights(W_prime, bits)
    acc, yt = linear_asym(qx, sx, mx, qw, sw)
    return {"codes_x": qx, "s_x": sx, "min_x": mx, "codes_w": qw, "s_w": sw,
            "acc": acc, "y_tilde": yt}


# ------------------------------------------------------------ packing
def pack_int4(codes) -> np.ndarray:
    """Two's-complement int4 pairs: byte j of a row holds element 2j in
    bits 0-3 and element 2j+1 in bits 4-7."""
    c = np.asarray(codes, dtype=np.int16)
    if c.shape[-1] % 2:
        raise ValueError("row length must be even")
    lo = c[..., 0::2] & 0xF
    hi = c[..., 1::2] & 0xF
    return (lo | (hi << 4)).astype(np.uint8)


def unpack_int4(packed) -> np.ndarray:
    p = np.asarray(packed, dtype=np.uint8).astype(np.int16)
    lo = p & 0xF
    hi = (p >> 4) & 0xF
    lo = np.where(lo >= 8, lo - 16, lo)
    hi = np.where(hi >= 8, hi - 16, hi)
    out = np.empty(p.shape[:-1] + (p.shape[-1] * 2,), dtype=np.int8)
    out[..., 0::2] = lo
    out[..., 1::2] = hi
    return out


# ------------------------------------------------------------ a3: GEMM
def w4a4_linear(codes_x, s_x, codes_w, s_w):
    """Q(W T^-1) Q(T x) as an integer product with per-token and
    per-output-channel scales (Sec. 3, eq. 5).
    acc[t, o] = sum_j qx[t, j] qw[o, j] exactly (fp64 holds every partial
    sum of these small integers exactly), then
    y_tilde = fl32(fl32(acc) * s_x[t]) * s_w[o] in fp32.
    Returns (acc int32 [n, d_out], y_tilde fp32 [n, d_out])."""
    qx = np.asarray(codes_x, dtype=np.float64)
    qw = np.asarray(codes_w, dtype=np.float64)
    acc = qx @ qw.T
    acc_i = acc.astype(np.int64)
    if not np.array_equal(acc_i.astype(np.float64), acc):
        raise AssertionError("integer product not exact")
    y = (acc.astype(np.float32) * _f32(s_x)[:, None]).astype(np.float32)
    y = (y * _f32(s_w)[None, :]).astype(np.float32)
    return acc_i.astype(np.int32), y


# ------------------------------------------------------------ a4: SQNR
def sqnr(y, y_tilde):
    """SQNR = E||W x||^2 / E||W x - W~ x~||^2 (Sec. 2, eq. 1) with the
    expectations replaced by sums over all tokens and outputs.
    Returns (S, E, dB) with S = sum y^2, E = sum (y - y~)^2 in fp64."""
    y = np.asarray(y, dtype=np.float64).ravel()
    yt = np.asarray(y_tilde, dtype=np.float64).ravel()
    S = float(np.dot(y, y))
    diff = y - yt
    E = float(np.dot(diff, diff))
    with np.errstate(divide="ignore", invalid="ignore"):
        dB = float(10.0 * np.log10(np.float64(S) / np.float64(E)))
    return S, E, dB


def to_db(v) -> float:
    return float(10.0 * np.log10(v))


# ----------------------------------------- decomposition (Sec. 2, App. A)
def parallel(a, b):
    """a || b = (1/a + 1/b)^-1 (Lemma 2.1)."""
    return 1.0 / (1.0 / a + 1.0 / b)


def n_intervals(bits: int) -> int:
    """Number of quantization intervals of the symmetric grid
    [-qmax, qmax]: 2^b - 2 (see the module readings)."""
    return 2 * qmax_of(bits)


def sym_range(v, axis=-1):
    """Symmetric range r(v) = 2 max_i |v_i| (Lemma 2.2)."""
    return 2.0 * np.max(np.abs(np.asarray(v, dtype=np.float64)), axis=axis)


def asym_range(v, axis=-1):
    """Asymmetric range r(v) = max_i v_i - min_i v_i (Lemma 2.2)."""
    v = np.asarray(v, dtype=np.float64)
    return np.max(v, axis=axis) - np.min(v, axis=axis)


def concentration_act(X, asymmetric: bool = False) -> float:
    """C(x) = E||x||^2 / E[r(x)^2] over the rows of X (Lemma 2.2), with the
    symmetric range by default or the asymmetric one on request."""
    X = np.atleast_2d(np.asarray(X, dtype=np.float64))
    r = asym_range(X, 1) if asymmetric else sym_range(X, 1)
    return float(np.mean(np.sum(X * X, axis=1)) / np.mean(r ** 2))


def concentration_weight(W) -> float:
    """C(W) = sum_i ||w_i||^2 / sum_i r(w_i)^2 over output rows (Lemma 2.3)."""
    W = np.asarray(W, dtype=np.float64)
    return float(np.sum(W * W) / np.sum(sym_range(W, 1) ** 2))


def alignment(X, W) -> float:
    """A(x, W) = E||W x||^2 / (||W||_F^2 E||x||^2) (Lemma 2.2)."""
    X = np.asarray(X, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    Y = X @ W.T
    return float(np.sum(Y * Y) / (np.sum(W * W) * np.sum(X * X)))


def alignment_from_moments(sigma_x, sigma_w) -> float:
    """The same A written with second moments:
    Tr(Sigma_w Sigma_x) / (Tr Sigma_w Tr Sigma_x)."""
    return float(np.trace(sigma_w @ sigma_x) /
                 (np.trace(sigma_w) * np.trace(sigma_x)))


def sqnr_act_only(X, W, bits: int) -> float:
    """Closed form of Lemma 2.2: 12 N(b)^2 C(x) A(x, W)."""
    return 12.0 * n_intervals(bits) ** 2 * concentration_act(X) * alignment(X, W)


def sqnr_weight_only(X, W, bits: int) -> float:
    """Closed form of Lemma 2.3: 12 N(b)^2 C(W) A(x, W)."""
    return 12.0 * n_intervals(bits) ** 2 * concentration_weight(W) * alignment(X, W)


def theorem_2_4(X, W, bits_x: int, bits_w: int) -> float:
    """Theorem 2.4: 12 (N(b_x)^2 C(x) || N(b_w)^2 C(W)) A(x, W)."""
    nx, nw = n_intervals(bits_x), n_intervals(bits_w)
    return 12.0 * parallel(nx ** 2 * concentration_act(X),
                           nw ** 2 * concentration_weight(W)) * alignment(X, W)


def max_alignment(sigma_x, sigma_w) -> float:
    """Maximum alignment over all invertible M (Sec. 4, eq. 9, corrected
    reading): sum sigma_i^2 / (sum sigma_i)^2 with sigma_i the singular
    values of W Sigma_x^(1/2), i.e. Tr(Sigma_y) / (Tr Sigma_y^(1/2))^2."""
    sxh = spd_power(sigma_x, 0.5)
    C = sxh @ sigma_w @ sxh
    lam = np.clip(np.linalg.eigvalsh(0.5 * (C + C.T)), 0.0, None)
    sig = np.sqrt(lam)
    return float(np.sum(sig ** 2) / np.sum(sig) ** 2)


# ------------------------------------------------------- full pipeline
def quantized_forward(X, T_blocks, W_prime, bits: int = 4):
    """The whole quantized layer on fp64 inputs: Q(T x), Q(W T^-1), the
    integer product and dequantization.  Returns a dict of every
    intermediate."""
    qx, sx = transform_quant(X, T_blocks, bits)
    qw, sw = quantize_weights(W_prime, bits)
    acc, yt = w4a4_linear(qx, sx, qw, sw)
    return {"codes_x": qx, "s_x": sx, "codes_w": qw, "s_w": sw,
            "acc": acc, "y_tilde": yt}


def reference_output(X, W) -> np.ndarray:
    """Full-precision layer output y = W x in fp64 (Sec. 2, eq. 1)."""
    return np.asarray(X, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T
