"""Seeded synthetic inputs for the CAT W4A4 linear-layer path.

This module only draws random numbers and lays them out; it holds none of
the method's arithmetic (no second moment, no transform, no quantizer, no
GEMM, no SQNR).  Both the CPU oracle's tests and the GPU path's tests, the
benchmark and the smoke check take their inputs from here, so the two sides
always see identical arrays.

The five layer configurations stand in for the LLM linear layers the paper
measures (Sec. 6, set-up; Sec. 3, layers of Llama and Qwen models): shapes copy Llama-3-8B attention / MLP
projections and a 70B-class MLP, and the value structure copies what the
paper describes for real activations -- heavy tails and outlier channels
(Sec. 3, concentration analysis) and massive-activation tokens (Fig. 2
caption).  No model weights or dataset items are used.

Readings of the configuration text (where it leaves a choice open):
  * LogNormal(mu, sigma) is parameterised by the underlying normal.
  * N(0, v) gives the variance v.
  * "x c outlier channels": those channels' scales are multiplied by c; the
    channels are drawn once per seed and shared by the calibration and the
    evaluation activations.
  * Draw order is fixed: channel scales -> outlier channels -> X_cal -> X -> W.
  * bf16 configurations round the fp32 draw to bf16 (round-to-nearest-even)
    and hand both sides exactly those bf16 values.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass

import numpy as np

__all__ = [
    "LayerConfig", "CONFIGS", "get_config", "make_layer", "to_bf16_bits",
    "bf16_bits_to_f32", "random_codes", "random_pair", "random_spd",
    "random_bf16_matrix",
]


@dataclass(frozen=True)
class LayerConfig:
    name: str
    d_in: int
    d_out: int
    k: int                 # CAT block size
    n_cal: int             # calibration tokens
    n: int                 # evaluation tokens
    dtype: str             # "f32" or "bf16": activation / transform storage
    act: str               # "lognormal", "lowrank" or "student_t"
    act_sigma: float = 0.0     # LogNormal sigma of the per-channel scale
    n_outlier: int = 0         # number of outlier channels
    outlier_mult: float = 1.0  # their scale multiplier
    w_row_sigma: float = 0.0   # LogNormal sigma of the per-row weight scale
    lowrank_rank: int = 0      # activation factor rank (lowrank)
    noise_frac: float = 0.0    # isotropic noise share of total variance
    w_lowrank_rank: int = 0    # rank of the aligned weight component
    t_df: float = 0.0          # Student-t degrees of freedom
    massive_frac: float = 0.0  # share of massive-activation token rows
    massive_mult: float = 1.0
    massive_channels: int = 0
    k_sweep: tuple = ()


CONFIGS = {
    "tiny": LayerConfig(
        name="tiny", d_in=256, d_out=256, k=32, n_cal=2048, n=512,
        dtype="f32", act="lognormal", act_sigma=0.5, n_outlier=4,
        outlier_mult=30.0, w_row_sigma=0.3),
    "attn4096": LayerConfig(
        name="attn4096", d_in=4096, d_out=4096, k=128, n_cal=16384, n=2048,
        dtype="bf16", act="lognormal", act_sigma=1.0, n_outlier=8,
        outlier_mult=50.0),
    "mlp_up": LayerConfig(
        name="mlp_up", d_in=4096, d_out=14336, k=128, n_cal=32768, n=8192,
        dtype="bf16", act="lowrank", lowrank_rank=64, noise_frac=0.1,
        w_lowrank_rank=32),
    "mlp_down": LayerConfig(
        name="mlp_down", d_in=14336, d_out=4096, k=256, n_cal=32768, n=8192,
        dtype="bf16", act="student_t", t_df=3.0, massive_frac=0.01,
        massive_mult=100.0, massive_channels=2),
    "stress": LayerConfig(
        name="stress", d_in=8192, d_out=28672, k=128, n_cal=65536, n=16384,
        dtype="bf16", act="lognormal", act_sigma=1.2, n_outlier=16,
        outlier_mult=40.0, k_sweep=(64, 128, 256, 512)),
}


def get_config(name: str, **overrides) -> LayerConfig:
    """A named configuration, optionally with fields replaced (e.g. a
    smaller token count for a test that keeps the layer's structure)."""
    cfg = CONFIGS[name]
    return dataclasses.replace(cfg, **overrides) if overrides else cfg


# ----------------------------------------------------------------- bf16 I/O
def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return the uint16
    bit patterns.  Inputs are finite by construction."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _round_storage(a32: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.ascontiguousarray(a32, dtype=np.float32)
    return bf16_bits_to_f32(to_bf16_bits(a32))


# ------------------------------------------------------------ activations
def _haar_orthonormal(rng, rows, cols):
    g = rng.standard_normal((rows, cols))
    q, r = np.linalg.qr(g)
    return q * np.sign(np.diag(r))[None, :]


class _ActSource:
    """Draws the shared per-layer activation structure once, then any
    number of token batches from it."""

    def __init__(self, cfg: LayerConfig, rng):
        self.cfg = cfg
        d = cfg.d_in
        self.scale = np.ones(d)
        self.outliers = np.zeros(0, dtype=np.int64)
        self.massive_channels = np.zeros(0, dtype=np.int64)
        if cfg.act == "lognormal":
            self.scale = rng.lognormal(mean=0.0, sigma=cfg.act_sigma, size=d)
            self.outliers = rng.choice(d, size=cfg.n_outlier, replace=False)
            self.scale[self.outliers] *= cfg.outlier_mult
        elif cfg.act == "lowrank":
            r = cfg.lowrank_rank
            self.factor = _haar_orthonormal(rng, d, r)
            lam = 1.0 / np.arange(1, r + 1)
            lam *= (1.0 - cfg.noise_frac) * d / lam.sum()
            self.factor_scale = np.sqrt(lam)
            self.noise_std = np.sqrt(cfg.noise_frac)
        elif cfg.act == "student_t":
            self.massive_channels = rng.choice(
                d, size=cfg.massive_channels, replace=False)
        else:
            raise ValueError(cfg.act)

    def draw(self, rng, n: int) -> np.ndarray:
        cfg, d = self.cfg, self.cfg.d_in
        out = np.empty((n, d), dtype=np.float32)
        chunk = max(1, (1 << 22) // d)
        for r0 in range(0, n, chunk):
            m = min(chunk, n - r0)
            if cfg.act == "lognormal":
                g = rng.standard_normal((m, d), dtype=np.float32)
                out[r0:r0 + m] = g * self.scale.astype(np.float32)[None, :]
            elif cfg.act == "lowrank":
                g = rng.standard_normal((m, cfg.lowrank_rank))
                e = rng.standard_normal((m, d), dtype=np.float32)
                low = (g * self.factor_scale[None, :]) @ self.factor.T
                out[r0:r0 + m] = low.astype(np.float32) + \
                    np.float32(self.noise_std) * e
            else:  # student_t: z / sqrt(chi2_df / df)
                z = rng.standard_normal((m, d), dtype=np.float32)
                chi2 = 2.0 * rng.standard_gamma(cfg.t_df / 2.0, size=(m, d),
                                                dtype=np.float32)
                out[r0:r0 + m] = z / np.sqrt(chi2 / np.float32(cfg.t_df))
        if cfg.act == "student_t" and cfg.massive_frac > 0:
            n_massive = int(round(cfg.massive_frac * n))
            rows = rng.choice(n, size=n_massive, replace=False)
            for c in self.massive_channels:
                out[rows, c] *= np.float32(cfg.massive_mult)
        return out


def _draw_weights(cfg: LayerConfig, rng) -> np.ndarray:
    d_in, d_out = cfg.d_in, cfg.d_out
    std = np.float32(1.0 / np.sqrt(d_in))
    W = np.empty((d_out, d_in), dtype=np.float32)
    chunk = max(1, (1 << 22) // d_in)
    for r0 in range(0, d_out, chunk):
        m = min(chunk, d_out - r0)
        W[r0:r0 + m] = rng.standard_normal((m, d_in), dtype=np.float32) * std
    if cfg.w_row_sigma > 0:
        rs = rng.lognormal(mean=0.0, sigma=cfg.w_row_sigma, size=d_out)
        W *= rs.astype(np.float32)[:, None]
    if cfg.w_lowrank_rank > 0:
        r = cfg.w_lowrank_rank
        U = _haar_orthonormal(rng, d_out, r)
        V = _haar_orthonormal(rng, d_in, r)
        # equal energy: ||alpha U V^T||_F = ||G||_F, and ||U V^T||_F = sqrt(r)
        alpha = np.linalg.norm(W.astype(np.float64)) / np.sqrt(r)
        for r0 in range(0, d_out, chunk):
            m = min(chunk, d_out - r0)
            W[r0:r0 + m] += (alpha * (U[r0:r0 + m] @ V.T)).astype(np.float32)
    return W


def make_layer(cfg: LayerConfig, seed: int = 0, with_cal: bool = True,
               with_eval: bool = True, with_weights: bool = True) -> dict:
    """Seeded synthetic layer: calibration activations ``X_cal`` [n_cal, d_in],
    evaluation activations ``X`` [n, d_in] (fp32 arrays holding exactly the
    storage-precision values) and weights ``W`` [d_out, d_in] (fp32).

    The draw order is fixed, so disabling a part still leaves the other
    parts identical to a full draw of the same seed, except that later
    parts are drawn from a generator positioned as if earlier ones had been
    drawn (skipped parts are drawn and discarded)."""
    rng = np.random.default_rng(seed)
    src = _ActSource(cfg, rng)
    out = {"cfg": cfg, "seed": seed, "outlier_channels": src.outliers,
           "massive_channels": src.massive_channels}
    xc = src.draw(rng, cfg.n_cal)
    if with_cal:
        out["X_cal"] = _round_storage(xc, cfg.dtype)
    del xc
    x = src.draw(rng, cfg.n)
    if with_eval:
        out["X"] = _round_storage(x, cfg.dtype)
    del x
    if with_weights:
        out["W"] = _draw_weights(cfg, rng)
    return out


# ------------------------------------------------- plain random test inputs
def random_codes(rows: int, cols: int, seed: int, qmax: int = 7) -> np.ndarray:
    """Integer codes uniform in [-qmax, qmax], int8, [rows, cols]."""
    rng = np.random.default_rng(seed)
    return rng.integers(-qmax, qmax + 1, size=(rows, cols), dtype=np.int8)


def random_pair(count: int, seed: int, noise: float = 0.05):
    """A signal y ~ N(0,1) and a perturbed copy y + noise*N(0,1), fp32."""
    rng = np.random.default_rng(seed)
    y = rng.standard_normal(count, dtype=np.float32)
    e = rng.standard_normal(count, dtype=np.float32)
    return y, (y + np.float32(noise) * e).astype(np.float32)


def random_spd(n: int, seed: int, cond: float = 1e3) -> np.ndarray:
    """A random symmetric positive definite matrix with a given condition
    number (log-uniform spectrum between 1/cond and 1)."""
    rng = np.random.default_rng(seed)
    q = _haar_orthonormal(rng, n, n)
    ev = np.exp(rng.uniform(np.log(1.0 / cond), 0.0, size=n))
    ev[0], ev[-1] = 1.0, 1.0 / cond
    a = (q * ev[None, :]) @ q.T
    return 0.5 * (a + a.T)


def random_bf16_matrix(rows: int, cols: int, seed: int,
                       scale: float = 1.0) -> np.ndarray:
    """N(0, scale^2) values rounded to bf16, returned as fp32."""
    rng = np.random.default_rng(seed)
    a = rng.standard_normal((rows, cols), dtype=np.float32) * np.float32(scale)
    return bf16_bits_to_f32(to_bf16_bits(a))
