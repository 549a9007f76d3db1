"""Helpers shared by the GPU parity tests: device transfers and the
comparison rules (integer exactness, the rounding-tie rule for codes,
relative Frobenius error)."""
import sys

import numpy as np

from oracle import cat_oracle as o


def torch_mod():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a HIP device (torch.cuda.is_available() is False)")
    return torch


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(a, dtype):
    """numpy -> device tensor.  dtype 'bf16' expects values already
    representable in bf16 (the conversion is then exact)."""
    torch = torch_mod()
    a = np.ascontiguousarray(a)
    if dtype == "bf16":
        t = torch.from_numpy(a.astype(np.float32)).to("cuda").to(torch.bfloat16)
        back = t.float().cpu().numpy()
        assert np.array_equal(back, a.astype(np.float32)), "value not representable in bf16"
        return t
    if dtype == "f32":
        return torch.from_numpy(a.astype(np.float32)).to("cuda")
    if dtype == "f64":
        return torch.from_numpy(a.astype(np.float64)).to("cuda")
    if dtype == "u8":
        return torch.from_numpy(a.astype(np.uint8)).to("cuda")
    if dtype == "i8":
        return torch.from_numpy(a.astype(np.int8)).to("cuda")
    if dtype == "i32":
        return torch.from_numpy(a.astype(np.int32)).to("cuda")
    raise ValueError(dtype)


def gemm_tile_rows(n, d_out):
    """Token rows per tile the integer GEMMs launch with on this device:
    128 when 256-row tiles would leave CUs idle and 128-row ones take no
    more rounds of the one-workgroup-per-CU grid, else 256."""
    torch = torch_mod()
    slots = torch.cuda.get_device_properties(0).multi_processor_count // 8 * 8
    tn = -(-d_out // 256)
    t256, t128 = -(-n // 256) * tn, -(-n // 128) * tn
    return 128 if t256 < slots and -(-t128 // slots) <= -(-t256 // slots) else 256


def check_tile_rows(n, d_out, rows):
    """On a 256-CU MI355X, asserts that the case runs on the expected tile
    height (elsewhere the rule may pick another, and the case still runs)."""
    torch = torch_mod()
    if torch.cuda.get_device_properties(0).multi_processor_count == 256:
        assert gemm_tile_rows(n, d_out) == rows


def host(t):
    torch = torch_mod()
    torch.cuda.synchronize()
    return t.cpu().numpy()


def rel_fro(a, ref):
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(a - ref) / den) if den > 0 else float(np.linalg.norm(a))


def check_codes(codes_gpu, X, T_blocks, bits=4, label=""):
    """Codes must equal the oracle's except at exact rounding ties: a
    mismatch must be off by one code and the oracle's exact multiplier
    u* = z * qmax / amax (fp64) must lie within 2^-20 max(1, |u*|) of a
    half-integer; at most 1e-6 of all INT4 codes, and 1e-6 * qmax / 7 of
    the 6- and 8-bit ones (at least one allowed for small inputs), may be
    such ties.
    Returns (n_mismatch, oracle codes, oracle scales)."""
    q_or, s_or = o.transform_quant(X, T_blocks, bits)
    # bits 4: packed INT4 pairs; 6 and 8: one int8 per code
    q_gpu = o.unpack_int4(codes_gpu) if bits == 4 else np.asarray(codes_gpu).view(np.int8)
    mism = q_gpu != q_or
    nm = int(mism.sum())
    if nm:
        Z = o.transform_rows(X, T_blocks)
        amax = np.abs(Z).max(axis=1, keepdims=True)
        with np.errstate(divide="ignore", invalid="ignore"):
            u = Z * (o.qmax_of(bits) / amax)
        um = np.abs(u[mism])
        tie_dist = np.abs(um - np.floor(um) - 0.5)
        is_tie = (np.abs(q_gpu[mism].astype(int) - q_or[mism].astype(int)) == 1) & \
                 (tie_dist <= 2.0 ** -20 * np.maximum(1.0, um))
        assert is_tie.all(), (
            f"{label}: {int((~is_tie).sum())} non-tie code mismatches of {q_or.size}; "
            f"first at {np.argwhere(mism)[:3].tolist()}")
        # INT4: at most 1e-6 of the codes.  A one-ulp difference in fp32 z
        # flips a rounding decision with probability proportional to
        # |u| = |z| qmax / amax, i.e. to qmax, so the 6- and 8-bit widths
        # get the same bar scaled by qmax / 7 (4.4e-6 and 1.8e-5).
        allowed = max(1, int(1e-6 * (o.qmax_of(bits) / 7.0) * q_or.size))
        assert nm <= allowed, f"{label}: {nm} tie mismatches > {allowed}"
    say(f"  {label}: codes {q_or.size}, tie mismatches {nm}")
    return nm, q_or, s_or
