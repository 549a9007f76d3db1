#!/usr/bin/env python3
"""Throughput of the CAT W4A4 linear-layer hot path on one MI355X.

One step = one pass of the whole path over one batch of N tokens of the
4096 -> 14336 MLP-up layer (block size 128, N = 8192), every part a HIP
kernel behind the C ABI:
  transform_quant  z = T x (block-diagonal, bf16 MFMA) + per-token INT4
  w4a4_linear      int4 x int4 GEMM on int8 MFMA + dequantization
  sqnr             fp64 reduction of sum y^2 and sum (y - y~)^2
  cov_accumulate   Sigma_x += X^T X over the batch (bf16 MFMA, full
                   symmetric 4096 x 4096)
Inputs are resident in HBM before timing starts.  Two input sets alternate
between steps so the 256 MiB last-level cache never holds a step's
activations when its transform_quant starts (the sqnr pass of the previous
step streams ~900 MiB in between).

Printed: one JSON line (rank 0) with the throughput, per-kernel times,
the roofline of the dominant kernel and the CPU oracle baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {  # MI355X published dense peaks
    "hbm_GBps": 8000.0,
    "int8_TOPS": 5033.2,
    "bf16_TFLOPS": 2516.6,
}
METRIC = ("CAT W4A4 linear tokens/s + TOPS (% int8 MFMA peak) at 4096→14336; quant GB/s")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--config", default="mlp_up")
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--wide-steps", type=int, default=10,
                   help="timed iterations of each 6- and 8-bit comparison pair")
    p.add_argument("--cpu-seconds", type=float, default=10.0,
                   help="minimum CPU time of the oracle sample")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="only run a plain device-to-device copy of MIB MiB (5 launches): "
                        "the known-size kernel that scales HBM byte counters")
    return p.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


GEMM_SOURCES = ("k_w4a4.hip", "device_common.h", "kernels.h")


def kernel_sources_sha():
    """Hash of the sources the W4A4 GEMM kernel is built from: the stored
    counter figures apply only while it matches."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2603_04359_amd", "csrc")
    for f in GEMM_SOURCES:
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary,
    or None when the kernel sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("sources_sha") != kernel_sources_sha():
        return None
    ent = rec.get("kernels", {}).get(kernel)
    return None if ent is None else ent.get("hbm_bytes_per_launch")


def cpu_baseline(lay, T_vals, codes_w, s_w, n_tokens, min_seconds):
    """The CPU oracle (test infrastructure, never the product path) timed on
    this host on a bounded sample of the same workload: 512-token chunks
    of the step's batch run through the oracle's Sigma_x, transform+quant,
    integer GEMM and SQNR, cycling over the batch, until at least
    `min_seconds` of oracle time have passed (and at most 4 passes)."""
    from oracle import cat_oracle as o
    try:
        import threadpoolctl
        threads = max(i["num_threads"] for i in threadpoolctl.threadpool_info()) \
            if threadpoolctl.threadpool_info() else 1
    except Exception:  # pragma: no cover
        threads = os.cpu_count()
    X = lay["X"]
    W32 = lay["W"]
    T = np.asarray(T_vals, dtype=np.float64)
    qw = o.unpack_int4(codes_w)
    chunk, done, t_total = 512, 0, 0.0
    while done < 4 * n_tokens and (t_total < min_seconds or done == 0):
        a = done % n_tokens
        xs = X[a:a + chunk].astype(np.float64)
        y = xs.astype(np.float32) @ W32.T   # signal: input of the SQNR step, not timed
        t0 = time.perf_counter()
        o.second_moment_sum(xs)
        qx, sx = o.transform_quant(xs, T)
        _, yt = o.w4a4_linear(qx, sx, qw, s_w)
        o.sqnr(y, yt)
        t_total += time.perf_counter() - t0
        done += xs.shape[0]
    return {"value": done / t_total, "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{done} tokens ({done / n_tokens:.2f} passes over one step's "
                      f"{n_tokens}-token batch) in 512-token chunks, {t_total:.1f} s of "
                      f"oracle time (fp64 numpy, os.cpu_count()={os.cpu_count()})"}


def copy_calibration(mib):
    """Five launches of torch's device copy of `mib` MiB: each reads and
    writes exactly mib*2^20 bytes, so FETCH_SIZE / WRITE_SIZE read under
    rocprofv3 for it give the factor from counter units to HBM bytes."""
    import torch
    dev = torch.device("cuda:0")
    src = torch.ones(mib << 18, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": mib << 20, "launches": 5}), flush=True)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); this build has no "
              "multi-GPU path: collectives and sharding are design-only.", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2603_04359_amd as cat
    from paper_2603_04359_amd import binding as B
    import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs an MI355X (no HIP device visible)", file=sys.stderr)
        sys.exit(3)
    torch.backends.cuda.matmul.allow_tf32 = False
    dev = torch.device("cuda:0")
    cfg = wl.get_config(args.config)
    d_in, d_out, k, n = cfg.d_in, cfg.d_out, cfg.k, cfg.n
    xdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    log(f"[bench] generating {cfg.name} layer (seed {args.seed})")
    lay = wl.make_layer(cfg, seed=args.seed)

    # ---------------- calibration + transform construction (untimed set-up)
    log("[bench] calibration: block-diagonal Sigma_x on the GPU")
    Xc = torch.from_numpy(lay["X_cal"]).to(dev).to(xdt)
    acc_blk = torch.zeros((d_in // k, k, k), dtype=torch.float32, device=dev)
    for a in range(0, cfg.n_cal, 8192):
        cat.cat_cov_accumulate(Xc[a:a + 8192], acc_blk, B.CAT_COV_BLOCK_DIAG, k)
    torch.cuda.synchronize()
    del Xc
    sx_blocks = acc_blk.double().cpu().numpy() / cfg.n_cal
    log("[bench] host transform construction")
    t0 = time.perf_counter()
    tdt = B.CAT_BF16 if cfg.dtype == "bf16" else B.CAT_F32
    T_host, _, Wp = cat.cat_build_transform(sx_blocks, lay["W"], k, B.CAT_BUILD_CAT, tdt)
    codes_w_h, s_w_h = cat.cat_quantize_weights(Wp, 4)
    t_build = time.perf_counter() - t0

    # ---------------- device-resident inputs (two alternating sets)
    X0 = torch.from_numpy(lay["X"]).to(dev).to(xdt)
    if tdt == B.CAT_BF16:
        T_dev = torch.from_numpy(T_host.view(np.int16)).to(dev).view(torch.bfloat16)
    else:
        T_dev = torch.from_numpy(T_host).to(dev)
    W_dev = torch.from_numpy(lay["W"]).to(dev)
    # y: the unquantized layer output (the SQNR signal), an input of the
    # sqnr step synthesised once here in fp32
    Xs = [X0, torch.roll(X0, shifts=1, dims=0).contiguous()]
    Ys = []
    for Xi in Xs:
        Ys.append(torch.matmul(Xi.float(), W_dev.t()).contiguous())
    del W_dev
    codes_w = torch.from_numpy(codes_w_h).to(dev)
    s_w = torch.from_numpy(s_w_h).to(dev)
    codes = torch.empty((n, d_in // 2), dtype=torch.uint8, device=dev)
    s_x = torch.empty(n, dtype=torch.float32, device=dev)
    ws_q = torch.empty(cat.cat_transform_quant_workspace_bytes(n, d_in, k), dtype=torch.uint8,
                       device=dev)
    y_t = torch.empty((n, d_out), dtype=torch.float32, device=dev)
    ws_s = torch.empty(cat.cat_sqnr_workspace_bytes(n * d_out), dtype=torch.uint8, device=dev)
    out = torch.empty(3, dtype=torch.float64, device=dev)
    sigma = torch.zeros((d_in, d_in), dtype=torch.float32, device=dev)
    ws_c = torch.empty(max(16, cat.cat_cov_workspace_bytes(
        B.CAT_BF16 if xdt == torch.bfloat16 else B.CAT_F32, n, d_in, B.CAT_COV_FULL, k)),
        dtype=torch.uint8, device=dev)

    def step(i, ev=None):
        Xi, Yi = Xs[i % 2], Ys[i % 2]
        if ev: ev[0].record()
        cat.cat_transform_quant(Xi, T_dev, k, codes, s_x, ws_q)
        if ev: ev[1].record()
        cat.cat_w4a4_linear(codes, s_x, codes_w, s_w, y_t)
        if ev: ev[2].record()
        cat.cat_sqnr(Yi, y_t, ws_s, out)
        if ev: ev[3].record()
        cat.cat_cov_accumulate(Xi, sigma, B.CAT_COV_FULL, k, ws_c)
        if ev: ev[4].record()

    log(f"[bench] warmup {args.warmup} steps")
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    sqnr_db = float(out[2].item())
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    log(f"[bench] timing {args.steps} steps")
    torch.cuda.synchronize()
    t_start.record()
    for i in range(args.steps):
        step(args.warmup + i, evs[i])
    t_end.record()
    torch.cuda.synchronize()
    ms_step = t_start.elapsed_time(t_end) / args.steps
    names = ["transform_quant", "w4a4_linear", "sqnr", "cov_accumulate"]
    per = {nm: float(np.mean([e[j].elapsed_time(e[j + 1]) for e in evs]))
           for j, nm in enumerate(names)}
    log("[bench] per-call ms: " + ", ".join(f"{k_}={v:.4f}" for k_, v in per.items()))

    # ---------------- algorithmic work per launch
    gemm_ops = 2.0 * n * d_in * d_out
    gemm_bytes = n * d_in / 2 + n * 4 + d_out * d_in / 2 + d_out * 4 + n * d_out * 4
    tq_bytes = n * d_in * (2 if xdt == torch.bfloat16 else 4) + n * d_in / 2 + n * 4 + \
        d_in * k * (2 if tdt == B.CAT_BF16 else 4)
    sq_bytes = 8.0 * n * d_out
    cov_flop = float(n) * d_in * (d_in + 1)
    t_g = per["w4a4_linear"] * 1e-3
    t_q = per["transform_quant"] * 1e-3
    t_s = per["sqnr"] * 1e-3
    t_c = per["cov_accumulate"] * 1e-3
    gemm_tops = gemm_ops / t_g / 1e12
    kernels = {
        "w4a4_linear": {"ms": per["w4a4_linear"], "TOPS": gemm_tops,
                        "frac_int8_peak": gemm_tops / PEAK["int8_TOPS"],
                        "tokens_per_s": n / t_g},
        "transform_quant": {"ms": per["transform_quant"], "GBps": tq_bytes / t_q / 1e9,
                            "frac_hbm_peak": tq_bytes / t_q / 1e9 / PEAK["hbm_GBps"],
                            "algorithmic_bytes": tq_bytes},
        "sqnr": {"ms": per["sqnr"], "GBps": sq_bytes / t_s / 1e9,
                 "frac_hbm_peak": sq_bytes / t_s / 1e9 / PEAK["hbm_GBps"]},
        "cov_accumulate": {"ms": per["cov_accumulate"], "TFLOPS": cov_flop / t_c / 1e12,
                           "frac_bf16_peak": cov_flop / t_c / 1e12 / PEAK["bf16_TFLOPS"]},
    }
    traffic = measured_traffic("w4a4_linear")
    roofline = {"bound": "mfma", "achieved": gemm_tops, "peak": PEAK["int8_TOPS"],
                "unit": "TFLOP/s", "frac": gemm_tops / PEAK["int8_TOPS"], "traffic": traffic,
                "kernel": "w4a4_linear (int8 MFMA, TOP/s)",
                "algorithmic_ops_per_launch": gemm_ops,
                "algorithmic_bytes_per_launch": gemm_bytes}
    rec = {
        "metric": METRIC,
        "value": n / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "dtypes": {"transform_quant": "bf16 MFMA -> int4", "w4a4_linear": "int4 codes on int8 MFMA -> int32 -> f32",
                   "sqnr": "f32 -> f64", "cov_accumulate": "bf16 MFMA -> f32"},
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: CAT W4A4 linear {d_in}->{d_out}, block {k}, "
                               f"{n} tokens per step (transform+quant, W4A4 GEMM, SQNR, "
                               f"Sigma_x accumulation over the batch)",
                   "d_in": d_in, "d_out": d_out, "block": k, "tokens_per_step": n,
                   "calibration_tokens": cfg.n_cal, "seed": args.seed},
        "linear_tokens_per_s": n / (t_q + t_g),
        "gemm_TOPS": gemm_tops,
        "quant_GBps": tq_bytes / t_q / 1e9,
        "sqnr_db": sqnr_db,
        "kernels": kernels,
        "roofline": roofline,
        "host_transform_build_s": t_build,
    }
    # ---------------- the W6A6 / W8A8 comparison widths (after the timed
    # steps; not part of the step): the same layer and tokens through
    # transform+quant at 6 or 8 bits and the int8-code GEMM
    wide = {"W4A4": {"sqnr_db": sqnr_db}}
    codes8 = torch.empty((n, d_in), dtype=torch.int8, device=dev)
    for bits in (6, 8):
        cw_h, sw_h = cat.cat_quantize_weights(Wp, bits)
        cw, sw = torch.from_numpy(cw_h).to(dev), torch.from_numpy(sw_h).to(dev)
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)]
              for _ in range(args.wide_steps)]
        for i in range(2 + args.wide_steps):
            e = ev[i - 2] if i >= 2 else None
            if e: e[0].record()
            cat.cat_transform_quant(Xs[i % 2], T_dev, k, codes8, s_x, ws_q, bits=bits)
            if e: e[1].record()
            cat.cat_int8_linear(codes8, s_x, cw, sw, y_t)
            if e: e[2].record()
        cat.cat_sqnr(Ys[(1 + args.wide_steps) % 2], y_t, ws_s, out)
        torch.cuda.synchronize()
        tq_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
        g_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
        tq_b = tq_bytes + n * d_in / 2          # one byte per code instead of half
        g_tops = gemm_ops / (g_ms * 1e-3) / 1e12
        wide[f"W{bits}A{bits}"] = {
            "sqnr_db": float(out[2].item()),
            "transform_quant": {"ms": tq_ms, "GBps": tq_b / (tq_ms * 1e-3) / 1e9,
                                "frac_hbm_peak": tq_b / (tq_ms * 1e-3) / 1e9 / PEAK["hbm_GBps"]},
            "int8_linear": {"ms": g_ms, "TOPS": g_tops, "frac_int8_peak": g_tops / PEAK["int8_TOPS"]},
            "linear_tokens_per_s": n / ((tq_ms + g_ms) * 1e-3)}
        log(f"[bench] W{bits}A{bits}: transform_quant {tq_ms:.4f} ms, int8_linear {g_ms:.4f} ms "
            f"({g_tops:.0f} TOP/s), SQNR {wide[f'W{bits}A{bits}']['sqnr_db']:.2f} dB")
    # ---------------- the Theorem 2.4 decomposition of the W4A4 layer from
    # device results (per-token scales, the batch's block second-moment
    # sums, sum y^2), after the timed steps
    cat.cat_transform_quant(Xs[0], T_dev, k, codes, s_x, ws_q)
    cat.cat_w4a4_linear(codes, s_x, codes_w, s_w, y_t)
    cat.cat_sqnr(Ys[0], y_t, ws_s, out)
    acc_e = torch.zeros((d_in // k, k, k), dtype=torch.float32, device=dev)
    cat.cat_cov_accumulate(Xs[0], acc_e, B.CAT_COV_BLOCK_DIAG, k)
    torch.cuda.synchronize()
    res = out.cpu().numpy()
    terms = cat.cat_sqnr_terms(s_x.cpu().numpy(), 4, acc_e.double().cpu().numpy(), T_host, tdt,
                               Wp, 4, float(res[0]))
    terms["measured_db"] = float(res[2])
    rec["theorem_2_4"] = terms
    log(f"[bench] Theorem 2.4: predicted {terms['sqnr_pred_db']:.2f} dB, measured {res[2]:.2f} dB")

    # ---------------- full-dimension Hadamard T = H_d blockdiag(M_b), INT4,
    # after the timed steps
    if cat.cat_transform_quant_full_workspace_bytes(n, d_in, k) and tdt == B.CAT_BF16 and \
            k in (128, 256):
        cw_h, sw_h = cat.cat_quantize_weights(cat.cat_full_hadamard_weights(Wp, k), 4)
        cw, sw = torch.from_numpy(cw_h).to(dev), torch.from_numpy(sw_h).to(dev)
        ws_f = torch.empty(cat.cat_transform_quant_full_workspace_bytes(n, d_in, k),
                           dtype=torch.uint8, device=dev)
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)]
              for _ in range(args.wide_steps)]
        for i in range(2 + args.wide_steps):
            e = ev[i - 2] if i >= 2 else None
            if e: e[0].record()
            cat.cat_transform_quant_full(Xs[i % 2], T_dev, k, codes, s_x, ws_f)
            if e: e[1].record()
            cat.cat_w4a4_linear(codes, s_x, cw, sw, y_t)
            if e: e[2].record()
        cat.cat_sqnr(Ys[(1 + args.wide_steps) % 2], y_t, ws_s, out)
        torch.cuda.synchronize()
        tq_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
        g_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
        rec_full = {"sqnr_db": float(out[2].item()), "transform_quant_full_ms": tq_ms,
                    "w4a4_linear_ms": g_ms, "linear_tokens_per_s": n / ((tq_ms + g_ms) * 1e-3)}
        log(f"[bench] full-dimension Hadamard: transform_quant {tq_ms:.4f} ms, SQNR "
            f"{rec_full['sqnr_db']:.2f} dB")
        del ws_f
    else:
        rec_full = None
    del Wp
    rec["wide_codes"] = wide
    rec["full_hadamard"] = rec_full

    # ---------------- asymmetric per-token activations (the paper's own
    # activation set-up), INT4, after the timed steps
    zmin = torch.empty(n, dtype=torch.float32, device=dev)
    rsum = torch.from_numpy(cat.cat_weight_code_sums(codes_w_h)).to(dev)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.wide_steps)]
    for i in range(2 + args.wide_steps):
        e = ev[i - 2] if i >= 2 else None
        if e: e[0].record()
        cat.cat_transform_quant_asym(Xs[i % 2], T_dev, k, codes, s_x, zmin, ws_q)
        if e: e[1].record()
        cat.cat_w4a4_linear_asym(codes, s_x, zmin, codes_w, s_w, rsum, y_t)
        if e: e[2].record()
    cat.cat_sqnr(Ys[(1 + args.wide_steps) % 2], y_t, ws_s, out)
    torch.cuda.synchronize()
    tq_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    g_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    g_tops = gemm_ops / (g_ms * 1e-3) / 1e12
    rec["asymmetric_activations"] = {
        "sqnr_db": float(out[2].item()), "sqnr_db_symmetric": sqnr_db,
        "transform_quant": {"ms": tq_ms, "GBps": (tq_bytes + 4 * n) / (tq_ms * 1e-3) / 1e9},
        "w4a4_linear": {"ms": g_ms, "TOPS": g_tops, "frac_int8_peak": g_tops / PEAK["int8_TOPS"]},
        "linear_tokens_per_s": n / ((tq_ms + g_ms) * 1e-3)}
    log(f"[bench] asymmetric INT4: transform_quant {tq_ms:.4f} ms, w4a4_linear {g_ms:.4f} ms, "
        f"SQNR {rec['asymmetric_activations']['sqnr_db']:.2f} dB")

    if not args.no_cpu_baseline:
        log("[bench] CPU oracle baseline")
        T_vals = wl.bf16_bits_to_f32(T_host) if tdt == B.CAT_BF16 else T_host
        rec["cpu_baseline"] = cpu_baseline(lay, T_vals, codes_w_h, s_w_h, n, args.cpu_seconds)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
