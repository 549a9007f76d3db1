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

The chain (calibration on the GPU, host transform construction, the four
device calls, the fp64 reference output y) is paper_2603_04359_amd.pipeline,
the same code the full-size layer tests check against the oracle.

Printed: one JSON line with the throughput, per-kernel times (mean, median,
min), the roofline of the dominant kernel, the CPU oracle baseline, and,
after the timed steps, the widened paths and a report over the other layer
configurations (tiny: SQNR per transform; attention and MLP-down: kernel
times and SQNR; stress: block-size sweep and 4/6/8-bit widths).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import threading
import time

# explicit thread counts for the CPU oracle's BLAS (the host's share of cores)
_CORES = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
for _v in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
    os.environ.setdefault(_v, str(_CORES))

import numpy as np  # noqa: E402

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
    p.add_argument("--no-report", action="store_true",
                   help="skip the widened paths and the other configurations after the steps")
    p.add_argument("--no-configs", action="store_true",
                   help="keep the widened paths of the metric layer, skip the other configurations")
    p.add_argument("--wide-steps", type=int, default=10,
                   help="timed iterations of each pair measured after the steps")
    p.add_argument("--cpu-seconds", type=float, default=10.0,
                   help="minimum oracle time of each CPU baseline sample")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="only run a plain device-to-device copy of MIB MiB (5 launches): "
                        "the known-size kernel that scales HBM byte counters")
    return p.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


GEMM_SOURCES = ("k_w4a4.hip", "device_common.h")   # the GEMM kernel and its device helpers


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


def stats(ms):
    ms = np.asarray(ms, dtype=np.float64)
    return {"mean": float(ms.mean()), "median": float(np.median(ms)), "min": float(ms.min()),
            "max": float(ms.max())}


# ------------------------------------------------------------ CPU baseline
def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(lay, T_vals, codes_w, s_w, n_tokens, min_seconds):
    """The CPU oracle (test infrastructure, never the product path) timed on
    this host on a bounded sample of the same workload: 512-token chunks
    of the step's batch through the oracle's Sigma_x, transform+quant,
    integer GEMM and SQNR (each timed), cycling over the batch, until at
    least `min_seconds` of oracle time have passed (at most 4 passes).
    Run twice: with every core of this process's affinity set, then with
    the BLAS pools limited to one thread."""
    from oracle import cat_oracle as o
    import threadpoolctl

    X = lay["X"]
    W64 = lay["W"].astype(np.float64)
    T = np.asarray(T_vals, dtype=np.float64)
    qw = o.unpack_int4(codes_w)

    def sample(limit):
        chunk, done, info = 512, 0, []
        part = {"second_moment": 0.0, "transform_quant": 0.0, "w4a4_linear": 0.0, "sqnr": 0.0}
        while done < 4 * n_tokens and (sum(part.values()) < min_seconds or done == 0):
            a = done % n_tokens
            xs = X[a:a + chunk].astype(np.float64)
            y = xs @ W64.T          # signal: input of the SQNR step, not timed
            with threadpoolctl.threadpool_limits(limits=limit):
                info = threadpoolctl.threadpool_info()
                t0 = time.perf_counter()
                o.second_moment_sum(xs)
                t1 = time.perf_counter()
                qx, sx = o.transform_quant(xs, T)
                t2 = time.perf_counter()
                _, yt = o.w4a4_linear(qx, sx, qw, s_w)
                t3 = time.perf_counter()
                o.sqnr(y, yt)
                t4 = time.perf_counter()
            for key, dt in zip(part, (t1 - t0, t2 - t1, t3 - t2, t4 - t3)):
                part[key] += dt
            done += xs.shape[0]
        total = sum(part.values())
        threads = max([i.get("num_threads", 1) for i in info] or [1])
        return done, total, part, threads, info

    done, total, part, threads, info = sample(None)
    d1, t1, p1, _, _ = sample(1)
    blas = [{k: i.get(k) for k in ("internal_api", "version", "num_threads", "threading_layer")}
            for i in info]
    return {"value": done / total, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{done} tokens ({done / n_tokens:.2f} passes over one step's "
                      f"{n_tokens}-token batch) in 512-token chunks, {total:.1f} s of oracle "
                      f"time (fp64 numpy); one-thread run: {d1} tokens in {t1:.1f} s",
            "seconds_per_part": part,
            "one_thread": {"value": d1 / t1, "unit": "tokens/s", "cores": 1,
                           "seconds_per_part": p1},
            "host": {"cpu_model": _cpu_model(), "os_cpu_count": os.cpu_count(),
                     "affinity_cores": _CORES, "blas": blas,
                     "env": {v: os.environ.get(v) for v in
                             ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")}}}


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


# --------------------------------------------- measured reference rates
def reference_rates(torch, n, d_in, d_out, iters=10):
    """Measured ceilings beside the published peaks, none of them part of
    the path: a 1 GiB device copy (HBM), hipBLASLt's int8 GEMM at the
    metric layer's shape through torch._int_mm (int8 operands, int32
    output, no dequantization) and a bf16 X^T X matmul at the batch's Sigma_x
    shape through torch.mm."""
    dev = torch.device("cuda:0")
    out = {}

    def timed(fn):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(iters + 1)]
        for i in range(iters):
            ev[i].record()
            fn()
        ev[iters].record()
        torch.cuda.synchronize()
        return stats([ev[i].elapsed_time(ev[i + 1]) for i in range(iters)])

    src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    st = timed(lambda: dst.copy_(src))
    out["hbm_copy"] = {"ms": st, "GBps": 2.0 * (1 << 30) / (st["median"] * 1e-3) / 1e9,
                       "bytes": "1 GiB read + 1 GiB written per call"}
    del src, dst
    g = torch.Generator(device=dev)
    g.manual_seed(1)
    a = torch.randint(-7, 8, (n, d_in), dtype=torch.int8, device=dev, generator=g)
    b = torch.randint(-7, 8, (d_in, d_out), dtype=torch.int8, device=dev, generator=g)
    try:
        st = timed(lambda: torch._int_mm(a, b))
        out["int8_gemm_hipblaslt"] = {"ms": st, "TOPS": gemm_ops_of(n, d_in, d_out) /
                                      (st["median"] * 1e-3) / 1e12,
                                      "shape": f"{n}x{d_in} @ {d_in}x{d_out}, int8 -> int32"}
    except RuntimeError as e:            # a torch build without the int8 path
        out["int8_gemm_hipblaslt"] = {"error": str(e)[:200]}
    del a, b
    x = torch.randn((n, d_in), dtype=torch.float32, device=dev, generator=g).to(torch.bfloat16)
    xt = x.t().contiguous()
    st = timed(lambda: torch.mm(xt, x))
    out["bf16_xtx_hipblaslt"] = {"ms": st, "TFLOPS": 2.0 * n * d_in * d_in /
                                 (st["median"] * 1e-3) / 1e12,
                                 "shape": f"{d_in}x{n} @ {n}x{d_in}, bf16 (full square)"}
    del x, xt
    torch.cuda.empty_cache()
    return out


# ------------------------------------------------------------ GPU clocks
class ClockSampler:
    """Samples the graphics and memory clocks of this process's GPU through
    amd-smi (matched by PCI address) every 2 ms on a side thread.  Reports
    nothing if the monitoring library is unavailable."""

    def __init__(self, torch):
        self.samples, self.handle, self.smi = [], None, None
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            props = torch.cuda.get_device_properties(0)
            want = f"{props.pci_domain_id:04x}:{props.pci_bus_id:02x}:{props.pci_device_id:02x}"
            for h in amdsmi.amdsmi_get_processor_handles():
                if amdsmi.amdsmi_get_gpu_device_bdf(h).lower().startswith(want):
                    self.handle = h
            self.smi = amdsmi
        except Exception:  # monitoring is optional
            self.handle = None

    def _read(self):
        gfx = self.smi.amdsmi_get_clock_info(self.handle, self.smi.AmdSmiClkType.GFX)
        mem = self.smi.amdsmi_get_clock_info(self.handle, self.smi.AmdSmiClkType.MEM)
        return gfx.get("clk"), mem.get("clk")

    def __enter__(self):
        self._stop = threading.Event()
        if self.handle is not None:
            def run():
                while not self._stop.is_set():
                    try:
                        self.samples.append(self._read())
                    except Exception:
                        return
                    time.sleep(0.002)
            self._thr = threading.Thread(target=run, daemon=True)
            self._thr.start()
        return self

    def __exit__(self, *a):
        self._stop.set()
        if self.handle is not None:
            self._thr.join(timeout=1.0)

    def summary(self):
        s = [x for x in self.samples if x[0] is not None]
        if not s:
            return None
        g = np.array([x[0] for x in s], dtype=np.float64)
        m = np.array([x[1] for x in s], dtype=np.float64)
        return {"samples": len(s), "gfx_MHz": {"median": float(np.median(g)), "min": float(g.min()),
                                               "max": float(g.max())},
                "mem_MHz": {"median": float(np.median(m)), "min": float(m.min()),
                            "max": float(m.max())}}


# ------------------------------------------------------------ helpers
def timed_pairs(torch, calls, iters):
    """Run `calls` (a list of callables) `iters` + 2 times; returns per-call
    event-timed ms of the last `iters` iterations."""
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)]
          for _ in range(iters)]
    for i in range(2 + iters):
        e = ev[i - 2] if i >= 2 else None
        for j, c in enumerate(calls):
            if e:
                e[j].record()
            c(i)
        if e:
            e[-1].record()
    torch.cuda.synchronize()
    return [[e[j].elapsed_time(e[j + 1]) for e in ev] for j in range(len(calls))]


def tq_bytes_of(n, d_in, k, x_bytes=2, t_bytes=2, code_bytes=0.5):
    return n * d_in * x_bytes + n * d_in * code_bytes + n * 4 + d_in * k * t_bytes


def gemm_ops_of(n, d_in, d_out):
    return 2.0 * n * d_in * d_out


def kernel_line(ms, work, unit, peak):
    """Event-timed ms statistics of one kernel and its rate at the median
    time in `unit` (GB/s, TOP/s or TFLOP/s), with the fraction of `peak`."""
    st = stats(ms)
    scale = 1e9 if unit == "GB/s" else 1e12
    rate = work / (st["median"] * 1e-3) / scale
    return {"ms": st, "rate": rate, "unit": unit, "frac_peak": rate / peak}


# --------------------------------------------- report: other configurations
def report_tiny(torch, cat, B, P, wl, seed):
    """Tiny fp32 layer: SQNR of the whole GPU chain for T = I, the block
    Hadamard H_32, the full Hadamard H_256 (one 256-block) and CAT (k = 32),
    at 4, 6 and 8 bits."""
    cfg = wl.get_config("tiny")
    lay = wl.make_layer(cfg, seed=seed)
    dev = torch.device("cuda:0")
    Xc = P.to_device(lay["X_cal"], "f32")
    X = P.to_device(lay["X"], "f32")
    y = P.reference_output(X, lay["W"])
    out = {}
    for label, k, flags in (("I", 32, 0), ("H_32 block", 32, B.CAT_BUILD_HADAMARD),
                            ("H_256 full", 256, B.CAT_BUILD_HADAMARD),
                            ("CAT_32", 32, B.CAT_BUILD_CAT)):
        sig = P.calibrate_blocks(Xc, k) if flags & B.CAT_BUILD_ALIGN else None
        layer = P.build_layer(sig, lay["W"], k, B.CAT_F32, flags=flags, bits=(4, 6, 8), device=dev)
        run = P.LayerRunner(layer, cfg.n, cfg.d_in, cfg.d_out, device=dev)
        for bits in (4, 6, 8):
            out.setdefault(f"W{bits}A{bits}", {})[label] = float(run.run(X, y, bits)[2])
    return {"workload": "tiny: 256->256 fp32, 2048 calibration / 512 eval tokens, seed "
                        f"{seed}", "sqnr_db": out}


def report_layer(torch, cat, B, P, wl, name, k, seed, iters):
    """A layer's four kernels at its full size: median event-timed ms and
    rate of transform+quant, the W4A4 GEMM, SQNR and the full Sigma_x of the
    batch, plus the chain's SQNR."""
    cfg = wl.get_config(name, k=k)
    n, d_in, d_out = cfg.n, cfg.d_in, cfg.d_out
    lay = wl.make_layer(cfg, seed=seed)
    Xc = P.to_device(lay["X_cal"], "bf16")
    sig = P.calibrate_blocks(Xc, k)
    del Xc, lay["X_cal"]
    torch.cuda.empty_cache()
    layer = P.build_layer(sig, lay["W"], k, B.CAT_BF16)
    X0 = P.to_device(lay["X"], "bf16")
    Xs = [X0, torch.roll(X0, shifts=1, dims=0).contiguous()]
    Ys = [P.reference_output(Xi, lay["W"]) for Xi in Xs]
    run = P.LayerRunner(layer, n, d_in, d_out)
    sigma = torch.zeros((d_in, d_in), dtype=torch.float32, device="cuda")
    ws_c = torch.empty(max(16, cat.cat_cov_workspace_bytes(B.CAT_BF16, n, d_in, B.CAT_COV_FULL,
                                                           1)), dtype=torch.uint8, device="cuda")
    ms = timed_pairs(torch, [lambda i: run.transform_quant(Xs[i % 2]), lambda i: run.linear(),
                             lambda i: run.sqnr(Ys[i % 2]),
                             lambda i: cat.cat_cov_accumulate(Xs[i % 2], sigma, B.CAT_COV_FULL,
                                                              1, ws_c)], iters)
    db = float(run.run(X0, Ys[0])[2])
    res = {"workload": f"{name}: {d_in}->{d_out}, block {k}, {n} tokens, "
                       f"{cfg.n_cal} calibration tokens, seed {seed}",
           "sqnr_db": db,
           "transform_quant": kernel_line(ms[0], tq_bytes_of(n, d_in, k), "GB/s",
                                          PEAK["hbm_GBps"]),
           "w4a4_linear": kernel_line(ms[1], gemm_ops_of(n, d_in, d_out), "TOP/s",
                                      PEAK["int8_TOPS"]),
           "sqnr": kernel_line(ms[2], 8.0 * n * d_out, "GB/s", PEAK["hbm_GBps"]),
           "cov_accumulate_full": kernel_line(ms[3], float(n) * d_in * (d_in + 1), "TFLOP/s",
                                              PEAK["bf16_TFLOPS"])}
    res["linear_tokens_per_s"] = n / ((res["transform_quant"]["ms"]["median"] +
                                       res["w4a4_linear"]["ms"]["median"]) * 1e-3)
    return res


def report_stress(torch, cat, B, P, wl, seed, iters):
    """Stress layer (8192 -> 28672, 16384 tokens): transform+quant time and
    the chain's SQNR for every block size of the sweep, the GEMM time, and
    the 4/6/8-bit widths at k = 128."""
    cfg = wl.get_config("stress")
    n, d_in, d_out = cfg.n, cfg.d_in, cfg.d_out
    lay = wl.make_layer(cfg, seed=seed)
    Xc = P.to_device(lay["X_cal"], "bf16")
    del lay["X_cal"]
    X0 = P.to_device(lay["X"], "bf16")
    Xs = [X0, torch.roll(X0, shifts=1, dims=0).contiguous()]
    y0 = P.reference_output(X0, lay["W"])
    sweep, widths, gemm = {}, {}, None
    for k in cfg.k_sweep:
        t0 = time.perf_counter()
        sig = P.calibrate_blocks(Xc, k)
        bits = (4, 6, 8) if k == 128 else (4,)
        layer = P.build_layer(sig, lay["W"], k, B.CAT_BF16, bits=bits)
        t_build = time.perf_counter() - t0
        run = P.LayerRunner(layer, n, d_in, d_out)
        ms = timed_pairs(torch, [lambda i: run.transform_quant(Xs[i % 2])], iters)
        db = float(run.run(X0, y0)[2])
        sweep[str(k)] = {"sqnr_db": db, "host_build_s": t_build,
                         "transform_quant": kernel_line(ms[0], tq_bytes_of(n, d_in, k), "GB/s",
                                                        PEAK["hbm_GBps"])}
        if k == 128:
            ms = timed_pairs(torch, [lambda i: run.linear()], iters)
            gemm = kernel_line(ms[0], gemm_ops_of(n, d_in, d_out), "TOP/s", PEAK["int8_TOPS"])
            widths["W4A4"] = {"sqnr_db": db}
            for b in (6, 8):
                ms = timed_pairs(torch, [lambda i, b=b: run.transform_quant(Xs[i % 2], b),
                                         lambda i, b=b: run.linear(b)], iters)
                widths[f"W{b}A{b}"] = {
                    "sqnr_db": float(run.run(X0, y0, b)[2]),
                    "transform_quant": kernel_line(ms[0], tq_bytes_of(n, d_in, k, code_bytes=1),
                                                   "GB/s", PEAK["hbm_GBps"]),
                    "int8_linear": kernel_line(ms[1], gemm_ops_of(n, d_in, d_out), "TOP/s",
                                               PEAK["int8_TOPS"])}
        del run, layer
        torch.cuda.empty_cache()
    return {"workload": f"stress: {d_in}->{d_out}, {n} tokens, {cfg.n_cal} calibration tokens, "
                        f"seed {seed}", "k_sweep": sweep, "w4a4_linear_k128": gemm,
            "widths_k128": widths}


# ------------------------------------------------------------------ main
def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the library has no "
              "multi-GPU path: collectives and sharding are design-only.", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2603_04359_amd as cat
    from paper_2603_04359_amd import binding as B
    from paper_2603_04359_amd import pipeline as P
    import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs an MI355X (no HIP device visible)", file=sys.stderr)
        sys.exit(3)
    torch.backends.cuda.matmul.allow_tf32 = False
    dev = torch.device("cuda:0")
    cfg = wl.get_config(args.config)
    d_in, d_out, k, n = cfg.d_in, cfg.d_out, cfg.k, cfg.n
    xdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    tdt = B.CAT_BF16 if cfg.dtype == "bf16" else B.CAT_F32
    log(f"[bench] generating {cfg.name} layer (seed {args.seed})")
    lay = wl.make_layer(cfg, seed=args.seed)

    # ---------------- calibration + transform construction (untimed set-up)
    log("[bench] calibration: block-diagonal Sigma_x on the GPU")
    Xc = P.to_device(lay["X_cal"], cfg.dtype)
    sig = P.calibrate_blocks(Xc, k)
    del Xc
    log("[bench] host transform construction")
    t0 = time.perf_counter()
    layer = P.build_layer(sig, lay["W"], k, tdt, bits=(4, 6, 8))
    t_build = time.perf_counter() - t0

    # ---------------- device-resident inputs (two alternating sets)
    X0 = P.to_device(lay["X"], cfg.dtype)
    Xs = [X0, torch.roll(X0, shifts=1, dims=0).contiguous()]
    # y: the unquantized layer output (the SQNR signal), fp64 on the device
    # and stored as fp32; an input of the sqnr step, formed once here
    Ys = [P.reference_output(Xi, lay["W"]) for Xi in Xs]
    run = P.LayerRunner(layer, n, d_in, d_out)
    sigma = torch.zeros((d_in, d_in), dtype=torch.float32, device=dev)
    ws_c = torch.empty(max(16, cat.cat_cov_workspace_bytes(
        B.CAT_BF16 if xdt == torch.bfloat16 else B.CAT_F32, n, d_in, B.CAT_COV_FULL, k)),
        dtype=torch.uint8, device=dev)

    def step(i, ev=None):
        Xi, Yi = Xs[i % 2], Ys[i % 2]
        if ev: ev[0].record()
        run.transform_quant(Xi)
        if ev: ev[1].record()
        run.linear()
        if ev: ev[2].record()
        run.sqnr(Yi)
        if ev: ev[3].record()
        cat.cat_cov_accumulate(Xi, sigma, B.CAT_COV_FULL, k, ws_c)
        if ev: ev[4].record()

    log(f"[bench] warmup {args.warmup} steps")
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    log(f"[bench] timing {args.steps} steps")
    clocks = ClockSampler(torch)
    torch.cuda.synchronize()
    with clocks:
        # a ~1 ms device spin ahead of the start event: while it runs the host
        # enqueues the first steps, so the first timed call does not include
        # the host's launch latency after the synchronize (it measured 113 us
        # against 32 us for transform_quant)
        if hasattr(torch.cuda, "_sleep"):
            torch.cuda._sleep(2_000_000)
        t_start.record()
        for i in range(args.steps):
            step(args.warmup + i, evs[i])
        t_end.record()
        torch.cuda.synchronize()
        # a sustained GEMM window after the steps, so the clock sampler sees
        # the power state of the dominant kernel over ~0.5 s
        if clocks.handle is not None:
            for _ in range(max(1, int(500 / 0.4))):
                run.linear()
            torch.cuda.synchronize()
    ms_step = t_start.elapsed_time(t_end) / args.steps
    names = ["transform_quant", "w4a4_linear", "sqnr", "cov_accumulate"]
    per_ms = {nm: [e[j].elapsed_time(e[j + 1]) for e in evs] for j, nm in enumerate(names)}
    per = {nm: float(np.mean(v)) for nm, v in per_ms.items()}
    log("[bench] per-call ms (mean): " + ", ".join(f"{k_}={v:.4f}" for k_, v in per.items()))

    # the chain's SQNR on the first input set (the value the full-size layer
    # test compares with the oracle's chain)
    sqnr_db = float(run.run(X0, Ys[0])[2])

    # ---------------- algorithmic work per launch
    gemm_ops = gemm_ops_of(n, d_in, d_out)
    gemm_bytes = n * d_in / 2 + n * 4 + d_out * d_in / 2 + d_out * 4 + n * d_out * 4
    tq_bytes = tq_bytes_of(n, d_in, k, 2 if xdt == torch.bfloat16 else 4,
                           2 if tdt == B.CAT_BF16 else 4)
    sq_bytes = 8.0 * n * d_out
    cov_flop = float(n) * d_in * (d_in + 1)
    t_g = per["w4a4_linear"] * 1e-3
    t_q = per["transform_quant"] * 1e-3
    t_s = per["sqnr"] * 1e-3
    t_c = per["cov_accumulate"] * 1e-3
    gemm_tops = gemm_ops / t_g / 1e12
    kernels = {
        "w4a4_linear": {"ms": per["w4a4_linear"], "ms_stats": stats(per_ms["w4a4_linear"]),
                        "TOPS": gemm_tops, "frac_int8_peak": gemm_tops / PEAK["int8_TOPS"],
                        "tokens_per_s": n / t_g},
        "transform_quant": {"ms": per["transform_quant"],
                            "ms_stats": stats(per_ms["transform_quant"]),
                            "GBps": tq_bytes / t_q / 1e9,
                            "frac_hbm_peak": tq_bytes / t_q / 1e9 / PEAK["hbm_GBps"],
                            "algorithmic_bytes": tq_bytes},
        "sqnr": {"ms": per["sqnr"], "ms_stats": stats(per_ms["sqnr"]),
                 "GBps": sq_bytes / t_s / 1e9,
                 "frac_hbm_peak": sq_bytes / t_s / 1e9 / PEAK["hbm_GBps"]},
        "cov_accumulate": {"ms": per["cov_accumulate"], "ms_stats": stats(per_ms["cov_accumulate"]),
                           "TFLOPS": cov_flop / t_c / 1e12,
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
        "dtypes": {"transform_quant": "bf16 MFMA -> int4",
                   "w4a4_linear": "int4 codes on int8 MFMA -> int32 -> f32",
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
        "clocks": clocks.summary(),
        "host_transform_build_s": t_build,
    }

    if not args.no_report:
        widened(rec, torch, cat, B, P, layer, run, Xs, Ys, lay, n, d_in, d_out, k, tdt,
                tq_bytes, gemm_ops, args.wide_steps)
        log("[bench] measured reference rates (device copy, hipBLASLt int8 GEMM, bf16 X^T X)")
        rec["references"] = reference_rates(torch, n, d_in, d_out)
    if not args.no_report and not args.no_configs:
        # free the metric layer before the other configurations
        del run, Xs, Ys, X0, sigma, ws_c
        torch.cuda.empty_cache()
        rep = {}
        log("[bench] report: tiny layer transforms")
        rep["tiny"] = report_tiny(torch, cat, B, P, wl, args.seed)
        for name, kk in (("attn4096", 128), ("mlp_down", 256)):
            log(f"[bench] report: {name}")
            rep[name] = report_layer(torch, cat, B, P, wl, name, kk, args.seed, args.wide_steps)
            torch.cuda.empty_cache()
        log("[bench] report: stress block-size sweep and widths")
        rep["stress"] = report_stress(torch, cat, B, P, wl, args.seed, args.wide_steps)
        rec["configs_report"] = rep

    if not args.no_cpu_baseline:
        log("[bench] CPU oracle baseline (all cores, then one thread)")
        T_vals = wl.bf16_bits_to_f32(layer["T_host"]) if tdt == B.CAT_BF16 else layer["T_host"]
        rec["cpu_baseline"] = cpu_baseline(lay, T_vals, layer["weights"][4]["codes_host"],
                                           layer["weights"][4]["s_host"], n, args.cpu_seconds)
    print(json.dumps(rec), flush=True)


def widened(rec, torch, cat, B, P, layer, run, Xs, Ys, lay, n, d_in, d_out, k, tdt, tq_bytes,
            gemm_ops, iters):
    """After the timed steps (same layer and batch, not part of the step):
    the W6A6 / W8A8 widths, the Theorem 2.4 terms, the full-dimension
    Hadamard and asymmetric activations."""
    T_dev, Wp = layer["T"], layer["W_prime"]
    wide = {"W4A4": {"sqnr_db": rec["sqnr_db"]}}
    for bits in (6, 8):
        ms = timed_pairs(torch, [lambda i, b=bits: run.transform_quant(Xs[i % 2], b),
                                 lambda i, b=bits: run.linear(b)], iters)
        db = float(run.run(Xs[0], Ys[0], bits)[2])
        tq_ms, g_ms = float(np.mean(ms[0])), float(np.mean(ms[1]))
        tq_b = tq_bytes + n * d_in / 2          # one byte per code instead of half
        g_tops = gemm_ops / (g_ms * 1e-3) / 1e12
        wide[f"W{bits}A{bits}"] = {
            "sqnr_db": db,
            "transform_quant": {"ms": tq_ms, "ms_stats": stats(ms[0]),
                                "GBps": tq_b / (tq_ms * 1e-3) / 1e9,
                                "frac_hbm_peak": tq_b / (tq_ms * 1e-3) / 1e9 / PEAK["hbm_GBps"]},
            "int8_linear": {"ms": g_ms, "ms_stats": stats(ms[1]), "TOPS": g_tops,
                            "frac_int8_peak": g_tops / PEAK["int8_TOPS"]},
            "linear_tokens_per_s": n / ((tq_ms + g_ms) * 1e-3)}
        log(f"[bench] W{bits}A{bits}: transform_quant {tq_ms:.4f} ms, int8_linear {g_ms:.4f} ms "
            f"({g_tops:.0f} TOP/s), SQNR {db:.2f} dB")
    rec["wide_codes"] = wide

    # the Theorem 2.4 decomposition of the W4A4 layer from device results
    # (per-token scales, the batch's block second-moment sums, sum y^2)
    res = run.run(Xs[0], Ys[0], 4)
    acc_e = torch.zeros((d_in // k, k, k), dtype=torch.float32, device="cuda")
    cat.cat_cov_accumulate(Xs[0], acc_e, B.CAT_COV_BLOCK_DIAG, k)
    torch.cuda.synchronize()
    terms = cat.cat_sqnr_terms(run.s_x.cpu().numpy(), 4, acc_e.double().cpu().numpy(),
                               layer["T_host"], tdt, Wp, 4, float(res[0]))
    terms["measured_db"] = float(res[2])
    rec["theorem_2_4"] = terms
    log(f"[bench] Theorem 2.4: predicted {terms['sqnr_pred_db']:.2f} dB, measured {res[2]:.2f} dB")

    # full-dimension Hadamard T = H_d blockdiag(M_b), INT4
    rec_full = None
    if cat.cat_transform_quant_full_workspace_bytes(n, d_in, k) and tdt == B.CAT_BF16 and \
            k in (128, 256):
        cw_h, sw_h = cat.cat_quantize_weights(cat.cat_full_hadamard_weights(Wp, k), 4)
        cw, sw = torch.from_numpy(cw_h).cuda(), torch.from_numpy(sw_h).cuda()
        ws_f = torch.empty(cat.cat_transform_quant_full_workspace_bytes(n, d_in, k),
                           dtype=torch.uint8, device="cuda")
        ms = timed_pairs(torch, [
            lambda i: cat.cat_transform_quant_full(Xs[i % 2], T_dev, k, run.codes4, run.s_x, ws_f),
            lambda i: cat.cat_w4a4_linear(run.codes4, run.s_x, cw, sw, run.y_t)], iters)
        cat.cat_transform_quant_full(Xs[0], T_dev, k, run.codes4, run.s_x, ws_f)
        cat.cat_w4a4_linear(run.codes4, run.s_x, cw, sw, run.y_t)
        run.sqnr(Ys[0])
        torch.cuda.synchronize()
        tq_ms, g_ms = float(np.mean(ms[0])), float(np.mean(ms[1]))
        rec_full = {"sqnr_db": float(run.out[2].item()), "transform_quant_full_ms": tq_ms,
                    "transform_quant_full_ms_stats": stats(ms[0]),
                    "w4a4_linear_ms": g_ms, "linear_tokens_per_s": n / ((tq_ms + g_ms) * 1e-3)}
        log(f"[bench] full-dimension Hadamard: transform_quant {tq_ms:.4f} ms, SQNR "
            f"{rec_full['sqnr_db']:.2f} dB")
        del ws_f
    rec["full_hadamard"] = rec_full

    # asymmetric per-token activations (the paper's own activation set-up)
    w4 = layer["weights"][4]
    zmin = torch.empty(n, dtype=torch.float32, device="cuda")
    rsum = torch.from_numpy(cat.cat_weight_code_sums(w4["codes_host"])).cuda()
    ms = timed_pairs(torch, [
        lambda i: cat.cat_transform_quant_asym(Xs[i % 2], T_dev, k, run.codes4, run.s_x, zmin,
                                               run.ws_q),
        lambda i: cat.cat_w4a4_linear_asym(run.codes4, run.s_x, zmin, w4["codes"], w4["s"], rsum,
                                           run.y_t)], iters)
    cat.cat_transform_quant_asym(Xs[0], T_dev, k, run.codes4, run.s_x, zmin, run.ws_q)
    cat.cat_w4a4_linear_asym(run.codes4, run.s_x, zmin, w4["codes"], w4["s"], rsum, run.y_t)
    run.sqnr(Ys[0])
    torch.cuda.synchronize()
    tq_ms, g_ms = float(np.mean(ms[0])), float(np.mean(ms[1]))
    g_tops = gemm_ops / (g_ms * 1e-3) / 1e12
    rec["asymmetric_activations"] = {
        "sqnr_db": float(run.out[2].item()), "sqnr_db_symmetric": rec["sqnr_db"],
        "transform_quant": {"ms": tq_ms, "ms_stats": stats(ms[0]),
                            "GBps": (tq_bytes + 4 * n) / (tq_ms * 1e-3) / 1e9},
        "w4a4_linear": {"ms": g_ms, "ms_stats": stats(ms[1]), "TOPS": g_tops,
                        "frac_int8_peak": g_tops / PEAK["int8_TOPS"]},
        "linear_tokens_per_s": n / ((tq_ms + g_ms) * 1e-3)}
    log(f"[bench] asymmetric INT4: transform_quant {tq_ms:.4f} ms, w4a4_linear {g_ms:.4f} ms, "
        f"SQNR {rec['asymmetric_activations']['sqnr_db']:.2f} dB")


if __name__ == "__main__":
    main()
