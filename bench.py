"""Benchmark of the IF4 quantized-linear hot path on one MI355X.

One step = one forward pass of an IF4 linear layer at the MLP up-projection
shape: quantize the bf16 activations A [8192, 4096] and weights W
[14336, 4096] along K (tensor max pass + quantize pass each), then the
IF4 x IF4 GEMM Y = A_hat W_hat^T with bf16 output.  Inputs are resident in
HBM before timing starts.  `value` is the step's whole-job throughput,
2*M*N*K / step time.

Also reported (one JSON line): per-kernel times from HIP events on the
launch stream, the roofline of the dominant kernel (the GEMM, MFMA-bound) and
of the quantizer (HBM-bound), the same kernels in NVFP4 mode, and the CPU
oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "IF4 quantize GB/s (%HBM peak) + IF4 GEMM TFLOP/s (%MFMA peak), 1 MI355X"
HBM_PEAK_GBS = 8000.0
FP16_MFMA_PEAK_TFLOPS = 2500.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-rows", type=int, default=0,
                   help="activation rows in the CPU oracle's GEMM sample (0: all)")
    p.add_argument("--traffic-from", metavar="DIR",
                   help="read rocprofv3 FETCH_SIZE/WRITE_SIZE counter CSVs of a --mode step run "
                        "(DIR/pmc_FETCH_SIZE, DIR/pmc_WRITE_SIZE) and write profiles/hbm_traffic.json")
    p.add_argument("--format", choices=["if4", "nvfp4", "if3", "if6_e2m3", "if6_e3m2", "nvint4",
                                        "nvfp4_46", "if4_bs8", "if3_bs8", "nvfp4_bs8"], default="if4",
                   help="format of the --mode step run")
    p.add_argument("--small", action="store_true", help="1/8-size shapes (quick checks)")
    p.add_argument("--mode", choices=["full", "step", "copy", "wgrad", "bitwidth", "dual", "dequant"], default="full",
                   help="step: only the timed IF4 step (for counter runs); copy: a plain 1 GiB "
                        "device copy, the reference for scaling the HBM byte counters")
    return p.parse_args()


def main():
    args = parse()
    if args.traffic_from:
        record_traffic(args.traffic_from)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the kernels run on one "
              "GPU's share of the work; no path across several GPUs is built.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2603_28765_amd import ops, workloads

    torch.cuda.set_device(0)
    if args.mode == "copy":
        n = 1 << 30
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"mode": "copy", "bytes_read_per_launch": n, "bytes_written_per_launch": n}))
        return
    if args.mode == "wgrad":
        print(json.dumps({"mode": "wgrad", **wgrad_times(ops, workloads, torch)}))
        return
    if args.mode == "bitwidth":
        print(json.dumps({"mode": "bitwidth", **bitwidth_times(ops, workloads, torch)}))
        return
    if args.mode == "dual":
        print(json.dumps({"mode": "dual", **dual_times(ops, workloads, torch)}))
        return
    if args.mode == "dequant":
        print(json.dumps({"mode": "dequant", **dequant_times(ops, workloads, torch)}))
        return
    div = 8 if args.small else 1
    M, N, K = 8192 // div, 14336 // div, 4096 // div
    w = workloads.fwd_mlp(M, N, K)
    A = w.tensors["A"].cuda()
    W = w.tensors["W"].cuda()
    dev = A.device

    def alloc(fmt, rows, cols):
        return ops.Packed(fmt, torch.empty((rows, cols * ops.BITS[fmt] // 8), dtype=torch.uint8, device=dev),
                          torch.empty((rows, cols // ops.GSIZE[fmt]), dtype=torch.uint8, device=dev),
                          torch.empty(1, dtype=torch.float32, device=dev), rows, cols)

    ws = torch.empty(4096, dtype=torch.uint8, device=dev)
    Y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)

    def run(fmt, pa, pw, ev=None):
        if ev: ev[0].record()
        ops.ifx_quantize(fmt, A, out=pa, workspace=ws)
        if ev: ev[1].record()
        ops.ifx_quantize(fmt, W, out=pw, workspace=ws)
        if ev: ev[2].record()
        ops.ifx_gemm(pa, pw, ops.BF16, Y)
        if ev: ev[3].record()

    def timed(fmt, steps, warmup):
        pa, pw = alloc(fmt, M, K), alloc(fmt, N, K)
        for _ in range(warmup):
            run(fmt, pa, pw)
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
        t0 = time.perf_counter()
        for i in range(steps):
            run(fmt, pa, pw, evs[i])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        qa = np.mean([e[0].elapsed_time(e[1]) for e in evs]) * 1e-3
        qw = np.mean([e[1].elapsed_time(e[2]) for e in evs]) * 1e-3
        gm = np.mean([e[2].elapsed_time(e[3]) for e in evs]) * 1e-3
        step = np.mean([e[0].elapsed_time(e[3]) for e in evs]) * 1e-3
        return {"wall_s": wall, "step_s": step, "quant_A_s": qa, "quant_W_s": qw, "gemm_s": gm}

    # single-pass quantize kernel alone (alpha supplied): the HBM-bound kernel.
    # Launches run back to back between two events and cycle through COPIES
    # copies of x and of the outputs: a copy was last touched COPIES - 1
    # launches earlier (over 256 MB of other traffic), so every launch reads
    # x from HBM, not from the 256 MB infinity cache, and no per-launch event
    # or cache flush sits between the launches.
    COPIES = 5

    def timed_scale_in(fmt, x, steps, warmup):
        q = ops.if4_quantize if fmt == ops.IF4 else ops.nvfp4_quantize
        xs = [x.clone() for _ in range(COPIES)]
        ps = [alloc(fmt, x.shape[0], x.shape[1]) for _ in range(COPIES)]
        q(x, out=ps[0], workspace=ws)
        ts = ps[0].tensor_scale.clone()
        n = max(2 * steps, 8 * COPIES)
        for i in range(max(warmup, COPIES)):
            q(xs[i % COPIES], flags=ops.SCALE_IN, tensor_scale=ts, out=ps[i % COPIES])
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(n):
            q(xs[i % COPIES], flags=ops.SCALE_IN, tensor_scale=ts, out=ps[i % COPIES])
        e1.record()
        torch.cuda.synchronize()
        del xs, ps
        return e0.elapsed_time(e1) * 1e-3 / n

    if args.mode == "step":
        fmt = {v: k for k, v in ops.FORMAT_NAMES.items()}[args.format]
        r = timed(fmt, args.steps, args.warmup)
        print(json.dumps({"mode": "step", "format": args.format, "ms_per_step": r["step_s"] * 1e3,
                          "gemm_us": r["gemm_s"] * 1e6, "quant_A_us": r["quant_A_s"] * 1e6,
                          "quant_W_us": r["quant_W_s"] * 1e6}))
        return
    res = timed(ops.IF4, args.steps, args.warmup)
    res_nv = timed(ops.NVFP4, max(5, args.steps // 2), 2)
    n_a, n_w = M * K, N * K
    flops = 2.0 * M * N * K
    qbytes_2pass = lambda n: n * (2 + 2 + 0.5 + 1 / 16)  # read for max, read + write codes/scales
    qbytes_1pass = lambda n: n * (2 + 0.5 + 1 / 16)
    t_w_1p = timed_scale_in(ops.IF4, W, max(5, args.steps // 2), 2)
    t_w_1p_nv = timed_scale_in(ops.NVFP4, W, max(5, args.steps // 2), 2)

    gemm_tflops = flops / res["gemm_s"] / 1e12
    out = {
        "metric": METRIC,
        "value": round(flops / res["step_s"] / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(res["step_s"] * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp16",
        "data": "synthetic (seeded; activations t(4) x lognormal channel scales, weights N(0,0.02^2))",
        "config": {"workload": f"fwd_mlp_up_{M}x{N}x{K}", "format": "IF4", "M": M, "N": N, "K": K,
                   "quantize": "row-wise along K, round-to-nearest, alpha from tensor max",
                   "out": "bf16"},
        "roofline": {"bound": "mfma", "achieved": round(gemm_tflops, 2),
                     "peak": FP16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(gemm_tflops / FP16_MFMA_PEAK_TFLOPS, 4),
                     "traffic": recorded_traffic("gemm", (M, N, K)),
                     "traffic_unit": "HBM bytes per launch", "kernel": "gemm_tn_fast<IF4, bf16 out>"},
        "roofline_quantize": {
            "bound": "hbm", "kernel": "quantize_rows<IF4> (alpha supplied, single pass, W)",
            "achieved": round(qbytes_1pass(n_w) / t_w_1p / 1e9, 1), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(qbytes_1pass(n_w) / t_w_1p / 1e9 / HBM_PEAK_GBS, 4),
            "traffic": recorded_traffic("quantize_W", (N, K)), "traffic_unit": "HBM bytes per launch"},
        "components": {
            "if4": {"quant_A_us": round(res["quant_A_s"] * 1e6, 2),
                    "quant_A_GBps_2pass": round(qbytes_2pass(n_a) / res["quant_A_s"] / 1e9, 1),
                    "quant_W_us": round(res["quant_W_s"] * 1e6, 2),
                    "quant_W_GBps_2pass": round(qbytes_2pass(n_w) / res["quant_W_s"] / 1e9, 1),
                    "quant_W_1pass_us": round(t_w_1p * 1e6, 2),
                    "gemm_us": round(res["gemm_s"] * 1e6, 2),
                    "gemm_TFLOPs": round(gemm_tflops, 2)},
            "nvfp4": {"quant_A_us": round(res_nv["quant_A_s"] * 1e6, 2),
                      "quant_W_us": round(res_nv["quant_W_s"] * 1e6, 2),
                      "quant_W_1pass_us": round(t_w_1p_nv * 1e6, 2),
                      "quant_W_1pass_GBps": round(qbytes_1pass(n_w) / t_w_1p_nv / 1e9, 1),
                      "gemm_us": round(res_nv["gemm_s"] * 1e6, 2),
                      "gemm_TFLOPs": round(flops / res_nv["gemm_s"] / 1e12, 2),
                      "step_ms": round(res_nv["step_s"] * 1e3, 4)},
        },
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, M, N, K, args.cpu_rows or M)
    print(json.dumps(out), flush=True)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
# Kernels whose HBM traffic bench.py reports: record key -> (kernel name in
# the profiler, which of its dispatches per step, sources it is built from).
TRAFFIC_KERNELS = {
    "gemm": ("ifq::gemm_tn_fast<0, true>", None,
             ("paper_2603_28765_amd/csrc/gemm.hip", "paper_2603_28765_amd/csrc/device.h")),
    "quantize_W": ("ifq::quantize_rows<0, false, false>", 1,
                   ("paper_2603_28765_amd/csrc/quantize.hip", "paper_2603_28765_amd/csrc/device.h")),
}
# Per-dispatch calibration of the byte counters against a plain 1 GiB device
# copy (bench.py --mode copy): FETCH_SIZE reads back half the bytes read,
# WRITE_SIZE the bytes written.
FETCH_SCALE, WRITE_SCALE = 2.0, 1.0


def _event_time(torch, fn, steps, warmup, flush=None):
    """Mean time of fn() in seconds from HIP events on the current stream;
    with `flush`, a 512 MiB buffer is rewritten before every launch so the
    kernel reads from HBM."""
    times = []
    for i in range(warmup + steps):
        if flush is not None:
            flush.fill_(i & 0xFF)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        if i >= warmup:
            times.append(e0.elapsed_time(e1) * 1e-3)
    return float(sum(times) / len(times))


def _steady_time(torch, fn, steps=10, warmup=20):
    """Mean time of fn() in seconds under sustained load, as in the timed
    step: `warmup` launches back to back (the GEMM's power-management
    transient settles within them), then `steps` launches back to back, each
    between two HIP events, with one synchronisation at the end."""
    for _ in range(warmup):
        fn()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for e0, e1 in evs:
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    return float(sum(e0.elapsed_time(e1) for e0, e1 in evs) / steps * 1e-3)


def wgrad_times(ops, workloads, torch):
    """Weight gradient dW = dY^T X (dY 8192 x 14336, X 8192 x 4096, both
    quantized along the token axis with RHT, SR and the 16/17 margin; fp32
    out): quantizer times (two-pass, and single-pass with alpha supplied and
    a cache flush) and the GEMM M = 14336, N = 4096, K = 8192."""
    w = workloads.wgrad()
    dy, x = w.tensors["dY"].cuda(), w.tensors["X"].cuda()
    ws = torch.empty(4096, dtype=torch.uint8, device="cuda")
    fl = ops.AXIS_STRIDED | ops.RHT | ops.SR | ops.MARGIN_16_17
    signs = w.info["rht_signs"]
    sd, sx = w.info["sr_seed_dY"], w.info["sr_seed_X"]
    pdy = ops.if4_quantize(dy, fl, signs, sd, workspace=ws)
    px = ops.if4_quantize(x, fl, signs, sx, workspace=ws)
    flush = torch.empty(512 * 1024 * 1024, dtype=torch.uint8, device="cuda")
    t_dy = _event_time(torch, lambda: ops.if4_quantize(dy, fl, signs, sd, out=pdy, workspace=ws), 10, 2, flush)
    t_dy1 = _event_time(torch, lambda: ops.if4_quantize(dy, fl | ops.SCALE_IN, signs, sd,
                                                        tensor_scale=pdy.tensor_scale, out=pdy), 10, 2, flush)
    t_x = _event_time(torch, lambda: ops.if4_quantize(x, fl, signs, sx, out=px, workspace=ws), 10, 2, flush)
    del flush
    M, N, K = w.info["M"], w.info["N"], w.info["K"]
    out = torch.empty((M, N), dtype=torch.float32, device="cuda")
    t_g = _steady_time(torch, lambda: ops.if4_gemm(pdy, px, ops.F32, out), 20)
    n_dy = dy.numel()
    return {"workload": f"wgrad_{M}x{N}x{K}", "quant_dY_us": round(t_dy * 1e6, 1),
            "quant_dY_1pass_us": round(t_dy1 * 1e6, 1),
            "quant_dY_1pass_GBps": round(n_dy * 2.5625 / t_dy1 / 1e9, 1),
            "quant_X_us": round(t_x * 1e6, 1), "gemm_us": round(t_g * 1e6, 1),
            "gemm_TFLOPs": round(2.0 * M * N * K / t_g / 1e12, 1)}


def bitwidth_times(ops, workloads, torch):
    """Bit-width study: A, B 8192 x 8192 (N(0,1), 0.05 % of elements x100)
    quantized along K in every format (both passes, cache flushed), then the
    8192^3 GEMM with bf16 out under sustained load."""
    w = workloads.bitwidth()
    a, b = w.tensors["A"].cuda(), w.tensors["B"].cuda()
    n = a.shape[0]
    ws = torch.empty(4096, dtype=torch.uint8, device="cuda")
    out = torch.empty((n, n), dtype=torch.bfloat16, device="cuda")
    res = {"workload": f"bitwidth_{n}^3"}
    flush = torch.empty(512 * 1024 * 1024, dtype=torch.uint8, device="cuda")
    for fmt, name in ops.FORMAT_NAMES.items():
        pa, pb = ops.ifx_quantize(fmt, a, workspace=ws), ops.ifx_quantize(fmt, b, workspace=ws)
        t_q = _event_time(torch, lambda: ops.ifx_quantize(fmt, a, out=pa, workspace=ws), 5, 2, flush)
        t_g = _steady_time(torch, lambda: ops.ifx_gemm(pa, pb, ops.BF16, out), 10)
        res[name] = {"quant_us": round(t_q * 1e6, 1), "gemm_us": round(t_g * 1e6, 1),
                     "gemm_TFLOPs": round(2.0 * n ** 3 / t_g / 1e12, 1)}
        del pa, pb
    return res


def dual_times(ops, workloads, torch):
    """Training-step quantization of one linear layer's tensors in both
    layouts (X 8192 x 4096 and W 14336 x 4096 with RTN, RHT on X's token
    side; dY 8192 x 14336 with SR, RHT + SR + margin on its token side): two
    separate quantizer calls against one dual call, each with a cache flush;
    and the activation-gradient GEMM dX = dY W (M = 8192, N = 4096,
    K = 14336, dY row-wise, W along its rows), bf16 out."""
    wg = workloads.wgrad()
    fw = workloads.fwd_mlp()
    dy, x, W = wg.tensors["dY"].cuda(), fw.tensors["A"].cuda(), fw.tensors["W"].cuda()
    signs = wg.info["rht_signs"]
    flush = torch.empty(512 * 1024 * 1024, dtype=torch.uint8, device="cuda")
    res = {}
    for name, t, rf, cf in (("X", x, 0, ops.RHT), ("W", W, 0, 0),
                            ("dY", dy, ops.SR, ops.RHT | ops.SR | ops.MARGIN_16_17)):
        pr, pc = ops.ifx_quantize_dual(ops.IF4, t, rf, cf, signs, 1, 2)
        ws = torch.empty(4096, dtype=torch.uint8, device="cuda")
        sep = _event_time(torch, lambda: (ops.if4_quantize(t, rf, signs, 1, out=pr, workspace=ws),
                                          ops.if4_quantize(t, cf | ops.AXIS_STRIDED, signs, 2, out=pc,
                                                           workspace=ws)), 10, 2, flush)
        dual = _event_time(torch, lambda: ops.ifx_quantize_dual(ops.IF4, t, rf, cf, signs, 1, 2, out_row=pr,
                                                                out_col=pc, workspace=ws), 10, 2, flush)
        res[name] = {"shape": list(t.shape), "separate_us": round(sep * 1e6, 1), "dual_us": round(dual * 1e6, 1)}
    del flush
    pdy, _ = ops.ifx_quantize_dual(ops.IF4, dy, ops.SR, ops.RHT | ops.SR | ops.MARGIN_16_17, signs, 1, 2)
    _, pw = ops.ifx_quantize_dual(ops.IF4, W)
    M, N, K = dy.shape[0], W.shape[1], dy.shape[1]
    out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    t_g = _steady_time(torch, lambda: ops.if4_gemm(pdy, pw, ops.BF16, out), 20)
    res["dgrad"] = {"workload": f"dgrad_{M}x{N}x{K}", "gemm_us": round(t_g * 1e6, 1),
                    "gemm_TFLOPs": round(2.0 * M * N * K / t_g / 1e12, 1)}
    return res


def dequant_times(ops, workloads, torch):
    """Standalone dequantizer on the weights W 14336 x 4096 in every format,
    bf16 and fp32 out, cache flushed before every launch.  Algorithmic bytes
    per element: codes b/8 + scales 1/G read, 2 or 4 written."""
    W = workloads.fwd_mlp().tensors["W"].cuda()
    n = W.numel()
    ws = torch.empty(4096, dtype=torch.uint8, device="cuda")
    flush = torch.empty(512 * 1024 * 1024, dtype=torch.uint8, device="cuda")
    res = {"workload": f"dequant_{W.shape[0]}x{W.shape[1]}"}
    for fmt, name in ops.FORMAT_NAMES.items():
        p = ops.ifx_quantize(fmt, W, workspace=ws)
        read = ops.BITS[fmt] / 8 + 1 / ops.GSIZE[fmt]
        r = {}
        for dt, tag, wb in ((ops.BF16, "bf16", 2), (ops.F32, "fp32", 4)):
            out = ops.ifx_dequantize(p, dt)
            t = _event_time(torch, lambda: ops.ifx_dequantize(p, dt, out), 10, 2, flush)
            r[tag + "_us"] = round(t * 1e6, 1)
            r[tag + "_GBps"] = round(n * (read + wb) / t / 1e9, 1)
            del out
        res[name] = r
        del p
    del flush
    return res


def _sources_digest(files):
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_traffic(key, shape):
    """Counter-measured HBM bytes per launch of kernel `key`, or None when the
    record is missing, was taken at another shape, or the kernel's sources
    changed since."""
    try:
        with open(TRAFFIC_FILE) as fh:
            rec = json.load(fh)[key]
    except (OSError, KeyError, ValueError):
        return None
    if rec.get("sha256") != _sources_digest(TRAFFIC_KERNELS[key][2]) or rec.get("shape") != list(shape):
        return None
    return int(rec["fetch_bytes"] + rec["write_bytes"])


def record_traffic(d):
    import csv

    def per_dispatch(sub, kernel, which):
        vals = []
        for root, _, files in os.walk(os.path.join(d, sub)):
            for f in sorted(files):
                if f.endswith("counter_collection.csv"):
                    with open(os.path.join(root, f)) as fh:
                        vals += [float(r["Counter_Value"]) for r in csv.DictReader(fh)
                                 if r["Kernel_Name"].replace("void ", "").startswith(kernel)]
        if which is not None:  # every second dispatch: the W operand of each step
            vals = vals[which::2]
        if not vals:
            raise SystemExit(f"no {kernel} dispatches under {os.path.join(d, sub)}")
        return sum(vals) / len(vals) * 1024.0

    shapes = {"gemm": [8192, 14336, 4096], "quantize_W": [14336, 4096]}
    rec = {}
    for key, (kernel, which, sources) in TRAFFIC_KERNELS.items():
        rec[key] = {"kernel": kernel, "shape": shapes[key], "sources": list(sources),
                    "sha256": _sources_digest(sources),
                    "fetch_bytes": round(per_dispatch("pmc_FETCH_SIZE", kernel, which) * FETCH_SCALE),
                    "write_bytes": round(per_dispatch("pmc_WRITE_SIZE", kernel, which) * WRITE_SCALE),
                    "calibration": {"FETCH_SIZE": FETCH_SCALE, "WRITE_SIZE": WRITE_SCALE}}
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    print(json.dumps(rec))


def cpu_baseline(w, M, N, K, rows):
    """The CPU oracle on a bounded sample of the same step: the C oracle
    quantizes all of A and W (one thread; the step's whole quantize work),
    then its reference GEMM (dequantize to fp64, numpy BLAS product) runs for
    `rows` rows of A against all of W.  The product's time is scaled by
    M/rows; the quantize time and W's dequantize are taken as measured."""
    import numpy as np
    import torch

    import oracle as O
    from threadpoolctl import threadpool_info

    def bits(t):
        return t.contiguous().view(torch.int16).numpy().view(np.uint16)

    a, wt = bits(w.tensors["A"]), bits(w.tensors["W"])
    t0 = time.perf_counter()
    ca, sa, aa = O.quantize(a, O.FMT_IF4)
    cw, sw, aw = O.quantize(wt, O.FMT_IF4)
    t_q = time.perf_counter() - t0
    t1 = time.perf_counter()
    Wd = O.dequantize(cw, sw, aw, O.FMT_IF4, np.float64)
    t_dw = time.perf_counter() - t1
    t2 = time.perf_counter()
    Ad = O.dequantize(ca[:rows], sa[:rows], aa, O.FMT_IF4, np.float64)
    _ = Ad @ Wd.T
    t_g = time.perf_counter() - t2
    blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    t_full = t_q + t_dw + t_g * M / rows
    flops = 2.0 * M * N * K
    return {"value": round(flops / t_full / 1e12, 6), "unit": "TFLOP/s",
            "cores": int(blas_threads), "kind": "oracle",
            "sample": f"IF4 quantize of all of A and W (C oracle, 1 thread, {t_q:.2f} s), "
                      f"fp64 dequantize of W ({t_dw:.2f} s), reference GEMM of {rows} of {M} rows of A "
                      f"against all {N} rows of W (numpy BLAS, {blas_threads} threads, {t_g:.2f} s, "
                      f"scaled by M/{rows})",
            "seconds": round(t_q + t_dw + t_g, 2)}


if __name__ == "__main__":
    main()
