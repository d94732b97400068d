"""Benchmark of the IF4 quantized-linear hot path on one MI355X.

One step = one forward pass of an IF4 linear layer at the MLP up-projection
shape: quantize the bf16 activations A [8192, 4096] and weights W
[14336, 4096] along K (tensor max pass + quantize pass each), then the
IF4 x IF4 GEMM Y = A_hat W_hat^T with bf16 output.  Inputs are resident in
HBM before timing starts.  `value` is the step's whole-job throughput,
2*M*N*K / step time.

Also reported (one JSON line on stdout; progress lines go to stderr):
per-kernel times from HIP events on the launch stream, the roofline of the
dominant kernel (the GEMM, MFMA-bound) and of the quantizer (HBM-bound), the
same kernels in NVFP4 mode, the other measured workloads (the 8192^2
quantizer sweep with and without the RHT, the weight-gradient quantizers and
GEMM, the bit-width GEMMs at 8192^3, the dequantizer), and the CPU oracle
timed on a bounded sample of the step, single- and multi-threaded.
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
    p.add_argument("--no-workloads", action="store_true",
                   help="skip the other measured workloads (quantizer sweep, weight gradient, "
                        "bit-width GEMMs, dequantizer) in the default run")
    p.add_argument("--cpu-rows", type=int, default=0,
                   help="activation rows in the CPU oracle's GEMM sample (0: all)")
    p.add_argument("--traffic-from", metavar="DIR",
                   help="read rocprofv3 FETCH_SIZE/WRITE_SIZE counter CSVs of a --mode step run "
                        "(DIR/pmc_FETCH_SIZE, DIR/pmc_WRITE_SIZE) and write profiles/hbm_traffic.json")
    p.add_argument("--format", choices=["if4", "nvfp4", "if3", "if6_e2m3", "if6_e3m2", "nvint4",
                                        "nvfp4_46", "if4_bs8", "if3_bs8", "nvfp4_bs8"], default="if4",
                   help="format of the --mode step run")
    p.add_argument("--small", action="store_true", help="1/8-size shapes (quick checks)")
    p.add_argument("--mode", choices=["full", "step", "copy", "sweep", "wgrad", "bitwidth", "dual",
                                      "dequant", "context"], default="full",
                   help="step: only the timed IF4 step (for counter runs); copy: a plain 1 GiB "
                        "device copy, the reference for scaling the HBM byte counters; sweep, "
                        "wgrad, bitwidth, dequant: one of the other workloads alone; context: "
                        "a device copy and a library FP16 GEMM at the step's sizes")
    return p.parse_args()


def log(msg):
    print(f"bench: {msg}", file=sys.stderr, flush=True)


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
    single = {"sweep": quant_sweep_times, "wgrad": wgrad_times, "bitwidth": bitwidth_times,
              "dual": dual_times, "dequant": dequant_times, "context": context_times}
    if args.mode in single:
        print(json.dumps({"mode": args.mode, **single[args.mode](ops, workloads, torch)}))
        return
    div = 8 if args.small else 1
    M, N, K = 8192 // div, 14336 // div, 4096 // div
    t_gen = time.perf_counter()
    w = workloads.fwd_mlp(M, N, K)
    A = w.tensors["A"].cuda()
    W = w.tensors["W"].cuda()
    dev = A.device
    log(f"forward workload {M}x{N}x{K} generated ({time.perf_counter() - t_gen:.1f} s)")

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
        pa, pw = alloc(ops, torch, fmt, M, K), alloc(ops, torch, fmt, N, K)
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

    if args.mode == "step":
        fmt = {v: k for k, v in ops.FORMAT_NAMES.items()}[args.format]
        r = timed(fmt, args.steps, args.warmup)
        print(json.dumps({"mode": "step", "format": args.format, "ms_per_step": r["step_s"] * 1e3,
                          "gemm_us": r["gemm_s"] * 1e6, "quant_A_us": r["quant_A_s"] * 1e6,
                          "quant_W_us": r["quant_W_s"] * 1e6}))
        return
    # The other measured workloads run first: the step is then timed with
    # the device already under sustained load, as in serving or training,
    # rather than inside the power-management transient of a cold start.
    extra = {}
    if not args.no_workloads and not args.small:
        for key, fn in (("quant_sweep", quant_sweep_times), ("wgrad", wgrad_times),
                        ("bitwidth", bitwidth_times), ("dequant", dequant_times),
                        ("context", context_times)):
            t0 = time.perf_counter()
            extra[key] = fn(ops, workloads, torch)
            torch.cuda.empty_cache()
            log(f"{key} workload timed ({time.perf_counter() - t0:.1f} s)")
    res = timed(ops.IF4, args.steps, args.warmup)
    log(f"IF4 step timed: {res['step_s'] * 1e3:.3f} ms (GEMM {res['gemm_s'] * 1e6:.1f} us)")
    res_nv = timed(ops.NVFP4, max(5, args.steps // 2), 2)
    n_a, n_w = M * K, N * K
    flops = 2.0 * M * N * K
    qbytes_2pass = lambda n: n * (2 + 2 + 0.5 + 1 / 16)  # read for max, read + write codes/scales
    qbytes_1pass = lambda n: n * (2 + 0.5 + 1 / 16)
    t_w_1p = single_pass_time(ops, torch, ops.IF4, W, 0, max(5, args.steps // 2))
    t_w_1p_nv = single_pass_time(ops, torch, ops.NVFP4, W, 0, max(5, args.steps // 2))
    log(f"single-pass quantizer on W timed: IF4 {t_w_1p * 1e6:.1f} us, NVFP4 {t_w_1p_nv * 1e6:.1f} us")

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
                      "quant_W_1pass_frac": round(qbytes_1pass(n_w) / t_w_1p_nv / 1e9 / HBM_PEAK_GBS, 4),
                      "gemm_us": round(res_nv["gemm_s"] * 1e6, 2),
                      "gemm_TFLOPs": round(flops / res_nv["gemm_s"] / 1e12, 2),
                      "gemm_frac": round(flops / res_nv["gemm_s"] / 1e12 / FP16_MFMA_PEAK_TFLOPS, 4),
                      "step_ms": round(res_nv["step_s"] * 1e3, 4)},
        },
    }
    del A, W, Y
    torch.cuda.empty_cache()
    if extra:
        out["workloads"] = extra
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, M, N, K, args.cpu_rows or M)
        log("cpu baseline timed")
    print(json.dumps(out), flush=True)


def alloc(ops, torch, fmt, rows, cols, dev="cuda"):
    return ops.Packed(fmt, torch.empty((rows, cols * ops.BITS[fmt] // 8), dtype=torch.uint8, device=dev),
                      torch.empty((rows, cols // ops.GSIZE[fmt]), dtype=torch.uint8, device=dev),
                      torch.empty(1, dtype=torch.float32, device=dev), rows, cols)


def rotating_time(torch, fns, n, warmup=None, min_warm_s=0.02):
    """Mean time of one launch in seconds, for launches that cycle through
    len(fns) copies of their data: fns[i % len(fns)]() runs n times back to
    back between two HIP events on the current stream, with no per-launch
    event or cache flush between the launches.  With enough copies a copy
    was last touched after more than the 256 MB infinity cache of other
    traffic, so every launch reads its input from HBM.  Warm-up: batches of
    max(len(fns), warmup) launches until at least min_warm_s of them have
    run, so that the timed launches find the clocks settled under this
    load (the first milliseconds after a change of workload run slower)."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    batch, warm, i = max(len(fns), warmup or 0), 0.0, 0
    while warm < min_warm_s and i < 100000:
        e0.record()
        for _ in range(batch):
            fns[i % len(fns)]()
            i += 1
        e1.record()
        torch.cuda.synchronize()
        warm += e0.elapsed_time(e1) * 1e-3
    e0.record()
    for k in range(n):  # the rotation continues where the warm-up stopped
        fns[(i + k) % len(fns)]()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e-3 / n


def _copies_for(nbytes_per_launch, floor=3):
    """Copies needed so that a copy's last use lies over 600 MB of other
    traffic in the past (well beyond the 256 MB infinity cache)."""
    return max(floor, int(600e6 // max(nbytes_per_launch, 1)) + 2)


def single_pass_time(ops, torch, fmt, x, flags, steps, signs=0, seed=0):
    """The quantize pass alone (alpha supplied): back-to-back launches over
    rotating copies of x and of the outputs."""
    R, Kq = (x.shape[1], x.shape[0]) if flags & ops.AXIS_STRIDED else (x.shape[0], x.shape[1])
    n = x.numel()
    copies = _copies_for(n * (2 + ops.BITS[fmt] / 8 + 1 / ops.GSIZE[fmt]), 5)
    p0 = ops.ifx_quantize(fmt, x, flags, signs, seed)
    ts = p0.tensor_scale.clone()
    xs = [x] + [x.clone() for _ in range(copies - 1)]
    ps = [alloc(ops, torch, fmt, R, Kq) for _ in range(copies)]
    fns = [lambda i=i: ops.ifx_quantize(fmt, xs[i], flags | ops.SCALE_IN, signs, seed, tensor_scale=ts,
                                        out=ps[i]) for i in range(copies)]
    t = rotating_time(torch, fns, max(2 * steps, 8 * copies), 5)
    del xs, ps, p0
    return t


def two_pass_time(ops, torch, fmt, x, flags, steps, signs=0, seed=0):
    """Tensor-max pass + quantize pass (alpha from Eq. 1), back to back over
    rotating copies."""
    R, Kq = (x.shape[1], x.shape[0]) if flags & ops.AXIS_STRIDED else (x.shape[0], x.shape[1])
    n = x.numel()
    copies = _copies_for(n * (4 + ops.BITS[fmt] / 8 + 1 / ops.GSIZE[fmt]), 4)
    xs = [x] + [x.clone() for _ in range(copies - 1)]
    ps = [alloc(ops, torch, fmt, R, Kq) for _ in range(copies)]
    wss = [torch.empty(4096, dtype=torch.uint8, device="cuda") for _ in range(copies)]
    fns = [lambda i=i: ops.ifx_quantize(fmt, xs[i], flags, signs, seed, out=ps[i], workspace=wss[i])
           for i in range(copies)]
    t = rotating_time(torch, fns, max(2 * steps, 8 * copies), 5)
    del xs, ps
    return t


def _quant_record(ops, fmt, n, t1, t2):
    b = 2 + ops.BITS[fmt] / 8 + 1 / ops.GSIZE[fmt]
    r = {"1pass_us": round(t1 * 1e6, 2), "1pass_GBps": round(n * b / t1 / 1e9, 1),
         "1pass_frac": round(n * b / t1 / 1e9 / HBM_PEAK_GBS, 4)}
    if t2 is not None:
        r.update({"2pass_us": round(t2 * 1e6, 2),
                  "2pass_GBps_algorithmic": round(n * b / t2 / 1e9, 1),
                  "2pass_GBps_traffic": round(n * (b + 2) / t2 / 1e9, 1)})
    return r


def quant_sweep_times(ops, workloads, torch):
    """Quantizer bandwidth sweep: X 8192 x 8192 t(3) * 0.5 with 0.1 % of
    columns x50, row-wise, IF4 and NVFP4, with and without the fused 16-point
    RHT: the quantize pass alone (alpha supplied) and both passes (alpha
    from the tensor maximum), each over rotating copies (read from HBM).
    Algorithmic bytes per element: 2 read, 0.5 + 1/16 written."""
    w = workloads.quant_sweep()
    x = w.tensors["X"].cuda()
    signs = w.info["rht_signs"]
    n = x.numel()
    res = {"workload": f"quant_sweep_{x.shape[0]}x{x.shape[1]}",
           "bytes_per_element": {"1pass": 2.5625, "2pass_traffic": 4.5625}}
    for fmt in (ops.IF4, ops.NVFP4):
        for rht in (False, True):
            fl = ops.RHT if rht else 0
            t1 = single_pass_time(ops, torch, fmt, x, fl, 20, signs)
            t2 = two_pass_time(ops, torch, fmt, x, fl, 20, signs)
            res[f"{ops.FORMAT_NAMES[fmt]}{'_rht' if rht else ''}"] = _quant_record(ops, fmt, n, t1, t2)
    return res


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


def _gemm_record(M, N, K, t):
    tf = 2.0 * M * N * K / t / 1e12
    return {"gemm_us": round(t * 1e6, 1), "gemm_TFLOPs": round(tf, 1),
            "gemm_frac": round(tf / FP16_MFMA_PEAK_TFLOPS, 4)}


def wgrad_times(ops, workloads, torch):
    """Weight gradient dW = dY^T X (dY 8192 x 14336, X 8192 x 4096, both
    quantized along the token axis with RHT, SR and the 16/17 margin; fp32
    out): each quantizer's pass alone (alpha supplied) and both passes, over
    rotating copies, and the GEMM M = 14336, N = 4096, K = 8192 under
    sustained load, in IF4 and NVFP4."""
    w = workloads.wgrad()
    dy, x = w.tensors["dY"].cuda(), w.tensors["X"].cuda()
    fl = ops.AXIS_STRIDED | ops.RHT | ops.SR | ops.MARGIN_16_17
    signs = w.info["rht_signs"]
    sd, sx = w.info["sr_seed_dY"], w.info["sr_seed_X"]
    M, N, K = w.info["M"], w.info["N"], w.info["K"]
    res = {"workload": f"wgrad_{M}x{N}x{K}",
           "quantize": "strided (token axis), RHT + SR + 16/17 margin"}
    out = torch.empty((M, N), dtype=torch.float32, device="cuda")
    for fmt in (ops.IF4, ops.NVFP4):
        r = {}
        for name, t, seed in (("dY", dy, sd), ("X", x, sx)):
            t1 = single_pass_time(ops, torch, fmt, t, fl, 10, signs, seed)
            t2 = two_pass_time(ops, torch, fmt, t, fl, 10, signs, seed)
            r[f"quant_{name}"] = _quant_record(ops, fmt, t.numel(), t1, t2)
        pdy = ops.ifx_quantize(fmt, dy, fl, signs, sd)
        px = ops.ifx_quantize(fmt, x, fl, signs, sx)
        r.update(_gemm_record(M, N, K, _steady_time(torch, lambda: ops.ifx_gemm(pdy, px, ops.F32, out), 10)))
        res[ops.FORMAT_NAMES[fmt]] = r
        del pdy, px
    return res


def bitwidth_times(ops, workloads, torch):
    """Bit-width study: A, B 8192 x 8192 (N(0,1), 0.05 % of elements x100)
    quantized along K in every format (both passes, rotating copies of A),
    then the 8192^3 GEMM with bf16 out under sustained load."""
    w = workloads.bitwidth()
    a, b = w.tensors["A"].cuda(), w.tensors["B"].cuda()
    n = a.shape[0]
    out = torch.empty((n, n), dtype=torch.bfloat16, device="cuda")
    res = {"workload": f"bitwidth_{n}^3"}
    for fmt, name in ops.FORMAT_NAMES.items():
        pa, pb = ops.ifx_quantize(fmt, a), ops.ifx_quantize(fmt, b)
        t_q = two_pass_time(ops, torch, fmt, a, 0, 10)
        t_g = _steady_time(torch, lambda: ops.ifx_gemm(pa, pb, ops.BF16, out), 10)
        r = {"quant_2pass_us": round(t_q * 1e6, 1)}
        r.update(_gemm_record(n, n, n, t_g))
        res[name] = r
        del pa, pb
    return res


def dequant_times(ops, workloads, torch):
    """Standalone dequantizer on the weights W 14336 x 4096, bf16 and fp32
    out, over rotating copies of the packed input and of the output.
    Algorithmic bytes per element: codes b/8 + scales 1/G read, 2 or 4
    written."""
    W = workloads.fwd_mlp().tensors["W"].cuda()
    n = W.numel()
    res = {"workload": f"dequant_{W.shape[0]}x{W.shape[1]}"}
    for fmt in (ops.IF4, ops.NVFP4, ops.NVINT4, ops.IF3, ops.IF6_E2M3):
        p = ops.ifx_quantize(fmt, W)
        read = ops.BITS[fmt] / 8 + 1 / ops.GSIZE[fmt]
        r = {}
        for dt, tag, wb in ((ops.BF16, "bf16", 2), (ops.F32, "fp32", 4)):
            copies = _copies_for(n * (read + wb), 4)
            ps = [p] + [ops.Packed(fmt, p.codes.clone(), p.scales.clone(), p.tensor_scale.clone(), p.rows, p.cols)
                        for _ in range(copies - 1)]
            outs = [ops.ifx_dequantize(q, dt) for q in ps]
            fns = [lambda i=i: ops.ifx_dequantize(ps[i], dt, outs[i]) for i in range(copies)]
            t = rotating_time(torch, fns, 8 * copies, 5)
            r[tag + "_us"] = round(t * 1e6, 1)
            r[tag + "_GBps"] = round(n * (read + wb) / t / 1e9, 1)
            r[tag + "_frac"] = round(n * (read + wb) / t / 1e9 / HBM_PEAK_GBS, 4)
            del ps, outs
        res[ops.FORMAT_NAMES[fmt]] = r
        del p
    return res


def context_times(ops, workloads, torch):
    """Context for the fractions, not a result of this library: a plain
    device-to-device copy of 117 MB (the size of W's bf16 data) over
    rotating buffers; the library FP16 GEMM (torch.matmul, hipBLASLt) at the
    step's 8192 x 14336 x 4096 on N(0,1) FP16 operands under sustained load;
    and this library's IF4 GEMM at that shape on all-zero operands (the same
    instructions with no operand bit activity: the part's clock under the
    GEMM depends on the data)."""
    n = 14336 * 4096 * 2
    copies = _copies_for(2 * n, 4)
    srcs = [torch.ones(n, dtype=torch.uint8, device="cuda") for _ in range(copies)]
    dsts = [torch.empty(n, dtype=torch.uint8, device="cuda") for _ in range(copies)]
    t = rotating_time(torch, [lambda i=i: dsts[i].copy_(srcs[i]) for i in range(copies)], 8 * copies, 5)
    del srcs, dsts
    g = torch.Generator(device="cuda").manual_seed(1)
    a = torch.randn((8192, 4096), generator=g, device="cuda", dtype=torch.float16)
    bt = torch.randn((14336, 4096), generator=g, device="cuda", dtype=torch.float16)
    b = bt.t()
    c = torch.empty((8192, 14336), device="cuda", dtype=torch.float16)
    tg = _steady_time(torch, lambda: torch.mm(a, b, out=c), 10)
    del a, bt, b
    za = ops.if4_quantize(torch.zeros((8192, 4096), dtype=torch.bfloat16, device="cuda"))
    zw = ops.if4_quantize(torch.zeros((14336, 4096), dtype=torch.bfloat16, device="cuda"))
    cz = c.view(torch.bfloat16)
    tz = _steady_time(torch, lambda: ops.if4_gemm(za, zw, ops.BF16, cz), 10)
    del c, cz, za, zw
    return {"copy_117MB_GBps": round(2 * n / t / 1e9, 1),
            "copy_117MB_frac": round(2 * n / t / 1e9 / HBM_PEAK_GBS, 4),
            "fp16_matmul_8192x14336x4096_us": round(tg * 1e6, 1),
            "fp16_matmul_TFLOPs": round(2.0 * 8192 * 14336 * 4096 / tg / 1e12, 1),
            "fp16_matmul_frac": round(2.0 * 8192 * 14336 * 4096 / tg / 1e12 / FP16_MFMA_PEAK_TFLOPS, 4),
            "if4_gemm_zero_operands_us": round(tz * 1e6, 1),
            "if4_gemm_zero_operands_TFLOPs": round(2.0 * 8192 * 14336 * 4096 / tz / 1e12, 1)}


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
# Kernels whose HBM traffic bench.py reports: record key -> (kernel name in
# the profiler, which of its dispatches per step, sources it is built from).
TRAFFIC_KERNELS = {
    "gemm": ("ifq::gemm_tn_fast<0, true>", None,
             ("paper_2603_28765_amd/csrc/gemm.hip", "paper_2603_28765_amd/csrc/device.h")),
    "quantize_W": ("ifq::quantize_rows<0, false, false, true>", 1,
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
    """The CPU oracle on the same step, no extrapolation of the quantize work:

    - quantize A and W to IF4 with the C oracle on one thread (alpha from the
      whole tensor, as the oracle does it), and again with threads over row
      blocks on the cores this process may use (alpha from the tensor
      maximum first, then each block quantized with that alpha: row groups
      are independent given alpha, so the result is the same bytes, which
      is checked);
    - dequantize W to fp64 (threads over row blocks) and run the reference
      GEMM (numpy BLAS, fp64) for `rows` rows of A against all of W; the
      product's time is scaled by M/rows.

    `value` uses the multi-threaded legs; each leg reports its threads."""
    import concurrent.futures as cf

    import numpy as np
    import torch

    import oracle as O
    from threadpoolctl import threadpool_info

    def bits(t):
        return t.contiguous().view(torch.int16).numpy().view(np.uint16)

    a, wt = bits(w.tensors["A"]), bits(w.tensors["W"])
    nthreads = max(1, min(len(os.sched_getaffinity(0)), 16))

    t0 = time.perf_counter()
    ca, sa, aa = O.quantize(a, O.FMT_IF4)
    cw, sw, aw = O.quantize(wt, O.FMT_IF4)
    t_q1 = time.perf_counter() - t0

    def blocks(n):
        step = -(-n // (4 * nthreads))
        return [(r, min(n, r + step)) for r in range(0, n, step)]

    def quantize_mt(x, pool):
        alpha = O.tensor_scale(O.FMT_IF4, float(np.abs(O.bf16_to_f32(x)).max()))
        parts = list(pool.map(lambda rr: O.quantize(np.ascontiguousarray(x[rr[0]:rr[1]]), O.FMT_IF4,
                                                    O.SCALE_IN, tensor_scale=alpha), blocks(x.shape[0])))
        return np.concatenate([p[0] for p in parts]), np.concatenate([p[1] for p in parts]), alpha

    with cf.ThreadPoolExecutor(nthreads) as pool:
        t1 = time.perf_counter()
        qa = quantize_mt(a, pool)
        qw = quantize_mt(wt, pool)
        t_qm = time.perf_counter() - t1
        same = all(np.array_equal(u, v) for u, v in ((qa[0], ca), (qa[1], sa), (qw[0], cw), (qw[1], sw))) \
            and qa[2] == aa and qw[2] == aw
        t2 = time.perf_counter()
        Wd = np.concatenate(list(pool.map(lambda rr: O.dequantize(cw[rr[0]:rr[1]], sw[rr[0]:rr[1]], aw, O.FMT_IF4,
                                                                  np.float64), blocks(N))))
        t_dw = time.perf_counter() - t2
    t3 = time.perf_counter()
    Ad = O.dequantize(ca[:rows], sa[:rows], aa, O.FMT_IF4, np.float64)
    _ = Ad @ Wd.T
    t_g = time.perf_counter() - t3
    blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    flops = 2.0 * M * N * K
    t_full = t_qm + t_dw + t_g * M / rows
    t_full1 = t_q1 + t_dw + t_g * M / rows
    return {"value": round(flops / t_full / 1e12, 6), "unit": "TFLOP/s",
            "cores": int(max(nthreads, blas_threads)), "kind": "oracle",
            "sample": f"the whole step on the CPU: IF4 quantize of all of A and W (C oracle, "
                      f"{nthreads} threads over row blocks, {t_qm:.2f} s; on 1 thread {t_q1:.2f} s), fp64 "
                      f"dequantize of W ({nthreads} threads, {t_dw:.2f} s), reference GEMM of {rows} of {M} "
                      f"rows of A against all {N} rows of W (numpy BLAS, {blas_threads} threads, {t_g:.2f} s, "
                      f"scaled by M/{rows})",
            "legs": {"quantize_threads": nthreads, "quantize_s": round(t_qm, 3),
                     "quantize_1thread_s": round(t_q1, 3), "quantize_results_identical": bool(same),
                     "dequantize_W_threads": nthreads, "dequantize_W_s": round(t_dw, 3),
                     "gemm_ref_threads": int(blas_threads), "gemm_ref_s": round(t_g, 3),
                     "gemm_ref_rows": rows},
            "value_with_1thread_quantize": round(flops / t_full1 / 1e12, 6),
            "seconds": round(t_q1 + t_qm + t_dw + t_g, 2)}


if __name__ == "__main__":
    main()
