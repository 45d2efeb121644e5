#!/usr/bin/env python3
"""Throughput of the NOBLE-CosNet linear layer (forward + backward) on one MI355X.

A step is the forward of every projection of the workload in order, then the
backward of each in reverse order, on one stream (inputs already resident in
HBM).  The default workload is the largest one-GPU configuration: a slice of
four 1.5B-style decoder blocks, T = 16 x 2048 tokens, d = 2048, r = 128,
six projections per block (Q, K, V and O 2048->2048, FFN up 2048->8192, FFN
down 8192->2048; Q, K and V read the same block input), 24 in all.

Reported: algorithmic TFLOP/s, 6 T [d_in d_out + r (d_in + d_out) + r^2] per
projection over the step time (no r^2 term for the one-application
activations, which have no M); the same step with r = 0 (plain linear, same
kernels) and the overhead over it; the roofline of the step's dominant launch
(the weight-gradient product of an FFN projection); and the fp64 oracle's
throughput on a bounded sample on the host cores.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                      [--activation NAME]   (CosNet by default)
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16 = 2.5e15   # dense bf16 MFMA, MI355X
PEAK_F32 = 157.3e12  # dense fp32 MFMA, MI355X
METRIC = "NOBLE linear fwd+bwd TFLOP/s, % bf16 MFMA peak, overhead vs plain GEMM"


def flop_alg(T, d_in, d_out, r, mixing=1, groups=1):
    """Forward + backward FLOPs: 6 T [d_in d_out + r (G d_in + d_out) + m G r^2]
    for G groups of rank r (each group maps d_in to d_out / G) with m = mixing
    r x r matrices per group (0, 1, or 2 for the 3-layer CosNet)."""
    G = groups
    return 6.0 * T * (d_in * d_out + r * (G * d_in + d_out) + int(mixing) * G * r * r)


def branch_floor(d_in, d_out, r, mixing=1, groups=1):
    """Branch FLOPs over the main product's."""
    G = groups
    return (r * (G * d_in + d_out) + int(mixing) * G * r * r) / (d_in * d_out)


TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "wgrad_ffn_up_T32768_traffic.md")
WGRAD_KERNEL = "noble::gemm_bf16_kernel<false, false, true, 0>"


# Sources of the roofline kernel (gemm_bf16_kernel): a traffic record stays
# valid while these files and the compiler flags are unchanged and the launch
# has the recorded workgroup count (which the host's plan sets).
ROOFLINE_SOURCES = ("noble_tiles.hpp", "noble_gemm.hpp", "noble_gemm_dma.hpp")


def kernel_source_hash() -> str:
    from paper_2603_06492_amd import _build
    h = hashlib.sha256()
    h.update(" ".join(_build.HIP_FLAGS).encode())
    d = os.path.join(ROOT, "paper_2603_06492_amd", "csrc")
    for f in ROOFLINE_SOURCES:
        h.update(f.encode())
        with open(os.path.join(d, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def recorded_traffic(kernel: str, workload: str, workgroups: int):
    """HBM bytes per launch of the roofline kernel from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary, or None when that record was taken on
    other kernel sources, another workload or another launch shape."""
    try:
        with open(TRAFFIC_RECORD) as fh:
            m = re.search(r"^traffic_record: (\{.*\})$", fh.read(), re.M)
        rec = json.loads(m.group(1))
    except (OSError, AttributeError, ValueError):
        return None
    if rec.get("source_sha256_16") != kernel_source_hash():
        return None
    if rec.get("workload") != workload or rec.get("kernel") != kernel or rec.get("workgroups") != workgroups:
        return None
    return rec.get("traffic_bytes")


class HipEvents:
    """hipEvent_t handles created and read through the HIP runtime (for the
    launch that the library brackets itself, noble_profile_next_wgrad)."""

    def __init__(self):
        import ctypes
        self.ct = ctypes
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self) -> int:
        ev = self.ct.c_void_p()
        if self.hip.hipEventCreate(self.ct.byref(ev)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return ev.value

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = self.ct.c_float()
        if self.hip.hipEventSynchronize(self.ct.c_void_p(b)) != 0 or \
                self.hip.hipEventElapsedTime(self.ct.byref(ms), self.ct.c_void_p(a), self.ct.c_void_p(b)) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def destroy(self, ev: int) -> None:
        self.hip.hipEventDestroy(self.ct.c_void_p(ev))


def _row_err(gpu, ref):
    """max over rows of max_j |gpu - ref| / (max_j |ref| + 1e-6)."""
    import numpy as np
    num = np.abs(gpu - ref).max(axis=1)
    den = np.abs(ref).max(axis=1) + 1e-6
    return float((num / den).max())


def cpu_baseline(workload: str, samples, gpu_rows, budget_s: float = 12.0, activation: str = "cosnet"):
    """fp64 oracle fwd+bwd on a prefix of the tokens of the bench's own
    projections (the same arrays the GPU ran on).  `samples[i]` holds the
    weights and the first rows of x and dy of projection i; `gpu_rows(i, n)`
    returns the GPU's y and dx rows [0, n).  Besides the oracle's rate it
    reports the row-wise parity error of y and dx on those rows (both depend
    only on their own tokens; the weight gradients, sums over every token,
    are checked by the tests)."""
    import oracle  # test infrastructure: only this leg of the bench uses it
    from paper_2603_06492_amd import inputs as inp
    from paper_2603_06492_amd import noble
    mixing = noble.layers(activation) - 1   # mixing matrices per group
    kw = dict(activation=activation)
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    cores = len(os.sched_getaffinity(0))
    shapes = inp.workload_shapes(workload)
    groups = inp.workload_groups(workload)
    T_full = shapes[0][1]

    def fwd(a, Ts, G):
        args = (a["x"][:Ts], a["W"], a["b"], a["W_down"], a["omega1"], a["phi1"], a["M"], a["omega2"], a["phi2"],
                a["W_up"])
        return oracle.forward_grouped(*args, G, **kw) if G > 1 else oracle.forward(*args, **kw)

    def bwd(a, Ts, G):
        args = (a["dy"][:Ts], a["x"][:Ts], a["W"], a["W_down"], a["omega1"], a["phi1"], a["M"], a["omega2"],
                a["phi2"], a["W_up"])
        return oracle.backward_grouped(*args, G, **kw) if G > 1 else oracle.backward(*args, **kw)
    T_max = min(T_full, samples[0]["x"].shape[0])
    Ts = 128
    while True:
        outs = []
        t0 = time.perf_counter()
        for a, G in zip(samples, groups):
            Y, _ = fwd(a, Ts, G)
            g = bwd(a, Ts, G)
            outs.append((Y, g["dx"]))
        dt = time.perf_counter() - t0
        if dt >= budget_s / 4 or Ts * 2 > T_max:
            break
        Ts *= 2
    # repeat the pass on the chosen sample until about `budget_s` of CPU work
    passes = 1
    while dt < budget_s:
        t0 = time.perf_counter()
        for a, G in zip(samples, groups):
            fwd(a, Ts, G)
            bwd(a, Ts, G)
        dt += time.perf_counter() - t0
        passes += 1
    parity = {"rows": Ts, "tol": 2e-2, "y": 0.0, "dx": 0.0}
    for i, (Y, dx) in enumerate(outs):
        gy, gdx = gpu_rows(i, Ts)
        parity["y"] = max(parity["y"], round(_row_err(gy, Y), 6))
        parity["dx"] = max(parity["dx"], round(_row_err(gdx, dx), 6))
    flops = passes * sum(flop_alg(Ts, di, do, r, mixing, G) for (_, _, di, do, r), G in zip(shapes, groups))
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(cores), "blas_threads": int(threads),
            "kind": "oracle",
            "sample": f"first {Ts} of {T_full} tokens of every projection (the bench's own arrays), "
                      f"numpy float64, {passes} fwd+bwd passes",
            "seconds": round(dt, 3), "parity_vs_gpu": parity}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llm1p5b_stack4_r128")
    ap.add_argument("--activation", default="cosnet",
                    help="bottleneck activation: cosnet (default), cos, tanh, tanh_m, leaky_relu, "
                         "leaky_relu_m, gelu, gelu_m, cosnet3")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-blas", action="store_true",
                    help="skip the hipBLASLt (torch.mm) context timings of the plain products")
    ap.add_argument("--proj-reps", type=int, default=50,
                    help="calls per per-projection median (fwd, bwd, plain fwd, plain bwd)")
    ap.add_argument("--roofline-launches", type=int, default=20,
                    help="timed weight-gradient launches of the dominant projection for the roofline entry")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one device-to-device copy of this many MiB (a kernel of known "
                         "traffic, for scaling FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the kernels run on a single MI355X and there is "
              "no multi-GPU path (rerun with --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2603_06492_amd import inputs as inp
    from paper_2603_06492_amd import noble
    from paper_2603_06492_amd.runner import DeviceProblem

    mixing = noble.layers(args.activation) - 1   # mixing matrices per group
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)

    wl = inp.WORKLOADS[args.workload]
    shapes = inp.workload_shapes(args.workload)
    groups = inp.workload_groups(args.workload)
    print(f"[bench] workload {args.workload}: {len(shapes)} projections, T={wl['T']}, r={wl['r']}",
          file=sys.stderr, flush=True)
    probs, plain, samples = [], [], []
    sample_rows = min(wl["T"], 8192)
    xsrc = inp.workload_x_source(args.workload)
    for i in range(len(shapes)):
        p = inp.draw_workload_projection(args.workload, i, layers=max(2, mixing + 1))
        dp = DeviceProblem(p, activation=args.activation, x_from=probs[xsrc[i]] if xsrc[i] != i else None)
        probs.append(dp)
        plain.append(DeviceProblem(p, branch=False, inputs_from=dp))
        if not args.no_cpu_baseline:
            samples.append({k: (v[:sample_rows] if k in ("x", "dy") else v) for k, v in p.arrays.items()})
        del p
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    def step(ps):
        for dp in ps:
            dp.fwd()
        for dp in reversed(ps):
            dp.bwd()

    def timed(ps, K, W):
        for _ in range(W):
            step(ps)
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        ev0.record(stream)
        for _ in range(K):
            step(ps)
        ev1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return ev0.elapsed_time(ev1) / K, wall / K * 1e3

    ms_noble, wall_noble = timed(probs, args.steps, args.warmup)
    print(f"[bench] noble step {ms_noble:.3f} ms", file=sys.stderr, flush=True)
    ms_plain, wall_plain = timed(plain, args.steps, args.warmup)
    print(f"[bench] plain step {ms_plain:.3f} ms", file=sys.stderr, flush=True)

    # Per-projection fwd / bwd times: median over `--proj-reps` calls, each
    # bracketed by HIP events on the launch stream, after warm-up calls.
    def median_ms(fn, reps):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(2 * reps)]
        for i in range(reps):
            evs[2 * i].record(stream)
            fn()
            evs[2 * i + 1].record(stream)
        torch.cuda.synchronize()
        d = sorted(evs[2 * i].elapsed_time(evs[2 * i + 1]) for i in range(reps))
        return d[reps // 2]

    # one entry per distinct projection shape (the blocks of a stack repeat)
    per, seen = [], {}
    for dp, d0 in zip(probs, plain):
        key = (dp.p.d_in, dp.p.d_out, dp.G)
        if key in seen:
            seen[key]["also"].append(dp.p.name.split("/")[-1])
            continue
        T, di, do, r, G = dp.p.T, dp.p.d_in, dp.p.d_out, dp.p.r, dp.G
        for _ in range(10):
            dp.fwd(); dp.bwd(); d0.fwd(); d0.bwd()
        torch.cuda.synchronize()
        tf = median_ms(dp.fwd, args.proj_reps)
        tb = median_ms(dp.bwd, args.proj_reps)
        pf = median_ms(d0.fwd, args.proj_reps)
        pb = median_ms(d0.bwd, args.proj_reps)
        fl = flop_alg(T, di, do, r, mixing, G)
        entry = {"projection": dp.p.name.split("/")[-1], "T": T, "d_in": di, "d_out": do, "r": r, "groups": G,
                 "fwd_ms": round(tf, 4), "bwd_ms": round(tb, 4), "plain_fwd_ms": round(pf, 4),
                 "plain_bwd_ms": round(pb, 4), "tflops": round(fl / ((tf + tb) * 1e-3) / 1e12, 2),
                 "pct_bf16_peak": round(100 * fl / ((tf + tb) * 1e-3) / PEAK_BF16, 2),
                 "main_gemm_pct_peak": round(100 * 6.0 * T * di * do / ((pf + pb) * 1e-3) / PEAK_BF16, 2),
                 "overhead": round((tf + tb) / (pf + pb) - 1, 4),
                 "overhead_floor": round(branch_floor(di, do, r, mixing, G), 4), "also": []}
        seen[key] = entry
        if not args.no_blas:
            # Context only: hipBLASLt (through torch.mm) on the same plain
            # products and operands, bf16 in and out: y = x W, dx = dy W^T,
            # dW = x^T dy.  Operands are made contiguous first.
            x, W, dy = dp.t["x"], dp.t["W"], dp.t["dy"]
            WT, xT = W.t().contiguous(), x.t().contiguous()
            for _ in range(3):
                torch.mm(x, W); torch.mm(dy, WT); torch.mm(xT, dy)
            bf = median_ms(lambda: torch.mm(x, W), args.proj_reps // 2)
            bdx = median_ms(lambda: torch.mm(dy, WT), args.proj_reps // 2)
            bdw = median_ms(lambda: torch.mm(xT, dy), args.proj_reps // 2)
            del WT, xT
            entry["hipblaslt_plain_ms"] = {"fwd": round(bf, 4), "dx": round(bdx, 4), "dW": round(bdw, 4),
                                           "main_pct_peak": round(100 * 6.0 * T * di * do / ((bf + bdx + bdw) * 1e-3)
                                                                  / PEAK_BF16, 2)}
        per.append(entry)

    # Roofline entry: the step's dominant launch, the weight-gradient product
    # of the projection with the most weight-gradient FLOPs (an FFN
    # projection): one grouped bf16 MFMA launch computing dW = x^T dy,
    # dW_down = x^T dH, dW_up = C2^T dy and dM = C1^T dH2 (and db's column
    # sums).  The library records a pair of HIP events on its stream right
    # before and after that launch (noble_profile_next_wgrad); `achieved` is
    # the launch's algorithmic FLOPs, 2 T (d_in d_out + d_in R + r d_out +
    # m G r^2), over the mean of those launch durations.
    def wgrad_flops(dp):
        T, di, do, r, G = dp.p.T, dp.p.d_in, dp.p.d_out, dp.p.r, dp.G
        return 2.0 * T * (di * do + G * r * di + r * do + mixing * G * r * r)
    dom = max(probs, key=wgrad_flops)
    hev = HipEvents()
    evs = [(hev.create(), hev.create()) for _ in range(args.roofline_launches)]
    for _ in range(3):
        dom.bwd()
    torch.cuda.synchronize()
    import ctypes
    wgs = ctypes.c_int64(0)
    for (a, b) in evs:
        noble.noble_profile_next_wgrad(a, b, wgs)
        dom.bwd()
    torch.cuda.synchronize()
    t_launch = sum(hev.elapsed_ms(a, b) for (a, b) in evs) / len(evs) * 1e-3
    for (a, b) in evs:
        hev.destroy(a)
        hev.destroy(b)
    wg_flops = wgrad_flops(dom)
    ach = wg_flops / t_launch / 1e12
    pname = dom.p.name.split("/")[-1]
    roofline = {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_BF16 / 1e12, "unit": "TFLOP/s",
                "frac": round(ach / (PEAK_BF16 / 1e12), 4),
                "traffic": recorded_traffic(WGRAD_KERNEL, f"{args.workload}/{pname}", wgs.value),
                "kernel": f"{WGRAD_KERNEL} (weight gradients dW, dW_down, dW_up, dM of "
                          f"{pname} T={dom.p.T} {dom.p.d_in}->{dom.p.d_out} r={dom.r}, {wgs.value} workgroups)",
                "avg_launch_us": round(t_launch * 1e6, 2), "flop_per_launch": wg_flops}

    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib * (1 << 20)
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    flops_step = sum(flop_alg(T, di, do, r, mixing, G) for (_, T, di, do, r), G in zip(shapes, groups))
    main_flops = sum(6.0 * T * di * do for (_, T, di, do, r) in shapes)
    value = flops_step / (ms_noble * 1e-3) / 1e12
    floor = sum(T * di * do * branch_floor(di, do, r, mixing, G) for (_, T, di, do, r), G in zip(shapes, groups)) / \
        sum(T * di * do for (_, T, di, do, r) in shapes)
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_noble, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl["dtype"],
        "data": "synthetic",
        "config": {"workload": args.workload, "T": wl["T"], "r": wl["r"], "activation": args.activation,
                   "projections": [f"{n} {di}->{do}" + (f" ({G} groups)" if G > 1 else "")
                                   for (n, _, di, do, _), G in zip(shapes, groups)]},
        "pct_bf16_peak": round(100 * value / (PEAK_BF16 / 1e12), 2),
        "plain_ms_per_step": round(ms_plain, 4),
        "overhead_vs_plain": round(ms_noble / ms_plain - 1, 4),
        "overhead_floor": round(floor, 4),
        "main_gemm_pct_peak": round(100 * main_flops / (ms_plain * 1e-3) / PEAK_BF16, 2),
        "wall_ms_per_step": round(wall_noble, 4),
        "roofline": roofline,
        "per_projection": per,
    }
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (fp64 oracle)", file=sys.stderr, flush=True)
        def gpu_rows(i, n):
            dp = probs[i]
            return (dp.y[:n].float().cpu().numpy().astype("float64"),
                    dp.g["dx"][:n].float().cpu().numpy().astype("float64"))
        out["cpu_baseline"] = cpu_baseline(args.workload, samples, gpu_rows, activation=args.activation)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
