#!/usr/bin/env python3
"""Throughput of the approximate-multiplier hot path on one MI355X.

One step = approx_gemm 4096x4096x4096 (Mitchell multiplier, M = 7, table in LDS) plus the
ResNet-style 3x3 convolution (batch 128, 64 -> 64 channels at 32x32, stride 1, pad 1, NHWC,
Mitchell M = 7) forward, backward-data and backward-weight.  Inputs are seeded synthetic
tensors resident in HBM before the timed region; outputs and workspaces are preallocated.
value = approximate multiply-accumulates per second over the timed steps (whole job).

Prints one JSON line.  Besides the contract fields it carries
  roofline      the GEMM kernel (the dominant one): algorithmic FLOP (2 per approx-MAC) per
                launch over its average launch duration, measured with HIP events recorded on
                its stream inside the timed region, against the FP32 vector peak
  kernels       per-kernel rates of the step (HIP events on the launch stream: the GEMM's
                inside the timed steps, the convolution passes' in as many repetitions of the
                step's three convolution calls right after), then, timed
                after the step: the 4096^3 GEMM with the M = 11 Mitchell table (sum-indexed: read
                from one array of 4096 factors),
                the three ResNet-50 layers (batch 32, each pass), the LeNet-5 stack (batch 64,
                exact bfloat16-truncation table), the step's GEMM and convolution passes with
                the native FP32 multiply in the same kernels, and the same four with the vendor
                FP32 libraries torch calls (hipBLASLt / MIOpen, TF32 off).  The ResNet-50 1x1
                passes run as GEMMs and may launch the step GEMM's kernel instance, so a kernel
                trace that is to time only the launches the roofline is quoted for is taken with
                --no-other-kernels.
  cpu_baseline  the CPU oracle timed on a seeded sample of the same step's outputs
  extra         (with --extra only) a GEMM size sweep, the direct-evaluation GEMMs, a
                post-ReLU input case, the exact-truncation table on the step and a LeNet-5
                training step through the autograd layers.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "approx-MACs/s (G/s) and % FP32 VALU peak: approx_gemm 4096³ + ResNet conv fwd+bwd"
FP32_VECTOR_PEAK_TFLOPS = 157.3   # MI355X published FP32 vector peak (dense)
FLOP_PER_APPROX_MAC = 2           # one multiply + one add
# The 157.3 TFLOP/s peak counts packed (two-wide) FP32 FMAs.  The plain per-lane rate is
# 256 CUs x 64 lanes x 2.4 GHz = 39.3 T lane-ops/s; one approx-MAC per lane-op is the second
# reading of "% of the FP32 vector peak", reported beside the first.
FP32_LANE_RATE_T = 256 * 64 * 2.4e9 / 1e12
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "gemm_4096_m7_traffic.txt")
# Device sources whose content the committed counters belong to (hashed in this order).
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2209_04161_amd", "csrc", f)
                  for f in ("amsim_common.h", "amsim_tab.h", "amsim_tab.hip", "amsim_kernels.hip", "amsim_plan.h")]


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def kernel_source_hash():
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def read_traffic():
    """HBM bytes per GEMM launch from the committed rocprofv3 --pmc summary, or None when the
    kernel source changed since the counters were taken."""
    if not os.path.exists(TRAFFIC_PROFILE):
        return None
    fields = {}
    with open(TRAFFIC_PROFILE) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    if fields.get("kernel_source_sha256") != kernel_source_hash():
        return None
    try:
        return float(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-fraction", type=float, default=0.1,
                    help="fraction of each part's outputs the CPU oracle computes for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--extra", action="store_true", help="also time the other workloads (see above)")
    ap.add_argument("--no-other-kernels", action="store_true",
                    help="time the step only (no M = 11 GEMM, ResNet-50, LeNet-5, native or vendor entries)")
    ap.add_argument("--no-extra", action="store_true", help="(the default; kept for older command lines)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 256 MiB device copy three times (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (each GPU would run "
              "its own shard of the batch/rows; see the design notes). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2209_04161_amd import binding as B
    from paper_2209_04161_amd import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    B.lib()  # fails loudly if the HIP library is not built
    dev = torch.device("cuda:0")
    m_bits = 7
    lut = B.device_lut(B.lut_build(m_bits, "mitchell"), dev)

    g = W.GEMM_LARGE
    M, N, K = g["M"], g["N"], g["K"]
    A_h, B_h = W.gemm_inputs(M, N, K, "normal", seed=5000)
    A = torch.from_numpy(A_h).to(dev)
    Bm = torch.from_numpy(B_h).to(dev)
    C = torch.empty((M, N), dtype=torch.float32, device=dev)
    ws_g = torch.empty(B.amsim_gemm_workspace_size(0, 0, M, N, K, m_bits), dtype=torch.uint8, device=dev)

    cv = W.RESNET_3X3["conv"]
    x_h, w_h, dy_h = W.resnet_conv_inputs(cv, seed=3000)
    x, w, dy = (torch.from_numpy(t).to(dev) for t in (x_h, w_h, dy_h))
    y = torch.empty_like(dy)
    dx = torch.empty_like(x)
    dw = torch.empty_like(w)
    ws_c = [torch.empty(max(1, B.amsim_conv2d_workspace_size(cv, p, m_bits)), dtype=torch.uint8, device=dev)
            for p in range(3)]

    gemm_macs = M * N * K
    conv_macs = W.conv_macs(cv)
    step_macs = gemm_macs + 3 * conv_macs

    def step():
        B.approx_gemm(A, Bm, lut, m_bits, out=C, workspace=ws_g)
        B.approx_conv2d_fwd(cv, x, w, lut, m_bits, out=y, workspace=ws_c[0])
        B.approx_conv2d_bwd_data(cv, dy, w, lut, m_bits, out=dx, workspace=ws_c[1])
        B.approx_conv2d_bwd_weight(cv, x, dy, lut, m_bits, out=dw, workspace=ws_c[2])

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log("warmup step %d done" % (i + 1))

    if args.calibrate_copy:
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("copy calibration: 3 copies of %d bytes" % (src.numel() * 4))
        del src, dst

    # Inside the timed steps only the dominant kernel (the GEMM's, which the roofline is quoted for)
    # is bracketed by timing events: each pair of events leaves the GPU idle for a few microseconds
    # around the kernel it times.  The convolution kernels are timed the same way right after, in
    # as many repetitions of the step's three convolution calls.
    B.amsim_profile_start(2 * args.steps + 8, kinds=["gemm"])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    B.amsim_profile_stop()
    elapsed = t1 - t0
    log("timed %d steps in %.3f s" % (args.steps, elapsed))
    timed = {"gemm": B.amsim_profile_read("gemm")}
    conv_kinds = ["conv_fwd", "conv_bwd_data", "conv_bwd_weight"]
    B.amsim_profile_start(4 * args.steps + 8, kinds=conv_kinds)
    for _ in range(args.steps):
        B.approx_conv2d_fwd(cv, x, w, lut, m_bits, out=y, workspace=ws_c[0])
        B.approx_conv2d_bwd_data(cv, dy, w, lut, m_bits, out=dx, workspace=ws_c[1])
        B.approx_conv2d_bwd_weight(cv, x, dy, lut, m_bits, out=dw, workspace=ws_c[2])
    torch.cuda.synchronize()
    B.amsim_profile_stop()
    for kind in conv_kinds:
        timed[kind] = B.amsim_profile_read(kind)

    value = step_macs * args.steps / elapsed / 1e9
    kernels = {}
    for kind, macs in (("gemm", gemm_macs), ("conv_fwd", conv_macs), ("conv_bwd_data", conv_macs),
                       ("conv_bwd_weight", conv_macs)):
        n, ms = timed[kind]
        avg = ms / max(n, 1)
        kernels[kind] = {"launches": n, "avg_ms": round(avg, 4),
                         "gmacs_per_s": round(macs / (avg * 1e-3) / 1e9, 1) if n else None,
                         "pct_fp32_vector_peak": round(100 * FLOP_PER_APPROX_MAC * macs / (avg * 1e-3) /
                                                       (FP32_VECTOR_PEAK_TFLOPS * 1e12), 2) if n else None,
                         "pct_fp32_lane_rate": round(100 * macs / (avg * 1e-3) / (FP32_LANE_RATE_T * 1e12), 2)
                         if n else None}
    g_avg_s = kernels["gemm"]["avg_ms"] * 1e-3
    achieved = FLOP_PER_APPROX_MAC * gemm_macs / g_avg_s / 1e12
    roofline = {"bound": "alu", "achieved": round(achieved, 3), "peak": FP32_VECTOR_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / FP32_VECTOR_PEAK_TFLOPS, 4),
                "traffic": read_traffic(),
                "traffic_source": "not measured in this run: HBM bytes per launch from the committed rocprofv3 "
                                  "FETCH_SIZE/WRITE_SIZE summary profiles/gemm_4096_m7_traffic.txt, used only while "
                                  "its kernel_source_sha256 matches the kernel sources (else null)",
                "kernel": "tab_kernel<OP_GEMM, 4, 8, 8, 8, 7, kTabApprox> (approx_gemm 4096^3, Mitchell M=7, bf16 pair path)"}

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "G approx-MAC/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "approx_gemm 4096x4096x4096 normal(0,1) + ResNet 3x3 conv 64->64 @32x32 batch 128 "
                               "fwd+bwd_data+bwd_weight (half-normal x, He-normal w, N(0,1) dy), Mitchell multiplier, "
                               "M=7 (65536-byte table in LDS)",
                   "approx_macs_per_step": step_macs, "m_bits": m_bits, "multiplier": "mitchell"},
        "pct_fp32_vector_peak": round(100 * FLOP_PER_APPROX_MAC * value * 1e9 / (FP32_VECTOR_PEAK_TFLOPS * 1e12), 2),
        "pct_fp32_lane_rate": round(100 * value * 1e9 / (FP32_LANE_RATE_T * 1e12), 2),
        "roofline": roofline,
        "kernels": kernels,
    }

    if not args.no_other_kernels:
        other = other_kernels(B, W, torch, dev, lut, m_bits, A, Bm, C, cv, (x, w, dy), ws_g, ws_c)
        native_step = sum(other["native_multiply"][k]["call_ms"] for k in ("gemm", "conv_fwd", "conv_bwd_data",
                                                                          "conv_bwd_weight"))
        vendor_step = sum(other["vendor_fp32"][k] for k in ("gemm_ms", "conv_fwd_ms", "conv_bwd_data_ms",
                                                           "conv_bwd_weight_ms"))
        other["step_time_ratios"] = {
            "what": "time of the step's four calls over the vendor FP32 libraries' time for the same four",
            "approx_over_vendor_fp32": round(out["ms_per_step"] / vendor_step, 2),
            "native_multiply_over_vendor_fp32": round(native_step / vendor_step, 2),
            "approx_over_native_multiply": round(out["ms_per_step"] / native_step, 2)}
        kernels.update(other)

    if args.extra and not args.no_extra:
        out["extra"] = extras(B, W, torch, np, dev, lut, m_bits, A, Bm, C)

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.cpu_fraction, A_h, B_h, cv, x_h, w_h, dy_h, m_bits)
        out["gpu_over_cpu"] = round(value / out["cpu_baseline"]["value"], 1)

    print(json.dumps(out), flush=True)


def _time_call(torch, fn, reps):
    fn()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps  # ms per call


def _rates(macs, ms):
    return {"gmacs_per_s": round(macs / ms / 1e6, 1),
            "pct_fp32_vector_peak": round(100 * FLOP_PER_APPROX_MAC * macs / (ms * 1e-3) /
                                          (FP32_VECTOR_PEAK_TFLOPS * 1e12), 2),
            "pct_fp32_lane_rate": round(100 * macs / (ms * 1e-3) / (FP32_LANE_RATE_T * 1e12), 2)}


def _time_main_kernel(B, torch, fn, reps, kind, macs):
    """Average main-kernel time (the library's HIP-event timer) and whole-call time (events on
    torch's stream, pre-passes included) of `reps` calls of fn, after one untimed call."""
    call_ms = _time_call(torch, fn, reps)
    B.amsim_profile_start(4 * reps + 4)
    for _ in range(reps):
        fn()
    torch.cuda.synchronize()
    B.amsim_profile_stop()
    n, tot = B.amsim_profile_read(kind)
    avg = tot / max(n, 1)
    r = {"launches": n, "avg_ms": round(avg, 4), "call_ms": round(call_ms, 4)}
    r.update(_rates(macs, avg))
    return r


def other_kernels(B, W, torch, dev, lut7, m7, A, Bm, C, cv, conv_t, ws_g, ws_c):
    """The other configurations, timed after the step (not part of `value`)."""
    ks = {}
    M, N, K = A.shape[0], Bm.shape[1], A.shape[1]
    # the step's GEMM with the M = 11 table (sum-indexed: one array of 2^12 factors in LDS)
    lut11 = B.device_lut(B.lut_build(11, "mitchell"), dev)
    ws = torch.empty(B.amsim_gemm_workspace_size(0, 0, M, N, K, 11), dtype=torch.uint8, device=dev)
    ks["gemm_4096_m11"] = _time_main_kernel(B, torch, lambda: B.approx_gemm(A, Bm, lut11, 11, out=C, workspace=ws),
                                            3, "gemm", M * N * K)
    del ws
    log("M=11 GEMM done")
    # ResNet-50 layers, batch 32, Mitchell M = 7, each pass
    for cfg in W.RESNET50_LAYERS:
        p = cfg["conv"]
        x_h, w_h, dy_h = W.resnet_conv_inputs(p, seed=4000, stem=(cfg is W.RESNET50_LAYERS[0]))
        x, w, dy = (torch.from_numpy(t).to(dev) for t in (x_h, w_h, dy_h))
        macs = W.conv_macs(p)
        for name, kind, fn in (("fwd", "conv_fwd", lambda: B.approx_conv2d_fwd(p, x, w, lut7, m7)),
                               ("bwd_data", "conv_bwd_data", lambda: B.approx_conv2d_bwd_data(p, dy, w, lut7, m7)),
                               ("bwd_weight", "conv_bwd_weight",
                                lambda: B.approx_conv2d_bwd_weight(p, x, dy, lut7, m7))):
            ks["%s_%s" % (cfg["name"], name)] = _time_main_kernel(B, torch, fn, 5, kind, macs)
        del x, w, dy
    log("ResNet-50 layers done")
    ks["lenet5_b64_fwd_bwd"] = lenet_stack(B, W, torch, dev)
    log("LeNet-5 stack done")
    ks["dense_batch1"] = dense_batch1(B, W, torch, dev, lut7, m7)
    log("batch-1 dense layers done")
    # the step with the native FP32 multiply in the same kernels
    x, w, dy = conv_t
    conv_macs = W.conv_macs(cv)
    nat = {}
    nat["gemm"] = _time_main_kernel(
        B, torch, lambda: B.approx_gemm_ex(A, Bm, lut7, m7, out=C, workspace=ws_g, multiply="native"), 5,
        "gemm_native", M * N * K)
    for name, fn in (("conv_fwd", lambda: B.approx_conv2d_fwd_ex(cv, x, w, lut7, m7, workspace=ws_c[0],
                                                                 multiply="native")),
                     ("conv_bwd_data", lambda: B.approx_conv2d_bwd_data_ex(cv, dy, w, lut7, m7, workspace=ws_c[1],
                                                                           multiply="native")),
                     ("conv_bwd_weight", lambda: B.approx_conv2d_bwd_weight_ex(cv, x, dy, lut7, m7,
                                                                               workspace=ws_c[2],
                                                                               multiply="native"))):
        nat[name] = _time_main_kernel(B, torch, fn, 5, name + "_native", conv_macs)
    ks["native_multiply"] = nat
    log("native-multiply step done")
    ks["vendor_fp32"] = native_fp32(torch, W, dev, A, Bm, C)
    log("vendor FP32 step done")
    return ks


def dense_batch1(B, W, torch, dev, lut, m_bits):
    """Dense layers at batch 1 (the vector kernels): the ResNet-50 classifier 2048 -> 1000 forward
    (1 x 2048 by 2048 x 1000), input gradient (1 x 1000 by the transposed weights) and weight
    gradient (2048 x 1 by 1 x 1000, single products), and a 1 x 8192 by 8192 x 8192 product whose
    8192^2 FP32 weights (256 MiB) set an HBM roofline: algorithmic bytes = the matrix, the vector
    and the result, once each."""
    r = {}
    x = torch.from_numpy(W.uniform((1, 2048), 0.0, 1.0, 6100)).to(dev)
    w = torch.from_numpy(W.glorot_uniform((2048, 1000), 2048, 1000, 6101)).to(dev)
    dy = torch.from_numpy(W.normal((1, 1000), 0.01, 6102)).to(dev)
    for name, fn in (("fc2048x1000_fwd", lambda: B.approx_gemm(x, w, lut, m_bits)),
                     ("fc2048x1000_bwd_data", lambda: B.approx_gemm(dy, w, lut, m_bits, trans_b=True)),
                     ("fc2048x1000_bwd_weight", lambda: B.approx_gemm(x, dy, lut, m_bits, trans_a=True))):
        ms = _time_call(torch, fn, 20)
        r[name] = {"call_ms": round(ms, 4), "gmacs_per_s": round(2048 * 1000 / ms / 1e6, 1)}
    n = 8192
    v = torch.from_numpy(W.normal((1, n), 1.0, 6103)).to(dev)
    big = torch.from_numpy(W.normal((n, n), 0.01, 6104)).to(dev)
    out = torch.empty((1, n), dtype=torch.float32, device=dev)
    ws = torch.empty(max(1, B.amsim_gemm_workspace_size(0, 0, 1, n, n, m_bits)), dtype=torch.uint8, device=dev)
    g = _time_main_kernel(B, torch, lambda: B.approx_gemm(v, big, lut, m_bits, out=out, workspace=ws), 10, "gemm",
                          n * n)
    nbytes = 4 * (n * n + 2 * n)
    g["algorithmic_bytes"] = nbytes
    g["hbm_gb_per_s"] = round(nbytes / (g["avg_ms"] * 1e-3) / 1e9, 1)
    g["frac_of_8000_gb_per_s"] = round(nbytes / (g["avg_ms"] * 1e-3) / 8e12, 3)
    r["gemv_1x8192x8192"] = g
    return r


def lenet_stack(B, W, torch, dev):
    """LeNet-5 stack, batch 64, exact bfloat16-truncation table: forward and backward of every
    approximate layer (whole calls, pre-passes included)."""
    cfg = W.LENET5
    mb = cfg["m_bits"]
    lutb = B.device_lut(B.lut_build(mb, "exact_trunc"), dev)
    c1, c2 = cfg["conv1"], cfg["conv2"]
    x0 = torch.from_numpy(W.uniform((64, 28, 28, 1), 0, 1, 6000)).to(dev)
    w1 = torch.from_numpy(W.glorot_uniform((5, 5, 1, 6), 25, 150, 6001)).to(dev)
    w2 = torch.from_numpy(W.glorot_uniform((5, 5, 6, 16), 150, 400, 6002)).to(dev)
    fcw = [torch.from_numpy(W.glorot_uniform((i, o), i, o, 6003 + j)).to(dev) for j, (i, o) in enumerate(cfg["fc"])]
    g = torch.Generator(device="cpu").manual_seed(6020)
    p1 = torch.rand((64, 14, 14, 6), generator=g).to(dev)
    dy1 = torch.randn((64, 28, 28, 6), generator=g).to(dev)
    dy2 = torch.randn((64, 10, 10, 16), generator=g).to(dev)
    acts = [torch.rand((64, i), generator=g).to(dev) for i, _ in cfg["fc"]]
    grads = [torch.randn((64, o), generator=g).to(dev) for _, o in cfg["fc"]]
    macs = 2 * W.conv_macs(c1) + 3 * W.conv_macs(c2) + 3 * sum(64 * i * o for i, o in cfg["fc"])

    def stack():
        B.approx_conv2d_fwd(c1, x0, w1, lutb, mb)
        B.approx_conv2d_fwd(c2, p1, w2, lutb, mb)
        for a, wj in zip(acts, fcw):
            B.approx_gemm(a, wj, lutb, mb)
        for a, gj, wj in zip(acts, grads, fcw):
            B.approx_gemm(a, gj, lutb, mb, trans_a=True)
            B.approx_gemm(gj, wj, lutb, mb, trans_b=True)
        B.approx_conv2d_bwd_weight(c2, p1, dy2, lutb, mb)
        B.approx_conv2d_bwd_data(c2, dy2, w2, lutb, mb)
        B.approx_conv2d_bwd_weight(c1, x0, dy1, lutb, mb)

    ms = _time_call(torch, stack, 10)
    r = {"call_ms": round(ms, 4), "approx_macs": macs, "calls": 14}
    r.update(_rates(macs, ms))
    # the same 14 calls captured once into a HIP graph and replayed: the host-side cost of the
    # calls (argument checks, planning, torch allocations, launches) leaves the timed region
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        stack()
    gms = _time_call(torch, graph.replay, 20)
    r["graph_replay"] = {"call_ms": round(gms, 4)}
    r["graph_replay"].update(_rates(macs, gms))
    return r


def extras(B, W, torch, np, dev, lut7, m7, A, Bm, C):
    """Rates of further workloads (not part of the timed step)."""
    ex = {}
    M, N, K = A.shape[0], Bm.shape[1], A.shape[1]
    lut11 = B.device_lut(B.lut_build(11, "mitchell"), dev)
    # the same GEMM at smaller sizes, with the M = 7 and the M = 11 table
    sweep = {}
    for n in (64, 512, 1024, 2048):
        a, b = (torch.from_numpy(t).to(dev) for t in W.gemm_inputs(n, n, n, "normal", seed=5100 + n))
        c = torch.empty((n, n), dtype=torch.float32, device=dev)
        for mb, lt in ((7, lut7), (11, lut11)):
            wsn = torch.empty(max(1, B.amsim_gemm_workspace_size(0, 0, n, n, n, mb)), dtype=torch.uint8, device=dev)
            ms = _time_call(torch, lambda: B.approx_gemm(a, b, lt, mb, out=c, workspace=wsn), 5 if mb == 7 else 2)
            sweep["n%d_m%d" % (n, mb)] = {"ms": round(ms, 3), "gmacs_per_s": round(n ** 3 / ms / 1e6, 1)}
    ex["gemm_sweep_mitchell"] = sweep
    log("GEMM size sweep done")
    # the 4096^3 GEMM without a table: Mitchell computed from the operands' bits, and the native
    # FP32 multiply, in the same simple register-tiled kernel (the paper's AMSim-vs-direct figure)
    d = {}
    for mode in ("mitchell", "native"):
        ms = _time_call(torch, lambda: B.approx_gemm_direct(A, Bm, mode, m7, out=C), 2)
        d[mode] = {"ms": round(ms, 2), "gmacs_per_s": round(M * N * K / ms / 1e6, 1)}
    ex["gemm_4096_direct"] = d
    log("direct GEMM done")
    # ResNet 3x3 with post-ReLU activations (about half exact zeros) instead of |N(0,1)|
    cv = W.RESNET_3X3["conv"]
    x_h, w_h, dy_h = W.resnet_conv_inputs(cv, seed=4500)
    x_h = np.maximum(W.normal(x_h.shape, 1.0, 4501), 0.0).astype(np.float32)
    x, w, dy = (torch.from_numpy(t).to(dev) for t in (x_h, w_h, dy_h))
    macs = W.conv_macs(cv)
    r = {"zero_fraction": round(float((x_h == 0).mean()), 3)}
    for name, fn in (("fwd", lambda: B.approx_conv2d_fwd(cv, x, w, lut7, m7)),
                     ("bwd_weight", lambda: B.approx_conv2d_bwd_weight(cv, x, dy, lut7, m7))):
        ms = _time_call(torch, fn, 5)
        r[name] = {"ms": round(ms, 3), "gmacs_per_s": round(macs / ms / 1e6, 1)}
    ex["resnet_3x3_relu_input"] = r
    log("ReLU-input ResNet 3x3 done")
    # the step's GEMM and ResNet 3x3 passes with the exact bfloat16-truncation table (2-byte
    # entries: the hi/lo path on the 8-wave 8-column tiles, the exact path elsewhere)
    lut_et = B.device_lut(B.lut_build(7, "exact_trunc"), dev)
    x_h, w_h, dy_h = W.resnet_conv_inputs(cv, seed=3000)
    x, w, dy = (torch.from_numpy(t).to(dev) for t in (x_h, w_h, dy_h))
    ms = _time_call(torch, lambda: B.approx_gemm(A, Bm, lut_et, 7, out=C), 2)
    r = {"gemm_4096": {"ms": round(ms, 2), "gmacs_per_s": round(M * N * K / ms / 1e6, 1)}}
    for name, fn in (("fwd", lambda: B.approx_conv2d_fwd(cv, x, w, lut_et, 7)),
                     ("bwd_data", lambda: B.approx_conv2d_bwd_data(cv, dy, w, lut_et, 7)),
                     ("bwd_weight", lambda: B.approx_conv2d_bwd_weight(cv, x, dy, lut_et, 7))):
        ms = _time_call(torch, fn, 5)
        r["resnet_3x3_" + name] = {"ms": round(ms, 3), "gmacs_per_s": round(macs / ms / 1e6, 1)}
    ex["exact_trunc_two_byte_table"] = r
    log("exact-truncation table done")
    cfg = W.LENET5
    lutb = B.device_lut(B.lut_build(cfg["m_bits"], "exact_trunc"), dev)
    ex["lenet5_b64_train_step_layers"] = lenet_train_step(torch, W, np, dev, lutb, cfg["m_bits"])
    log("LeNet-5 training step done")
    return ex


def lenet_train_step(torch, W, np, dev, lut, m_bits):
    """One training step (forward, autograd backward, SGD update) of LeNet-5 built from the
    autograd layers, batch 64: the per-batch training time the paper tabulates, on synthetic data."""
    from paper_2209_04161_amd import modules
    F = torch.nn.functional
    torch.manual_seed(0)
    net = torch.nn.ModuleList([modules.AMConv2d(1, 6, 5, lut, m_bits, padding="same"),
                               modules.AMConv2d(6, 16, 5, lut, m_bits),
                               modules.AMLinear(400, 120, lut, m_bits), modules.AMLinear(120, 84, lut, m_bits),
                               modules.AMLinear(84, 10, lut, m_bits)])
    x = torch.from_numpy(W.uniform((64, 28, 28, 1), 0.0, 1.0, 6000)).to(dev)
    labels = torch.from_numpy(np.random.default_rng(6010).integers(0, 10, 64)).to(dev)
    opt = torch.optim.SGD(net.parameters(), lr=0.01)

    def pool(t):
        return F.max_pool2d(t.permute(0, 3, 1, 2), 2).permute(0, 2, 3, 1).contiguous()

    def step():
        opt.zero_grad(set_to_none=True)
        h = pool(torch.relu(net[0](x)))
        h = pool(torch.relu(net[1](h))).reshape(64, 400)
        h = torch.relu(net[3](torch.relu(net[2](h))))
        F.cross_entropy(net[4](h), labels).backward()
        opt.step()

    return {"ms": round(_time_call(torch, step, 10), 3)}


def native_fp32(torch, W, dev, A, Bm, C):
    """The step's GEMM and ResNet 3x3 passes with the native FP32 multiply, in the vendor
    libraries torch calls (hipBLASLt/rocBLAS GEMM, MIOpen convolution): the paper's
    approximate-over-native ratio on this GPU.  Context only; nothing of the path runs here."""
    mm, cd = torch.backends.cuda.matmul.allow_tf32, torch.backends.cudnn.allow_tf32
    torch.backends.cuda.matmul.allow_tf32 = False  # full FP32 products
    torch.backends.cudnn.allow_tf32 = False
    try:
        out = {"what": "torch.matmul (hipBLASLt/rocBLAS) and MIOpen convolution in FP32 (TF32 off), whole calls",
               "gemm_ms": round(_time_call(torch, lambda: torch.matmul(A, Bm, out=C), 5), 4)}
        cv = W.RESNET_3X3["conv"]
        x_h, w_h, dy_h = W.resnet_conv_inputs(cv, seed=3000)
        # NHWC data viewed as NCHW (channels-last strides), HWIO weights as OIHW
        x = torch.from_numpy(x_h).to(dev).permute(0, 3, 1, 2)
        w = torch.from_numpy(w_h).to(dev).permute(3, 2, 0, 1).contiguous()
        dy = torch.from_numpy(dy_h).to(dev).permute(0, 3, 1, 2)
        pad = cv["pad_top"]
        F = torch.nn.functional
        for name, fn in (("conv_fwd_ms", lambda: F.conv2d(x, w, padding=pad)),
                         ("conv_bwd_data_ms", lambda: torch.nn.grad.conv2d_input(x.shape, w, dy, padding=pad)),
                         ("conv_bwd_weight_ms", lambda: torch.nn.grad.conv2d_weight(x, w.shape, dy, padding=pad))):
            out[name] = round(_time_call(torch, fn, 5), 4)
        return out
    finally:
        torch.backends.cuda.matmul.allow_tf32, torch.backends.cudnn.allow_tf32 = mm, cd


def cpu_baseline(frac, A_h, B_h, cv, x_h, w_h, dy_h, m_bits):
    """The CPU oracle (as it stands) on a seeded sample of every part of the step: the same
    fraction of each part's outputs, each output computed in full."""
    import numpy as np

    import oracle
    from paper_2209_04161_amd import workloads as W

    rng = np.random.default_rng(777)
    M, K = A_h.shape
    N = B_h.shape[1]
    oh, ow = W.conv_out_hw(cv)
    n_y = cv["n"] * oh * ow * cv["c_out"]
    n_dx = cv["n"] * cv["h"] * cv["w"] * cv["c_in"]
    n_dw = cv["kh"] * cv["kw"] * cv["c_in"] * cv["c_out"]
    k_fwd = cv["kh"] * cv["kw"] * cv["c_in"]
    k_bwd_w = cv["n"] * oh * ow
    parts = [("gemm", M * N, K), ("fwd", n_y, k_fwd), ("bwd_data", n_dx, k_fwd), ("bwd_weight", n_dw, k_bwd_w)]
    sample = {name: np.sort(rng.choice(total, max(1, int(round(frac * total))), replace=False))
              for name, total, _ in parts}
    macs = sum(sample[name].size * k for name, _, k in parts)
    log("cpu_baseline: oracle on %d outputs (%.3g approx-MACs)" % (sum(s.size for s in sample.values()), macs))
    t0 = time.perf_counter()
    oracle.gemm(oracle.MITCHELL, m_bits, A_h, B_h, idx=sample["gemm"])
    oracle.conv2d_fwd(oracle.MITCHELL, m_bits, cv, x_h, w_h, idx=sample["fwd"])
    oracle.conv2d_bwd_data(oracle.MITCHELL, m_bits, cv, dy_h, w_h, idx=sample["bwd_data"])
    oracle.conv2d_bwd_weight(oracle.MITCHELL, m_bits, cv, x_h, dy_h, idx=sample["bwd_weight"])
    dt = time.perf_counter() - t0
    log("cpu_baseline: %.1f s" % dt)
    return {"value": round(macs / dt / 1e9, 4), "unit": "G approx-MAC/s", "cores": oracle.num_threads(),
            "kind": "oracle", "seconds": round(dt, 2),
            "sample": "%.1f%% of the outputs of each part of the step (GEMM 4096^3, conv fwd, bwd_data, "
                      "bwd_weight), seeded uniform without replacement, each output computed in full: "
                      "%d approx-MACs" % (100 * frac, macs)}


if __name__ == "__main__":
    main()
