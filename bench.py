#!/usr/bin/env python3
"""Throughput of the Winograd convolution hot path on one MI355X (gfx950).

One step = one full layer through eq. (2) of Barabasz & Gregg (arXiv
1905.05233): kernel and input transforms (one launch), alpha'^2 batched
matrix-core contraction and output transform (separate kernels, or one fused
kernel where the library picks that path for the layer shape), on seeded
synthetic inputs already resident in HBM.  Default workload: conv3x3 stride 1 pad 1, N=8, C=K=128, H=W=56, fp32,
F(4x4,3x3) with points {0, 1, -1, 1/2, -1/2, inf}.

Prints one JSON line: direct-equivalent TFLOP/s (2 N H W C K 9 flops per
step), per-kernel average durations (HIP events on the launch stream), the
roofline of the dominant kernel, the rel-L2 error against fp64 direct
convolution, and the CPU oracle's throughput on the same workload.

    python bench.py [--steps K] [--warmup W] [--workload cfg2] [--plan 0]

``--workload cfg5`` runs the VGG-16-shaped stack instead (thirteen layers at
N = 32, ``--dtype`` bf16 or f16, the most accurate candidate plan per layer);
its step is one pass through the thirteen convolutions.
"""
import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "direct-equiv conv TFLOP/s + MFMA util/HBM GB/s; rel-L2 err vs fp64 direct"
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"f32": 157.3, "f16": 2500.0, "bf16": 2500.0}
KERNEL_NAMES = ("kernel_input_transform", "contract", "output_transform", "contract_output", "kernel_transform",
                "input_contract_output")
KERNEL_SOURCES = {"kernel_input_transform": "transforms.hip", "contract": "contract.hip",
                  "output_transform": "transforms.hip", "contract_output": "fused.hip",
                  "kernel_transform": "transforms.hip", "input_contract_output": "fused.hip"}


def algorithmic_work(wl, alpha, m):
    """Bytes / flops each kernel must move or compute for one layer."""
    s = 4 if wl.dtype == "f32" else 2
    th, tw = -(-wl.H // m), -(-wl.W // m)
    T = wl.N * th * tw
    a2 = alpha * alpha
    C, K = wl.C, wl.K
    return {
        # one launch: kernel transform (w in, U out) and input transform (x in, V out)
        "kernel_input_transform": {"bytes": 9 * C * K * s + a2 * C * K * s + wl.N * wl.H * wl.W * C * s
                                   + a2 * T * C * s},
        "contract": {"flops": 2 * a2 * T * C * K, "bytes": a2 * (T * C * s + K * C * s + T * K * 4)},
        "output_transform": {"bytes": a2 * T * K * 4 + wl.N * wl.H * wl.W * K * s},
        # fused: V and U in, y out, no M
        "contract_output": {"flops": 2 * a2 * T * C * K,
                            "bytes": a2 * (T * C * s + K * C * s) + wl.N * wl.H * wl.W * K * s},
        # fused_input path: kernel transform alone, then x and U in, y out (no V, no M)
        "kernel_transform": {"bytes": 9 * C * K * s + a2 * C * K * s},
        "input_contract_output": {"flops": 2 * a2 * T * C * K,
                                  "bytes": wl.N * wl.H * wl.W * C * s + a2 * K * C * s + wl.N * wl.H * wl.W * K * s},
        "T": T,
    }


def source_hash(name):
    with open(os.path.join(ROOT, "paper_1905_05233_amd", "csrc", name), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def load_traffic(kernel, workload_tag):
    """HBM bytes per launch from committed rocprofv3 counter summaries, if they
    were taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload_tag}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256_16") != source_hash(KERNEL_SOURCES[kernel]):
        return None
    return rec.get("hbm_bytes_per_launch")


def make_stages(plan, xd, wd, y, N_, H, W, C, K, stream):
    """Launchers of the stage kernels that conv2d runs for this layer (the
    path the plan takes for the shape; intermediates allocated here), in
    launch order, each returning the library's status."""
    import torch
    from paper_1905_05233_amd import _native as NAT
    lib = NAT.lib()
    g = plan.geometry(N_, H, W, C, K)
    a2 = plan.alpha ** 2
    dev = xd.device
    path = plan.conv_path(N_, H, W, C, K)
    fused = path == "fused"
    U = torch.empty((a2, K, g["Cp"]), dtype=xd.dtype, device=dev)
    V = torch.empty((a2, g["T"], g["Cp"]), dtype=xd.dtype, device=dev)
    M = None if fused else torch.empty((a2, g["T"], g["Kp"]), dtype=torch.float32, device=dev)
    xt = NAT.WgTensor(ctypes.c_void_p(xd.data_ptr()), N_, H, W, C)
    wt = NAT.WgTensor(ctypes.c_void_p(wd.data_ptr()), K, 3, 3, C)
    yt = NAT.WgTensor(ctypes.c_void_p(y.data_ptr()), N_, H, W, K)
    sh = ctypes.c_void_p(stream.cuda_stream)
    # the closures keep U, V, M and the tensor descriptors alive
    if path == "fused_input":
        return {
            "kernel_transform": lambda: lib.winograd_kernel_transform(plan._h, ctypes.byref(wt),
                                                                      ctypes.c_void_p(U.data_ptr()), sh),
            "input_contract_output": lambda: lib.winograd_input_contract_output(
                plan._h, ctypes.byref(xt), ctypes.c_void_p(U.data_ptr()), ctypes.byref(yt), sh),
        }
    stages = {
        "kernel_input_transform": lambda: lib.winograd_kernel_input_transform(
            plan._h, ctypes.byref(wt), ctypes.byref(xt), ctypes.c_void_p(U.data_ptr()), ctypes.c_void_p(V.data_ptr()),
            sh),
    }
    if fused:
        stages["contract_output"] = lambda: lib.winograd_contract_output(
            plan._h, ctypes.c_void_p(V.data_ptr()), ctypes.c_void_p(U.data_ptr()), C, ctypes.byref(yt), sh)
    else:
        stages["contract"] = lambda: lib.winograd_contract(plan._h, ctypes.c_void_p(V.data_ptr()),
                                                           ctypes.c_void_p(U.data_ptr()),
                                                           ctypes.c_void_p(M.data_ptr()), g["T"], C, K, sh)
        stages["output_transform"] = lambda: lib.winograd_output_transform(
            plan._h, ctypes.c_void_p(M.data_ptr()), ctypes.byref(yt), sh)
    return stages


def time_kernels(stages, reps, stream):
    """Average duration (us) of each stage kernel over ``reps`` back-to-back
    launches on ``stream``, bracketed by HIP events."""
    import torch
    from paper_1905_05233_amd import _native as NAT
    for fn in stages.values():
        NAT.check(fn())
    torch.cuda.synchronize()
    out = {}
    for name, fn in stages.items():
        for _ in range(3):
            fn()
        k0 = torch.cuda.Event(enable_timing=True)
        k1 = torch.cuda.Event(enable_timing=True)
        k0.record(stream)
        for _ in range(reps):
            fn()
        k1.record(stream)
        torch.cuda.synchronize()
        out[name] = 1e3 * k0.elapsed_time(k1) / reps
    return out


def roofline(dom, work, us, dtype):
    """Roofline record of kernel ``dom`` from its algorithmic work and time."""
    if dom in ("contract", "contract_output", "input_contract_output"):
        ai = work["flops"] / work["bytes"]
        ridge = MFMA_PEAK_TFLOPS[dtype] * 1e12 / (HBM_PEAK_GBS * 1e9)
        if ai >= ridge:
            roof = {"bound": "mfma", "achieved": round(work["flops"] / (us * 1e-6) / 1e12, 2),
                    "peak": MFMA_PEAK_TFLOPS[dtype], "unit": "TFLOP/s"}
        else:
            roof = {"bound": "hbm", "achieved": round(work["bytes"] / (us * 1e-6) / 1e9, 1), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(work["bytes"] / (us * 1e-6) / 1e9, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["kernel"] = dom
    return roof


def run_vgg(a):
    """cfg5: the VGG-16-shaped stack, N = 32, the most accurate candidate plan
    per layer; a step is one pass through the thirteen convolutions (the ReLU
    and pooling between them are not timed)."""
    import numpy as np
    import torch

    from paper_1905_05233_amd import workloads as WL
    from paper_1905_05233_amd.vgg import VggStack, relu_pool

    dtype = a.dtype or "bf16"
    N = 32
    stack = VggStack(dtype)
    x = stack.input(N)
    stream = torch.cuda.current_stream()
    for _ in range(a.warmup):
        stack.forward(x)
    torch.cuda.synchronize()
    per_layer = np.zeros(len(stack.layers))
    for _ in range(a.steps):
        _, ms = stack.timed_forward(x)
        per_layer += np.array(ms)
    per_layer /= a.steps
    ms_per_step = float(per_layer.sum())
    flops = stack.direct_flops(N)
    value = flops / (ms_per_step * 1e-3) / 1e12

    # per-kernel totals over the layers, each layer's stages timed back to back
    reps = max(5, a.steps // 5)
    tot_us = {k: 0.0 for k in KERNEL_NAMES}
    tot_work = {k: {"bytes": 0, "flops": 0} for k in KERNEL_NAMES}
    xi = x
    layers = []
    for i, L in enumerate(stack.layers):
        hw, C, K = L["hw"], L["C"], L["K"]
        y = torch.empty((N, hw, hw, K), dtype=stack.tdt, device=x.device)
        stages = make_stages(L["plan"], xi, L["w"], y, N, hw, hw, C, K, stream)
        kus = time_kernels(stages, reps, stream)
        wl = WL.Workload(f"vgg{i}", N=N, H=hw, W=hw, C=C, K=K, dtype=dtype, plans=(), x_dist="halfnormal")
        work = algorithmic_work(wl, L["plan"].alpha, L["plan"].m)
        for k in kus:
            tot_us[k] += kus[k]
            tot_work[k]["bytes"] += work[k]["bytes"]
            tot_work[k]["flops"] += work[k].get("flops", 0)
        layers.append({"layer": i, "H": hw, "C": C, "K": K, "moduli": L["spec"].moduli, "m": L["spec"].m,
                       "alpha": L["plan"].alpha, "path": L["plan"].conv_path(N, hw, hw, C, K),
                       "conv_ms": round(float(per_layer[i]), 4),
                       "kernels_us": {k: round(v, 2) for k, v in kus.items()}})
        xi = relu_pool(y, L["pool"])
    dom = max(KERNEL_NAMES, key=lambda k: tot_us[k])
    roof = roofline(dom, tot_work[dom], tot_us[dom], dtype)
    roof["traffic"] = None
    used = [k for k in KERNEL_NAMES if tot_us[k] > 0]
    kernels = {k: {"total_us": round(tot_us[k], 2), "algorithmic_bytes": tot_work[k]["bytes"],
                   "GB_s": round(tot_work[k]["bytes"] / (tot_us[k] * 1e-6) / 1e9, 1)} for k in used}
    for k in ("contract", "contract_output", "input_contract_output"):
        if k in kernels:
            kernels[k]["TFLOP_s"] = round(tot_work[k]["flops"] / (tot_us[k] * 1e-6) / 1e12, 2)
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s (direct-equivalent)",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype, "data": "synthetic",
        "config": {"workload": f"VGG-16-shaped stack of 13 conv3x3 s1 p1 NHWC layers, N={N}, {dtype}, "
                               f"most accurate candidate plan per layer (ReLU and 2x2 max-pool between "
                               f"stages, not timed)", "N": N, "layers": layers},
        "kernels": kernels, "roofline": roof,
    }
    if a.cpu_seconds > 0:
        from oracle import conv as OC
        from oracle import plan as OP
        t0 = time.perf_counter()
        done = 0
        xs = x[:1]
        for L in stack.layers:
            xa = xs.float().cpu().numpy()
            op = OP.build_plan(L["spec"].moduli, n_o=L["spec"].m, inner=L["spec"].inner)
            OC.winograd_emulated(xa, L["w"].float().cpu().numpy(), op, dtype)
            done += 2 * L["hw"] * L["hw"] * L["C"] * L["K"] * 9
            xs = relu_pool(L["plan"].conv2d(xs, L["w"]), L["pool"])
            if time.perf_counter() - t0 >= a.cpu_seconds:
                break
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": round(done / dt / 1e12, 6), "unit": "TFLOP/s (direct-equivalent)",
                               "cores": blas_threads(), "kind": "oracle",
                               "sample": f"image 0 through the stack's layers in order, as far as {a.cpu_seconds:g} s "
                                         f"allows, with the oracle's rounding-emulated Winograd ({dt:.1f} s)"}
    print(json.dumps(out), flush=True)
    return 0


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        n = [p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"]
        return max(n) if n else 1
    except Exception:
        return 1


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="cfg2")
    ap.add_argument("--plan", type=int, default=0)
    ap.add_argument("--dtype", default=None, choices=("f16", "bf16"),
                    help="storage dtype of the cfg5 VGG-16 stack (default bf16)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="CPU oracle time budget (0 disables the cpu_baseline leg)")
    ap.add_argument("--graph", action="store_true", help="replay each step from a captured HIP graph")
    ap.add_argument("--profile-kernel", default=None, choices=KERNEL_NAMES + ("copy",),
                    help="only launch this kernel, --steps times (for counter collection); 'copy' "
                         "launches a plain 256 MiB device copy to calibrate the byte counters")
    a = ap.parse_args(argv)

    if a.gpus != 1:
        print(f"bench.py: this library runs on one GPU; --gpus {a.gpus} is not supported "
              "(sharding is described in the design notes, not built)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_1905_05233_amd import _native as NAT
    from paper_1905_05233_amd import workloads as WL
    from paper_1905_05233_amd.winograd import Plan

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    dev = torch.device("cuda:0")
    if a.workload == "cfg5":
        return run_vgg(a)
    wl = WL.CONFIGS[a.workload]
    ps = wl.plans[a.plan]
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[wl.dtype]
    x32, w32 = wl.draw()
    xd = torch.from_numpy(x32).to(tdt).to(dev)
    wd = torch.from_numpy(w32).to(tdt).to(dev)
    y = torch.empty((wl.N, wl.H, wl.W, wl.K), dtype=tdt, device=dev)
    plan = Plan(ps.moduli, m=ps.m, dtype=wl.dtype, inner=ps.inner)
    work = algorithmic_work(wl, plan.alpha, plan.m)
    step = plan.bind_call(xd, wd, y)
    stream = torch.cuda.current_stream()

    stages = make_stages(plan, xd, wd, y, wl.N, wl.H, wl.W, wl.C, wl.K, stream)

    if a.profile_kernel == "copy":
        src = torch.empty(64 * 1024 * 1024, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(a.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"profiled": "copy", "bytes_read_per_launch": src.numel() * 4,
                          "bytes_written_per_launch": dst.numel() * 4, "launches": a.steps}))
        return 0
    if a.profile_kernel:
        if a.profile_kernel not in stages:
            print(f"bench.py: {a.profile_kernel} is not on this layer's path ({list(stages)})", file=sys.stderr)
            return 2
        for fn in stages.values():      # produce valid inputs for the profiled kernel
            NAT.check(fn())
        torch.cuda.synchronize()
        for _ in range(a.steps):
            NAT.check(stages[a.profile_kernel]())
        torch.cuda.synchronize()
        print(json.dumps({"profiled": a.profile_kernel, "launches": a.steps}))
        return 0

    # ---------------------------------------------------------- whole step
    run = step
    graph = None
    if a.graph:
        for _ in range(3):
            step()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        run = graph.replay
    for _ in range(a.warmup):
        run()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(a.steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / a.steps
    value = wl.direct_flops / (ms_per_step * 1e-3) / 1e12

    # ------------------------------------------- per-kernel event timing
    # Each kernel is launched --steps times back to back on the bench stream
    # between two HIP events (its inputs are valid: every stage ran first).
    kernel_us = time_kernels(stages, a.steps, stream)

    wtag = a.workload + (f"p{a.plan}" if a.plan else "")
    kernels = {}
    for name in stages:
        us = kernel_us[name]
        rec = {"avg_us": round(us, 3), "algorithmic_bytes": work[name]["bytes"],
               "GB_s": round(work[name]["bytes"] / (us * 1e-6) / 1e9, 1)}
        if "flops" in work[name]:
            rec["algorithmic_flops"] = work[name]["flops"]
            rec["TFLOP_s"] = round(work[name]["flops"] / (us * 1e-6) / 1e12, 2)
        kernels[name] = rec
    dom = max(stages, key=lambda n: kernel_us[n])
    roof = roofline(dom, work[dom], kernel_us[dom], wl.dtype)
    roof["traffic"] = load_traffic(dom, wtag)

    # --------------------------------------------- accuracy and CPU oracle
    step()
    torch.cuda.synchronize()
    y_gpu = y.float().cpu().numpy().astype(np.float64)
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s (direct-equivalent)",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": f"conv3x3 s1 p1 NHWC N={wl.N} C={wl.C} K={wl.K} H=W={wl.H} {wl.dtype} "
                               f"F({ps.m}x{ps.m},3x3) moduli {{{ps.moduli}}}",
                   "N": wl.N, "H": wl.H, "W": wl.W, "C": wl.C, "K": wl.K, "moduli": ps.moduli, "m": ps.m,
                   "alpha": plan.alpha, "tiles": work["T"], "graph": bool(a.graph),
                   "path": plan.conv_path(wl.N, wl.H, wl.W, wl.C, wl.K)},
        "kernels": kernels, "roofline": roof,
    }
    if a.cpu_seconds > 0:
        from oracle import conv as OC
        from oracle import fp as OF
        from oracle import plan as OP
        x, w = OF.to_dtype(x32, wl.dtype), OF.to_dtype(w32, wl.dtype)
        op = OP.build_plan(ps.moduli, n_o=ps.m, inner=ps.inner)
        t0 = time.perf_counter()
        reps = 0
        while True:
            yo = OC.winograd_emulated(x, w, op, wl.dtype)
            reps += 1
            if time.perf_counter() - t0 >= a.cpu_seconds:
                break
        dt = time.perf_counter() - t0
        y64 = OC.direct_f64(x, w)
        err_gpu = OC.rel_l2(y_gpu, y64)
        err_or = OC.rel_l2(yo, y64)
        out["rel_l2"] = {"gpu_vs_fp64_direct": err_gpu, "oracle_vs_fp64_direct": err_or, "cap": wl.cap,
                         "pass": bool(err_gpu <= min(2 * err_or, wl.cap))}
        out["cpu_baseline"] = {"value": round(wl.direct_flops * reps / dt / 1e12, 6),
                               "unit": "TFLOP/s (direct-equivalent)", "cores": blas_threads(), "kind": "oracle",
                               "sample": f"{reps} full layer(s) of the same workload through the oracle's "
                                         f"rounding-emulated Winograd (numpy; BLAS threads for the channel "
                                         f"sums, one thread elsewhere), {dt:.1f} s"}
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
