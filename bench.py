#!/usr/bin/env python3
"""Throughput of the Winograd convolution hot path on one MI355X (gfx950).

Default workload: the VGG-16-shaped stack of thirteen conv3x3 stride-1 pad-1
NHWC layers at N = 32 in bf16 (224^2 x 3 -> 64 up to 14^2 x 512 -> 512),
seeded half-normal input and He-initialised random weights, each layer on the
Winograd plan (Algorithms 1 and 2 of Barabasz & Gregg, arXiv 1905.05233)
that is most accurate against float64 direct convolution on its own input.
One step is one pass through the thirteen convolutions of eq. (2): kernel
and input transforms (one launch), then the alpha'^2 batched matrix-core
contraction and the output transform (separate kernels, or one fused kernel
where the library picks that path), inputs already resident in HBM.  The
ReLU and 2x2 max-pooling between layers (one HIP kernel each) run between the
timed convolutions; the whole pass including them is reported too.

Prints one JSON line: direct-equivalent TFLOP/s (2 N H W C K 9 flops per
layer) from HIP events around each convolution (warm caches; a device fill
before the first convolution keeps the GPU busy while the host enqueues it),
the same with the caches flushed before every layer, per-layer and per-kernel durations,
the roofline of the dominant (kernel, layer) launch (the first of the layers of
its shape, timed as their mean), each layer's rel-L2
error against float64 direct convolution, and the CPU oracle's throughput on
a bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--dtype bf16|f16]
    python bench.py --workload cfg2 [--plan 0]      # one configured layer

``--profile-kernel NAME [--profile-layer L]`` launches only that stage kernel
(of VGG layer L), ``--steps`` times, for rocprofv3 kernel traces and counters.
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
KERNEL_NAMES = ("kernel_input_transform", "input_transform", "contract", "output_transform", "contract_output",
                "kernel_transform", "input_contract_output")
KERNEL_SOURCES = {"kernel_input_transform": "transforms.hip", "input_transform": "transforms.hip",
                  "contract": "contract.hip",
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
        # later chunks of a chunked fused layer: the input transform alone
        "input_transform": {"bytes": wl.N * wl.H * wl.W * C * s + a2 * T * C * s},
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


def load_traffic(kernel, workload_tag, layer=None):
    """HBM bytes per launch from committed rocprofv3 counter summaries, if they
    were taken on the current kernel source; else None.  ``layer`` looks the
    launch up in the stack's per-layer table (``traffic_{tag}.json``)."""
    if layer is not None:
        path = os.path.join(ROOT, "profiles", f"traffic_{workload_tag}.json")
        if not os.path.exists(path):
            return None
        with open(path) as f:
            tab = json.load(f)
        src = KERNEL_SOURCES[kernel]
        if tab.get("sources", {}).get(src) != source_hash(src):
            return None
        for e in tab.get("entries", []):
            if e["layer"] == layer and e["kernel"] == kernel:
                return e["hbm_bytes_per_launch"]
        return None
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload_tag}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256_16") != source_hash(KERNEL_SOURCES[kernel]):
        return None
    return rec.get("hbm_bytes_per_launch")


def stage_counts(plan, N_, H, W, C, K):
    """{stage: (images per launch, launches per conv2d)} for the launches
    conv2d makes on this layer: a fused layer whose batch goes in chunks runs
    the kernel and input transforms on the first chunk, the input transform
    alone on each later one, and the fused kernel on every chunk (figures for
    a chunk of the largest size)."""
    path = plan.conv_path(N_, H, W, C, K)
    n_chunks, chunk = plan.conv_chunks(N_, H, W, C, K)
    if path == "fused_input":
        return {"kernel_transform": (N_, 1), "input_contract_output": (N_, 1)}
    if path == "fused":
        if n_chunks == 1:
            return {"kernel_input_transform": (N_, 1), "contract_output": (N_, 1)}
        return {"kernel_input_transform": (chunk, 1), "input_transform": (chunk, n_chunks - 1),
                "contract_output": (chunk, n_chunks)}
    return {"kernel_input_transform": (N_, 1), "contract": (N_, 1), "output_transform": (N_, 1)}


def make_stages(plan, xd, wd, y, N_, H, W, C, K, stream):
    """Launchers of the stage kernels that conv2d runs for this layer (the
    path the plan takes for the shape, each launch over as many images as
    conv2d gives it, see ``stage_counts``; intermediates allocated here), in
    launch order, each returning the library's status."""
    import torch
    from paper_1905_05233_amd import _native as NAT
    lib = NAT.lib()
    counts = stage_counts(plan, N_, H, W, C, K)
    if "input_transform" in counts:       # a chunked fused layer: launches over the first chunk
        N_ = counts["contract_output"][0]
        xd, y = xd[:N_], y[:N_]
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
    if "input_transform" in counts:
        stages["input_transform"] = lambda: lib.winograd_input_transform(
            plan._h, ctypes.byref(xt), ctypes.c_void_p(V.data_ptr()), sh)
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


def _vgg_layer_work(L, N, dtype):
    from paper_1905_05233_amd import workloads as WL
    wl = WL.Workload("vgg", N=N, H=L["hw"], W=L["hw"], C=L["C"], K=L["K"], dtype=dtype, plans=(),
                     x_dist="halfnormal")
    return algorithmic_work(wl, L["plan"].alpha, L["plan"].m)


def _vgg_cpu_baseline(stack, trace, budget_s):
    """The oracle on image 0 of the batch, layer by layer in order (each
    layer on the GPU's own input for it), until ``budget_s`` is used: the
    rounding-emulated Winograd of the layer's plan and, timed apart, the
    float64 direct convolution.  Returns the cpu_baseline record."""
    import numpy as np
    from oracle import conv as OC
    from oracle import plan as OP
    t_emu = t_dir = 0.0
    flops = 0
    done = []
    errs = {}
    for i, (L, (xi, _)) in enumerate(zip(stack.layers, trace)):
        if t_emu + t_dir >= budget_s:
            break
        x = xi[:1].float().cpu().numpy()
        w = L["w"].float().cpu().numpy()
        op = OP.build_plan(L["spec"].moduli, n_o=L["spec"].m, inner=L["spec"].inner)
        t0 = time.perf_counter()
        yo = OC.winograd_emulated(x, w, op, stack.dtype)
        t1 = time.perf_counter()
        y64 = OC.direct_f64(x, w)
        t2 = time.perf_counter()
        t_emu += t1 - t0
        t_dir += t2 - t1
        flops += 2 * L["hw"] * L["hw"] * L["C"] * L["K"] * 9
        done.append(i)
        errs[i] = OC.rel_l2(yo, y64)
    threads = blas_threads()
    return {
        "value": round(flops / t_emu / 1e12, 6), "unit": "TFLOP/s (direct-equivalent)", "cores": threads,
        "kind": "oracle",
        "sample": f"image 0 of the batch through layers {done[0]}..{done[-1]} in order (each on the GPU's input "
                  f"for it): the oracle's rounding-emulated Winograd of the layer's plan, {t_emu:.1f} s "
                  f"(numpy; BLAS threads for the channel sums, one thread elsewhere)",
        "cpu_count": os.cpu_count(), "blas_threads": threads,
        "fp64_direct": {"value": round(flops / t_dir / 1e12, 6), "unit": "TFLOP/s", "seconds": round(t_dir, 2),
                        "what": "the oracle's float64 direct convolution (9 shifted BLAS products) of the same "
                                "sample"},
        "oracle_rel_l2": {str(k): v for k, v in errs.items()},
    }


def run_vgg(a):
    """The VGG-16-shaped stack, N = 32: a step is one pass through the
    thirteen convolutions (the ReLU and pooling between them run in their own
    kernel, outside the per-convolution events)."""
    import numpy as np
    import torch

    from paper_1905_05233_amd import _native as NAT
    from paper_1905_05233_amd import layer_ops
    from paper_1905_05233_amd.vgg import VggStack

    dtype = a.dtype or "bf16"
    N = 32
    stack = VggStack(dtype)
    x = stack.input(N)
    stream = torch.cuda.current_stream()
    _, trace = stack.forward(x, keep=True)
    torch.cuda.synchronize()

    if a.profile_kernel == "each":
        # every stage kernel of every layer, --steps launches each, in order
        order = []
        for li, (L, (xi, yi)) in enumerate(zip(stack.layers, trace)):
            y = torch.empty_like(yi)
            stages = make_stages(L["plan"], xi, L["w"], y, N, L["hw"], L["hw"], L["C"], L["K"], stream)
            counts = stage_counts(L["plan"], N, L["hw"], L["hw"], L["C"], L["K"])
            for fn in stages.values():
                NAT.check(fn())
            torch.cuda.synchronize()
            for name, fn in stages.items():
                work = _vgg_layer_work(L, counts[name][0], dtype)
                for _ in range(a.steps):
                    NAT.check(fn())
                torch.cuda.synchronize()
                per = 2 if name == "kernel_input_transform" and L["plan"].tile_in > 8 else 1
                order.append({"layer": li, "kernel": name, "launches": a.steps, "dispatches": a.steps * per,
                              "bytes": work[name]["bytes"], "flops": work[name].get("flops", 0),
                              "images": counts[name][0], "per_conv": counts[name][1],
                              "shape": f"{L['hw']}x{L['hw']} {L['C']}->{L['K']}", "moduli": L["spec"].moduli})
        os.makedirs(os.path.dirname(os.path.abspath(a.order_out)), exist_ok=True)
        with open(a.order_out, "w") as f:
            json.dump({"dtype": dtype, "N": N, "order": order}, f)
        print(json.dumps({"profiled": "each", "groups": len(order), "order": a.order_out}))
        return 0

    if a.profile_kernel:
        li = a.profile_layer
        L = stack.layers[li]
        xi = trace[li][0]
        y = torch.empty((N, L["hw"], L["hw"], L["K"]), dtype=stack.tdt, device=x.device)
        stages = make_stages(L["plan"], xi, L["w"], y, N, L["hw"], L["hw"], L["C"], L["K"], stream)
        if a.profile_kernel not in stages:
            print(f"bench.py: {a.profile_kernel} is not on layer {li}'s path ({list(stages)})", file=sys.stderr)
            return 2
        for fn in stages.values():
            NAT.check(fn())
        torch.cuda.synchronize()
        for _ in range(a.steps):
            NAT.check(stages[a.profile_kernel]())
        torch.cuda.synchronize()
        print(json.dumps({"profiled": a.profile_kernel, "layer": li, "launches": a.steps}))
        return 0

    for _ in range(a.warmup):
        stack.forward(x)
    torch.cuda.synchronize()
    per_layer = np.zeros(len(stack.layers))
    lead = torch.empty(64 * 1024 * 1024, dtype=torch.float32, device=x.device)   # 256 MiB, see timed_forward
    for _ in range(a.steps):
        _, ms = stack.timed_forward(x, lead=lead)
        per_layer += np.array(ms)
    del lead
    per_layer /= a.steps
    ms_per_step = float(per_layer.sum())
    flops = stack.direct_flops(N)
    value = flops / (ms_per_step * 1e-3) / 1e12
    ms_pass = stack.timed_pass(x, a.steps)
    # cold caches: a 512 MiB buffer overwritten before every convolution
    flush = torch.empty(128 * 1024 * 1024, dtype=torch.float32, device=x.device)
    cold = np.zeros(len(stack.layers))
    for _ in range(a.steps):
        _, ms = stack.timed_forward(x, flush=flush)
        cold += np.array(ms)
    cold /= a.steps
    del flush

    # per-kernel durations, each layer's stages launched back to back
    reps = max(5, a.steps)
    layers, launches = [], []
    tot_us = {k: 0.0 for k in KERNEL_NAMES}
    tot_work = {k: {"bytes": 0, "flops": 0} for k in KERNEL_NAMES}
    for i, (L, (xi, yi)) in enumerate(zip(stack.layers, trace)):
        hw, C, K = L["hw"], L["C"], L["K"]
        y = torch.empty_like(yi)
        stages = make_stages(L["plan"], xi, L["w"], y, N, hw, hw, C, K, stream)
        counts = stage_counts(L["plan"], N, hw, hw, C, K)
        kus = time_kernels(stages, reps, stream)
        for k, us in kus.items():
            work = _vgg_layer_work(L, counts[k][0], dtype)[k]
            n_launch = counts[k][1]
            tot_us[k] += us * n_launch
            tot_work[k]["bytes"] += work["bytes"] * n_launch
            tot_work[k]["flops"] += work.get("flops", 0) * n_launch
            launches.append((us, k, i, work))
        # accuracy of image 0 against the library's float64 direct convolution
        ref = layer_ops.direct_conv_f64(xi[:1], L["w"])
        err = layer_ops.rel_l2(yi[:1].contiguous(), ref)
        layers.append({"layer": i, "H": hw, "C": C, "K": K, "moduli": L["spec"].moduli, "m": L["spec"].m,
                       "alpha": L["plan"].alpha, "path": L["plan"].conv_path(N, hw, hw, C, K),
                       "conv_ms": round(float(per_layer[i]), 4), "conv_ms_cold": round(float(cold[i]), 4),
                       "kernels_us": {k: round(v, 2) for k, v in kus.items()},
                       "launches": {k: {"images": counts[k][0], "per_conv": counts[k][1]} for k in kus},
                       "rel_l2_image0": err})
    # layers of one shape launch the same kernel on the same work: the
    # dominant launch is reported for the first of them, timed as their mean
    _, dom, dl, dwork = max(launches, key=lambda r: r[0])
    shape = lambda i: (stack.layers[i]["hw"], stack.layers[i]["C"], stack.layers[i]["K"])
    twins = [r for r in launches if r[1] == dom and shape(r[2]) == shape(dl)]
    us = float(np.mean([r[0] for r in twins]))
    dl = min(r[2] for r in twins)
    roof = roofline(dom, dwork, us, dtype)
    roof["layer"] = dl
    roof["layers_of_this_shape"] = sorted(r[2] for r in twins)
    roof["traffic"] = load_traffic(dom, f"vgg16_{dtype}", layer=dl)
    used = [k for k in KERNEL_NAMES if tot_us[k] > 0]
    kernels = {k: {"total_us": round(tot_us[k], 2), "algorithmic_bytes": tot_work[k]["bytes"],
                   "GB_s": round(tot_work[k]["bytes"] / (tot_us[k] * 1e-6) / 1e9, 1)} for k in used}
    for k in ("contract", "contract_output", "input_contract_output"):
        if k in kernels:
            kernels[k]["TFLOP_s"] = round(tot_work[k]["flops"] / (tot_us[k] * 1e-6) / 1e12, 2)
    errs = [r["rel_l2_image0"] for r in layers]
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s (direct-equivalent)",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype, "data": "synthetic",
        "config": {"workload": f"VGG-16-shaped stack of 13 conv3x3 s1 p1 NHWC layers (224x224x3->64 .. "
                               f"14x14x512->512), N={N}, {dtype}, the most accurate candidate plan per layer; "
                               f"stands in for the paper's ImageNet/VGG16 runs", "N": N, "layers": layers},
        "cold": {"ms_per_step": round(float(cold.sum()), 5),
                 "value": round(flops / (float(cold.sum()) * 1e-3) / 1e12, 2),
                 "how": "a 512 MiB device buffer overwritten before every convolution, outside its events"},
        "pass_with_relu_pool": {"ms": round(ms_pass, 5),
                                "value": round(flops / (ms_pass * 1e-3) / 1e12, 2),
                                "how": "HIP events around whole back-to-back passes: 13 convolutions and the "
                                       "ReLU/max-pool kernels"},
        "rel_l2": {"max_over_layers_image0": max(errs), "cap": 5e-2, "pass": bool(max(errs) <= 5e-2),
                   "reference": "the library's float64 direct convolution of the same layer input"},
        "kernels": kernels, "roofline": roof,
    }
    if a.cpu_seconds > 0:
        out["cpu_baseline"] = _vgg_cpu_baseline(stack, trace, a.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


STAGE_TRACE_NAMES = {"kernel_input_transform": ("kernel_input_transform<", "kernel_transform<", "input_transform<"),
                     "input_transform": ("input_transform<",),
                     "contract": ("contract_stream_kernel<", "contract_kernel<", "contract_pairwise_kernel<"),
                     "output_transform": ("output_transform<",),
                     "contract_output": ("contract_output_kernel<", "contract_output_unrolled_kernel<"),
                     "kernel_transform": ("kernel_transform<",), "input_contract_output": ("contract_output_kernel<",)}


def _read_csv(path):
    import csv
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _profile_groups(rows, info):
    """The dispatch rows of each recorded (layer, kernel) group of a
    ``--profile-kernel each`` run: the last dispatches of the library's
    kernels in dispatch order, each layer's uncounted first launch of each
    stage skipped."""
    warm = {}
    for g in info["order"]:
        warm[g["layer"]] = warm.get(g["layer"], 0) + g["dispatches"] // g["launches"]
    total = sum(g["dispatches"] for g in info["order"]) + sum(warm.values())
    rows = rows[len(rows) - total:]
    out, i, seen = [], 0, set()
    for g in info["order"]:
        if g["layer"] not in seen:
            seen.add(g["layer"])
            i += warm[g["layer"]]
        grp = rows[i:i + g["dispatches"]]
        i += g["dispatches"]
        for r in grp:
            if not any(n in r["Kernel_Name"] for n in STAGE_TRACE_NAMES[g["kernel"]]):
                raise SystemExit(f"trace does not follow the recorded order at {g}: {r['Kernel_Name'][:80]}")
        out.append(grp)
    return out


def summarize_trace(trace_csv, order_json, counters=None, table_out=None):
    """Markdown table (kernel x layer) of the average dispatch duration from a
    rocprofv3 kernel trace of ``bench.py --profile-kernel each``; with
    ``counters`` (FETCH_SIZE and WRITE_SIZE collections of the same mode and
    of the 256 MiB copy), also each group's HBM bytes per launch (medians,
    scaled by the copy's true bytes over its readings), written as well to
    ``table_out`` (JSON, with the kernel sources' hashes) for the bench line."""
    import statistics
    with open(order_json) as f:
        info = json.load(f)
    ours = lambda rows: [r for r in rows if "wg::" in r["Kernel_Name"]]   # noqa: E731
    trace = sorted(ours(_read_csv(trace_csv)), key=lambda r: int(r["Start_Timestamp"]))
    groups = _profile_groups(trace, info)
    traffic = None
    if counters:
        fetch_csv, write_csv, cf_csv, cw_csv = counters[:4]
        cinfo = info
        if len(counters) > 4:          # the counter runs' own launch order
            with open(counters[4]) as f:
                cinfo = json.load(f)
        by_id = lambda rows: sorted(ours(rows), key=lambda r: int(r["Dispatch_Id"]))   # noqa: E731
        fg = _profile_groups(by_id(_read_csv(fetch_csv)), cinfo)
        wg = _profile_groups(by_id(_read_csv(write_csv)), cinfo)
        true_bytes = 64 * 1024 * 1024 * 4
        cf = statistics.median(float(r["Counter_Value"]) for r in _read_csv(cf_csv) if "copyBuffer" in r["Kernel_Name"])
        cw = statistics.median(float(r["Counter_Value"]) for r in _read_csv(cw_csv) if "copyBuffer" in r["Kernel_Name"])
        rs, ws = true_bytes / (cf * 1024), true_bytes / (cw * 1024)
        traffic = [statistics.median(float(r["Counter_Value"]) for r in f) * 1024 * rs
                   + statistics.median(float(r["Counter_Value"]) for r in w) * 1024 * ws for f, w in zip(fg, wg)]
    dt = info["dtype"]
    if traffic and table_out:
        entries = [{"layer": g["layer"], "kernel": g["kernel"], "images": g.get("images"),
                    "algorithmic_bytes": g["bytes"], "hbm_bytes_per_launch": int(round(t))}
                   for g, t in zip(info["order"], traffic)]
        with open(table_out, "w") as f:
            json.dump({"workload": f"vgg16_{dt}", "sources": {n: source_hash(n) for n in sorted(set(KERNEL_SOURCES.values()))},
                       "read_scale": rs, "write_scale": ws, "entries": entries}, f, indent=1)
    head = ("| layer | shape | kernel | images per launch, launches per conv | dispatches | average (us) | "
            "algorithmic work | rate | fraction of peak |")
    sep = "|---|---|---|---|---|---|---|---|---|"
    if traffic:
        head += " HBM bytes per launch (counters) | traffic / algorithmic |"
        sep += "---|---|"
    lines = [head, sep]
    tot = 0.0
    for gi, (g, grp) in enumerate(zip(info["order"], groups)):
        us = sum(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in grp) / 1e3 / g["launches"]
        tot += us
        roof = roofline(g["kernel"], {"bytes": g["bytes"], "flops": g["flops"]}, us, dt)
        work = f"{g['bytes'] / 1e6:.1f} MB" + (f", {g['flops'] / 1e9:.2f} GFLOP" if g["flops"] else "")
        per = f"{g.get('images', '')}, {g.get('per_conv', '')}"
        line = (f"| {g['layer']} | {g['shape']} | `{g['kernel']}` | {per} | {g['dispatches']} | {us:.2f} | {work} | "
                f"{roof['achieved']} {roof['unit']} | {roof['frac']:.3f} ({roof['bound']}) |")
        if traffic:
            line += f" {traffic[gi] / 1e6:.1f} MB | {traffic[gi] / g['bytes']:.2f} |"
        lines.append(line)
    lines.append(f"| all | | | | | {tot:.2f} (sum over layers and kernels, one launch each) |"
                 + " |" * (len(sep.split("|")) - 8))
    return "\n".join(lines)


def summarize_counters(kernel, tag, fetch_csv, write_csv, copy_fetch_csv, copy_write_csv):
    """HBM bytes per dispatch of one kernel from rocprofv3 FETCH_SIZE and
    WRITE_SIZE runs (median over its dispatches), scaled by what the same
    counters read for a plain 256 MiB device copy; a traffic record as JSON."""
    import statistics

    def med(path, pick):
        vals = [float(r["Counter_Value"]) for r in _read_csv(path) if pick(r["Kernel_Name"])]
        return statistics.median(vals), len(vals)

    names = STAGE_TRACE_NAMES[kernel]
    ours = lambda n: "wg::" in n and any(x in n for x in names)   # noqa: E731
    copy = lambda n: "copyBuffer" in n                           # noqa: E731
    fk, nf = med(fetch_csv, ours)
    wk, nw = med(write_csv, ours)
    cf, _ = med(copy_fetch_csv, copy)
    cw, _ = med(copy_write_csv, copy)
    true_bytes = 64 * 1024 * 1024 * 4
    rs, ws = true_bytes / (cf * 1024), true_bytes / (cw * 1024)
    return {"kernel": kernel, "workload": tag, "fetch_kib": fk, "write_kib": wk, "dispatches": [nf, nw],
            "copy_fetch_kib": cf, "copy_write_kib": cw, "read_scale": rs, "write_scale": ws,
            "hbm_bytes_per_launch": int(round(fk * 1024 * rs + wk * 1024 * ws)),
            "source": KERNEL_SOURCES[kernel], "source_sha256_16": source_hash(KERNEL_SOURCES[kernel])}


def profile_copy(a, dev):
    """A plain 256 MiB device copy, --steps times: the calibration of the
    byte counters (its true traffic is known)."""
    import torch
    src = torch.empty(64 * 1024 * 1024, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(a.steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"profiled": "copy", "bytes_read_per_launch": src.numel() * 4,
                      "bytes_written_per_launch": dst.numel() * 4, "launches": a.steps}))
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
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="vgg16", choices=("vgg16", "cfg5", "cfg1", "cfg2", "cfg3", "cfg4"),
                    help="vgg16 (= cfg5, the default): the VGG-16-shaped stack; cfg1..cfg4: one layer")
    ap.add_argument("--plan", type=int, default=0)
    ap.add_argument("--dtype", default=None, choices=("f16", "bf16"),
                    help="storage dtype of the VGG-16 stack (default bf16)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="CPU oracle time budget (0 disables the cpu_baseline leg)")
    ap.add_argument("--graph", action="store_true", help="replay each step from a captured HIP graph")
    ap.add_argument("--profile-kernel", default=None, choices=KERNEL_NAMES + ("copy", "each"),
                    help="only launch this kernel, --steps times (for counter collection); 'copy' "
                         "launches a plain 256 MiB device copy to calibrate the byte counters; 'each' "
                         "launches every stage kernel of every VGG layer in turn (for a kernel trace)")
    ap.add_argument("--profile-layer", type=int, default=1, help="VGG layer of --profile-kernel (0..12)")
    ap.add_argument("--order-out", default="gpurun_out/vgg_profile_order.json",
                    help="where --profile-kernel each records its launch order")
    ap.add_argument("--summarize-trace", nargs="+", default=None,
                    metavar="TRACE_CSV ORDER_JSON [FETCH_CSV WRITE_CSV COPY_FETCH_CSV COPY_WRITE_CSV [ORDER_JSON]]",
                    help="print the kernel x layer table of a kernel trace of --profile-kernel each, with HBM "
                         "bytes from counter runs of the same mode if given (no GPU)")
    ap.add_argument("--summarize-counters", nargs=4, default=None,
                    metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="print the traffic record of --profile-kernel from counter runs (no GPU)")
    ap.add_argument("--traffic-tag", default="vgg16_bf16_l1", help="workload tag of --summarize-counters")
    ap.add_argument("--traffic-table-out", default=None,
                    help="with --summarize-trace and counter files: also write the per-launch HBM bytes table (JSON)")
    a = ap.parse_args(argv)

    if a.summarize_trace:
        if len(a.summarize_trace) not in (2, 6, 7):
            ap.error("--summarize-trace takes 2, 6 or 7 files")
        print(summarize_trace(a.summarize_trace[0], a.summarize_trace[1], a.summarize_trace[2:] or None,
                              a.traffic_table_out))
        return 0
    if a.summarize_counters:
        print(json.dumps(summarize_counters(a.profile_kernel, a.traffic_tag, *a.summarize_counters), indent=1))
        return 0

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
    if a.workload in ("vgg16", "cfg5"):
        if a.profile_kernel == "copy":
            return profile_copy(a, dev)
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
        return profile_copy(a, dev)
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
        t1 = time.perf_counter()
        y64 = OC.direct_f64(x, w)
        dt64 = time.perf_counter() - t1
        err_gpu = OC.rel_l2(y_gpu, y64)
        err_or = OC.rel_l2(yo, y64)
        out["rel_l2"] = {"gpu_vs_fp64_direct": err_gpu, "oracle_vs_fp64_direct": err_or, "cap": wl.cap,
                         "pass": bool(err_gpu <= min(2 * err_or, wl.cap))}
        out["cpu_baseline"] = {"value": round(wl.direct_flops * reps / dt / 1e12, 6),
                               "unit": "TFLOP/s (direct-equivalent)", "cores": blas_threads(), "kind": "oracle",
                               "sample": f"{reps} full layer(s) of the same workload through the oracle's "
                                         f"rounding-emulated Winograd (numpy; BLAS threads for the channel "
                                         f"sums, one thread elsewhere), {dt:.1f} s",
                               "cpu_count": os.cpu_count(), "blas_threads": blas_threads(),
                               "fp64_direct": {"value": round(wl.direct_flops / dt64 / 1e12, 6), "unit": "TFLOP/s",
                                               "seconds": round(dt64, 2)}}
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
