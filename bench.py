"""Throughput of the DeepPCR hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step = one pass of the whole path over one batch of synthetic input that
is already resident in HBM.  The default workload is the deep residual net
(L = 1024 blocks, width 128, batch 16): Newton + PCR forward pass, then the
transposed-PCR backward pass with parameter gradients.  Prints one JSON line:
layer-steps/s = B*L / (seconds per step), the roofline position of the PCR
level kernel (timed with HIP events on its own stream by the library's
instrumentation), and the CPU oracle timed on the host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0        # MI355X HBM3E, GB/s
PEAK_FP32_TFLOPS = 157.3     # MI355X dense fp32 (matrix and vector), TFLOP/s
RIDGE = PEAK_FP32_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--workload", default="resnet_fwd_bwd")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=10.0)
    # forward-only workloads: also time single calls on the host, through
    # the Python binding and through the C entry point
    p.add_argument("--call-latency", action="store_true")
    return p.parse_args()


def make_step(wl, dev):
    """Returns (step(), info) for the workload with inputs resident on `dev`."""
    import torch

    from paper_2309_16318_amd import deeppcr, synth

    d = synth.workload_inputs(wl)
    t = {k: torch.from_numpy(v).to(dev) for k, v in d.items()}
    B, L, w = wl.B, wl.L, wl.w
    # marks: per step, events on the launch stream before the forward, between
    # the passes and after the backward (the split of a forward + backward step)
    info = {"iters": None, "marks": []}

    def mark():
        e = torch.cuda.Event(enable_timing=True)
        e.record()
        return e
    if wl.kind == "pcr":
        ws = torch.empty(deeppcr.workspace_bytes(deeppcr.OP_PCR, B, L, w), dtype=torch.uint8,
                         device=dev)
        x = torch.empty_like(t["r"])

        if wl.chunks > 1:
            ws = torch.empty(deeppcr.lib().deeppcr_chunked_workspace_bytes(B, L, w, wl.chunks),
                             dtype=torch.uint8, device=dev)

        def step():
            e0 = mark()
            if wl.chunks > 1:
                deeppcr.pcr_solve_block_bidiag_chunked(t["J"], t["r"], wl.chunks, x,
                                                       transpose=wl.transpose, workspace=ws)
            else:
                deeppcr.pcr_solve_block_bidiag(t["J"], t["r"], x, transpose=wl.transpose,
                                               workspace=ws)
            e1 = mark()
            info["marks"].append((e0, e1, e1))
        return step, info

    if wl.kind == "diffusion":
        from paper_2309_16318_amd import generic

        p = {k: t[k] for k in ("W1", "b1", "W2", "b2", "temb")}
        step_fn, jac_fn = generic.denoising_steps(p, t["eps"])
        ws = torch.empty(deeppcr.workspace_bytes(deeppcr.OP_PCR, B, L, w), dtype=torch.uint8,
                         device=dev)

        def step():
            e0 = mark()
            res = generic.newton_generic(step_fn, jac_fn, t["zT"], L, tol=wl.tol,
                                         max_iter=wl.max_iter, workspace=ws)
            if res.status != deeppcr.OK:
                raise RuntimeError(f"sampler status {res.status}")
            info["iters"] = res.iters
            e1 = mark()
            info["marks"].append((e0, e1, e1))
        return step, info

    if wl.kind == "resnet":
        wsf = torch.empty(deeppcr.resnet_workspace_bytes(deeppcr.OP_FWD, B, L, w, wl.skip),
                          dtype=torch.uint8, device=dev)
        wsb = torch.empty(deeppcr.resnet_workspace_bytes(deeppcr.OP_BWD, B, L, w, wl.skip),
                          dtype=torch.uint8, device=dev)
        Z = torch.empty((B, L, w), dtype=torch.float32, device=dev)
        outs = dict(Lambda=torch.empty((B, L, w), dtype=torch.float32, device=dev),
                    dz0=torch.empty((B, w), dtype=torch.float32, device=dev),
                    dW=torch.empty((L, w, w), dtype=torch.float32, device=dev),
                    db=torch.empty((L, w), dtype=torch.float32, device=dev))

        def step():
            e0 = mark()
            res = deeppcr.deeppcr_resnet_forward(t["W"], t["bias"], t["z0"], wl.skip, wl.act, Z,
                                                 tol=wl.tol, max_iter=wl.max_iter,
                                                 workspace=wsf)
            if res.status != deeppcr.OK:
                raise RuntimeError(f"forward status {res.status}")
            info["iters"] = res.iters
            e1 = mark()
            deeppcr.deeppcr_resnet_backward(t["W"], t["z0"], Z, t["G"], wl.skip, wl.act,
                                            workspace=wsb, **outs)
            info["marks"].append((e0, e1, mark()))
        return step, info

    op_ws = {}
    Z = torch.empty((B, L, w), dtype=torch.float32, device=dev)
    if "fwd" in wl.passes:
        op_ws["fwd"] = torch.empty(deeppcr.workspace_bytes(deeppcr.OP_FWD, B, L, w),
                                   dtype=torch.uint8, device=dev)
    if "bwd" in wl.passes:
        op_ws["bwd"] = torch.empty(deeppcr.workspace_bytes(deeppcr.OP_BWD, B, L, w),
                                   dtype=torch.uint8, device=dev)
        outs = dict(Lambda=torch.empty((B, L, w), dtype=torch.float32, device=dev),
                    dz0=torch.empty((B, w), dtype=torch.float32, device=dev),
                    dW=torch.empty((L, w, w), dtype=torch.float32, device=dev),
                    db=torch.empty((L, w), dtype=torch.float32, device=dev))
        if "fwd" not in wl.passes:
            # backward alone: forward states from one Newton + PCR pass, outside the timing
            res = deeppcr.deeppcr_mlp_forward(t["W"], t["bias"], t["z0"], Z, layer=wl.layer,
                                              alpha=wl.alpha, tol=wl.tol, max_iter=wl.max_iter)
            if res.status != deeppcr.OK:
                raise RuntimeError(f"forward status {res.status}")

    def step():
        e0 = mark()
        if "fwd" in wl.passes:
            res = deeppcr.deeppcr_mlp_forward(t["W"], t["bias"], t["z0"], Z, layer=wl.layer,
                                              alpha=wl.alpha, tol=wl.tol, max_iter=wl.max_iter,
                                              workspace=op_ws["fwd"])
            if res.status != deeppcr.OK:
                raise RuntimeError(f"forward status {res.status}")
            info["iters"] = res.iters
        e1 = mark()
        if "bwd" in wl.passes:
            deeppcr.deeppcr_mlp_backward(t["W"], t["bias"], t["z0"], Z, t["G"], layer=wl.layer,
                                         alpha=wl.alpha, workspace=op_ws["bwd"], **outs)
        info["marks"].append((e0, e1, mark()))

    if wl.passes == ("fwd",):
        def c_call():
            # the C entry point alone: the same call with its arguments
            # marshalled once (no Python-side checks, stream lookup or result
            # object), timed on the host; it returns after the solve's
            # host wait, as every forward call does
            import ctypes

            f = deeppcr.lib().deeppcr_mlp_forward
            it, last = ctypes.c_int(0), ctypes.c_float(0.0)
            a = (ctypes.c_void_p(t["W"].data_ptr()), ctypes.c_void_p(t["bias"].data_ptr()),
                 ctypes.c_void_p(t["z0"].data_ptr()), ctypes.c_void_p(Z.data_ptr()), B, L, w,
                 int(wl.layer), float(wl.alpha), float(wl.tol), int(wl.max_iter), None,
                 ctypes.c_void_p(op_ws["fwd"].data_ptr()), op_ws["fwd"].numel(),
                 ctypes.byref(it), ctypes.byref(last),
                 ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
            return lambda: f(*a)

        def py_call():
            deeppcr.deeppcr_mlp_forward(t["W"], t["bias"], t["z0"], Z, layer=wl.layer,
                                        alpha=wl.alpha, tol=wl.tol, max_iter=wl.max_iter,
                                        workspace=op_ws["fwd"])
        info["c_call"] = c_call
        info["py_call"] = py_call
    return step, info


def call_latency_us(fn, n, reps=5):
    """Minimum over reps of the mean host time of n back-to-back calls."""
    for _ in range(min(n, 50)):
        fn()
    best = float("inf")
    for _ in range(reps):
        t0 = time.perf_counter()
        for _ in range(n):
            fn()
        best = min(best, (time.perf_counter() - t0) / n)
    return best * 1e6


def cpu_model():
    """The host CPU's model name (as lscpu reports it), from /proc/cpuinfo."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:  # pragma: no cover
        pass
    return None


def cpu_baseline(wl, budget_s):
    """The oracle (numpy float64, sequential substitution) on the same
    workload: one warm-up run, then the minimum of 5 timed runs (fewer if
    one run takes more than a fifth of `budget_s`), with all BLAS threads
    and again with one."""
    import oracle
    from paper_2309_16318_amd import synth

    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        cores = 1
    d = synth.workload_inputs(wl)
    B, L = wl.B, wl.L
    Zs = None
    if wl.kind == "mlp" and "fwd" not in wl.passes:
        Zs = oracle.seq_forward(wl.layer, wl.alpha, d["W"], d["bias"], d["z0"])

    def once():
        if wl.kind == "pcr":
            oracle.seq_solve(d["J"], d["r"], bool(wl.transpose))
            return
        if wl.kind == "diffusion":
            oracle.diffusion_oracle.seq_sample(d, d["zT"], d["eps"])
            return
        if wl.kind == "resnet":
            R = oracle.resnet_oracle
            Z = R.resnet_seq_forward(wl.act, wl.skip, d["W"], d["bias"], d["z0"])
            R.resnet_seq_backward(wl.act, wl.skip, d["W"], d["bias"], d["z0"], Z, d["G"])
            return
        Z = Zs
        if "fwd" in wl.passes:
            Z = oracle.seq_forward(wl.layer, wl.alpha, d["W"], d["bias"], d["z0"])
        if "bwd" in wl.passes:
            oracle.seq_backward(wl.layer, wl.alpha, d["W"], d["bias"], d["z0"], Z, d["G"])

    def best(budget):
        t0 = time.perf_counter()
        once()
        warm = time.perf_counter() - t0
        runs = 5 if warm * 5 <= budget else max(1, int(budget / warm))
        times = []
        for _ in range(runs):
            t0 = time.perf_counter()
            once()
            times.append(time.perf_counter() - t0)
        return min(times), runs

    t_all, runs = best(budget_s)
    # the same with one BLAS thread
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            t_one, _ = best(budget_s)
        one = B * L / t_one
    except Exception:  # pragma: no cover
        one = None
    parts = "+".join(("seq_solve",) if wl.kind == "pcr" else
                     ("resnet_seq_forward", "resnet_seq_backward") if wl.kind == "resnet" else
                     ("diffusion seq_sample",) if wl.kind == "diffusion" else
                     tuple(p for p, on in (("seq_forward", "fwd" in wl.passes),
                                           ("seq_backward", "bwd" in wl.passes)) if on))
    return {"value": B * L / t_all, "unit": "layer-steps/s", "cores": int(cores),
            "kind": "oracle",
            "sample": f"full workload ({parts}, numpy float64): 1 warm-up, then the minimum "
                      f"of {runs} runs ({t_all * 1e3:.1f} ms per run)",
            "value_1_thread": one, "host_cpu_count": os.cpu_count(), "host_cpu_model": cpu_model()}


def measured_traffic(workload):
    """HBM bytes per PCR-level launch from the committed rocprofv3 counter
    summary of this workload (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy
    of known size), or None if there is none or the kernel source changed
    since the counters were taken."""
    from paper_2309_16318_amd import pmc_traffic

    fn = os.path.join(ROOT, "profiles", f"pcr_level_hbm_traffic_{workload}.json")
    if not os.path.exists(fn):
        return None
    with open(fn) as f:
        t = json.load(f)
    if t.get("kernel_source_sha256") != pmc_traffic.kernel_source_sha256():
        return None
    return round(t["traffic_bytes_per_launch"])


def measured_mfma_util(workload):
    """Mean MfmaUtil (percent of cycles the MFMA units are busy) of the PCR
    level launches and of the tail pass, from the committed rocprofv3
    summary of this workload, or None if there is none or the kernel source
    changed since it was taken."""
    from paper_2309_16318_amd import pmc_traffic

    fn = os.path.join(ROOT, "profiles", f"pcr_level_mfma_util_{workload}.json")
    if not os.path.exists(fn):
        return None
    with open(fn) as f:
        t = json.load(f)
    if t.get("kernel_source_sha256") != pmc_traffic.kernel_source_sha256():
        return None
    return {"pcr_level_pct": t.get("pcr_level_mfma_util_pct"),
            "pcr_tail_pct": t.get("pcr_tail_mfma_util_pct")}


def roofline(cls, w, by_intensity=False):
    """Roofline position of one kernel class from the library's counts:
    algorithmic flops and bytes of its launches over their summed event
    time; MFMA-bound at an intensity above the ridge (or, for the PCR level
    class, at w >= 64, the widths the workload targets rate against MFMA)."""
    intensity = cls["flops"] / max(cls["bytes"], 1.0)
    tflops = cls["flops"] / (cls["ms"] * 1e-3) / 1e12
    gbs = cls["bytes"] / (cls["ms"] * 1e-3) / 1e9
    # both positions, so that a w <= 32 class placed on the MFMA side still
    # shows its fraction of the HBM peak (and the other way round)
    both = {"frac_of_mfma_peak": round(tflops / PEAK_FP32_TFLOPS, 4),
            "frac_of_hbm_peak": round(gbs / PEAK_HBM_GBS, 4)}
    if intensity >= RIDGE or (w >= 64 and not by_intensity):
        return {"bound": "mfma", "achieved": round(tflops, 3), "peak": PEAK_FP32_TFLOPS,
                "unit": "TFLOP/s", "frac": round(tflops / PEAK_FP32_TFLOPS, 4), **both}
    return {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4), **both}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2309_16318_amd import deeppcr, synth

    wl = synth.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    deeppcr.lib()
    step, info = make_step(wl, dev)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    deeppcr.profile_reset()
    # only the classes placed on the roofline are timed: every event is a
    # marker between two kernels and costs the stream a few microseconds
    timed_classes = (deeppcr.KCLASS_PCR_LEVEL, deeppcr.KCLASS_PCR_TAIL)
    deeppcr.profile_select(timed_classes)
    deeppcr.profile_enable(True)
    torch.cuda.synchronize()
    info["marks"].clear()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    deeppcr.profile_enable(False)
    prof = {deeppcr.KCLASS_NAMES[c]: deeppcr.profile_read(c) for c in timed_classes}

    ms_step = el * 1e3 / args.steps
    value = wl.B * wl.L / (el / args.steps)
    roof = roofline(prof["pcr_level"], wl.w)
    roof["traffic"] = measured_traffic(wl.name)
    roof["mfma_util"] = measured_mfma_util(wl.name)
    roof["alg_bytes_per_launch"] = round(prof["pcr_level"]["bytes"] /
                                         max(prof["pcr_level"]["launches"], 1))
    roof["kernel"] = "pcr_level"
    roof["avg_launch_us"] = round(prof["pcr_level"]["ms"] * 1e3 /
                                  max(prof["pcr_level"]["launches"], 1), 3)
    roof["launches"] = prof["pcr_level"]["launches"]

    layer_names = ["tanh_mlp", "tanh_residual", "sigmoid_mlp", "sigmoid_residual", "relu_mlp",
                   "relu_residual"]
    if wl.kind == "mlp":
        layer = layer_names[wl.layer]
    elif wl.kind == "resnet":
        layer = f"{['tanh', 'sigmoid', 'relu'][wl.act]}_preact_skip{wl.skip}"
    elif wl.kind == "diffusion":
        layer = f"denoising_step_tanh_denoiser_h{wl.hidden}"
    else:
        layer = None
    cfg = {"workload": wl.name, "B": wl.B, "L": wl.L, "w": wl.w,
           "layer": layer, "alpha": wl.alpha if wl.kind == "mlp" else None,
           "passes": list(wl.passes), "newton_iters": info["iters"],
           **({"skip": wl.skip, "unknowns_per_system": wl.L // wl.skip}
              if wl.kind == "resnet" else {}),
           **({"row_chunks": wl.chunks} if wl.chunks > 1 else {}),
           "newton_tol": wl.tol if "fwd" in wl.passes else None,
           "parallelism": "single-gpu"}
    out = {
        "metric": "layer-steps/sec (B*L/s) for Newton+PCR forward and PCR backward",
        "value": round(value, 1), "unit": "layer-steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": cfg, "roofline": roof,
        "kernel_ms_per_step": {k: round(v["ms"] / args.steps, 4) for k, v in prof.items()},
    }
    tail = prof["pcr_tail"]
    if tail["launches"] > 0:
        # the last levels' pass (substitution along the chains), timed as a
        # class of its own
        out["roofline_tail"] = {"kernel": "chunk_chain" if wl.chunks > 1 else "pcr_chain_subst",
                                **roofline(tail, wl.w, by_intensity=True),
                                "avg_launch_us": round(tail["ms"] * 1e3 / tail["launches"], 3),
                                "launches": tail["launches"]}
    if info["marks"]:
        # device time of each step (first to last mark on the launch stream)
        per = sorted(a.elapsed_time(c) for a, _, c in info["marks"])
        out["step_ms_min"] = round(per[0], 4)
        out["step_ms_median"] = round(per[len(per) // 2], 4)
    if "fwd" in wl.passes and "bwd" in wl.passes and info["marks"]:
        # device time between the marks on the launch stream, per step
        n = len(info["marks"])
        out["pass_ms_per_step"] = {
            "fwd": round(sum(a.elapsed_time(b) for a, b, _ in info["marks"]) / n, 4),
            "bwd": round(sum(b.elapsed_time(c) for _, b, c in info["marks"]) / n, 4)}
    if args.call_latency and "c_call" in info:
        # latency-bound forward: per-call host time through the Python
        # binding and through the C entry point directly, beside the
        # solve's own device time (event-timed launches above)
        n = max(10, int(200.0 / max(ms_step, 1e-3)))
        out["call_latency_us"] = {
            "python_binding": round(call_latency_us(info["py_call"], n), 2),
            "c_entry": round(call_latency_us(info["c_call"](), n), 2),
            "pcr_level_event": roof["avg_launch_us"]}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
