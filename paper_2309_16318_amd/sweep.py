"""Depth x width sweep: DeepPCR against the sequential pass on the same GPU.

Reproduces the shape of the paper's single-pass experiment (Sec. 4.1 and
App. C: random MLPs, forward and backward passes, timings over depth L and
width w, break-even depth) on one MI355X.  For every (w, L):

  * forward  — Newton + PCR (tolerance 1e-5, at most 20 iterations) against
    the sequential layer loop, both as one fused launch and as one launch per
    layer (the shape of an eager framework's loop, the paper's baseline);
  * backward — one transposed PCR solve (adjoints only, as the sequential
    pass computes) against the sequential adjoint loop, both launch shapes.

With --resnet-skip s the same is done for the collapsed-skip ResNet of
App. A.3 (DeepPCR on the block chain against the sequential GPU pass), and
with --diffusion for the diffusion-style sampler of App. A.4 (DeepPCR with
PyTorch-evaluated steps against a PyTorch step loop).

Each timing is the minimum over `--reps` runs (the paper's statistic).
Prints one JSON line per point (so a long run shows progress) and writes the
whole table to `--out`.

    python -m paper_2309_16318_amd.sweep --layer 0 --batch 1 --out sweep.json
"""
from __future__ import annotations

import argparse
import json
import time


def _time_min(fn, reps, torch):
    best = float("inf")
    for _ in range(reps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        fn()
        torch.cuda.synchronize()
        best = min(best, time.perf_counter() - t0)
    return best


def run_point(w, L, B, layer, alpha, reps, dev):
    import torch

    from paper_2309_16318_amd import deeppcr, synth

    d = synth.mlp_inputs(B, L, w, seed=0)
    t = {k: torch.from_numpy(v).to(dev) for k, v in d.items()}
    Z = torch.empty((B, L, w), dtype=torch.float32, device=dev)
    Zs = torch.empty_like(Z)
    lam = torch.empty_like(Z)
    dz0 = torch.empty((B, w), dtype=torch.float32, device=dev)
    dW = torch.empty((L, w, w), dtype=torch.float32, device=dev)
    db = torch.empty((L, w), dtype=torch.float32, device=dev)
    wsf = torch.empty(deeppcr.workspace_bytes(deeppcr.OP_FWD, B, L, w), dtype=torch.uint8,
                      device=dev)
    wsb = torch.empty(deeppcr.workspace_bytes(deeppcr.OP_BWD, B, L, w), dtype=torch.uint8,
                      device=dev)
    info = {}

    def fwd():
        r = deeppcr.deeppcr_mlp_forward(t["W"], t["bias"], t["z0"], Z, layer=layer, alpha=alpha,
                                        tol=1e-5, max_iter=20, workspace=wsf)
        info["iters"], info["status"] = r.iters, r.status

    def seq_f(per_layer):
        return lambda: deeppcr.deeppcr_seq_forward(t["W"], t["bias"], t["z0"], Zs, layer=layer,
                                                   alpha=alpha, launch_per_layer=per_layer)

    def bwd():
        deeppcr.deeppcr_mlp_backward(t["W"], t["bias"], t["z0"], Zs, t["G"], layer=layer,
                                     alpha=alpha, Lambda=lam, dz0=dz0, dW=dW, db=db,
                                     workspace=wsb)

    def seq_b(per_layer):
        return lambda: deeppcr.deeppcr_seq_backward(t["W"], t["bias"], t["z0"], Zs, t["G"],
                                                    layer=layer, alpha=alpha, Lambda=lam,
                                                    dz0=dz0, launch_per_layer=per_layer)

    out = {"w": w, "L": L, "B": B}
    out["seq_fwd_fused_ms"] = _time_min(seq_f(False), reps, torch) * 1e3
    out["seq_fwd_per_layer_ms"] = _time_min(seq_f(True), reps, torch) * 1e3
    out["deeppcr_fwd_ms"] = _time_min(fwd, reps, torch) * 1e3
    out["newton_iters"] = info["iters"]
    out["newton_status"] = info["status"]
    out["fwd_max_abs_diff"] = float((Z - Zs).abs().max())
    out["seq_bwd_fused_ms"] = _time_min(seq_b(False), reps, torch) * 1e3
    out["seq_bwd_per_layer_ms"] = _time_min(seq_b(True), reps, torch) * 1e3
    out["deeppcr_bwd_ms"] = _time_min(bwd, reps, torch) * 1e3
    for k in ("fwd", "bwd"):
        out[f"{k}_speedup_vs_fused"] = out[f"seq_{k}_fused_ms"] / out[f"deeppcr_{k}_ms"]
        out[f"{k}_speedup_vs_per_layer"] = out[f"seq_{k}_per_layer_ms"] / out[f"deeppcr_{k}_ms"]
    return out


def run_point_resnet(w, L, B, skip, act, reps, dev):
    """The collapsed-skip ResNet (App. A.3) at one (w, L): DeepPCR on the
    block chain against the sequential GPU pass (one launch for all layers)."""
    import torch

    from paper_2309_16318_amd import deeppcr, synth

    d = synth.resnet_inputs(B, L, w, seed=0)
    t = {k: torch.from_numpy(v).to(dev) for k, v in d.items()}
    Z = torch.empty((B, L, w), dtype=torch.float32, device=dev)
    Zs = torch.empty_like(Z)
    lam = torch.empty_like(Z)
    dz0 = torch.empty((B, w), dtype=torch.float32, device=dev)
    dW = torch.empty((L, w, w), dtype=torch.float32, device=dev)
    db = torch.empty((L, w), dtype=torch.float32, device=dev)
    wsf = torch.empty(deeppcr.resnet_workspace_bytes(deeppcr.OP_FWD, B, L, w, skip),
                      dtype=torch.uint8, device=dev)
    wsb = torch.empty(deeppcr.resnet_workspace_bytes(deeppcr.OP_BWD, B, L, w, skip),
                      dtype=torch.uint8, device=dev)
    info = {}

    def fwd():
        r = deeppcr.deeppcr_resnet_forward(t["W"], t["bias"], t["z0"], skip, act, Z, tol=1e-5,
                                           max_iter=20, workspace=wsf)
        info["iters"], info["status"] = r.iters, r.status

    def seq_f(per_layer):
        return lambda: deeppcr.deeppcr_resnet_seq_forward(t["W"], t["bias"], t["z0"], skip, act,
                                                          Zs, launch_per_layer=per_layer)

    def bwd():
        deeppcr.deeppcr_resnet_backward(t["W"], t["z0"], Zs, t["G"], skip, act, Lambda=lam,
                                        dz0=dz0, dW=dW, db=db, workspace=wsb)

    def seq_b(per_layer):
        return lambda: deeppcr.deeppcr_resnet_seq_backward(t["W"], t["z0"], Zs, t["G"], skip, act,
                                                           Lambda=lam, dz0=dz0,
                                                           launch_per_layer=per_layer)

    out = {"w": w, "L": L, "B": B, "skip": skip}
    out["seq_fwd_per_layer_ms"] = _time_min(seq_f(True), reps, torch) * 1e3
    out["seq_fwd_ms"] = _time_min(seq_f(False), reps, torch) * 1e3
    out["deeppcr_fwd_ms"] = _time_min(fwd, reps, torch) * 1e3
    out["newton_iters"] = info["iters"]
    out["newton_status"] = info["status"]
    out["fwd_max_abs_diff"] = float((Z - Zs).abs().max())
    out["seq_bwd_per_layer_ms"] = _time_min(seq_b(True), reps, torch) * 1e3
    out["seq_bwd_ms"] = _time_min(seq_b(False), reps, torch) * 1e3
    out["deeppcr_bwd_ms"] = _time_min(bwd, reps, torch) * 1e3
    for k in ("fwd", "bwd"):
        out[f"{k}_speedup"] = out[f"seq_{k}_ms"] / out[f"deeppcr_{k}_ms"]
        out[f"{k}_speedup_vs_per_layer"] = out[f"seq_{k}_per_layer_ms"] / out[f"deeppcr_{k}_ms"]
    return out


def run_point_diffusion(w, L, B, reps, dev):
    """The diffusion-style sampler (App. A.4) at one (w, L): DeepPCR with the
    step values and Jacobians evaluated in PyTorch against the same step
    applied L times in a PyTorch loop (the shape of the paper's baseline)."""
    import torch

    from paper_2309_16318_amd import deeppcr, generic, synth

    hd = 2 * w
    d = synth.diffusion_inputs(B, L, w, hd, seed=0)
    t = {k: torch.from_numpy(v).to(dev) for k, v in d.items()}
    p = {k: t[k] for k in ("W1", "b1", "W2", "b2", "temb")}
    step_fn, jac_fn = generic.denoising_steps(p, t["eps"])
    ws = torch.empty(deeppcr.workspace_bytes(deeppcr.OP_PCR, B, L, w), dtype=torch.uint8,
                     device=dev)
    info = {}

    def dpcr():
        r = generic.newton_generic(step_fn, jac_fn, t["zT"], L, tol=1e-5, max_iter=30,
                                   workspace=ws)
        info["iters"], info["status"], info["Z"] = r.iters, r.status, r.Z

    # the same step applied one at a time (schedule coefficients on the host,
    # so the loop never waits for the GPU)
    import numpy as np

    beta = np.linspace(1e-4, 0.02, L) if L > 1 else np.array([1e-4])
    alpha = 1.0 - beta
    alphabar = np.cumprod(alpha)
    coef = []
    for l in range(L):
        ti = L - l
        coef.append(((1.0 - alpha[ti - 1]) / np.sqrt(1.0 - alphabar[ti - 1]),
                     1.0 / np.sqrt(alpha[ti - 1]), np.sqrt(beta[ti - 1])))
    W1t, W2t = p["W1"].t().contiguous(), p["W2"].t().contiguous()
    out = torch.empty((B, L, w), dtype=torch.float32, device=dev)

    def seq():
        z = t["zT"]
        for l in range(L):
            c, isa, sb = coef[l]
            g = torch.tanh(z @ W1t + p["b1"] + p["temb"][L - l - 1]) @ W2t + p["b2"]
            z = (z - c * g) * isa + sb * t["eps"][:, l]
            out[:, l] = z

    res = {"w": w, "L": L, "B": B, "hidden": hd}
    res["seq_ms"] = _time_min(seq, reps, torch) * 1e3
    res["deeppcr_ms"] = _time_min(dpcr, reps, torch) * 1e3
    res["newton_iters"] = info["iters"]
    res["newton_status"] = info["status"]
    res["max_abs_diff"] = float((info["Z"] - out).abs().max())
    res["speedup"] = res["seq_ms"] / res["deeppcr_ms"]
    return res


def break_even(rows, key):
    """Smallest L per w from which DeepPCR stays faster (speedup > 1)."""
    res = {}
    for w in sorted({r["w"] for r in rows}):
        pts = sorted((r for r in rows if r["w"] == w), key=lambda r: r["L"])
        be = None
        for i, r in enumerate(pts):
            if all(p[key] > 1.0 for p in pts[i:]):
                be = r["L"]
                break
        res[w] = be
    return res


def main():
    import torch

    p = argparse.ArgumentParser()
    p.add_argument("--layer", type=int, default=0)
    p.add_argument("--alpha", type=float, default=1.0)
    p.add_argument("--batch", type=int, default=1)
    p.add_argument("--widths", default="2,4,8,16,32,64,128")
    p.add_argument("--depths", default=",".join(str(2 ** k) for k in range(1, 15)))
    p.add_argument("--reps", type=int, default=3)
    p.add_argument("--max-w2l", type=float, default=0.0,
                   help="> 0: skip the points with w^2 L above this (the operator storage and "
                        "the PCR work grow as w^2 L and w^3 L log L)")
    p.add_argument("--resnet-skip", type=int, default=0,
                   help="> 0: the collapsed-skip ResNet with this skip length (activation "
                        "--act), depths that are multiples of it")
    p.add_argument("--act", type=int, default=2)
    p.add_argument("--diffusion", action="store_true",
                   help="the diffusion-style sampler (denoiser width 2w) against a PyTorch "
                        "step loop")
    p.add_argument("--out", required=True)
    a = p.parse_args()
    dev = torch.device("cuda:0")
    rows = []
    if a.diffusion:
        for w in [int(x) for x in a.widths.split(",")]:
            for L in [int(x) for x in a.depths.split(",")]:
                r = run_point_diffusion(w, L, a.batch, a.reps, dev)
                rows.append(r)
                print(json.dumps(r), flush=True)
        summary = {"diffusion": True, "batch": a.batch, "reps": a.reps,
                   "break_even_L": {"speedup": break_even(rows, "speedup")},
                   "max_speedup": {"speedup": max(r["speedup"] for r in rows)}, "points": rows}
        with open(a.out, "w") as f:
            json.dump(summary, f, indent=1)
        print(json.dumps({k: v for k, v in summary.items() if k != "points"}), flush=True)
        return
    if a.resnet_skip > 0:
        for w in [int(x) for x in a.widths.split(",")]:
            for L in [int(x) for x in a.depths.split(",")]:
                if L % a.resnet_skip:
                    continue
                r = run_point_resnet(w, L, a.batch, a.resnet_skip, a.act, a.reps, dev)
                rows.append(r)
                print(json.dumps(r), flush=True)
        keys = ("fwd_speedup", "bwd_speedup", "fwd_speedup_vs_per_layer",
                "bwd_speedup_vs_per_layer")
        summary = {"resnet_skip": a.resnet_skip, "act": a.act, "batch": a.batch, "reps": a.reps,
                   "break_even_L": {k: break_even(rows, k) for k in keys},
                   "max_speedup": {k: max(r[k] for r in rows) for k in keys}, "points": rows}
        with open(a.out, "w") as f:
            json.dump(summary, f, indent=1)
        print(json.dumps({k: v for k, v in summary.items() if k != "points"}), flush=True)
        return
    for w in [int(x) for x in a.widths.split(",")]:
        for L in [int(x) for x in a.depths.split(",")]:
            if a.max_w2l > 0 and float(w) * w * L > a.max_w2l:
                continue
            r = run_point(w, L, a.batch, a.layer, a.alpha, a.reps, dev)
            rows.append(r)
            print(json.dumps(r), flush=True)
    summary = {"layer": a.layer, "alpha": a.alpha, "batch": a.batch, "reps": a.reps,
               "break_even_L": {k: break_even(rows, k) for k in
                                ("fwd_speedup_vs_fused", "fwd_speedup_vs_per_layer",
                                 "bwd_speedup_vs_fused", "bwd_speedup_vs_per_layer")},
               "max_speedup": {k: max(r[k] for r in rows) for k in
                               ("fwd_speedup_vs_fused", "fwd_speedup_vs_per_layer",
                                "bwd_speedup_vs_fused", "bwd_speedup_vs_per_layer")},
               "points": rows}
    with open(a.out, "w") as f:
        json.dump(summary, f, indent=1)
    print(json.dumps({k: v for k, v in summary.items() if k != "points"}), flush=True)


if __name__ == "__main__":
    main()
