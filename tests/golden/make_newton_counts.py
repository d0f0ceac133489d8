"""Writes newton_counts.json: the number of Newton solves the oracle needs on
the full-size forward workloads (Sec. 2, Eqs. 2-3 with the start of App. F.2
and the update rule max|dZ| < tol * max(1, max|Z|), tol = 1e-5, at most 20
solves), with the final max|dZ|.  The GPU tests compare their counts with
these (within one).  Calls only the oracle and the seeded input generators;
the largest workload takes a few minutes on the CPU."""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from oracle import resnet_oracle as R  # noqa: E402
from paper_2309_16318_amd import synth  # noqa: E402

out = {}
for name in ("tiny_fwd", "mlp_fwd", "resnet_fwd_bwd", "resnet_skip4_fwd_bwd"):
    wl = synth.WORKLOADS[name]
    d = synth.workload_inputs(wl)
    t0 = time.time()
    if wl.kind == "resnet":
        _, k, ok, hist = R.resnet_newton_forward(wl.act, wl.skip, d["W"], d["bias"], d["z0"],
                                                 wl.tol, wl.max_iter)
    else:
        _, k, ok, hist = oracle.newton_forward(wl.layer, wl.alpha, d["W"], d["bias"], d["z0"],
                                               wl.tol, wl.max_iter)
    out[name] = {"B": wl.B, "L": wl.L, "w": wl.w, "tol": wl.tol, "max_iter": wl.max_iter,
                 "solves": k, "converged": bool(ok), "max_update": hist}
    print(name, k, ok, f"{time.time() - t0:.1f} s", flush=True)
with open(os.path.join(HERE, "newton_counts.json"), "w") as f:
    json.dump(out, f, indent=1)
