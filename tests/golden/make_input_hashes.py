"""Writes input_hashes.json: sha256 of the seeded synthetic inputs of three
workloads each, so a change to the generators (order of draws, distributions,
rounding) is caught.  Calls only the input generators."""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from paper_2309_16318_amd import synth  # noqa: E402

out = {name: synth.digest(synth.workload_inputs(synth.WORKLOADS[name]))
       for name in ("tiny_fwd", "mlp_fwd", "resnet_skip4_fwd_bwd")}
with open(os.path.join(HERE, "input_hashes.json"), "w") as f:
    json.dump(out, f, indent=1)
print(out)
