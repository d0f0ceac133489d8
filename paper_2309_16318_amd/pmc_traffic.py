"""Summarise HBM traffic of the PCR level kernel from rocprofv3 counter runs.

Two counter runs of the same command are needed (FETCH_SIZE, then
WRITE_SIZE; rocprofv3 cannot collect both at once), plus the same two runs
over a plain device copy of known size (``python -m
paper_2309_16318_amd.hbm_probe``), whose counters give the scale factor from
counter units to bytes.  The result is written as JSON together with the
sha256 of the kernel source it was measured on, so that readers can tell
when the figures no longer describe the current kernel.

    python -m paper_2309_16318_amd.pmc_traffic --workload NAME \
        --fetch DIR --write DIR --copy-fetch DIR --copy-write DIR --out FILE

Each DIR is a rocprofv3 ``-f csv`` output directory.
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import hashlib
import json
import os

# the PCR level kernels and the register-strip helpers they are built from
KERNEL_SOURCES = [os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", f)
                  for f in ("pcr_level.hip", "strip.h")]


def code_digest(text: str) -> str:
    """sha256 of the source with // comments and all whitespace removed, so
    that edits to comments and layout do not mark the counters stale."""
    lines = []
    for line in text.splitlines():
        k = line.find("//")
        lines.append(line if k < 0 else line[:k])
    return hashlib.sha256("".join("".join(lines).split()).encode()).hexdigest()


def kernel_source_sha256() -> str:
    text = ""
    for fn in KERNEL_SOURCES:
        with open(fn, encoding="utf-8") as f:
            text += f.read() + "\n"
    return code_digest(text)


def _rows(d: str):
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {d}")
    for fn in files:
        with open(fn) as f:
            yield from csv.DictReader(f)


def per_kernel(d: str, counter: str) -> dict:
    """{kernel-name-prefix: (dispatches, summed counter value)}."""
    acc = collections.defaultdict(lambda: [0, 0.0])
    seen = set()
    for r in _rows(d):
        if r["Counter_Name"] != counter:
            continue
        key = (r["Dispatch_Id"], r["Counter_Name"])
        if key in seen:
            continue
        seen.add(key)
        name = r["Kernel_Name"].replace("deeppcr::(anonymous namespace)::", "")
        name = name.replace("void ", "").split("(")[0]
        a = acc[name]
        a[0] += 1
        a[1] += float(r["Counter_Value"])
    return dict(acc)


def copy_factor(d: str, counter: str, nbytes: int) -> float:
    """bytes per counter unit, from the copy kernel of `nbytes` per launch."""
    k = per_kernel(d, counter)
    name = max(k, key=lambda n: k[n][1])
    n, total = k[name]
    return nbytes / (total / n)


def main():
    p = argparse.ArgumentParser()
    p.add_argument("--workload", required=True)
    p.add_argument("--fetch", required=True)
    p.add_argument("--write", required=True)
    p.add_argument("--copy-fetch", required=True)
    p.add_argument("--copy-write", required=True)
    p.add_argument("--copy-bytes", type=int, default=1 << 30)
    p.add_argument("--out", required=True)
    a = p.parse_args()
    ff = copy_factor(a.copy_fetch, "FETCH_SIZE", a.copy_bytes)
    wf = copy_factor(a.copy_write, "WRITE_SIZE", a.copy_bytes)
    fetch = per_kernel(a.fetch, "FETCH_SIZE")
    write = per_kernel(a.write, "WRITE_SIZE")
    kernels = {}
    for name in fetch:
        if "pcr_level" not in name or name not in write:
            continue
        n = fetch[name][0]
        kernels[name] = {"launches": n,
                         "read_bytes_per_launch": fetch[name][1] * ff / n,
                         "write_bytes_per_launch": write[name][1] * wf / write[name][0]}
    # The tail pass is timed as a class of its own, so the per-launch average
    # that goes with the PCR-level roofline leaves it out.
    level = {k: v for k, v in kernels.items() if not k.startswith("pcr_level_tail")}
    n_all = sum(v["launches"] for v in level.values())
    rd = sum(v["read_bytes_per_launch"] * v["launches"] for v in level.values()) / n_all
    wr = sum(v["write_bytes_per_launch"] * v["launches"] for v in level.values()) / n_all
    out = {"workload": a.workload, "kernel_source_sha256": kernel_source_sha256(),
           "fetch_bytes_per_counter_unit": ff, "write_bytes_per_counter_unit": wf,
           "pcr_level_launches": n_all, "read_bytes_per_launch": rd,
           "write_bytes_per_launch": wr, "traffic_bytes_per_launch": rd + wr,
           "by_kernel": kernels}
    os.makedirs(os.path.dirname(os.path.abspath(a.out)), exist_ok=True)
    with open(a.out, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps({k: v for k, v in out.items() if k != "by_kernel"}))


if __name__ == "__main__":
    main()
