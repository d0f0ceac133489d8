"""Summaries of rocprofv3 counter runs of the PCR level kernels.

HBM traffic.  Two counter runs of the same command are needed (FETCH_SIZE,
then WRITE_SIZE; rocprofv3 cannot collect both at once), plus the same two
runs over kernels of known traffic (``probe``), whose counters give the
scale factor from counter units to bytes: a plain device copy sets the
factor, and an elementwise add (two inputs read, one output written) checks
it (``calibrate``).  MFMA use: one run with the MfmaUtil metric and SQ cycle
counters (``mfma``).  Each summary is written as JSON together with the
sha256 of the kernel source it was measured on, so that readers can tell
when the figures no longer describe the current kernel.

    python -m paper_2309_16318_amd.pmc_traffic probe [--mib 1024]
    python -m paper_2309_16318_amd.pmc_traffic calibrate --fetch DIR --write DIR --out FILE
    python -m paper_2309_16318_amd.pmc_traffic --workload NAME \
        --fetch DIR --write DIR --copy-fetch DIR --copy-write DIR --out FILE
    python -m paper_2309_16318_amd.pmc_traffic mfma --workload NAME --dir DIR --out FILE

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

# the PCR level kernels, the register-strip helpers they are built from and
# the substitution pass of the last levels
KERNEL_SOURCES = [os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", f)
                  for f in ("pcr_level.hip", "strip.h", "chain.hip")]

# kernels of the last levels' pass (timed as a class of their own)
TAIL_PREFIXES = ("pcr_chain_subst", "pcr_level_tail")


def is_tail(name: str) -> bool:
    return name.startswith(TAIL_PREFIXES)


def is_pcr(name: str) -> bool:
    """A kernel of the PCR sweep: a level pass or the last levels' pass."""
    return "pcr_level" in name or is_tail(name)


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


def kernel_key(name: str) -> str:
    """Kernel name without namespace, return type and argument list."""
    name = name.replace("deeppcr::(anonymous namespace)::", "")
    return name.replace("void ", "").split("(")[0]


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
        a = acc[kernel_key(r["Kernel_Name"])]
        a[0] += 1
        a[1] += float(r["Counter_Value"])
    return dict(acc)


def copy_factor(d: str, counter: str, nbytes: int) -> float:
    """bytes per counter unit, from the copy kernel of `nbytes` per launch."""
    k = per_kernel(d, counter)
    name = max(k, key=lambda n: k[n][1])
    n, total = k[name]
    return nbytes / (total / n)


# ------------------------------------------------------------- calibration
# The probe's kernels: a device copy of `mib` MiB (mib MiB read and written)
# and an elementwise add c = a + b of three mib/4 MiB tensors (mib/2 MiB
# read, mib/4 MiB written).
def probe_bytes(mib: int) -> dict:
    n = mib << 20
    return {"copy": {"read": n, "write": n}, "add": {"read": n // 2, "write": n // 4}}


def probe(argv=None) -> None:
    """Runs the calibration kernels on cuda:0 (under rocprofv3 --pmc)."""
    import torch

    p = argparse.ArgumentParser(prog="pmc_traffic probe")
    p.add_argument("--mib", type=int, default=1024)
    p.add_argument("--reps", type=int, default=3)
    a = p.parse_args(argv)
    n = a.mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    x = torch.ones(n // 4, dtype=torch.float32, device="cuda:0")
    y = torch.ones_like(x)
    z = torch.empty_like(x)
    for _ in range(a.reps):
        dst.copy_(src)
        torch.add(x, y, out=z)
    torch.cuda.synchronize()
    print(json.dumps({"mib": a.mib, "reps": a.reps, "bytes": probe_bytes(a.mib)}), flush=True)


def _copy_and_add(k: dict) -> tuple:
    """Names of the copy kernel (rocclr's copyBuffer) and of the add."""
    copy = next(n for n in k if "copyBuffer" in n)
    add = max((n for n in k if n != copy and "add" in n.lower()), key=lambda n: k[n][1])
    return copy, add


def calibrate(argv=None) -> dict:
    """Scale factors from the probe's copy, checked on its add."""
    p = argparse.ArgumentParser(prog="pmc_traffic calibrate")
    p.add_argument("--fetch", required=True)
    p.add_argument("--write", required=True)
    p.add_argument("--mib", type=int, default=1024)
    p.add_argument("--out")
    a = p.parse_args(argv)
    want = probe_bytes(a.mib)
    f, w = per_kernel(a.fetch, "FETCH_SIZE"), per_kernel(a.write, "WRITE_SIZE")
    cf, af = _copy_and_add(f)
    cw, aw = _copy_and_add(w)
    ff = want["copy"]["read"] / (f[cf][1] / f[cf][0])
    wf = want["copy"]["write"] / (w[cw][1] / w[cw][0])
    add_read = f[af][1] / f[af][0] * ff
    add_write = w[aw][1] / w[aw][0] * wf
    out = {"copy_kernel": cf, "add_kernel": af,
           "fetch_bytes_per_counter_unit": ff, "write_bytes_per_counter_unit": wf,
           "add_read_bytes": add_read, "add_read_expected": want["add"]["read"],
           "add_read_ratio": add_read / want["add"]["read"],
           "add_write_bytes": add_write, "add_write_expected": want["add"]["write"],
           "add_write_ratio": add_write / want["add"]["write"]}
    if a.out:
        with open(a.out, "w") as fo:
            json.dump(out, fo, indent=1)
    print(json.dumps(out))
    return out


# -------------------------------------------------------------- MFMA use
def per_kernel_all(d: str) -> dict:
    """{kernel: {counter: [dispatches, summed value]}} over every counter."""
    acc = collections.defaultdict(lambda: collections.defaultdict(lambda: [0, 0.0]))
    seen = set()
    for r in _rows(d):
        key = (r["Dispatch_Id"], r["Counter_Name"])
        if key in seen:
            continue
        seen.add(key)
        a = acc[kernel_key(r["Kernel_Name"])][r["Counter_Name"]]
        a[0] += 1
        a[1] += float(r["Counter_Value"])
    return {k: dict(v) for k, v in acc.items()}


def mfma(argv=None) -> dict:
    """Per PCR kernel: mean MfmaUtil (percent of the cycles the MFMA units
    are busy) and mean SQ cycle counters per dispatch; plus the
    dispatch-weighted MfmaUtil of the level class (pair and single-level
    passes) and of the tail pass."""
    p = argparse.ArgumentParser(prog="pmc_traffic mfma")
    p.add_argument("--workload", required=True)
    p.add_argument("--dir", required=True)
    p.add_argument("--out", required=True)
    a = p.parse_args(argv)
    allk = per_kernel_all(a.dir)
    kernels = {}
    for name, cs in allk.items():
        if not is_pcr(name) or "MfmaUtil" not in cs:
            continue
        kernels[name] = {"launches": cs["MfmaUtil"][0],
                         **{c: v[1] / v[0] for c, v in cs.items()}}

    def weighted(sel):
        ks = [v for n, v in kernels.items() if sel(n)]
        n = sum(v["launches"] for v in ks)
        return (sum(v["MfmaUtil"] * v["launches"] for v in ks) / n) if n else None
    out = {"workload": a.workload, "kernel_source_sha256": kernel_source_sha256(),
           "pcr_level_mfma_util_pct": weighted(lambda n: not is_tail(n)),
           "pcr_tail_mfma_util_pct": weighted(is_tail),
           "by_kernel": kernels}
    os.makedirs(os.path.dirname(os.path.abspath(a.out)), exist_ok=True)
    with open(a.out, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps({k: v for k, v in out.items() if k != "by_kernel"}))
    return out


def main():
    import sys

    cmds = {"probe": probe, "calibrate": calibrate, "mfma": mfma}
    if len(sys.argv) > 1 and sys.argv[1] in cmds:
        cmds[sys.argv[1]](sys.argv[2:])
        return
    traffic()


def traffic():
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
        if not is_pcr(name) or name not in write:
            continue
        n = fetch[name][0]
        kernels[name] = {"launches": n,
                         "read_bytes_per_launch": fetch[name][1] * ff / n,
                         "write_bytes_per_launch": write[name][1] * wf / write[name][0]}
    # The tail pass is timed as a class of its own, so the per-launch average
    # that goes with the PCR-level roofline leaves it out.
    level = {k: v for k, v in kernels.items() if not is_tail(k)}
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
