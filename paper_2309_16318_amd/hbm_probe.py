"""Plain device-to-device copy of a known size, for calibrating HBM byte
counters (FETCH_SIZE / WRITE_SIZE) against a kernel whose traffic is known.

    python -m paper_2309_16318_amd.hbm_probe [--mib 1024] [--reps 3]

Each repetition copies `mib` MiB with one copy launch; the script prints the
bytes each launch must read and write, and the achieved copy bandwidth.
"""
import argparse
import json
import time


def main():
    import torch

    p = argparse.ArgumentParser()
    p.add_argument("--mib", type=int, default=1024)
    p.add_argument("--reps", type=int, default=3)
    a = p.parse_args()
    n = a.mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(a.reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    nbytes = n * 4
    print(json.dumps({"bytes_read_per_copy": nbytes, "bytes_written_per_copy": nbytes,
                      "copies_timed": a.reps, "copy_GBps": 2 * nbytes * a.reps / el / 1e9}))


if __name__ == "__main__":
    main()
