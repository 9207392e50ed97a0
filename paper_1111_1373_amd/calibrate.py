"""Counter calibration run: a streaming copy of exactly known size.

    python paper_1111_1373_amd/calibrate.py [--mib 1024] [--reps 5]

Launches the library's copy kernel (dt_probe_copy) `reps` times on a buffer of `mib`
MiB and prints the bytes each launch reads and writes, and the bandwidth it reaches.
Under a hardware-counter profiler, FETCH_SIZE and WRITE_SIZE of these dispatches divided
by the known byte counts give the scale factors applied to the tree kernels' counters.
"""
import argparse
import json
import os
import sys

if __package__ in (None, ""):   # run as a script: make the package importable
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import torch  # noqa: E402

from paper_1111_1373_amd import dtree as dt  # noqa: E402


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--mib", type=int, default=1024)
    ap.add_argument("--reps", type=int, default=5)
    args = ap.parse_args()
    n = args.mib << 20
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    dt.probe_copy(src, dst)
    torch.cuda.synchronize()
    times = []
    for _ in range(args.reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        dt.probe_copy(src, dst)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) * 1e-3)
    assert torch.equal(src, dst)
    avg = sum(times) / len(times)
    print(json.dumps({"bytes_read_per_launch": n, "bytes_written_per_launch": n,
                      "launches": args.reps + 1, "avg_us": avg * 1e6,
                      "copy_gbps_read_plus_write": 2 * n / avg / 1e9}))


if __name__ == "__main__":
    main()
