"""A plain device copy of known size, for calibrating the HBM byte counters.

Run under `rocprofv3 --pmc FETCH_SIZE` (then `WRITE_SIZE`): the elementwise copy
kernel reads and writes exactly `--mib` MiB per launch, so the counter's reading
for it gives the factor that turns the counter into bytes.

Usage: python -m paper_2608_15171_amd.calibrate [--mib 1024] [--launches 3]
"""
from __future__ import annotations

import argparse
import json


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--mib", type=int, default=1024)
    ap.add_argument("--launches", type=int, default=3)
    args = ap.parse_args()
    import torch
    n = args.mib * 1024 * 1024 // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(args.launches):
        torch.mul(x, 1.0, out=y)          # reads and writes n * 4 bytes
    torch.cuda.synchronize()
    print(json.dumps({"bytes_read_per_launch": n * 4, "bytes_written_per_launch": n * 4,
                      "launches": args.launches, "kernel": "vectorized_elementwise_kernel (mul)"}))


if __name__ == "__main__":
    main()
