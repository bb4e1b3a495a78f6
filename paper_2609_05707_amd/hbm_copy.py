"""Calibration copy for rocprofv3 memory counters.

Run a plain device-to-device copy of a known size under
``rocprofv3 --pmc FETCH_SIZE`` (then ``WRITE_SIZE``): the counters of this copy,
which reads and writes exactly ``--mib`` MiB, give the factor that turns the
counter units of the same run into bytes.

Usage: python -m paper_2609_05707_amd.hbm_copy [--mib 256] [--reps 3]
"""
from __future__ import annotations

import argparse


def main() -> None:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--mib", type=int, default=256)
    ap.add_argument("--reps", type=int, default=3)
    args = ap.parse_args()
    import torch
    n = args.mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(args.reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"copied {args.mib} MiB x {args.reps}", flush=True)


if __name__ == "__main__":
    main()
