"""Plain device copy of a known size, for calibrating rocprofv3 byte counters.

Run under ``rocprofv3 --pmc FETCH_SIZE`` (then ``WRITE_SIZE``): every
dispatch of the copy kernel reads and writes exactly --mib MiB, so the counter
value per dispatch fixes the factor between the counter and bytes moved.
"""
import argparse

import torch


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--mib", type=int, default=512)
    ap.add_argument("--reps", type=int, default=5)
    a = ap.parse_args()
    n = a.mib * 1024 * 1024 // 4
    x = torch.arange(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(a.reps):
        y.copy_(x)
    torch.cuda.synchronize()
    print(f"copied {a.mib} MiB x {a.reps}", flush=True)


if __name__ == "__main__":
    main()
