"""Plain device copy of a known size, for calibrating HBM traffic counters.

    python -m paper_2609_18935_amd.calibrate_copy [MiB]

Copies a buffer of the given size (default 256 MiB) with torch a few times. Run
under `rocprofv3 --pmc FETCH_SIZE` (then `WRITE_SIZE`) to read what the counters
report for exactly that many bytes read and written; the ratio scales the
counters of the library's kernels to bytes.
"""
import sys

import torch


def main():
    mib = int(sys.argv[1]) if len(sys.argv) > 1 else 256
    n = mib << 20
    a = torch.ones(n, dtype=torch.uint8, device="cuda:0")
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(f"copied {mib} MiB x 5")


if __name__ == "__main__":
    main()
