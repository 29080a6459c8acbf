"""Plain device-to-device copy of a known size, for calibrating HBM byte counters.

Run under ``rocprofv3 --pmc FETCH_SIZE`` (or ``WRITE_SIZE``): the counter value of the
copy kernel divided by the bytes it must move gives the scale factor applied to the
same counter read for the library's kernels.
"""
import sys

import torch


def main(mib: int = 1024, reps: int = 3):
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(f"copied {mib} MiB x {reps}: {mib * (1 << 20)} bytes read and written per copy", flush=True)


if __name__ == "__main__":
    main(int(sys.argv[1]) if len(sys.argv) > 1 else 1024)
