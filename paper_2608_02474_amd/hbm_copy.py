"""Device-to-device copy of a known size, used to calibrate the HBM byte
counters (FETCH_SIZE / WRITE_SIZE) that the profiler reports per dispatch:
the counters of this copy, divided by its exact byte count, give the factor
that turns a kernel's counter readings into bytes.

    python -m paper_2608_02474_amd.hbm_copy [--mib 1024]
"""
import argparse

import torch


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--mib", type=int, default=1024)
    a = ap.parse_args()
    n = a.mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda:0")
    src.fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    print(f"copied {n} bytes (read {n}, wrote {n})", flush=True)


if __name__ == "__main__":
    main()
