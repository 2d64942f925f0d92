"""A plain device-to-device copy of known size (256 MiB read, 256 MiB written).

Profiled with rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE, it gives the factor
that converts those counters to bytes on this device (see the profiles/
summaries that report HBM traffic).

    python paper_2609_29219_amd/measure_copy.py
"""
import torch

if __name__ == "__main__":
    a = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print("copied 3 x 256 MiB", flush=True)
