"""A plain device-to-device copy of known size, for normalising the
FETCH_SIZE / WRITE_SIZE counters of the GEMM kernels:

    rocprofv3 --pmc FETCH_SIZE -- python paper_2609_10549_amd/copy_probe.py

copies 256 MiB five times with torch's copy kernel (no library code)."""
import torch

BYTES = 256 << 20


def main():
    src = torch.empty(BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"copied {BYTES} bytes x5")


if __name__ == "__main__":
    main()
