"""The plain GEMM of the library on the two GPT-3 175B rank-share shapes,
for profiler runs of the GEMM core (kernel traces, matrix-core and LDS
counters):

    rocprofv3 --kernel-trace --stats -- python3 -m paper_2609_10549_amd.gemm_probe

Runs compass_gemm on 8192x6144x12288 (AllGather shape) and on
8192x12288x6144 with the fp32 partial (ReduceScatter shape), `--reps`
launches each after a warm-up, on random bf16 operands, and prints the
median time and rate of each from HIP events."""
from __future__ import annotations

import argparse
import json

import torch

from . import calibrate as CAL
from . import compass as C

SHAPES = {"ag": (8192, 6144, 12288), "rs": (8192, 12288, 6144)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--only", choices=sorted(SHAPES), default=None)
    args = ap.parse_args()
    torch.cuda.set_device(0)
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    out = {}
    for name, (M, N, K) in SHAPES.items():
        if args.only and name != args.only:
            continue
        A = torch.randn((M, K), device="cuda", generator=g).to(torch.bfloat16).view(torch.int16)
        W = (0.02 * torch.randn((N, K), device="cuda", generator=g)).to(torch.bfloat16).view(torch.int16)
        Cm = torch.empty((M, N), dtype=torch.int16, device="cuda")
        P = torch.randn((M, N), device="cuda", generator=g) if name == "rs" else None
        t = CAL.time_call(lambda: C.compass_gemm(A, W, Cm, P), reps=args.reps, warmup=5)
        out[name] = {"MNK": [M, N, K], "partial": P is not None, "us": round(t * 1e6, 2),
                     "tflops": round(2.0 * M * N * K / t / 1e12, 1)}
        print(json.dumps({name: out[name]}), flush=True)
        del A, W, Cm, P
        torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
