"""Latency of the arrival flags: from the copy side publishing a partition's
flag (a release store into pinned host memory, once its copies have landed
and its due time has passed) to the GEMM kernel's first tile passing the
gate of that partition.

    python -m paper_2609_10549_amd.flag_latency [--out result.json]

Runs the fused AllGather of the GPT-3 shape (8192 x 6144 x 12288, double
ring, directions paced 400 / 100 GB/s) with the copy-side trace (host clock)
and the tile trace (the GPU's 100 MHz counter) in a child process. The two
clocks are not synchronised, so the measurement pairs two one-way delays of
the same signalling path:

  d_start: the kernel's first workgroup writes the start word (GPU time of
           the first ticket) -> the copy side sees it (host time);
  d_flag(q): the copy side stores flag q (host time) -> a workgroup that was
           already waiting at q's gate passes it (GPU time).

(host start seen - host flag q) + (GPU gate pass of q - GPU first ticket)
equals d_start + d_flag(q) exactly, whatever the clocks' offset, so each
partition with a tile that had taken its ticket before the flag was stored
and waited at the gate (its gate wait above `min_wait_us`) gives that sum, an
upper bound of its flag latency. Reported: the sums per partition and their
median and maximum; --keep copies the two raw traces to a directory."""
from __future__ import annotations

import argparse
import csv
import json
import os
import subprocess
import sys
import tempfile

import numpy as np

M, N, K, n = 8192, 6144, 12288, 8
RATES = (400e9, 100e9)


def child(trace_npy: str) -> None:
    import torch

    from . import compass as C
    torch.cuda.set_device(0)
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    rows = M // n
    gathered = torch.randn((M, K), device="cuda", generator=g).to(torch.bfloat16).view(torch.int16)
    shards = [gathered[0:rows] if q == 0 else
              torch.randn((rows, K), device="cuda", generator=g).to(torch.bfloat16).view(torch.int16)
              for q in range(n)]
    W = (0.02 * torch.randn((N, K), device="cuda", generator=g)).to(torch.bfloat16).view(torch.int16)
    Cm = torch.empty((M, N), dtype=torch.int16, device="cuda")
    prob = C.ag_problem(shards, gathered, W, Cm, 0, "double")
    lk = C.links(*RATES)
    for _ in range(3):
        C.compass_ag_gemm(prob, lk)
    C.compass_sync()
    C.compass_set_option(C.OPT_TILE_TRACE, 8192)
    C.compass_ag_gemm(prob, lk)
    C.compass_sync()
    np.save(trace_npy, C.compass_tile_trace(8192))
    C.compass_set_option(C.OPT_TILE_TRACE, 0)


def analyse(copy_csv: str, tiles: np.ndarray, min_wait_us: float = 5.0, tile_rows: int | None = None) -> dict:
    rows = list(csv.DictReader(open(copy_csv)))
    epoch = max(int(r["epoch"]) for r in rows)   # the traced (last) call
    ev = [r for r in rows if int(r["epoch"]) == epoch]
    start_seen = min(float(r["t_s"]) for r in ev if r["event"] == "start_seen")
    flags = {int(r["item"]): float(r["t_s"]) for r in ev if r["event"] == "flag"}
    rec = tiles.astype(np.int64)
    rt, tick, gate = rec[:, 1] >> 16, rec[:, 4], rec[:, 5]
    first_tick = tick.min()
    bm = tile_rows or M // int(rt.max() + 1)      # rows per row tile (every row tile is traced)
    half = M // n // 2
    part = (rt * bm) // half                      # double ring: partition = 2 c + h = row // (M / 2n)
    out = {}
    for q, t_flag in sorted(flags.items()):
        host_us = (start_seen - t_flag) * 1e6
        # tiles of q that began waiting before the flag was stored: a tile's
        # ticket at GPU time t (relative to the first ticket) happened before
        # the store when t + host_us < d_start, so t + host_us < 0 is a safe
        # test whatever d_start >= 0 is; they also waited at the gate
        began = (tick - first_tick) / 100.0 + host_us < 0.0
        m = (part == q) & began & ((gate - tick) / 100.0 > min_wait_us)
        if not m.any():
            continue
        gpu_us = (gate[m].min() - first_tick) / 100.0
        out[q] = round(gpu_us + host_us, 2)
    s = np.array(list(out.values()))
    return {"epoch": epoch, "sum_us_by_partition": out, "partitions": len(out),
            "median_us": float(np.median(s)) if len(s) else None, "max_us": float(s.max()) if len(s) else None,
            "min_wait_us": min_wait_us}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=None)
    ap.add_argument("--keep", default=None, help="directory to keep the raw copy-side and tile traces in")
    ap.add_argument("--child", default=None, help=argparse.SUPPRESS)
    args = ap.parse_args()
    if args.child:
        child(args.child)
        return
    with tempfile.TemporaryDirectory() as td:
        trace_csv = os.path.join(td, "copy.csv")
        tiles_npy = os.path.join(td, "tiles.npy")
        env = dict(os.environ, COMPASS_TRACE=trace_csv)
        rc = subprocess.call([sys.executable, "-u", "-m", "paper_2609_10549_amd.flag_latency", "--child", tiles_npy],
                             env=env)
        if rc != 0:
            raise SystemExit(f"child failed with status {rc}")
        res = analyse(trace_csv, np.load(tiles_npy))
        if args.keep:
            import shutil
            os.makedirs(args.keep, exist_ok=True)
            shutil.copy(trace_csv, os.path.join(args.keep, "flag_latency_copy.csv"))
            shutil.copy(tiles_npy, os.path.join(args.keep, "flag_latency_tiles.npy"))
    res.update(shape=[M, N, K, n], rates_Bps=list(RATES))
    print(json.dumps(res, indent=1))
    if args.out:
        with open(args.out, "w") as f:
            json.dump(res, f, indent=1)


if __name__ == "__main__":
    main()
