"""Offline calibration of the Compass model on this GPU (Section IV-C:
one-time linear regression of the overhead parameters).

    python -m paper_2609_10549_amd.calibrate [--out calibration.json] [--quick]

Measures, through the C ABI only:
  * plain GEMM times over a set of shapes          -> T_comp = a + b * 2MNK
  * InterDecom times at d = 2..16 with the GEMM-alone and transfer-alone
    times of the same workload                     -> eta(d) = alpha + beta d
  * fused (IntraFusion) times with the same base   -> overhead alpha_f + beta_f m
and fits them with compass_calibrate. The shapes are one TP = 8 rank's share
of Table IV workloads at evaluation scale (M >= 4096), disjoint from the
study's and the benchmark's workloads.
"""
from __future__ import annotations

import argparse
import json
import time
import os

import numpy as np
import torch

from . import compass as C

HERE = os.path.dirname(os.path.abspath(__file__))
DEFAULT_OUT = os.path.join(HERE, "calibration.json")

# (pattern, M, N, K, n): one TP = 8 rank's share of Table IV workloads at
# evaluation scale (M >= 4096): AllGather M x N_int/8 x H, ReduceScatter
# M x H x N_int/8, with (N_int, H) in {(8192, 8192), (16384, 16384),
# (4096, 16384)}. None of them is a shape of the model and selector study
# (its (N_int, H) pairs are (8192, 4096), (16384, 4096), (16384, 8192)) or of
# the benchmark's workloads, so every evaluation of the fitted model is out
# of sample.
SHAPES = [
    ("ag", 4096, 1024, 8192, 8), ("ag", 16384, 1024, 8192, 8), ("ag", 8192, 2048, 16384, 8),
    ("ag", 8192, 512, 16384, 8),
    ("rs", 4096, 8192, 1024, 8), ("rs", 16384, 8192, 1024, 8), ("rs", 8192, 16384, 2048, 8),
    ("rs", 8192, 16384, 512, 8),
]
QUICK = [SHAPES[0], SHAPES[2], SHAPES[4], SHAPES[6]]


def _rand_bits(shape, gen):
    # small random bf16 patterns (values in about [-2, 2]); calibration only needs timing
    x = torch.randn(shape, device="cuda", generator=gen, dtype=torch.float32)
    return x.to(torch.bfloat16).view(torch.int16)


class Buffers:
    def __init__(self, pattern, M, N, K, n, ring, rank=0):
        g = torch.Generator(device="cuda")
        g.manual_seed(M * 7 + N * 3 + K)
        rows = M // n
        self.pattern = pattern
        self.W = _rand_bits((N, K), g)
        self.C = torch.empty((M, N), dtype=torch.int16, device="cuda")
        if pattern == "ag":
            self.gathered = _rand_bits((M, K), g)
            self.shards = [self.gathered[q * rows:(q + 1) * rows] if q == rank else _rand_bits((rows, K), g)
                           for q in range(n)]
            self.problem = C.ag_problem(self.shards, self.gathered, self.W, self.C, rank, ring)
            self.A = self.gathered
            self.P = None
        else:
            self.A = _rand_bits((M, K), g)
            self.stage = torch.randn((M, N), device="cuda", generator=g)
            self.partials = [torch.randn((rows, N), device="cuda", generator=g) for _ in range(n)]
            self.send = [None if q == rank else torch.empty((rows, N), dtype=torch.int16, device="cuda")
                         for q in range(n)]
            self.problem = C.rs_problem(self.A, self.W, self.partials, self.stage, self.C, self.send, rank, ring)
            self.P = self.stage


def time_call(fn, reps=5, warmup=2, min_warm_s=0.1) -> float:
    """Median seconds of fn() measured with HIP events on the current stream,
    after at least `warmup` calls and `min_warm_s` seconds of them (a GPU
    that was idle runs a millisecond-long GEMM 10-15 % slower for its first
    few milliseconds of work)."""
    t0 = time.perf_counter()
    done = 0
    while done < warmup or time.perf_counter() - t0 < min_warm_s:
        fn()
        done += 1
        if done >= warmup:
            C.compass_sync()
            torch.cuda.synchronize()
    C.compass_sync()
    out = []
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        b.synchronize()
        out.append(a.elapsed_time(b) * 1e-3)
    C.compass_sync()
    return float(np.median(out))


def time_interleaved(fns: dict, reps=7, min_warm_s=0.1) -> dict:
    """Median seconds of each fn() in `fns`, timed in rounds that call every
    one of them once, so that all see the same clock and thermal state (the
    overlap metrics divide differences of these times)."""
    t0 = time.perf_counter()
    while True:
        for fn in fns.values():
            fn()
        C.compass_sync()
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= min_warm_s:
            break
    out = {k: [] for k in fns}
    for _ in range(reps):
        for k, fn in fns.items():
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            b.synchronize()
            out[k].append(a.elapsed_time(b) * 1e-3)
    C.compass_sync()
    return {k: float(np.median(v)) for k, v in out.items()}


def ring_bytes_per_link(pattern, M, N, K, n, ring):
    """Bytes one ring link carries in the whole collective (n-1 steps)."""
    div = n if ring == "single" else 2 * n
    per = M * K * 2 / div if pattern == "ag" else M * N * 4 / div
    return (n - 1) * per


def measure_shape(shape, ds=(2, 4, 8, 16), lam_targets=(0.5, 1.0, 2.0), ring="double", verbose=True):
    """Samples of one shape: GEMM alone, and per lambda target the transfer
    alone, the fused operator and InterDecom at every d that splits it."""
    pat, M, N, K, n = shape
    samples, rows_out = [], []
    buf = Buffers(pat, M, N, K, n, ring)
    w = dict(pattern=C.PATTERNS[pat], M=M, N=N, K=K, n=n)
    tg = time_call(lambda: C.compass_gemm(buf.A, buf.W, buf.C, buf.P))
    samples.append(dict(kind=0, w=w, d=1, t_meas=tg, t_comp=tg, t_comm=0.0))
    per_link = ring_bytes_per_link(pat, M, N, K, n, ring)
    for lam in lam_targets:
        rate = per_link / (tg / lam)
        lk = C.links(rate, rate)
        tx = time_call(lambda: C.compass_transfer(buf.problem, lk))
        tf = time_call(lambda: (C.compass_ag_gemm if pat == "ag" else C.compass_gemm_rs)(buf.problem, lk))
        samples.append(dict(kind=2, w=w, d=1, t_meas=tf, t_comp=tg, t_comm=tx))
        rec = dict(pattern=pat, M=M, N=N, K=K, n=n, lam_target=lam, rate=rate, t_gemm=tg, t_xfer=tx, t_fused=tf)
        for d in ds:
            if (M // n) % (2 * d if ring == "double" else d):
                continue
            td = time_call(lambda: C.compass_decomp_gemm(buf.problem, d, lk))
            samples.append(dict(kind=1, w=w, d=d, t_meas=td, t_comp=tg, t_comm=tx))
            rec[f"t_decomp_{d}"] = td
        rows_out.append(rec)
        if verbose:
            print(json.dumps(rec), flush=True)
    return samples, rows_out


def fit(samples):
    """compass_calibrate over sample dicts (host only)."""
    st = [C.compass_sample(kind=x["kind"], w=C.compass_workload(**x["w"]), d=x["d"], t_meas=x["t_meas"],
                           t_comp=x["t_comp"], t_comm=x["t_comm"]) for x in samples]
    return C.compass_calibrate(st, C.compass_calib(d_max=16))


def run(shapes, verbose=True):
    """Measure every shape in a child process of its own (a fresh device
    heap per shape, so that one shape's allocations do not shape the next
    one's copy speed), then fit."""
    import subprocess
    import sys
    import tempfile
    samples, rows = [], []
    for shape in shapes:
        with tempfile.NamedTemporaryFile(suffix=".json") as tf:
            rc = subprocess.call([sys.executable, "-u", "-m", "paper_2609_10549_amd.calibrate", "--shape",
                                  json.dumps(list(shape)), "--out", tf.name] + ([] if verbose else ["--quiet"]))
            if rc != 0:
                raise SystemExit(f"calibration of {shape} failed with status {rc}")
            with open(tf.name) as f:
                d = json.load(f)
        samples += d["samples"]
        rows += d["measurements"]
    return fit(samples), rows


def calib_to_dict(cal) -> dict:
    return {k: getattr(cal, k) for k, _ in cal._fields_}


def load(path: str = DEFAULT_OUT):
    """The stored calibration as a compass_calib, or None."""
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)["calib"]
    return C.compass_calib(**d)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=DEFAULT_OUT)
    ap.add_argument("--quick", action="store_true")
    ap.add_argument("--shape", default=None, help="measure one shape (JSON list) in this process")
    ap.add_argument("--quiet", action="store_true")
    args = ap.parse_args()
    if args.shape is not None:
        torch.cuda.set_device(0)
        samples, rows = measure_shape(tuple(json.loads(args.shape)), verbose=not args.quiet)
        with open(args.out, "w") as f:
            json.dump({"samples": samples, "measurements": rows}, f)
        return
    cal, rows = run(QUICK if args.quick else SHAPES)
    d = calib_to_dict(cal)
    import subprocess
    import sys
    device = subprocess.run([sys.executable, "-c", "import torch; print(torch.cuda.get_device_name(0))"],
                            capture_output=True, text=True).stdout.strip()
    with open(args.out, "w") as f:
        json.dump({"calib": d, "measurements": rows, "device": device}, f, indent=1)
    print(json.dumps(d))


if __name__ == "__main__":
    main()
