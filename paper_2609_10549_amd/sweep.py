"""Measurement study around the benchmark step, on one GPU:

    python -m paper_2609_10549_amd.sweep [--out sweep.json] [--quick]

* InterDecom sweep on the QKV-projection shape (AllGather, 4096 tokens,
  hidden 8192, TP = 8 share N = 3072, single ring): T(d) for
  d = 1, 2, 4, 8, 16, the fused operator, compass_pick_strategy's choice (with
  the stored calibration), the measured best d, the regret of the predicted
  d* and the gap of the fixed d = 4 heuristic (Section V-B, Fig. 8).
* Overlap at the comp/comm ratios of the paper's Table I (lambda = 0.72,
  0.89, 4.39, 5.17) and at lambda = 1 for the two MLP operators of the
  benchmark step (AllGather 8192x2048x4096 double ring, ReduceScatter
  8192x4096x2048 single ring). A lambda whose link rate the copy engines
  cannot reach is reported once at the engines' ceiling (unpaced). The
  compute-dominated ratios (lambda > 2) need more flops per link byte than
  those shapes have: they are measured on the Table IV shapes with the
  largest N (AllGather 8192x16384x4096) and the largest K (ReduceScatter
  8192x4096x16384), as far as the ceiling allows.
* The GPT-3 175B shapes (8192 tokens, hidden 12288, TP = 8) over a double
  ring whose directions run at 4 : 1, with chunks split in halves and split
  in proportion to the rates (fused, unfused, InterDecom d = 2, 4, 8).
* Cross-NUMA AllGather (Section III-A): the fc1 shape over two NUMA domains
  of four ranks, the single ring (every step at the cross-domain rate B, and
  with per-hop rates: two slow hops at B, the rest at 200 GB/s) against the
  AlltoAll pattern (own-domain links at 200 GB/s, all cross-domain flows
  sharing B): transfer alone, fused and unfused, their effective bandwidths
  and the model's T_comm.
* Sub-chunk arrival flags: the benchmark's two operators and the GPT-3
  AllGather with 1, 2, 4 (and 8) arrival flags per partition.
* torch.matmul (hipBLASLt) on every GEMM shape, for context.

Timing only: the inputs are seeded random bf16 on the GPU (parity is the
tests' job). Every number is the median of several HIP-event-timed calls.
"""
from __future__ import annotations

import argparse
import json

import torch

from . import calibrate as CAL
from . import compass as C

LAMBDAS = (0.72, 0.89, 1.0, 4.39, 5.17)
CEILING_FRACTION = 0.95


def _fused(pat):
    return C.compass_ag_gemm if pat == "ag" else C.compass_gemm_rs


def _matmul_time(buf, reps=10):
    A = buf.A.view(torch.bfloat16)
    B = buf.W.view(torch.bfloat16).t().contiguous()   # K x N, row-major
    return CAL.time_call(lambda: torch.matmul(A, B), reps=reps)


def _pick(pat, M, N, K, n, ring, fwd, bwd, cal):
    w = C.compass_workload(pattern=C.PATTERNS[pat], M=M, N=N, K=K, n=n)
    t = C.compass_topology(ring=C.RINGS[ring], fwd_Bps=fwd, bwd_Bps=bwd, step_latency_s=0.0)
    return C.compass_pick_strategy(w, t, cal)


def overlap_point(buf, pat, lk, reps=7):
    t = CAL.time_interleaved({"g": lambda: C.compass_gemm(buf.A, buf.W, buf.C, buf.P),
                              "x": lambda: C.compass_transfer(buf.problem, lk),
                              "f": lambda: _fused(pat)(buf.problem, lk),
                              "s": lambda: C.compass_sequential(buf.problem, lk)}, reps=reps)
    tg, tx, tf, ts = t["g"], t["x"], t["f"], t["s"]
    ideal = ts - max(tg, tx)
    E = (ts - tf) / ideal if ideal > 0 else None
    h = (tg + tx - tf) / tx
    return dict(t_gemm_us=tg * 1e6, t_xfer_us=tx * 1e6, t_fused_us=tf * 1e6, t_seq_us=ts * 1e6, lam=tg / tx,
                E=E, h=h)


def lambda_study(pat, M, N, K, n, ring, lambdas, verbose):
    buf = CAL.Buffers(pat, M, N, K, n, ring)
    tg = CAL.time_call(lambda: C.compass_gemm(buf.A, buf.W, buf.C, buf.P), reps=10)
    tm = _matmul_time(buf)
    per_link = CAL.ring_bytes_per_link(pat, M, N, K, n, ring)
    unpaced = C.links(0.0, 0.0)
    cap = per_link / CAL.time_call(lambda: C.compass_transfer(buf.problem, unpaced), reps=5)
    out = dict(pattern=pat, M=M, N=N, K=K, n=n, ring=ring, t_gemm_us=tg * 1e6,
               gemm_tflops=2.0 * M * N * K / tg / 1e12, torch_matmul_us=tm * 1e6,
               ceiling_Bps_per_ring=cap, points=[])
    ceiling_done = False
    for lam in lambdas:
        rate = per_link * lam / tg
        if rate < CEILING_FRACTION * cap:
            pt = overlap_point(buf, pat, C.links(rate, rate))
            pt.update(lam_target=lam, rate_Bps=rate)
        elif not ceiling_done:
            pt = overlap_point(buf, pat, unpaced)
            pt.update(lam_target=lam, rate_Bps=0.0, note="rate above the copy-engine ceiling: unpaced")
            ceiling_done = True
        else:
            continue
        out["points"].append(pt)
        if verbose:
            print(json.dumps({k: (round(v, 4) if isinstance(v, float) else v) for k, v in pt.items()}), flush=True)
    del buf
    torch.cuda.empty_cache()
    return out


def decomp_study(cal, lam, verbose):
    pat, M, N, K, n, ring = "ag", 4096, 3072, 8192, 8, "single"
    buf = CAL.Buffers(pat, M, N, K, n, ring)
    tg = CAL.time_call(lambda: C.compass_gemm(buf.A, buf.W, buf.C, buf.P), reps=10)
    per_link = CAL.ring_bytes_per_link(pat, M, N, K, n, ring)
    unpaced = C.links(0.0, 0.0)
    cap = per_link / CAL.time_call(lambda: C.compass_transfer(buf.problem, unpaced), reps=5)
    rate = per_link * lam / tg
    lk = C.links(rate, rate) if rate < CEILING_FRACTION * cap else unpaced
    fns = {"g": lambda: C.compass_gemm(buf.A, buf.W, buf.C, buf.P),
           "x": lambda: C.compass_transfer(buf.problem, lk),
           "f": lambda: C.compass_ag_gemm(buf.problem, lk)}
    for d in (1, 2, 4, 8, 16):
        fns[d] = (lambda d=d: C.compass_decomp_gemm(buf.problem, d, lk))
    t = CAL.time_interleaved(fns, reps=7)
    tg, tx, tf = t["g"], t["x"], t["f"]
    times = {d: t[d] for d in (1, 2, 4, 8, 16)}
    eff = per_link / tx
    ch = _pick(pat, M, N, K, n, ring, eff, eff, cal)
    d_meas = min(times, key=times.get)
    d_star = ch.d_star
    out = dict(shape=[M, N, K, n, ring], lam_target=lam, rate_Bps=lk.fwd_Bps, t_gemm_us=tg * 1e6,
               t_xfer_us=tx * 1e6, lam=tg / tx, t_decomp_us={str(d): t * 1e6 for d, t in times.items()},
               t_fused_us=tf * 1e6, d_meas=d_meas, d_star=d_star,
               strategy_pick="intra_fusion" if ch.strategy == C.INTRA_FUSION else "inter_decom",
               strategy_meas="intra_fusion" if tf < times[d_meas] else "inter_decom",
               regret_d_star=(times[d_star] / times[d_meas] - 1.0) if d_star in times else None,
               gap_d4=times[4] / times[d_meas] - 1.0,
               model_t_decomp_us=ch.t_decomp * 1e6, model_t_fusion_us=ch.t_fusion * 1e6)
    if verbose:
        print(json.dumps(out), flush=True)
    del buf
    torch.cuda.empty_cache()
    return out


GPT3_SHAPES = {"ag": (8192, 6144, 12288), "rs": (8192, 12288, 6144)}


def gpt3_study(pats, verbose, cal=None):
    """GPT-3 175B shapes over a double ring whose forward direction runs at 4x
    the backward one: chunks split in halves (the paper's double ring) and
    split in proportion to the rates; fused, unfused and InterDecom at
    d = 2, 4, 8, and the selector's pick for each ring."""
    import types
    res = []
    for pat in pats:
        M, N, K = GPT3_SHAPES[pat]
        n = 8
        buf = CAL.Buffers(pat, M, N, K, n, "double")
        tg = CAL.time_call(lambda: C.compass_gemm(buf.A, buf.W, buf.C, buf.P), reps=5)
        tm = _matmul_time(buf, reps=5)
        per_link = CAL.ring_bytes_per_link(pat, M, N, K, n, "double")
        unpaced = C.links(0.0, 0.0)
        cap = per_link / CAL.time_call(lambda: C.compass_transfer(buf.problem, unpaced), reps=3)
        # the slow direction at the rate that balances the GEMM on halves,
        # capped so the fast one (4x) stays below the ceiling
        bwd = min(per_link / tg, CEILING_FRACTION * cap / 4.0)
        lk = C.links(4.0 * bwd, bwd)
        for ring in ("double", "double_split"):
            if ring == "double":
                prob = buf.problem
            elif pat == "ag":
                prob = C.ag_problem(buf.shards, buf.gathered, buf.W, buf.C, 0, ring)
            else:
                prob = C.rs_problem(buf.A, buf.W, buf.partials, buf.stage, buf.C, buf.send, 0, ring)
            view = types.SimpleNamespace(A=buf.A, W=buf.W, C=buf.C, P=buf.P, problem=prob)
            pt = overlap_point(view, pat, lk, reps=5)
            dec = CAL.time_interleaved({d: (lambda d=d: C.compass_decomp_gemm(prob, d, lk)) for d in (2, 4, 8)},
                                       reps=5)
            pt.update(pattern=pat, ring=ring, M=M, N=N, K=K, fwd_Bps=4.0 * bwd, bwd_Bps=bwd,
                      gemm_tflops=2.0 * M * N * K / (pt["t_gemm_us"] * 1e-6) / 1e12, torch_matmul_us=tm * 1e6,
                      fused_tflops=2.0 * M * N * K / (pt["t_fused_us"] * 1e-6) / 1e12,
                      t_decomp_us={str(d): t * 1e6 for d, t in dec.items()})
            if cal is not None:
                ch = _pick(pat, M, N, K, n, ring, 4.0 * bwd, bwd, cal)
                pt.update(pick="intra_fusion" if ch.strategy == C.INTRA_FUSION else "inter_decom",
                          pick_d=ch.d_star, model_t_comm_us=ch.t_comm * 1e6)
            res.append(pt)
            if verbose:
                print(json.dumps({k: (round(v, 4) if isinstance(v, float) else v) for k, v in pt.items()}),
                      flush=True)
        del buf
        torch.cuda.empty_cache()
    return res


NUMA_INTRA_BPS = 200e9
NUMA_CROSS_BPS = (50e9, 100e9)


def numa_study(verbose):
    """The single ring against the AlltoAll pattern on the cross-NUMA
    topology of Section III-A (n = 8, two domains of four ranks), on the
    fc1 AllGather shape. Single ring: every step at the cross-domain rate B
    (its slowest hop; the paper's step model), and with per-hop rates (hops
    3 -> 4 and 7 -> 0 at B, the rest at 200 GB/s) seen from rank 0, right
    after a slow hop, and from rank 3, three fast hops downstream of one.
    AlltoAll: own-domain chunks over direct links at 200 GB/s while the 16
    flows into the domain share B."""
    import types
    pat, M, N, K, n = "ag", 8192, 2048, 4096, 8
    S = M * K * 2.0
    res = []
    bufs = {r: CAL.Buffers(pat, M, N, K, n, "single", rank=r) for r in (0, 3)}
    for cross in NUMA_CROSS_BPS:
        hops = [cross if q in (3, 7) else NUMA_INTRA_BPS for q in range(n)]
        cases = (("single", 0, "single", C.links(cross, cross)),
                 ("single_hops", 0, "single", C.links(NUMA_INTRA_BPS, hop_Bps=hops)),
                 ("single_hops", 3, "single", C.links(NUMA_INTRA_BPS, hop_Bps=hops)),
                 ("alltoall", 0, "alltoall", C.links(NUMA_INTRA_BPS, cross)))
        for name, rank, ring, lk in cases:
            buf = bufs[rank]
            prob = buf.problem if ring == "single" else \
                C.ag_problem(buf.shards, buf.gathered, buf.W, buf.C, rank, ring)
            view = types.SimpleNamespace(A=buf.A, W=buf.W, C=buf.C, P=buf.P, problem=prob)
            pt = overlap_point(view, pat, lk, reps=5)
            if name == "single_hops":
                model = C.compass_ring_arrival_times(n, rank, S / n, hops)[-1]
            else:
                w = C.compass_workload(pattern=C.PATTERNS[pat], M=M, N=N, K=K, n=n)
                t = C.compass_topology(ring=C.RINGS[ring], fwd_Bps=lk.fwd_Bps, bwd_Bps=lk.bwd_Bps,
                                       step_latency_s=0.0)
                model = C.compass_model_t_comm(w, t)
            pt.update(pattern=pat, ring=name, rank=rank, M=M, N=N, K=K, n=n, cross_Bps=cross,
                      intra_Bps=cross if name == "single" else NUMA_INTRA_BPS,
                      model_t_comm_us=model * 1e6, eff_bw_Bps=S / (pt["t_xfer_us"] * 1e-6),
                      eff_bw_model_Bps=S / model)
            res.append(pt)
            if verbose:
                print(json.dumps({k: (round(v, 4) if isinstance(v, float) else v) for k, v in pt.items()}),
                      flush=True)
    del bufs
    torch.cuda.empty_cache()
    return res


SUBCHUNK_CASES = (("ag", 8192, 2048, 4096, "double", 0.0, 0.0), ("ag", 8192, 2048, 4096, "double", 150e9, 150e9),
                  ("ag", 8192, 2048, 4096, "double", 216e9, 216e9), ("rs", 8192, 4096, 2048, "single", 0.0, 0.0),
                  ("rs", 8192, 4096, 2048, "single", 150e9, 150e9),
                  ("ag", 8192, 6144, 12288, "double_split", 257e9, 64e9))


def subchunk_study(verbose):
    """Sub-chunk arrival flags: transfer and fused times of the benchmark's
    two operators and the GPT-3 AllGather against the number of flags per
    partition (1, 2, 4, and 8 where the 64-partition limit allows)."""
    res = []
    for pat, M, N, K, ring, fwd, bwd in SUBCHUNK_CASES:
        buf = CAL.Buffers(pat, M, N, K, 8, ring)
        fns = {"g": lambda: C.compass_gemm(buf.A, buf.W, buf.C, buf.P)}
        subs = [s for s in (1, 2, 4, 8) if (16 if ring != "single" else 8) * s <= 64]
        for sub in subs:
            lk = C.links(fwd, bwd, sub_chunks=sub)
            fns[("x", sub)] = (lambda lk=lk: C.compass_transfer(buf.problem, lk))
            fns[("f", sub)] = (lambda lk=lk: _fused(pat)(buf.problem, lk))
        t = CAL.time_interleaved(fns, reps=7)
        pt = dict(pattern=pat, M=M, N=N, K=K, ring=ring, fwd_Bps=fwd, bwd_Bps=bwd, t_gemm_us=t["g"] * 1e6,
                  t_xfer_us={str(s): t[("x", s)] * 1e6 for s in subs},
                  t_fused_us={str(s): t[("f", s)] * 1e6 for s in subs})
        res.append(pt)
        if verbose:
            print(json.dumps(pt), flush=True)
        del buf
        torch.cuda.empty_cache()
    return res


STUDIES = ("decomp", "mlp", "high", "gpt3_ag", "gpt3_rs", "numa", "subchunk")


def run_study(name, quick, cal):
    lams = (0.72, 1.0) if quick else LAMBDAS
    low = tuple(x for x in lams if x <= 2.0)
    high = tuple(x for x in lams if x > 2.0)
    if name == "decomp":
        return {"decomp": [decomp_study(cal, lam, True) for lam in ((1.0,) if quick else (0.72, 1.0))]}
    if name == "mlp":
        return {"mlp_fc1_ag": lambda_study("ag", 8192, 2048, 4096, 8, "double", low, True),
                "mlp_fc2_rs": lambda_study("rs", 8192, 4096, 2048, 8, "single", low, True)}
    if name == "high":
        if not high:
            return {}
        return {"high_lambda_ag": lambda_study("ag", 8192, 16384, 4096, 8, "double", high, True),
                "high_lambda_rs": lambda_study("rs", 8192, 4096, 16384, 8, "single", high, True)}
    if name == "subchunk":
        return {"subchunk_flags": subchunk_study(True)}
    if name == "numa":
        return {"numa_single_vs_alltoall": numa_study(True)}
    if name.startswith("gpt3_"):
        pat = name[len("gpt3_"):]
        return {} if quick else {f"gpt3_4to1_{pat}": gpt3_study((pat,), True, cal)}
    raise ValueError(name)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=None)
    ap.add_argument("--quick", action="store_true")
    ap.add_argument("--only", choices=STUDIES, default=None,
                    help="run one study in this process (the default runs each in a child process, "
                         "so that one study's allocations do not shape the next one's memory)")
    args = ap.parse_args()
    if args.only is None:
        import subprocess
        import sys
        import tempfile
        result = {}
        for name in STUDIES:
            with tempfile.NamedTemporaryFile(suffix=".json") as tf:
                cmd = [sys.executable, "-u", "-m", "paper_2609_10549_amd.sweep", "--only", name, "--out", tf.name]
                if args.quick:
                    cmd.append("--quick")
                rc = subprocess.call(cmd)
                if rc != 0:
                    raise SystemExit(f"study {name} failed with status {rc}")
                with open(tf.name) as f:
                    result.update(json.load(f))
        if args.out:
            with open(args.out, "w") as f:
                json.dump(result, f, indent=1)
        print("sweep done", flush=True)
        return
    torch.cuda.set_device(0)
    cal = CAL.load()
    if cal is None:
        raise SystemExit("no stored calibration (run python -m paper_2609_10549_amd.calibrate first)")
    result = {"device": torch.cuda.get_device_name(0)}
    result.update(run_study(args.only, args.quick, cal))
    if args.out:
        with open(args.out, "w") as f:
            json.dump(result, f, indent=1)


if __name__ == "__main__":
    main()
