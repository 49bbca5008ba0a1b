#!/usr/bin/env python3
"""Benchmark of the Compass hot path on one MI355X.

One step = one tensor-parallel rank's share (TP = 8) of the GPT-3 175B MLP
shapes, 8192 tokens, hidden 12288:
  AllGather + GEMM   M=8192, N=6144, K=12288 (A gathered from 8 row chunks of
                     1024 x 12288)
  GEMM + ReduceScatter  M=8192, N=12288, K=6144, every 1024-row chunk summed
                     with an fp32 incoming partial before its bf16 store
both over the paper's double ring (every chunk split in halves, one half per
ring direction), the two directions paced at a 4 : 1 fast : slow rate ratio
(NVLink-like against PCIe-like). The slow direction runs at the rate that
makes its transfer as long as the GEMM alone (lambda = 1), lowered where the
copy engines cannot carry it. For each operator compass_pick_strategy
(Algorithm 1, calibrated model) chooses TA-IntraFusion or ODP-InterDecom(d*),
and the chosen operator runs through the C ABI with the other ranks emulated
by paced SDMA copies from separate HBM buffers. Inputs are seeded synthetic
tensors already resident in HBM. The value is whole-step throughput:
2*M*N*K of both GEMMs per second.

Reported beside it (untimed): per operator the GEMM-alone, transfer-alone,
unfused and fused times with the overlap efficiency; the same workload over
the double ring split in proportion to the rates; the fc1 / fc2 MLP pair of
the smaller TP = 8 shapes (8192 x 2048 x 4096 double ring, 8192 x 4096 x
2048 single ring); the fp64 CPU oracle on a sample of the step.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5]
    (--remote host, remote buffers in pinned host memory for a PCIe-inclusive
    rate, is disabled: see the message it prints)
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6      # 256 CUs x 4096 flop/clk x 2.4 GHz, dense
RATE_RATIO = 4.0               # fast : slow ring direction
LAMBDA_TARGET = 1.0            # link rates chosen so transfer time ~ GEMM time
LINK_CAP_FRACTION = 0.95       # MLP pair: paced only below this fraction of the unpaced copy rate
RATE_SLACK = 1.05              # a paced transfer within 5 % of its link time counts as carried


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--strategy", choices=["auto", "fusion", "decomp", "sequential"], default="auto")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-mlp", action="store_true", help="skip the fc1 / fc2 MLP pair under ops")
    ap.add_argument("--profile-only", action="store_true",
                    help="run only the timed steps (for rocprofv3); print the JSON line")
    ap.add_argument("--remote", choices=["device", "host"], default="device",
                    help="where the other ranks' shards, partials and send buffers live: device (HBM, the "
                         "reported configuration) or pinned host memory (every transfer crosses PCIe; "
                         "a PCIe-inclusive rate, never the headline)")
    ap.add_argument("--rates", default=None,
                    help="slow-ring rates of the AllGather and the ReduceScatter in GB/s, comma-separated "
                         "(the fast ring runs 4x): skips the rate search, so that a profiled run uses the "
                         "rates an unprofiled one found")
    return ap.parse_args()


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def main():
    args = parse()
    if args.remote == "host":
        # the PCIe-inclusive run of this workload (every remote shard, partial
        # and send buffer in pinned host memory, four copy directions paced
        # 4 : 1) ended in a kernel-side wait bound during its warm-up; the
        # cause is not found, so the mode stays off
        print("bench.py --remote host: disabled (the pinned-host run of this workload hit a kernel-side wait "
              "bound; cause not found)", file=sys.stderr)
        sys.exit(2)
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_10549_amd import calibrate as CAL
    from paper_2609_10549_amd import compass as C
    from synth import make_config_inputs

    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    rank = 0

    def bits(x):
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(dev)

    # ---------------------------------------------------------------- inputs (config 5)
    say("bench: generating inputs")
    ag_in = make_config_inputs(5, "ag")
    rs_in = make_config_inputs(5, "rs")
    n = ag_in["n"]
    ag = AGBuffers(C, torch, bits, ag_in, rank, "double", args.remote)
    rs = RSBuffers(C, torch, bits, rs_in, rank, "double", args.remote)
    torch.cuda.synchronize()
    flops_ag = 2.0 * ag.M * ag.N * ag.K
    flops_rs = 2.0 * rs.M * rs.N * rs.K

    # ---------------------------------------------------------------- base times and link rates
    say("bench: GEMM-alone times, 4:1 link rates")
    t_gemm_ag = CAL.time_call(lambda: C.compass_gemm(ag.gathered, ag.W, ag.C), reps=7, warmup=3)
    t_gemm_rs = CAL.time_call(lambda: C.compass_gemm(rs.A, rs.W, rs.C, rs.stage), reps=7, warmup=3)
    per_link_ag = CAL.ring_bytes_per_link("ag", ag.M, ag.N, ag.K, n, "double")
    per_link_rs = CAL.ring_bytes_per_link("rs", rs.M, rs.N, rs.K, n, "double")
    fixed = [float(x) * 1e9 for x in args.rates.split(",")] if args.rates else [None, None]
    lk_ag, tx_ag, hist_ag = balanced_rates(C, CAL, per_link_ag, t_gemm_ag,
                                           lambda lk: C.compass_transfer(ag.problem, lk), fixed[0])
    lk_rs, tx_rs, hist_rs = balanced_rates(C, CAL, per_link_rs, t_gemm_rs,
                                           lambda lk: C.compass_transfer(rs.problem, lk), fixed[1])

    # ---------------------------------------------------------------- strategy (Algorithm 1)
    cal = CAL.load()
    if cal is None:
        say("bench: no stored calibration, calibrating (quick)")
        cal, _ = CAL.run(CAL.QUICK, verbose=False)

    def choose(pattern, M, N, K, ring, lk):
        w = C.compass_workload(pattern=C.PATTERNS[pattern], M=M, N=N, K=K, n=n)
        t = C.compass_topology(ring=C.RINGS[ring], fwd_Bps=lk.fwd_Bps, bwd_Bps=lk.bwd_Bps, step_latency_s=0.0)
        return C.compass_pick_strategy(w, t, cal)

    ch_ag = choose("ag", ag.M, ag.N, ag.K, "double", lk_ag)
    ch_rs = choose("rs", rs.M, rs.N, rs.K, "double", lk_rs)
    s_ag, d_ag, f_ag = op_for(C, args.strategy, ch_ag, C.compass_ag_gemm, ag.problem, lk_ag)
    s_rs, d_rs, f_rs = op_for(C, args.strategy, ch_rs, C.compass_gemm_rs, rs.problem, lk_rs)

    # ---------------------------------------------------------------- timed steps
    say(f"bench: warmup {args.warmup}, AG {s_ag} d={d_ag}, RS {s_rs} d={d_rs}")
    for _ in range(args.warmup):
        f_ag()
        f_rs()
    C.compass_sync()
    torch.cuda.synchronize()
    C.compass_set_option(C.OPT_KERNEL_TIMING, 1)   # HIP events around every GEMM launch
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    say(f"bench: timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        ev[k][0].record()
        f_ag()
        ev[k][1].record()
        f_rs()
        ev[k][2].record()
    torch.cuda.synchronize()
    C.compass_sync()
    wall = time.perf_counter() - t0
    kt = C.compass_kernel_times(4 * args.steps * 32)
    C.compass_set_option(C.OPT_KERNEL_TIMING, 0)
    op_ag = [ev[k][0].elapsed_time(ev[k][1]) * 1e-3 for k in range(args.steps)]
    op_rs = [ev[k][1].elapsed_time(ev[k][2]) * 1e-3 for k in range(args.steps)]
    ms_per_step = wall / args.steps * 1e3
    t_op_ag, t_op_rs = float(np.mean(op_ag)), float(np.mean(op_rs))
    value = (flops_ag + flops_rs) / (wall / args.steps) / 1e12
    say(f"bench: {value:.1f} TFLOP/s, {ms_per_step:.3f} ms per step")

    # dominant kernel: the GEMM launches with the larger total time; each
    # step launches d_ag kernels for the AllGather, then d_rs for the
    # ReduceScatter
    per = d_ag + d_rs
    done = len(kt) // per              # the runtime records at most 512 launches
    assert done >= 1, (len(kt), per)
    k_ag = [kt[i * per + j] for i in range(done) for j in range(d_ag)]
    k_rs = [kt[i * per + d_ag + j] for i in range(done) for j in range(d_rs)]
    if sum(k_ag) >= sum(k_rs):
        dom = dict(name=f"gemm_kernel, GPT-3 AllGather ({s_ag}, d={d_ag})", flops=flops_ag / d_ag,
                   t=float(np.mean(k_ag)) * 1e-6, tag="gpt3_ag", t_link=tx_ag)
    else:
        dom = dict(name=f"gemm_kernel, GPT-3 ReduceScatter ({s_rs}, d={d_rs})", flops=flops_rs / d_rs,
                   t=float(np.mean(k_rs)) * 1e-6, tag="gpt3_rs", t_link=tx_rs)
    achieved = dom["flops"] / dom["t"] / 1e12
    # context for the fraction: the matrix cores' sustained bf16 rate with no
    # memory traffic (the clock drops below its 2.4 GHz maximum under load),
    # and the transfer-alone time that bounds a fused operator at lambda < 1
    C.compass_probe_mfma(8192)
    probe_tf, probe_ghz = C.compass_probe_mfma(65536)
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": stored_traffic(dom["tag"]),
                "kernel": dom["name"], "kernel_us": round(dom["t"] * 1e6, 2),
                "kernel_us_ag": round(float(np.mean(k_ag)), 2), "kernel_us_rs": round(float(np.mean(k_rs)), 2),
                "peak_sustained_probe": round(probe_tf, 1), "sclk_GHz_probe": round(probe_ghz, 3),
                "frac_of_sustained": round(achieved / probe_tf, 4),
                "link_floor_us": round(dom["t_link"] * 1e6, 2),
                "link_floor_over_kernel": round(dom["t_link"] / dom["t"], 4)}

    rnd = lambda x, k=4: None if x is None else round(x, k)  # noqa: E731
    result = {
        "metric": "AG-GEMM/GEMM-RS TFLOP/s + overlap efficiency vs unfused GEMM+copy, 1 GPU",
        "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "gpt3_175b_tp8_double_ring_4to1 (config 5): AG-GEMM 8192x6144x12288 + "
                               "GEMM-RS 8192x12288x6144 (MxNxK), one TP=8 rank's share, double ring split in "
                               "halves, ring directions paced 4:1",
                   "tokens": 8192, "hidden": 12288, "parallelism": "tp8 (one rank emulated)",
                   "remote": "device (HBM)" if args.remote == "device" else
                             "pinned host memory (PCIe-inclusive, not the headline configuration)",
                   "links_Bps": {"ag": [rnd(lk_ag.fwd_Bps, 0), rnd(lk_ag.bwd_Bps, 0)],
                                 "rs": [rnd(lk_rs.fwd_Bps, 0), rnd(lk_rs.bwd_Bps, 0)]},
                   "strategy": {"ag": [s_ag, d_ag], "rs": [s_rs, d_rs]}},
        "roofline": roofline,
    }
    if args.profile_only:
        print(json.dumps(result))
        return

    # ---------------------------------------------------------------- overlap efficiency (untimed region)
    say("bench: unfused and fused references (halves, then split by rate)")
    ops = {}
    ops["gpt3_ag"] = overlap_op(C, CAL, "ag", ag, ag.problem, lk_ag, flops_ag, t_op_ag, s_ag, d_ag, ch_ag,
                                per_link_ag, hist_ag)
    ops["gpt3_rs"] = overlap_op(C, CAL, "rs", rs, rs.problem, lk_rs, flops_rs, t_op_rs, s_rs, d_rs, ch_rs,
                                per_link_rs, hist_rs)
    # the same workload with each chunk's rows split between the directions in
    # proportion to their rates (an extension, not the paper's design)
    ag_split = C.ag_problem(ag.shards, ag.gathered, ag.W, ag.C, rank, "double_split")
    rs_split = C.rs_problem(rs.A, rs.W, rs.partials, rs.stage, rs.C, rs.sends, rank, "double_split")
    ops["gpt3_ag_split_by_rate"] = overlap_op(C, CAL, "ag", ag, ag_split, lk_ag, flops_ag, None, "intra_fusion", 1,
                                              choose("ag", ag.M, ag.N, ag.K, "double_split", lk_ag), None, None)
    ops["gpt3_rs_split_by_rate"] = overlap_op(C, CAL, "rs", rs, rs_split, lk_rs, flops_rs, None, "intra_fusion", 1,
                                              choose("rs", rs.M, rs.N, rs.K, "double_split", lk_rs), None, None)
    result["ops"] = ops
    del ag, rs, ag_split, rs_split
    torch.cuda.empty_cache()

    if not args.no_mlp:
        say("bench: fc1 / fc2 MLP pair")
        ops.update(mlp_pair(C, CAL, torch, np, bits, make_config_inputs, args.strategy, cal, rank))

    # ---------------------------------------------------------------- CPU baseline (the oracle)
    if not args.no_cpu_baseline:
        say("bench: CPU oracle baseline")
        result["cpu_baseline"] = cpu_baseline(ag_in, rs_in)
    print(json.dumps(result))


def pinned(torch, x):
    """A copy of host array or tensor `x` in newly allocated pinned host memory."""
    t = x if isinstance(x, torch.Tensor) else torch.from_numpy(x)
    out = torch.empty(t.shape, dtype=t.dtype, pin_memory=True)
    out.copy_(t)
    return out


class AGBuffers:
    """Buffers of one AllGather+GEMM: the local shard in place in the gathered
    buffer, the other ranks' shards in separate device allocations (remote =
    "host": in pinned host memory)."""

    def __init__(self, C, torch, bits, inp, rank, ring, remote="device"):
        import numpy as np
        self.M, self.N, self.K, n = inp["M"], inp["N"], inp["K"], inp["n"]
        rows = self.M // n
        self.gathered = torch.empty((self.M, self.K), dtype=torch.int16, device="cuda")
        self.gathered[rank * rows:(rank + 1) * rows] = bits(inp["shards"][rank])

        def far(x):
            return bits(x) if remote == "device" else pinned(torch, np.ascontiguousarray(x).view(np.int16))
        self.shards = [self.gathered[rank * rows:(rank + 1) * rows] if q == rank else far(inp["shards"][q])
                       for q in range(n)]
        self.W = bits(inp["W"])
        self.C = torch.empty((self.M, self.N), dtype=torch.int16, device="cuda")
        self.problem = C.ag_problem(self.shards, self.gathered, self.W, self.C, rank, ring)


class RSBuffers:
    """Buffers of one GEMM+ReduceScatter: A, W, the output, the fp32 landing
    buffer, and the other ranks' partials and send destinations in separate
    device allocations (remote = "host": in pinned host memory; the operator
    moves the first step's partials into place itself)."""

    def __init__(self, C, torch, bits, inp, rank, ring, remote="device"):
        self.M, self.N, self.K, n = inp["M"], inp["N"], inp["K"], inp["n"]
        rows = self.M // n
        self.A = bits(inp["A"])
        self.W = bits(inp["W"])
        self.C = torch.empty((self.M, self.N), dtype=torch.int16, device="cuda")
        self.stage = torch.empty((self.M, self.N), dtype=torch.float32, device="cuda")
        if remote == "device":
            self.partials = [torch.from_numpy(p).to("cuda") for p in inp["P_in"]]
            self.sends = [None if q == rank else torch.empty((rows, self.N), dtype=torch.int16, device="cuda")
                          for q in range(n)]
        else:
            self.partials = [pinned(torch, p) for p in inp["P_in"]]
            self.sends = [None if q == rank else torch.empty((rows, self.N), dtype=torch.int16, pin_memory=True)
                          for q in range(n)]
        self.problem = C.rs_problem(self.A, self.W, self.partials, self.stage, self.C, self.sends, rank, ring)


def balanced_rates(C, CAL, per_link, t_gemm, transfer, fixed=None):
    """4 : 1 ring rates for the double ring in halves: the slow direction at
    the rate that makes its transfer (per_link bytes) as long as the GEMM
    alone, the fast one at four times that; lowered to what the copy engines
    deliver while a paced transfer takes more than 5 % over its link time
    (`fixed`: that slow rate, no search). Returns (links, transfer-alone
    time, [(slow rate, measured time), ...])."""
    bwd = fixed if fixed else per_link / (t_gemm / LAMBDA_TARGET)
    hist = []
    for _ in range(1 if fixed else 4):
        lk = C.links(RATE_RATIO * bwd, bwd)
        tx = CAL.time_call(lambda: transfer(lk), reps=3)
        hist.append((bwd, tx))
        want = per_link / bwd
        if tx <= RATE_SLACK * want:
            break
        bwd *= want / tx
    say(f"bench: 4:1 rates {lk.fwd_Bps / 1e9:.1f} / {lk.bwd_Bps / 1e9:.1f} GB/s, transfer {tx * 1e6:.0f} us "
        f"(GEMM alone {t_gemm * 1e6:.0f} us)")
    return lk, tx, hist


def op_for(C, strategy, choice, fused, prob, lk):
    if strategy == "fusion" or (strategy == "auto" and choice.strategy == C.INTRA_FUSION):
        return ("intra_fusion", 1, lambda: fused(prob, lk))
    if strategy == "sequential":
        return ("sequential", 1, lambda: C.compass_sequential(prob, lk))
    d = max(choice.d_star, 2) if strategy == "decomp" else choice.d_star
    return ("inter_decom", d, lambda: C.compass_decomp_gemm(prob, d, lk))


def overlap_op(C, CAL, pattern, buf, prob, lk, flops, t_op, strategy, d, choice, per_link, hist):
    """GEMM alone, transfer alone, unfused and fused, timed in interleaved
    rounds so that the differences the metrics take see one clock state."""
    fused = C.compass_ag_gemm if pattern == "ag" else C.compass_gemm_rs
    if pattern == "ag":
        g = lambda: C.compass_gemm(buf.gathered, buf.W, buf.C)  # noqa: E731
    else:
        g = lambda: C.compass_gemm(buf.A, buf.W, buf.C, buf.stage)  # noqa: E731
    r = CAL.time_interleaved({"g": g, "x": lambda: C.compass_transfer(prob, lk),
                              "s": lambda: C.compass_sequential(prob, lk), "f": lambda: fused(prob, lk)})
    tg, tx, ts, tf = r["g"], r["x"], r["s"], r["f"]
    ideal = ts - max(tg, tx)
    rnd = lambda x, k=4: None if x is None else round(x, k)  # noqa: E731
    out = {"strategy": strategy, "d": d, "shape_MNK": [buf.M, buf.N, buf.K],
           "t_gemm_us": rnd(tg * 1e6, 2), "gemm_tflops": rnd(flops / tg / 1e12, 1),
           "t_xfer_us": rnd(tx * 1e6, 2), "t_fused_us": rnd(tf * 1e6, 2), "fused_tflops": rnd(flops / tf / 1e12, 1),
           "t_unfused_us": rnd(ts * 1e6, 2), "lambda": rnd(tg / tx, 3),
           "overlap_efficiency": rnd((ts - tf) / ideal if ideal > 0 else None),
           "transfer_hidden": rnd((tg + tx - tf) / tx),
           "link_rate_Bps": [rnd(lk.fwd_Bps, 0), rnd(lk.bwd_Bps, 0)],
           "model": {"strategy": "intra_fusion" if choice.strategy == C.INTRA_FUSION else "inter_decom",
                     "d_star": choice.d_star, "t_fusion_us": rnd(choice.t_fusion * 1e6, 2),
                     "t_decomp_us": rnd(choice.t_decomp * 1e6, 2), "lambda": rnd(choice.lambda_, 3)}}
    if t_op is not None:
        out["t_op_us"] = rnd(t_op * 1e6, 2)
        out["tflops"] = rnd(flops / t_op / 1e12, 1)
    if per_link is not None:
        out["link_Bps_slow_ring"] = rnd(per_link / tx, 0)
        out["rate_search"] = [[rnd(b, 0), rnd(t * 1e6, 1)] for b, t in hist]
    return out


def mlp_pair(C, CAL, torch, np, bits, make_config_inputs, strategy, cal, rank):
    """The fc1 / fc2 pair of configurations 2 and 3 (8192 tokens, hidden
    4096, TP = 8): equal link rates for lambda ~ 1 where the copy engines
    carry them, else unpaced at their ceiling."""
    out = {}
    for key, idx, pattern, ring in (("fc1_ag", 2, "ag", "double"), ("fc2_rs", 3, "rs", "single")):
        inp = make_config_inputs(idx)
        n = inp["n"]
        if pattern == "ag":
            buf = AGBuffers(C, torch, bits, inp, rank, ring)
            g = lambda: C.compass_gemm(buf.gathered, buf.W, buf.C)  # noqa: E731
        else:
            buf = RSBuffers(C, torch, bits, inp, rank, ring)
            g = lambda: C.compass_gemm(buf.A, buf.W, buf.C, buf.stage)  # noqa: E731
        flops = 2.0 * buf.M * buf.N * buf.K
        tg = CAL.time_call(g, reps=10, warmup=3)
        per_link = CAL.ring_bytes_per_link(pattern, buf.M, buf.N, buf.K, n, ring)
        unpaced = C.links(0.0, 0.0)
        cap = per_link / CAL.time_call(lambda: C.compass_transfer(buf.problem, unpaced), reps=5)
        rate = per_link / (tg / LAMBDA_TARGET)
        lk = C.links(rate, rate) if rate < LINK_CAP_FRACTION * cap else unpaced
        w = C.compass_workload(pattern=C.PATTERNS[pattern], M=buf.M, N=buf.N, K=buf.K, n=n)
        tx = CAL.time_call(lambda: C.compass_transfer(buf.problem, lk), reps=5)
        eff = per_link / tx
        t = C.compass_topology(ring=C.RINGS[ring], fwd_Bps=eff, bwd_Bps=eff, step_latency_s=0.0)
        ch = C.compass_pick_strategy(w, t, cal)
        fused = C.compass_ag_gemm if pattern == "ag" else C.compass_gemm_rs
        s, d, f = op_for(C, strategy, ch, fused, buf.problem, lk)
        t_op = CAL.time_call(f, reps=10, warmup=3)
        o = overlap_op(C, CAL, pattern, buf, buf.problem, lk, flops, t_op, s, d, ch, None, None)
        o["link_Bps_per_ring"] = round(per_link / o["t_xfer_us"] * 1e6, 0)
        o["link_ceiling_Bps_per_ring"] = round(cap, 0)
        out[key] = o
        del buf
        torch.cuda.empty_cache()
    return out


def stored_traffic(tag):
    """HBM bytes per launch of the dominant kernel from the committed counter
    runs (profiles/traffic_<tag>.json), or None when absent or taken with a
    different kernel source."""
    from paper_2609_10549_amd import profile_summary as PS
    path = os.path.join(ROOT, "profiles", f"traffic_{tag}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_hash") != PS.kernel_source_hash():
        return None
    return round(rec["traffic_bytes_per_launch"], 0)


def cpu_baseline(ag_in, rs_in, rows: int = 128, rows_1t: int = 32) -> dict:
    """The fp64 oracle on a bounded sample of the same step: the first
    `rows` rows of every AllGather shard gathered and multiplied, and the same
    rows of every ReduceScatter chunk multiplied and reduced (rows / 1024 of
    the step); repeated until about 10 s of CPU work. Scaled to TFLOP/s of
    the sampled flops."""
    import numpy as np

    import oracle as O

    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        threads = max([i.get("num_threads", 1) for i in info] or [1])
        if info:
            blas = f"{info[0].get('internal_api', '?')} {info[0].get('version', '')}".strip()
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
        threadpool_limits = None
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    n = ag_in["n"]
    chunk = rs_in["M"] // n

    def sample(r):
        sh = [s[:r] for s in ag_in["shards"]]
        idx = np.concatenate([np.arange(c * chunk, c * chunk + r) for c in range(n)])
        A2, P2 = rs_in["A"][idx], [p[:r] for p in rs_in["P_in"]]
        fl = 2.0 * (n * r) * ag_in["N"] * ag_in["K"] + 2.0 * (n * r) * rs_in["N"] * rs_in["K"]

        def run():
            O.ag_gemm([O.bf16_to_f64(s) for s in sh], O.bf16_to_f64(ag_in["W"]))
            O.gemm_rs(O.bf16_to_f64(A2), O.bf16_to_f64(rs_in["W"]), [p.astype(np.float64) for p in P2], n)
        return fl, run

    flops, run = sample(rows)
    times = []
    t_all = time.perf_counter()
    while True:
        t0 = time.perf_counter()
        run()
        times.append(time.perf_counter() - t0)
        if time.perf_counter() - t_all > 10.0 or len(times) >= 50:
            break
    t = float(np.median(times))
    t1 = None
    if threadpool_limits is not None:
        fl1, run1 = sample(rows_1t)
        with threadpool_limits(limits=1, user_api="blas"):
            t0 = time.perf_counter()
            run1()
            t1 = time.perf_counter() - t0
    return {"value": round(flops / t / 1e12, 5), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{rows} rows of each of the {n} AllGather shards and ReduceScatter chunks "
                      f"({rows}/{chunk} of a config-5 step, {flops / 1e9:.0f} GFLOP), fp64 numpy, "
                      f"median of {len(times)} runs",
            "seconds": round(t, 4), "cpu_model": cpu_model, "blas": blas,
            "value_1_thread": None if t1 is None else round(fl1 / t1 / 1e12, 5),
            "sample_1_thread": f"{rows_1t} rows of each shard and chunk, one run"}


if __name__ == "__main__":
    main()
