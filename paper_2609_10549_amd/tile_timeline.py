"""Where the time of one fused operator goes, tile by tile: the tile trace
of one call (the GPU's 100 MHz counter at each work item's ticket, gate,
main-loop end and epilogue end) beside the copy side's trace of the same
call (when each partition's data landed and its flag was published).

    python -m paper_2609_10549_amd.tile_timeline --workload gpt3_ag [--rates 398,99.5]
        [--opt NAME=VALUE ...] [--out file.md]

Workloads (seeded random bf16 operands on the GPU, rank 0):
  fc1_ag   AllGather 8192 x 2048 x 4096, double ring, links unpaced
  fc2_rs   ReduceScatter 8192 x 4096 x 2048, single ring, links unpaced
  gpt3_ag  AllGather 8192 x 6144 x 12288, double ring, directions paced 4 : 1
  gpt3_rs  ReduceScatter 8192 x 12288 x 6144, double ring, directions paced 4 : 1
(--rates: the fast and the slow direction in GB/s for the paced ones).

The two clocks are not synchronised: host times are placed on the GPU's
time axis by taking the copy side's "start seen" (the moment it saw the
kernel's first workgroup start) as the first ticket. That puts a host event
at most the start word's one-way delay (about a microsecond, measured by
flag_latency) too early.

Before the traced call, five untraced ones are timed by HIP events around
the GEMM launch and by the host clock from the call to its synchronised end
(the operator's whole cost: staging, copy-side submission, kernel, join); the
launch span below runs from the first ticket to the last epilogue end.

Reported per partition (the row range one arrival flag covers): its flag
time, its tiles' first gate pass and last epilogue end, and the mean wait,
main-loop and epilogue time of its tiles; then the whole launch's span, the
tail after the last arrival, and the work items' time split into waiting at
the gate, main loop and epilogue. AllGather tiles wait before their main
loop (for the rows they read); ReduceScatter tiles wait in the epilogue (for
the incoming partial of their rows), and for them the send start of each
partition (when the copy side saw its last tile done) is reported too.

Occupancy: the launch's workgroup slots (the most items ever in flight at
once, from ticket to epilogue end) against time, in bins: per bin the mean
number of items in flight and how many of them wait at the gate, run the
main loop or the epilogue, and the idle slot time before and after the last
arrival flag (a slot is idle between the end of one item and the next
ticket, and after its last item until the launch's end), and per XCD (the
record's XCC_ID) its items and when its last item ended."""
from __future__ import annotations

import argparse
import csv
import json
import os
import subprocess
import sys
import tempfile
import time

import numpy as np

WORKLOADS = {
    "fc1_ag": ("ag", 8192, 2048, 4096, 8, "double", None),
    "fc2_rs": ("rs", 8192, 4096, 2048, 8, "single", None),
    "gpt3_ag": ("ag", 8192, 6144, 12288, 8, "double", (398e9, 99.5e9)),
    "gpt3_rs": ("rs", 8192, 12288, 6144, 8, "double", (710e9, 177.5e9)),
}
TRACE_CAP = 16384


def child(name: str, rates, tiles_npy: str, opts=(), slice_bytes: int = 0) -> None:
    import torch

    from . import calibrate as CAL
    from . import compass as C
    pat, M, N, K, n, ring, _ = WORKLOADS[name]
    torch.cuda.set_device(0)
    for key, value in opts:
        C.compass_set_option(getattr(C, "OPT_" + key), value)
    buf = CAL.Buffers(pat, M, N, K, n, ring)
    lk = C.links(*(rates or (0.0, 0.0)), slice_bytes=slice_bytes)
    op = C.compass_ag_gemm if pat == "ag" else C.compass_gemm_rs
    # warm up for a quarter of a second: an idle GPU runs its first
    # milliseconds of GEMM work at a lower clock
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < 0.25:
        op(buf.problem, lk)
        C.compass_sync()
    # five untraced calls, timed by the host clock (call to synchronised
    # end) and by HIP events around the GEMM launch, then the traced one
    C.compass_set_option(C.OPT_KERNEL_TIMING, 1)
    C.compass_kernel_times()
    wall = []
    for _ in range(5):
        t1 = time.perf_counter()
        op(buf.problem, lk)
        C.compass_sync()
        wall.append((time.perf_counter() - t1) * 1e6)
    kern = C.compass_kernel_times()
    C.compass_set_option(C.OPT_TILE_TRACE, TRACE_CAP)
    op(buf.problem, lk)
    C.compass_sync()
    kern_traced = C.compass_kernel_times()
    C.compass_set_option(C.OPT_KERNEL_TIMING, 0)
    np.save(tiles_npy, C.compass_tile_trace(TRACE_CAP))
    C.compass_set_option(C.OPT_TILE_TRACE, 0)
    with open(tiles_npy + ".json", "w") as f:
        json.dump({"op_wall_us": float(np.median(wall)), "kernel_event_us": float(np.median(kern)),
                   "kernel_event_us_traced": float(kern_traced[-1])}, f)


def occupancy(tick, gate, loop, end, pattern: str, bin_us: float, t_split_us: float, xcc=None) -> dict:
    """Items in flight per time bin (microseconds from the first ticket) and
    the idle slot time before and after `t_split_us`; tick..end in 100 MHz
    counter ticks."""
    t0 = tick.min()
    t = lambda x: (x.astype(np.float64) - t0) / 100.0  # noqa: E731
    a, e = t(tick), t(end)
    if pattern == "ag":
        phases = [("wait", a, t(gate)), ("main", t(gate), t(loop)), ("epilogue", t(loop), e)]
    else:
        phases = [("main", a, t(loop)), ("wait", t(loop), t(gate)), ("epilogue", t(gate), e)]
    ev = np.concatenate([np.stack([a, np.ones_like(a)], 1), np.stack([e, -np.ones_like(e)], 1)])
    ev = ev[np.lexsort((ev[:, 1], ev[:, 0]))]     # ends before starts at equal times
    slots = int(np.cumsum(ev[:, 1]).max())
    span = float(e.max())

    def overlap(lo, hi, b0, b1):
        return np.clip(np.minimum(hi, b1) - np.maximum(lo, b0), 0.0, None).sum()

    bins = []
    edges = np.arange(0.0, span + bin_us, bin_us)
    for b0 in edges[:-1].tolist():
        b1 = min(b0 + bin_us, span)
        w = b1 - b0
        if w <= 0:
            continue
        row = {"from_us": round(float(b0), 1), "in_flight": round(float(overlap(a, e, b0, b1)) / w, 1)}
        for name, lo, hi in phases:
            row[name] = round(float(overlap(lo, hi, b0, b1)) / w, 1)
        bins.append(row)
    busy_before = float(overlap(a, e, 0.0, t_split_us))
    busy_after = float(overlap(a, e, t_split_us, span))
    before, after = slots * min(t_split_us, span), slots * max(span - t_split_us, 0.0)
    per_xcd = []
    if xcc is not None:
        for x in sorted(set(xcc.tolist())):
            m = xcc == x
            per_xcd.append({"xcd": int(x), "items": int(m.sum()), "last_end_us": round(float(e[m].max()), 1),
                            "busy_us": round(float((e[m] - a[m]).sum()), 1)})
    return {"slots": slots, "bin_us": bin_us, "bins": bins, "per_xcd": per_xcd,
            "busy_share": round(float((e - a).sum()) / (slots * span), 3),
            "idle_slot_us_before_last_flag": round(before - busy_before, 1),
            "idle_slot_us_after_last_flag": round(after - busy_after, 1)}


def analyse(copy_csv: str, tiles: np.ndarray, pattern: str, M: int, n: int, ring: str,
            tile_rows: int | None = None, bin_us: float = 50.0) -> dict:
    """Per-partition and whole-launch figures (microseconds from the first
    ticket) of the traced (last) call in `copy_csv` and its tile records."""
    rows_ = list(csv.DictReader(open(copy_csv)))
    epoch = max(int(r["epoch"]) for r in rows_)
    ev = [r for r in rows_ if int(r["epoch"]) == epoch]
    t0_host = min(float(r["t_s"]) for r in ev if r["event"] == "start_seen")
    host = lambda t: (float(t) - t0_host) * 1e6  # noqa: E731
    flags = {int(r["item"]): host(r["t_s"]) for r in ev if r["event"] == "flag"}
    opened = {int(r["item"]): host(r["t_s"]) for r in ev if r["event"] == "gate_open"}
    rec = tiles.astype(np.int64)
    rt, tick, gate, loop, end = rec[:, 1] >> 16, rec[:, 4], rec[:, 5], rec[:, 6], rec[:, 7]
    t0 = tick.min()
    us = lambda x: (x - t0) / 100.0  # noqa: E731
    bm = tile_rows or M // int(rt.max() + 1)
    span_rows = M // (2 * n) if ring.startswith("double") else M // n
    part = (rt * bm) // span_rows
    if pattern == "ag":
        wait, main, epi = (gate - tick) / 100.0, (loop - gate) / 100.0, (end - loop) / 100.0
    else:
        main, wait, epi = (loop - tick) / 100.0, (gate - loop) / 100.0, (end - gate) / 100.0
    per = []
    for q in sorted(set(part.tolist())):
        m = part == q
        per.append({"partition": q, "items": int(m.sum()), "flag_us": round(flags[q], 1) if q in flags else None,
                    "first_gate_us": round(float(us(gate[m].min())), 1),
                    "last_end_us": round(float(us(end[m].max())), 1),
                    "wait_us": round(float(wait[m].mean()), 1), "main_us": round(float(main[m].mean()), 1),
                    "epilogue_us": round(float(epi[m].mean()), 1)})
        if pattern == "rs":
            per[-1]["send_start_us"] = round(opened[q], 1) if q in opened else None
    span = float(us(end.max()))
    last_flag = max(flags.values()) if flags else 0.0
    tot = float((end - tick).sum()) / 100.0
    out = {"pattern": pattern, "items": int(len(rec)), "tile_rows": bm, "span_us": round(span, 1),
           "last_flag_us": round(last_flag, 1), "tail_after_last_flag_us": round(span - last_flag, 1),
           "share_wait": round(float(wait.sum()) / tot, 3), "share_main": round(float(main.sum()) / tot, 3),
           "share_epilogue": round(float(epi.sum()) / tot, 3),
           "mean_main_us": round(float(main.mean()), 1), "partitions": per,
           "occupancy": occupancy(tick, gate, loop, end, pattern, bin_us, last_flag, rec[:, 3])}
    # the tiles of the last-arriving partitions (the last ring step)
    if flags:
        last = sorted(flags, key=flags.get)[-(2 if ring.startswith("double") else 1):]
        m = np.isin(part, last)
        if m.any():
            out["last_step"] = {"partitions": last, "items": int(m.sum()),
                                "flags_us": [round(flags[q], 1) for q in last],
                                "first_gate_us": round(float(us(gate[m].min())), 1),
                                "last_gate_us": round(float(us(gate[m].max())), 1),
                                "mean_main_us": round(float(main[m].mean()), 1),
                                "max_main_us": round(float(main[m].max()), 1),
                                "mean_epilogue_us": round(float(epi[m].mean()), 1),
                                "last_end_us": round(float(us(end[m].max())), 1)}
    return out


def markdown(name: str, res: dict, command: str) -> str:
    pat, M, N, K, n, ring, _ = WORKLOADS[name]
    L = [f"# Tile timeline: {name} ({'AllGather' if pat == 'ag' else 'ReduceScatter'} "
         f"{M}x{N}x{K}, n = {n}, {ring} ring)", "",
         f"Command: `{command}`", "",
         f"Rates (fast / slow direction): {res.get('rates', 'unpaced')}. Times in µs from the launch's first "
         "ticket; host events placed by the copy side's start-seen time (≤ ~1 µs early).", "",
         f"* work items: {res['items']} ({res['tile_rows']}-row tiles), launch span {res['span_us']} µs"
         + (f" (first ticket to last epilogue end; the traced launch by HIP events "
            f"{res['times']['kernel_event_us_traced']} µs; five untraced calls, median: launch "
            f"{res['times']['kernel_event_us']} µs by HIP events, {res['times']['op_wall_us']} µs from the call to "
            f"its synchronised end)" if "times" in res else ""),
         f"* last arrival flag at {res['last_flag_us']} µs; tail after it {res['tail_after_last_flag_us']} µs",
         f"* work-item time: {100 * res['share_wait']:.1f} % waiting at the gate, {100 * res['share_main']:.1f} % "
         f"main loop, {100 * res['share_epilogue']:.1f} % epilogue (mean main loop {res['mean_main_us']} µs)"]
    if "last_step" in res:
        s = res["last_step"]
        L.append(f"* last ring step (partitions {s['partitions']}, flags at {s['flags_us']} µs): {s['items']} items, "
                 f"gates passed {s['first_gate_us']}–{s['last_gate_us']} µs, main loop mean {s['mean_main_us']} / "
                 f"max {s['max_main_us']} µs, epilogue mean {s['mean_epilogue_us']} µs, last end {s['last_end_us']} µs")
    oc = res["occupancy"]
    L.append(f"* occupancy: {oc['slots']} workgroup slots busy {100 * oc['busy_share']:.1f} % of the span; idle slot "
             f"time {oc['idle_slot_us_before_last_flag']} µs before the last flag, "
             f"{oc['idle_slot_us_after_last_flag']} µs after it (÷ {oc['slots']}: "
             f"{oc['idle_slot_us_before_last_flag'] / oc['slots']:.1f} / "
             f"{oc['idle_slot_us_after_last_flag'] / oc['slots']:.1f} µs of the whole launch)")
    if oc["per_xcd"]:
        L.append("* per XCD (items, busy µs, last end µs): " + "; ".join(
            f"{x['xcd']}: {x['items']}, {x['busy_us']:.0f}, {x['last_end_us']}" for x in oc["per_xcd"]))
    L += ["", "| partition | items | flag | first gate | last end | wait | main loop | epilogue |"
          + (" send start |" if pat == "rs" else ""),
          "|---|---|---|---|---|---|---|---|" + ("---|" if pat == "rs" else "")]
    for p in res["partitions"]:
        L.append(f"| {p['partition']} | {p['items']} | {p['flag_us']} | {p['first_gate_us']} | {p['last_end_us']} | "
                 f"{p['wait_us']} | {p['main_us']} | {p['epilogue_us']} |"
                 + (f" {p['send_start_us']} |" if pat == "rs" else ""))
    L += ["", f"Items in flight per {oc['bin_us']:g} µs bin (mean over the bin):", "",
          "| from µs | in flight | waiting | main loop | epilogue |", "|---|---|---|---|---|"]
    for b in oc["bins"]:
        L.append(f"| {b['from_us']} | {b['in_flight']} | {b['wait']} | {b['main']} | {b['epilogue']} |")
    return "\n".join(L) + "\n"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", choices=sorted(WORKLOADS), required=True)
    ap.add_argument("--rates", default=None, help="fast,slow direction rates in GB/s (paced workloads)")
    ap.add_argument("--opt", action="append", default=[],
                    help="library option NAME=VALUE (NAME as in OPT_NAME of the binding), repeatable")
    ap.add_argument("--slice-bytes", type=int, default=0, help="largest single copy (links.slice_bytes; 0: default)")
    ap.add_argument("--out", default=None, help="markdown summary file")
    ap.add_argument("--keep", default=None, help="directory to keep the raw copy-side and tile traces in")
    ap.add_argument("--child", default=None, help=argparse.SUPPRESS)
    args = ap.parse_args()
    pat, M, N, K, n, ring, rates = WORKLOADS[args.workload]
    if args.rates:
        rates = tuple(float(x) * 1e9 for x in args.rates.split(","))
    opts = [(kv.split("=")[0].upper(), int(kv.split("=")[1])) for kv in args.opt]
    if args.child:
        child(args.workload, rates, args.child, opts, args.slice_bytes)
        return
    with tempfile.TemporaryDirectory() as td:
        trace_csv = os.path.join(td, "copy.csv")
        tiles_npy = os.path.join(td, "tiles.npy")
        cmd = [sys.executable, "-u", "-m", "paper_2609_10549_amd.tile_timeline", "--workload", args.workload,
               "--child", tiles_npy]
        if args.rates:
            cmd += ["--rates", args.rates]
        for kv in args.opt:
            cmd += ["--opt", kv]
        if args.slice_bytes:
            cmd += ["--slice-bytes", str(args.slice_bytes)]
        rc = subprocess.call(cmd, env=dict(os.environ, COMPASS_TRACE=trace_csv))
        if rc != 0:
            raise SystemExit(f"child failed with status {rc}")
        res = analyse(trace_csv, np.load(tiles_npy), pat, M, n, ring)
        with open(tiles_npy + ".json") as f:
            res["times"] = {k: round(v, 1) for k, v in json.load(f).items()}
        if args.keep:
            import shutil
            os.makedirs(args.keep, exist_ok=True)
            shutil.copy(trace_csv, os.path.join(args.keep, f"{args.workload}_copy.csv"))
            shutil.copy(tiles_npy, os.path.join(args.keep, f"{args.workload}_tiles.npy"))
            shutil.copy(tiles_npy + ".json", os.path.join(args.keep, f"{args.workload}_times.json"))
    res["rates"] = "unpaced" if not rates else f"{rates[0] / 1e9:g} / {rates[1] / 1e9:g} GB/s"
    command = "python -m paper_2609_10549_amd.tile_timeline " + " ".join(
        a for a in sys.argv[1:] if not a.startswith(("--out", "--keep")) and a not in (args.out, args.keep))
    text = markdown(args.workload, res, command.strip())
    print(text, flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)


if __name__ == "__main__":
    main()
