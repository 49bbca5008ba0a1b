"""Summarise rocprofv3 CSV output into the text kept under profiles/.

    python -m paper_2609_10549_amd.profile_summary trace <kernel_trace.csv> <last_n> <out.md> <command...>
    python -m paper_2609_10549_amd.profile_summary traffic [--last=N] <fetch_dir> <write_dir> <copy_fetch_dir> \
        <copy_write_dir> <kernel substring> <out.json> [command that made each dir ...]
    python -m paper_2609_10549_amd.profile_summary mfma <counter_dir> <copy_trace_dir> <last_n> <out.md> \
        "<kernel>:<bytes>;..." <command...>
    python -m paper_2609_10549_amd.profile_summary counters <out.md> <kernel substring> <title> \
        <counter_dir>... -- <command of each dir>...

`trace` averages the last `last_n` dispatches of every kernel (the timed
steps of `bench.py --profile-only`). `traffic` converts the FETCH_SIZE and
WRITE_SIZE counters (KiB per dispatch) of one kernel into bytes per launch,
each scaled by what the same counter reads for a plain 256 MiB copy kernel,
and records a hash of the kernel source the counters were taken with. `mfma`
reports MfmaUtil (matrix-core busy cycles over active cycles of every SIMD)
and the bf16 MFMA work of every GEMM kernel, averaged over its last `last_n`
dispatches, with the shader clock, and the SDMA side from a memory-copy
trace: device-to-device copies attributed to the operator whose GEMM
dispatch window they start in, the bytes of each operator given by its
kernel name. `counters` averages
every counter of the given runs over the dispatches of one kernel and
derives utilisations per cycle of the kernel (GRBM_GUI_ACTIVE): LDS active
(SQ_LDS_IDX_ACTIVE per CU), LDS bank-conflict stalls, MFMA busy
(SQ_VALU_MFMA_BUSY_CYCLES per SIMD), the texture address and data units'
busy cycles (TA_TA_BUSY, TD_TD_BUSY per CU) and the waves' LDS issue wait."""
from __future__ import annotations

import csv
import glob
import hashlib
import json
import os
import sys
from collections import defaultdict

HERE = os.path.dirname(os.path.abspath(__file__))
KERNEL_SRC = os.path.join(HERE, "csrc", "kernels.hip")
COPY_BYTES = 256 << 20


def kernel_source_hash() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def trace(path, last_n, out, command):
    rows = list(csv.DictReader(open(path)))
    by = defaultdict(list)
    for r in rows:
        by[r["Kernel_Name"]].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    lines = [f"# Kernel trace, timed steps of bench.py", "", f"Command: `{command}`", "",
             f"Last {last_n} dispatches of each kernel (microseconds):", "",
             "| kernel | dispatches | avg us | min us | max us |", "|---|---|---|---|---|"]
    for name, v in sorted(by.items(), key=lambda kv: -sum(kv[1][-last_n:])):
        w = v[-last_n:]
        short = name.split("(")[0].replace("void ", "")
        lines.append(f"| `{short}` | {len(w)} | {sum(w)/len(w):.1f} | {min(w):.1f} | {max(w):.1f} |")
    lines += ["", f"Kernel source hash: {kernel_source_hash()}"]
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")


def _counter(d, name, kernel_sub):
    vals = defaultdict(float)
    for path in glob.glob(os.path.join(d, "*counter_collection.csv")):
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == name and kernel_sub in r["Kernel_Name"]:
                vals[r["Dispatch_Id"]] += float(r["Counter_Value"])
    return [vals[k] for k in sorted(vals, key=int)]


def traffic(fetch_dir, write_dir, cfetch_dir, cwrite_dir, kernel_sub, out, *commands, last_n=0):
    """HBM bytes per launch of kernel_sub (its last `last_n` dispatches if
    positive: the timed steps)."""
    fk = _counter(fetch_dir, "FETCH_SIZE", kernel_sub)
    wk = _counter(write_dir, "WRITE_SIZE", kernel_sub)
    if last_n > 0:
        fk, wk = fk[-last_n:], wk[-last_n:]
    cf = _counter(cfetch_dir, "FETCH_SIZE", "copy")
    cw = _counter(cwrite_dir, "WRITE_SIZE", "copy")
    # the copy reads and writes COPY_BYTES per dispatch
    f_scale = COPY_BYTES / (sum(cf) / len(cf) * 1024.0)
    w_scale = COPY_BYTES / (sum(cw) / len(cw) * 1024.0)
    fetch = sum(fk) / len(fk) * 1024.0 * f_scale
    write = sum(wk) / len(wk) * 1024.0 * w_scale
    rec = {"kernel": kernel_sub, "fetch_bytes_per_launch": fetch, "write_bytes_per_launch": write,
           "traffic_bytes_per_launch": fetch + write, "fetch_scale": f_scale, "write_scale": w_scale,
           "dispatches": [len(fk), len(wk)], "kernel_source_hash": kernel_source_hash(),
           "commands": list(commands)}
    with open(out, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))




def mfma(counter_dir, copy_dir, last_n, out, op_bytes, command):
    """MfmaUtil of the GEMM kernels (last `last_n` dispatches each) and the
    SDMA copies of the last `last_n` operators. `copy_dir` holds a memory-copy
    trace and a kernel trace of the same run; every copy is attributed to the
    operator whose GEMM dispatch window it starts in (from that dispatch's
    start to the next GEMM dispatch's start: the copy side starts after the
    kernel's first workgroup, and stream order puts the next operator's
    kernel after this one's copies). `op_bytes` maps a GEMM kernel name to
    the bytes its operator moves, as name:bytes pairs separated by ";"."""
    sizes = dict(x.rsplit(":", 1) for x in op_bytes.split(";"))
    sizes = {k: int(v) for k, v in sizes.items()}
    by = defaultdict(lambda: defaultdict(list))
    for path in glob.glob(os.path.join(counter_dir, "*counter_collection.csv")):
        for r in csv.DictReader(open(path)):
            dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            by[r["Kernel_Name"].split("(")[0].replace("void ", "")][r["Counter_Name"]].append(
                (int(r["Dispatch_Id"]), float(r["Counter_Value"]), dur))
    lines = ["# Matrix-core utilisation and SDMA copies, timed steps of bench.py --profile-only", "",
             f"Command: `{command}`", "",
             f"GEMM kernels, last {last_n} dispatches each. MfmaUtil = SQ_VALU_MFMA_BUSY_CYCLES summed over SIMDs / "
             "(GRBM_GUI_ACTIVE x SIMDs); the shader clock is SQ_BUSY_CYCLES per shader engine over the dispatch "
             "duration:", "",
             "| kernel | dispatches | avg us | MfmaUtil % | shader clock GHz | bf16 MFMA GFLOP per dispatch |",
             "|---|---|---|---|---|---|"]
    for name, d in sorted(by.items()):
        if "gemm_kernel" not in name:
            continue
        util = sorted(d["MfmaUtil"])[-last_n:]
        mops = sorted(d["SQ_INSTS_VALU_MFMA_MOPS_BF16"])[-last_n:]
        busy = sorted(d.get("SQ_BUSY_CYCLES", []))[-last_n:]
        avg_us = sum(x[2] for x in util) / len(util)
        clk = (sum(x[1] for x in busy) / len(busy) / SE_NUM / (avg_us * 1e3)) if busy else float("nan")
        lines.append(f"| `{name}` | {len(util)} | {avg_us:.1f} | {sum(x[1] for x in util) / len(util):.1f} | "
                     f"{clk:.2f} | {sum(x[1] for x in mops) / len(mops) * 512 / 1e9:.1f} |")
    copies = []
    for path in glob.glob(os.path.join(copy_dir, "*memory_copy_trace.csv")):
        for r in csv.DictReader(open(path)):
            if r["Direction"].endswith("DEVICE_TO_DEVICE"):
                copies.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    copies.sort()
    gemms = []
    for path in glob.glob(os.path.join(copy_dir, "*kernel_trace.csv")):
        for r in csv.DictReader(open(path)):
            if "gemm_kernel" in r["Kernel_Name"]:
                gemms.append((int(r["Start_Timestamp"]), r["Kernel_Name"].split("(")[0].replace("void ", "")))
    gemms.sort()
    ops = []
    for i, (t0, name) in enumerate(gemms):
        t1 = gemms[i + 1][0] if i + 1 < len(gemms) else float("inf")
        cs = [c for c in copies if t0 <= c[0] < t1]
        if cs and name in sizes:
            ops.append((name, cs))
    tail = ops[-last_n:]
    lines += ["", f"SDMA device-to-device copies of the last {len(tail)} operators (each attributed to its GEMM "
              "dispatch window); per-copy durations are the engines' own, the span runs from the operator's "
              "first copy start to its last copy end:", "",
              "| operator kernel | MiB moved | copies | copy p10 / p50 / p90 us | span us | aggregate GB/s |",
              "|---|---|---|---|---|---|"]
    for name, cs in tail:
        dur = sorted((e - b) / 1e3 for b, e in cs)
        pct = lambda q: dur[min(len(dur) - 1, int(q * len(dur)))]  # noqa: E731
        span = (max(e for _, e in cs) - min(b for b, _ in cs)) / 1e3
        v = sizes[name]
        lines.append(f"| `{name}` | {v / 2**20:.0f} | {len(cs)} | {pct(0.1):.1f} / {pct(0.5):.1f} / {pct(0.9):.1f} | "
                     f"{span:.1f} | {v / span / 1e3:.1f} |")
    lines += ["", "The memory-copy tracer intercepts every copy call on the host, which stretches a span against "
              "an untraced run (the benchmark's own transfer-alone times are the reference).", "",
              f"Kernel source hash: {kernel_source_hash()}"]
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")


CU_NUM = 256
SIMD_NUM = 4 * CU_NUM
XCC_NUM = 8
SE_NUM = 32


def _dispatch_means(dirs, kernel_sub):
    """{counter: mean per dispatch} over every run directory, for the
    dispatches whose kernel name contains kernel_sub; `duration_us` is the
    mean dispatch duration of the first directory (each run perturbs it)."""
    acc = defaultdict(lambda: defaultdict(float))
    dur = {}
    for i, d in enumerate(dirs):
        for path in glob.glob(os.path.join(d, "*counter_collection.csv")):
            for r in csv.DictReader(open(path)):
                if kernel_sub in r["Kernel_Name"]:
                    acc[r["Counter_Name"]][(d, r["Dispatch_Id"])] += float(r["Counter_Value"])
                    if i == 0 and "Start_Timestamp" in r:
                        dur[r["Dispatch_Id"]] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    out = {k: sum(v.values()) / len(v) for k, v in acc.items() if v}
    if dur:
        out["duration_us"] = sum(dur.values()) / len(dur)
    return out


def counters(out, kernel_sub, title, dirs, commands):
    m = _dispatch_means(dirs, kernel_sub)
    lines = [f"# {title}", "", "Commands:", ""] + [f"* `{c}`" for c in commands] + [
        "", f"Kernel: dispatches whose name contains `{kernel_sub}`; every counter averaged per dispatch.", "",
        "| counter | mean per dispatch |", "|---|---|"]
    for k in sorted(m):
        lines.append(f"| `{k}` | {m[k]:.4g} |")
    # GRBM_GUI_ACTIVE comes summed over the 8 XCDs: per-XCD kernel cycles
    # (rocprof's own MfmaUtil / LdsUtil take the per-XCD maximum)
    gui = m.get("GRBM_GUI_ACTIVE", 0.0) / XCC_NUM
    if gui:
        der = []
        if "SQ_LDS_IDX_ACTIVE" in m:
            der.append(("LDS indexed-access active (SQ_LDS_IDX_ACTIVE / (GRBM_GUI_ACTIVE x CUs))", m["SQ_LDS_IDX_ACTIVE"] / (gui * CU_NUM)))
        if "SQ_LDS_BANK_CONFLICT" in m:
            der.append(("LDS bank-conflict stall (SQ_LDS_BANK_CONFLICT / (GRBM_GUI_ACTIVE x CUs))",
                        m["SQ_LDS_BANK_CONFLICT"] / (gui * CU_NUM)))
        if "SQ_VALU_MFMA_BUSY_CYCLES" in m:
            der.append(("MFMA busy (SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE x SIMDs))",
                        m["SQ_VALU_MFMA_BUSY_CYCLES"] / (gui * SIMD_NUM)))
        if "TA_TA_BUSY_sum" in m:
            der.append(("texture address busy (TA_TA_BUSY / (GRBM_GUI_ACTIVE x CUs))", m["TA_TA_BUSY_sum"] / (gui * CU_NUM)))
        if "TD_TD_BUSY_sum" in m:
            der.append(("texture data busy (TD_TD_BUSY / (GRBM_GUI_ACTIVE x CUs))", m["TD_TD_BUSY_sum"] / (gui * CU_NUM)))
        if "SQ_BUSY_CYCLES" in m and m.get("duration_us"):
            der.append(("shader clock, GHz (SQ_BUSY_CYCLES per shader engine / kernel time)",
                        m["SQ_BUSY_CYCLES"] / SE_NUM / (m["duration_us"] * 1e3)))
        if "SQ_WAIT_INST_LDS" in m and "SQ_BUSY_CYCLES" in m:
            der.append(("wave-cycles waiting to issue LDS per busy cycle (SQ_WAIT_INST_LDS x 4 / SQ_BUSY_CYCLES)",
                        4 * m["SQ_WAIT_INST_LDS"] / m["SQ_BUSY_CYCLES"]))
        if der:
            lines += ["", "Derived, per cycle of the kernel:", "", "| quantity | value |", "|---|---|"]
            lines += [f"| {name} | {v:.3f} |" for name, v in der]
    lines += ["", f"Kernel source hash: {kernel_source_hash()}"]
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    if sys.argv[1] == "counters":
        sep = sys.argv.index("--")
        counters(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5:sep], sys.argv[sep + 1:])
    elif sys.argv[1] == "trace":
        trace(sys.argv[2], int(sys.argv[3]), sys.argv[4], " ".join(sys.argv[5:]))
    elif sys.argv[1] == "mfma":
        mfma(sys.argv[2], sys.argv[3], int(sys.argv[4]), sys.argv[5], sys.argv[6], " ".join(sys.argv[7:]))
    else:
        args = sys.argv[2:]
        last = 0
        if args and args[0].startswith("--last="):
            last = int(args[0].split("=", 1)[1])
            args = args[1:]
        traffic(*args, last_n=last)
