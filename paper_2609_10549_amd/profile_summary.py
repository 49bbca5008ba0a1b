"""Summarise rocprofv3 CSV output into the text kept under profiles/.

    python -m paper_2609_10549_amd.profile_summary trace <kernel_trace.csv> <last_n> <out.md> <command...>
    python -m paper_2609_10549_amd.profile_summary traffic <fetch_dir> <write_dir> <copy_fetch_dir> \
        <copy_write_dir> <kernel substring> <out.json> [command that made each dir ...]

`trace` averages the last `last_n` dispatches of every kernel (the timed
steps of `bench.py --profile-only`). `traffic` converts the FETCH_SIZE and
WRITE_SIZE counters (KiB per dispatch) of one kernel into bytes per launch,
each scaled by what the same counter reads for a plain 256 MiB copy kernel,
and records a hash of the kernel source the counters were taken with."""
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


def traffic(fetch_dir, write_dir, cfetch_dir, cwrite_dir, kernel_sub, out, *commands):
    fk = _counter(fetch_dir, "FETCH_SIZE", kernel_sub)
    wk = _counter(write_dir, "WRITE_SIZE", kernel_sub)
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


if __name__ == "__main__":
    if sys.argv[1] == "trace":
        trace(sys.argv[2], int(sys.argv[3]), sys.argv[4], " ".join(sys.argv[5:]))
    else:
        traffic(*sys.argv[2:])
