"""Model and selector study over a Table IV subset on one GPU (the methodology
of Section IV's Table II and fusion-model check, Fig. 4's d landscape and
Section V-C's selector accuracy, on the emulated links):

    python -m paper_2609_10549_amd.selector_study [--out study.json] [--quick]

Workloads: one rank's share of every combination of pattern (AllGather+GEMM,
GEMM+ReduceScatter), TP in {4, 8}, sequence length M in {4096, 8192, 16384}
and (intermediate N, hidden K) in {(8192, 4096), (16384, 4096), (16384, 8192)}
(Table IV values), double ring. The rank's GEMM is M x N/TP x K for the
AllGather (column-parallel weight) and M x K x N/TP for the ReduceScatter
(row-parallel input, output M x K). None of these shapes is a calibration
shape. Every workload runs at two link settings: paced at 100 GB/s per ring
direction, and unpaced (the copy engines' ceiling).

Per point, in interleaved rounds: GEMM alone, transfer alone, the fused
operator (IntraFusion), InterDecom at d = 1 (sequential), 2, 4, 8, 16.
Reported:
  * Eq. 2 with the calibrated eta(d) (overhead-aware) and with eta = 1
    (overhead-agnostic) against the measured T(d): MAE by d;
  * Eq. 7-8 with the calibrated (alpha_f, beta_f) and with no overhead term
    against the measured fused time: MAE;
  * the d landscape: penalty of each d against the best d, how often d = 4
    and the model's d* are best, the regret of d*;
  * compass_pick_strategy (stored calibration, the measured link rate as
    the topology) against the measured best strategy: accuracy and the
    slowdown of its picks;
  * the same MAE, d* regret and selector accuracy with the model refitted on
    half of the study's workloads and evaluated on the other half (two-fold
    cross-validation), and refitted on all workloads but the evaluated one
    (leave one workload out), i.e. calibrated for this workload range.
The model inputs are the measured GEMM-alone and transfer-alone times, so the
errors are those of the overhead models. Timing only (seeded random bf16).
"""
from __future__ import annotations

import argparse
import itertools
import json
import subprocess
import sys
import tempfile

import numpy as np
import torch

from . import calibrate as CAL
from . import compass as C

DS = (1, 2, 4, 8, 16)
RATES = (100e9, 0.0)   # per ring direction; 0 = unpaced


def workloads(quick: bool = False):
    out = []
    pats = ("ag", "rs")
    tps = (8,) if quick else (4, 8)
    ms = (8192,) if quick else (4096, 8192, 16384)
    nks = ((16384, 4096),) if quick else ((8192, 4096), (16384, 4096), (16384, 8192))
    for pat, tp, M, (Nint, H) in itertools.product(pats, tps, ms, nks):
        if pat == "ag":
            out.append(dict(pattern=pat, M=M, N=Nint // tp, K=H, n=tp))
        else:
            out.append(dict(pattern=pat, M=M, N=H, K=Nint // tp, n=tp))
    return out


def measure(w: dict, cal) -> list:
    pat, M, N, K, n = w["pattern"], w["M"], w["N"], w["K"], w["n"]
    ring = "double"
    buf = CAL.Buffers(pat, M, N, K, n, ring)
    fused = C.compass_ag_gemm if pat == "ag" else C.compass_gemm_rs
    per_link = CAL.ring_bytes_per_link(pat, M, N, K, n, ring)
    cw = C.compass_workload(pattern=C.PATTERNS[pat], M=M, N=N, K=K, n=n)
    points = []
    for rate in RATES:
        lk = C.links(rate, rate)
        fns = {"g": lambda: C.compass_gemm(buf.A, buf.W, buf.C, buf.P),
               "x": lambda: C.compass_transfer(buf.problem, lk),
               "f": lambda: fused(buf.problem, lk)}
        for d in DS:
            if (M // n) % (2 * d) == 0:
                fns[d] = (lambda d=d: C.compass_decomp_gemm(buf.problem, d, lk))
        t = CAL.time_interleaved(fns, reps=5)
        tg, tx, tf = t["g"], t["x"], t["f"]
        td = {d: t[d] for d in DS if d in t}
        eff = per_link / tx                      # achieved rate per ring
        topo = C.compass_topology(ring=C.RINGS[ring], fwd_Bps=eff, bwd_Bps=eff, step_latency_s=0.0)
        ch = C.compass_pick_strategy(cw, topo, cal)
        step = tx / (n - 1)
        pt = dict(w=w, rate_Bps=rate, eff_Bps=eff, t_gemm=tg, t_xfer=tx, t_fused=tf,
                  t_decomp={str(d): v for d, v in td.items()},
                  model_aware={str(d): C.compass_model_t_decomp(tg, tx, d, cal.alpha_decomp, cal.beta_decomp)
                               for d in td},
                  model_agnostic={str(d): C.compass_model_t_decomp(tg, tx, d, 1.0, 0.0) for d in td},
                  model_fusion_aware=C.compass_model_t_fusion(cw, tg, step, cal.alpha_fusion, cal.beta_fusion),
                  model_fusion_agnostic=C.compass_model_t_fusion(cw, tg, step, 0.0, 0.0),
                  pick_strategy="intra_fusion" if ch.strategy == C.INTRA_FUSION else "inter_decom",
                  pick_d=ch.d_star, lam=tg / tx)
        points.append(pt)
        print(json.dumps({"M": M, "N": N, "K": K, "n": n, "pat": pat, "rate": rate, "lam": round(tg / tx, 3),
                          "fused_us": round(tf * 1e6, 1),
                          "decomp_us": {d: round(v * 1e6, 1) for d, v in td.items()},
                          "pick": [pt["pick_strategy"], ch.d_star]}), flush=True)
    del buf
    torch.cuda.empty_cache()
    return points


def summarize(points: list) -> dict:
    mae = {}
    for d in DS[1:]:
        aw = [abs(p["model_aware"][str(d)] - p["t_decomp"][str(d)]) for p in points if str(d) in p["t_decomp"]]
        ag = [abs(p["model_agnostic"][str(d)] - p["t_decomp"][str(d)]) for p in points if str(d) in p["t_decomp"]]
        tm = [p["t_decomp"][str(d)] for p in points if str(d) in p["t_decomp"]]
        if not tm:
            continue
        mae[str(d)] = dict(aware_us=1e6 * float(np.mean(aw)), agnostic_us=1e6 * float(np.mean(ag)),
                           mean_time_us=1e6 * float(np.mean(tm)), cases=len(aw))
    all_aw = [abs(p["model_aware"][k] - p["t_decomp"][k]) for p in points for k in p["t_decomp"] if k != "1"]
    all_ag = [abs(p["model_agnostic"][k] - p["t_decomp"][k]) for p in points for k in p["t_decomp"] if k != "1"]
    mae["overall"] = dict(aware_us=1e6 * float(np.mean(all_aw)), agnostic_us=1e6 * float(np.mean(all_ag)))
    fus = dict(aware_us=1e6 * float(np.mean([abs(p["model_fusion_aware"] - p["t_fused"]) for p in points])),
               agnostic_us=1e6 * float(np.mean([abs(p["model_fusion_agnostic"] - p["t_fused"]) for p in points])),
               mean_time_us=1e6 * float(np.mean([p["t_fused"] for p in points])))
    # d landscape over d >= 2 (InterDecom proper)
    pen, d4_best, dstar_best, regret, dbest = [], 0, 0, [], {}
    for p in points:
        td = {int(k): v for k, v in p["t_decomp"].items() if k != "1"}
        best_d = min(td, key=td.get)
        dbest[best_d] = dbest.get(best_d, 0) + 1
        pen += [v / td[best_d] - 1.0 for d, v in td.items() if d != best_d]
        d4_best += best_d == 4
        ds = max(2, p["pick_d"])
        if ds in td:
            dstar_best += ds == best_d
            regret.append(td[ds] / td[best_d] - 1.0)
    land = dict(mean_penalty_suboptimal=float(np.mean(pen)), max_penalty=float(np.max(pen)),
                d4_best_fraction=d4_best / len(points), dstar_best_fraction=dstar_best / len(points),
                mean_regret_dstar=float(np.mean(regret)), best_d_histogram={str(k): v for k, v in sorted(dbest.items())})
    # strategy selection: fused vs the best InterDecom (d >= 2)
    correct, slow, fusion_wins = 0, [], 0
    for p in points:
        td = {int(k): v for k, v in p["t_decomp"].items() if k != "1"}
        t_dec = min(td.values())
        best = "intra_fusion" if p["t_fused"] < t_dec else "inter_decom"
        fusion_wins += best == "intra_fusion"
        correct += p["pick_strategy"] == best
        d_pick = max(2, p["pick_d"])
        t_pick = p["t_fused"] if p["pick_strategy"] == "intra_fusion" else td.get(d_pick, t_dec)
        slow.append(t_pick / min(p["t_fused"], t_dec) - 1.0)
    sel = dict(accuracy=correct / len(points), fusion_best_fraction=fusion_wins / len(points),
               mean_slowdown_of_pick=float(np.mean(slow)), max_slowdown_of_pick=float(np.max(slow)),
               cases=len(points))
    return dict(decomp_mae=mae, fusion_mae=fus, landscape=land, selector=sel)


def _samples(points):
    """compass_calibrate samples from measured points (GEMM alone, InterDecom
    at d >= 2, fused), with the measured GEMM-alone / transfer-alone times."""
    out = []
    for p in points:
        w = C.compass_workload(pattern=C.PATTERNS[p["w"]["pattern"]], M=p["w"]["M"], N=p["w"]["N"],
                               K=p["w"]["K"], n=p["w"]["n"])
        out.append(C.compass_sample(kind=0, w=w, d=1, t_meas=p["t_gemm"], t_comp=p["t_gemm"], t_comm=0.0))
        out.append(C.compass_sample(kind=2, w=w, d=1, t_meas=p["t_fused"], t_comp=p["t_gemm"],
                                    t_comm=p["t_xfer"]))
        for k, v in p["t_decomp"].items():
            if k != "1":
                out.append(C.compass_sample(kind=1, w=w, d=int(k), t_meas=v, t_comp=p["t_gemm"],
                                            t_comm=p["t_xfer"]))
    return out


def cross_validated(points, folds: int = 2) -> dict:
    """Refit the model on the other folds' workloads (k-fold over workloads)
    and evaluate each fold's points with its held-out fit: InterDecom and
    fusion MAE, the d* regret and the selector's accuracy."""
    keys = sorted({json.dumps(p["w"], sort_keys=True) for p in points})
    fold_of = {k: i % folds for i, k in enumerate(keys)}
    aw, fu, correct, regret, fits = [], [], 0, [], []
    aw_by_d = {}
    for f in range(folds):
        train = [p for p in points if fold_of[json.dumps(p["w"], sort_keys=True)] != f]
        test = [p for p in points if fold_of[json.dumps(p["w"], sort_keys=True)] == f]
        cal = C.compass_calibrate(_samples(train), C.compass_calib(d_max=16))
        fits.append(dict(alpha_decomp=cal.alpha_decomp, beta_decomp=cal.beta_decomp,
                         alpha_fusion=cal.alpha_fusion, beta_fusion=cal.beta_fusion))
        for p in test:
            w = C.compass_workload(pattern=C.PATTERNS[p["w"]["pattern"]], M=p["w"]["M"], N=p["w"]["N"],
                                   K=p["w"]["K"], n=p["w"]["n"])
            for k, v in p["t_decomp"].items():
                if k != "1":
                    e = abs(C.compass_model_t_decomp(p["t_gemm"], p["t_xfer"], int(k), cal.alpha_decomp,
                                                     cal.beta_decomp) - v)
                    aw.append(e)
                    aw_by_d.setdefault(k, []).append(e)
            step = p["t_xfer"] / (p["w"]["n"] - 1)
            fu.append(abs(C.compass_model_t_fusion(w, p["t_gemm"], step, cal.alpha_fusion, cal.beta_fusion)
                          - p["t_fused"]))
            topo = C.compass_topology(ring=C.RING_DOUBLE, fwd_Bps=p["eff_Bps"], bwd_Bps=p["eff_Bps"],
                                      step_latency_s=0.0)
            ch = C.compass_pick_strategy(w, topo, cal)
            td = {int(k): v for k, v in p["t_decomp"].items() if k != "1"}
            best = "intra_fusion" if p["t_fused"] < min(td.values()) else "inter_decom"
            pick = "intra_fusion" if ch.strategy == C.INTRA_FUSION else "inter_decom"
            correct += pick == best
            ds = max(2, ch.d_star)
            if ds in td:
                regret.append(td[ds] / min(td.values()) - 1.0)
    # For comparison only (not the paper's model): Eq. 2 with eta = 1 plus a
    # fixed cost c0 per extra sub-operator, c0 fitted by least squares on the
    # other folds
    fc = []
    for f in range(folds):
        def rows(sel):
            out = []
            for p in points:
                if (fold_of[json.dumps(p["w"], sort_keys=True)] == f) != sel:
                    continue
                for k, v in p["t_decomp"].items():
                    d = int(k)
                    if d >= 2:
                        base = C.compass_model_t_decomp(p["t_gemm"], p["t_xfer"], d, 1.0, 0.0)
                        out.append((d - 1, base, v))
            return np.array(out)
        tr, te = rows(False), rows(True)
        c0 = float(tr[:, 0] @ (tr[:, 2] - tr[:, 1]) / (tr[:, 0] @ tr[:, 0]))
        fc += list(np.abs(te[:, 1] + c0 * te[:, 0] - te[:, 2]))
        fits[f]["fixed_cost_per_subop_us"] = 1e6 * c0
    return dict(folds=folds, fits=fits, decomp_mae_aware_us=1e6 * float(np.mean(aw)),
                decomp_mae_aware_by_d_us={k: 1e6 * float(np.mean(v)) for k, v in sorted(aw_by_d.items(), key=lambda kv: int(kv[0]))},
                decomp_mae_fixed_cost_us=1e6 * float(np.mean(fc)),
                fusion_mae_aware_us=1e6 * float(np.mean(fu)), selector_accuracy=correct / len(points),
                mean_regret_dstar=float(np.mean(regret)))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=None)
    ap.add_argument("--quick", action="store_true")
    ap.add_argument("--only", type=int, default=None, help="measure workload #i in this process")
    args = ap.parse_args()
    ws = workloads(args.quick)
    if args.only is not None:
        torch.cuda.set_device(0)
        cal = CAL.load()
        if cal is None:
            raise SystemExit("no stored calibration (run python -m paper_2609_10549_amd.calibrate first)")
        pts = measure(ws[args.only], cal)
        with open(args.out, "w") as f:
            json.dump(pts, f)
        return
    points = []
    for i in range(len(ws)):
        # each workload in a child process: a fresh device heap (copy speed)
        with tempfile.NamedTemporaryFile(suffix=".json") as tf:
            cmd = [sys.executable, "-u", "-m", "paper_2609_10549_amd.selector_study", "--only", str(i),
                   "--out", tf.name] + (["--quick"] if args.quick else [])
            rc = subprocess.call(cmd)
            if rc != 0:
                raise SystemExit(f"workload {i} failed with status {rc}")
            with open(tf.name) as f:
                points += json.load(f)
    summary = summarize(points)
    summary["cross_validated"] = cross_validated(points)
    n_work = len({json.dumps(p["w"], sort_keys=True) for p in points})
    summary["leave_one_out"] = cross_validated(points, folds=n_work)
    print(json.dumps(summary, indent=1), flush=True)
    if args.out:
        with open(args.out, "w") as f:
            json.dump(dict(summary=summary, points=points), f, indent=1)


if __name__ == "__main__":
    main()
