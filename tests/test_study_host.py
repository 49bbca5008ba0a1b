"""Host-side checks of the selector study's summary arithmetic on hand-made
points (no GPU): MAE by d, the d landscape and the selector accuracy."""
import pytest

from paper_2609_10549_amd.selector_study import summarize, workloads


def _pt(t_fused, t_dec, aware, agnostic, pick, d_pick, fa=None, fg=None):
    return dict(t_fused=t_fused, t_decomp={str(k): v for k, v in t_dec.items()},
                model_aware={str(k): v for k, v in aware.items()},
                model_agnostic={str(k): v for k, v in agnostic.items()},
                model_fusion_aware=t_fused if fa is None else fa,
                model_fusion_agnostic=t_fused if fg is None else fg,
                pick_strategy=pick, pick_d=d_pick)


def test_summary_by_hand():
    p1 = _pt(10.0, {1: 20.0, 2: 12.0, 4: 11.0}, {2: 13.0, 4: 11.0}, {2: 9.0, 4: 7.0},
             "intra_fusion", 4, fa=11.0, fg=8.0)
    p2 = _pt(30.0, {1: 40.0, 2: 25.0, 4: 27.0}, {2: 24.0, 4: 27.0}, {2: 20.0, 4: 19.0},
             "intra_fusion", 2, fa=30.0, fg=26.0)
    s = summarize([p1, p2])
    m = s["decomp_mae"]
    assert m["2"]["aware_us"] == pytest.approx(1e6 * (1.0 + 1.0) / 2)
    assert m["2"]["agnostic_us"] == pytest.approx(1e6 * (3.0 + 5.0) / 2)
    assert m["4"]["aware_us"] == pytest.approx(0.0)
    assert m["4"]["agnostic_us"] == pytest.approx(1e6 * (4.0 + 8.0) / 2)
    assert m["overall"]["aware_us"] == pytest.approx(1e6 * 2.0 / 4)
    assert s["fusion_mae"]["aware_us"] == pytest.approx(1e6 * 0.5)
    assert s["fusion_mae"]["agnostic_us"] == pytest.approx(1e6 * (2.0 + 4.0) / 2)
    land = s["landscape"]
    # p1: best d = 4, penalty of d=2 is 12/11-1; p2: best d = 2, penalty 27/25-1
    assert land["mean_penalty_suboptimal"] == pytest.approx((12 / 11 - 1 + 27 / 25 - 1) / 2)
    assert land["d4_best_fraction"] == pytest.approx(0.5)
    assert land["dstar_best_fraction"] == pytest.approx(1.0)
    assert land["best_d_histogram"] == {"2": 1, "4": 1}
    sel = s["selector"]
    # p1: fused 10 < 11 -> fusion best, picked fusion; p2: 30 > 25 -> decomp best, picked fusion
    assert sel["accuracy"] == pytest.approx(0.5)
    assert sel["fusion_best_fraction"] == pytest.approx(0.5)
    assert sel["max_slowdown_of_pick"] == pytest.approx(30 / 25 - 1)


def test_study_grid_is_the_table4_subset():
    ws = workloads()
    assert len(ws) == 2 * 2 * 3 * 3
    ag = [w for w in ws if w["pattern"] == "ag"]
    rs = [w for w in ws if w["pattern"] == "rs"]
    # AllGather: column-parallel weight, N/TP columns; ReduceScatter: row-parallel input, N/TP deep
    assert {(w["N"] * w["n"], w["K"]) for w in ag} == {(8192, 4096), (16384, 4096), (16384, 8192)}
    assert {(w["K"] * w["n"], w["N"]) for w in rs} == {(8192, 4096), (16384, 4096), (16384, 8192)}
    for w in ws:
        assert w["M"] % (2 * w["n"]) == 0
