"""Pins of the performance models (Eq. 2-8, Algorithm 1) and the
calibration fits: printed closed forms and Table I, brute-force minima,
special cases named by the paper, hand-computed selector cases, and recovery
of planted regression parameters."""
import math
import os
import random

import numpy as np
import pytest

import oracle as O


def _rows(path):
    with open(path) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


def test_ring_bandwidth_closed_forms(golden_dir):
    for ring, n, num, den in _rows(os.path.join(golden_dir, "ring_bandwidth.txt")):
        B = 12.5e9
        got = O.effective_bandwidth(ring, int(n), B)
        assert got == pytest.approx(B * int(num) / int(den), rel=1e-12)


def test_table1_sequential_is_d1(golden_dir):
    for tp, pat, comp, comm, total in _rows(os.path.join(golden_dir, "table1_sequential.txt")):
        Tc, Tm, Tt = float(comp), float(comm), float(total)
        for alpha, beta in [(1.0, 0.0), (0.7, 0.05), (1.3, 0.2)]:
            t1 = O.t_decomp(Tc, Tm, 1, alpha, beta)
            assert t1 == pytest.approx(Tc + Tm, abs=1e-12)
            assert abs(t1 - Tt) <= 0.011


def test_table4_counts(golden_dir):
    want = {k: int(v) for k, v in _rows(os.path.join(golden_dir, "table4_counts.txt"))}
    assert len(O.table4_workloads()) == want["all"]
    assert len(O.table4_workloads(pattern="ag")) == want["ag"]
    assert len(O.table4_workloads(pattern="ag", world=8)) == want["ag_tp8"]


def test_eq2_by_hand():
    # Tc=8, Tm=4, d=4, eta = 0.9 + 0.05*4 = 1.1: 3 * 2 * 1.1 + 2 + 1 = 9.6
    assert O.t_decomp(8.0, 4.0, 4, 0.9, 0.05) == pytest.approx(9.6, rel=1e-15)
    # comm-bound: Tc=2, Tm=6, d=2, eta=1: 1*3*1 + 1 + 3 = 7
    assert O.t_decomp(2.0, 6.0, 2, 1.0, 0.0) == pytest.approx(7.0, rel=1e-15)


def test_overhead_agnostic_special_case():
    # eta == 1 (alpha=1, beta=0) gives the overhead-agnostic pipeline model
    for Tc, Tm in [(5.0, 2.0), (1.0, 3.0)]:
        for d in [1, 2, 4, 8, 16]:
            agn = (d - 1) * max(Tc, Tm) / d + (Tc + Tm) / d
            assert O.t_decomp(Tc, Tm, d, 1.0, 0.0) == pytest.approx(agn, rel=1e-14)


def _dense_argmin(Tc, Tm, alpha, beta):
    ds = np.linspace(1.0, 200.0, 400001)
    T = np.array([O.t_decomp(Tc, Tm, d, alpha, beta) for d in ds[::50]])
    i = int(np.argmin(T)) * 50
    lo, hi = max(0, i - 60), min(len(ds), i + 60)
    Tf = np.array([O.t_decomp(Tc, Tm, d, alpha, beta) for d in ds[lo:hi]])
    return ds[lo + int(np.argmin(Tf))]


def test_eq5_stationary_point_is_minimum():
    rng = random.Random(5)
    for _ in range(25):
        lam = math.exp(rng.uniform(math.log(0.05), math.log(20.0)))
        Tm = 1.0
        Tc = lam * Tm
        alpha = rng.uniform(0.6, 1.2)
        beta = rng.uniform(0.002, 0.2)
        x = O.d_continuous(lam, alpha, beta)
        if not 1.0 < x < 190.0:
            continue
        assert _dense_argmin(Tc, Tm, alpha, beta) == pytest.approx(x, abs=2e-3 * max(1.0, x))


def test_eq5_literal_matches_when_compute_bound():
    for lam in [1.0, 1.5, 4.0, 10.0]:
        assert O.d_continuous(lam, 0.9, 0.03, literal=True) == O.d_continuous(lam, 0.9, 0.03)
    # when communication dominates the printed form differs
    assert O.d_continuous(0.25, 0.9, 0.03, literal=True) != O.d_continuous(0.25, 0.9, 0.03)


def test_convexity_second_difference():
    for Tc, Tm, a, b in [(5.0, 1.0, 0.9, 0.05), (1.0, 5.0, 1.1, 0.02), (2.0, 2.0, 0.8, 0.1)]:
        ds = np.arange(1.5, 64.0, 0.25)
        T = np.array([O.t_decomp(Tc, Tm, d, a, b) for d in ds])
        assert np.all(np.diff(T, 2) > 0)


@pytest.mark.parametrize("x,want", [(0.3, 1), (1.0, 1), (1.4, 1), (1.5, 2), (2.8, 2), (2.9, 4),
                                    (3.0, 4), (5.6, 4), (5.7, 8), (2 ** 3.5, 8), (100.0, 128)])
def test_p2_log_rounding(x, want):
    assert O.p2(x) == want


def test_p2_is_argmin_over_powers_of_two():
    rng = random.Random(9)
    for _ in range(200):
        A = rng.uniform(0.01, 5.0)
        C = rng.uniform(0.01, 500.0)
        x = math.sqrt(C / A)
        powers = [2 ** k for k in range(0, 12)]
        f = [A * d + C / d for d in powers]
        best = powers[int(np.argmin(f))]
        assert O.p2(x) == best


def test_d_candidate_matches_bruteforce_over_powers():
    rng = random.Random(11)
    for _ in range(100):
        lam = math.exp(rng.uniform(math.log(0.05), math.log(20.0)))
        alpha = rng.uniform(0.6, 1.1)
        beta = rng.uniform(0.002, 0.3)
        Tc, Tm = lam, 1.0
        cands = [1, 2, 4, 8, 16]
        T = [O.t_decomp(Tc, Tm, d, alpha, beta) for d in cands]
        # within one regime Eq. 2 is A*d + B + C/d for every d >= 1 (d = 1
        # included), so P2 of the stationary point is the discrete argmin
        best = cands[int(np.argmin(T))]
        assert O.d_candidate(lam, alpha, beta, 16) == best


def test_d_final_rule():
    # Eq. 4: a candidate that is no faster than d=1 is dropped
    Tc, Tm = 10.0, 0.1
    alpha, beta = 1.5, 0.5          # heavy overhead: splitting never pays
    assert O.d_final(Tc, Tm, alpha, beta) == 1
    Tc, Tm = 4.0, 4.0
    alpha, beta = 0.9, 0.02
    d = O.d_final(Tc, Tm, alpha, beta)
    assert d > 1 and O.t_decomp(Tc, Tm, d, alpha, beta) < Tc + Tm


def test_d_degenerate_parameters():
    assert O.d_candidate(2.0, 0.9, 0.0, 16) == 16        # beta <= 0 -> d_max
    assert O.d_candidate(2.0, 3.0, 0.1, 16) == 1         # 1 - alpha + r <= 0 -> 1


def test_eq7_eq8_by_hand():
    # n=4 chunks: comp 2 each, comm 0,3,1,3 -> 3 + 2 + 3 + 2 (chunk 1) = 10;
    # overhead (4-1)*(0.5 + 0.001*1000) = 4.5
    got = O.t_fusion([2.0, 2.0, 2.0, 2.0], [0.0, 3.0, 1.0, 3.0], 0.5, 0.001, 1000.0)
    assert got == pytest.approx(14.5, rel=1e-15)
    # no overhead and compute-bound: everything but nothing exposed = n * comp
    assert O.t_fusion([1.0] * 8, [0.0] + [0.5] * 7, 0.0, 0.0, 0.0) == pytest.approx(8.0)
    # comm-bound: (n-1) * comm + comp of chunk 1
    assert O.t_fusion([1.0] * 8, [0.0] + [2.0] * 7, 0.0, 0.0, 0.0) == pytest.approx(15.0)


def test_eq8_volume():
    assert O.fusion_m("ag", 8, 4, 16) == 8 * 16
    assert O.fusion_m("rs", 8, 4, 16) == 8 * 4


def test_algorithm1_tie_goes_to_interdecom():
    assert O.select_strategy(5.0, 5.0) == ("inter_decom", 5.0)
    assert O.select_strategy(4.999, 5.0) == ("intra_fusion", 4.999)
    assert O.select_strategy(6.0, 5.0) == ("inter_decom", 5.0)


def test_pick_strategy_by_hand():
    # AllGather, single ring, n=4, M=1024, K=1024 -> S = 2 MiB, per step S/4 =
    # 524288 B at 524288 B/s -> 1 s/step, 3 steps -> Tm = 3 s (tau = 0).
    # T_comp = 0 + 1e-9 * 2*M*N*K with N=2048 -> 2*1024*2048*1024*1e-9 = 4.294967296 s.
    r = O.pick_strategy("ag", "single", 1024, 2048, 1024, 4, 524288.0, 524288.0, 0.0,
                        0.0, 1e-9, 1.0, 0.0, 0.0, 0.0, d_max=16)
    Tc = 4.294967296
    assert r["t_comm"] == pytest.approx(3.0, rel=1e-15)
    assert r["t_comp"] == pytest.approx(Tc, rel=1e-12)
    # agnostic eta -> beta=0 -> d_cand = d_max (16); rows 256 divisible by 16
    assert r["d_cand"] == 16 and r["d_star"] == 16
    t16 = 15 * Tc / 16 + (Tc + 3.0) / 16
    assert r["t_decomp"] == pytest.approx(t16, rel=1e-12)
    # fusion: chunk 1 comp Tc/4 + 3 * max(Tc/4, 1) with no overhead
    tf = Tc / 4 + 3 * max(Tc / 4, 1.0)
    assert r["t_fusion"] == pytest.approx(tf, rel=1e-12)
    assert r["strategy"] == ("intra_fusion" if tf < t16 else "inter_decom")


def test_fit_line_recovers_planted():
    rng = np.random.default_rng(3)
    x = rng.uniform(1, 16, size=40)
    y = 0.85 + 0.031 * x
    a, b = O.fit_line(x, y)
    assert a == pytest.approx(0.85, abs=1e-12) and b == pytest.approx(0.031, abs=1e-13)
    y2 = y + rng.normal(0, 1e-3, size=40)
    a2, b2 = O.fit_line(x, y2)
    assert abs(a2 - 0.85) < 5e-3 and abs(b2 - 0.031) < 5e-4


def test_eta_observed_inverts_eq2():
    for Tc, Tm, d, a, b in [(5.0, 2.0, 4, 0.9, 0.05), (1.0, 3.0, 8, 1.1, 0.01)]:
        t = O.t_decomp(Tc, Tm, d, a, b)
        assert O.eta_observed(t, Tc, Tm, d) == pytest.approx(O.eta(d, a, b), rel=1e-12)


def test_fusion_overhead_observed_inverts_eq7():
    comp = [1.0] * 8
    comm = [0.0] + [1.3] * 7
    t = O.t_fusion(comp, comm, 0.02, 1e-6, 5000.0)
    assert O.fusion_overhead_observed(t, comp, comm) == pytest.approx(0.02 + 1e-6 * 5000.0, rel=1e-12)


def test_calibration_eta_fit_from_measurements():
    # synthetic "measurements" built from a known eta(d), then the two-step
    # procedure (invert Eq. 2 per point, fit Eq. 3) must recover it
    alpha, beta = 0.93, 0.041
    xs, ys = [], []
    for Tc, Tm in [(3.0, 1.0), (1.0, 2.0), (2.0, 2.5)]:
        for d in [2, 4, 8, 16]:
            t = O.t_decomp(Tc, Tm, d, alpha, beta)
            xs.append(d)
            ys.append(O.eta_observed(t, Tc, Tm, d))
    a, b = O.fit_line(xs, ys)
    assert a == pytest.approx(alpha, abs=1e-12) and b == pytest.approx(beta, abs=1e-12)


def test_proportional_double_ring_comm_by_hand():
    # AllGather n = 8, M x K = 8192 x 4096 bf16: a step moves one 8 MiB chunk.
    # Split 1:4 between a 50 GB/s backward and a 200 GB/s forward ring, both
    # finish a step after 8 MiB / 250 GB/s; the halved double ring waits for
    # its 4 MiB on the slow ring.
    chunk = 8192 * 4096 * 2 / 8
    got = O.t_comm(O.AG, O.DOUBLE_SPLIT, 8192, 1, 4096, 8, 200e9, 50e9)
    assert got == pytest.approx(7 * chunk / 250e9, rel=1e-14)
    assert O.t_comm(O.AG, O.DOUBLE, 8192, 1, 4096, 8, 200e9, 50e9) == pytest.approx(7 * chunk / 2 / 50e9, rel=1e-14)
    # ReduceScatter: the fp32 partial in (twice the bf16 sum out) sets the step
    chunk_in = 8192 * 4096 * 4 / 8
    got = O.t_comm(O.RS, O.DOUBLE_SPLIT, 8192, 4096, 2048, 8, 200e9, 50e9, tau=1e-6)
    assert got == pytest.approx(7 * (chunk_in / 250e9 + 1e-6), rel=1e-14)


def test_proportional_double_ring_reduces_to_halves_at_equal_rates():
    rng = random.Random(11)
    for _ in range(50):
        pat = rng.choice([O.AG, O.RS])
        n = rng.choice([2, 4, 8, 16])
        M, N, K = n * 2 * rng.randint(1, 64) * 8, rng.randint(1, 64) * 64, rng.randint(1, 64) * 64
        B = rng.uniform(1e9, 500e9)
        a = O.t_comm(pat, O.DOUBLE_SPLIT, M, N, K, n, B, B)
        b = O.t_comm(pat, O.DOUBLE, M, N, K, n, B, B)
        assert a == pytest.approx(b, rel=1e-13)
        # and never slower than halves at unequal rates
        f = rng.uniform(0.05, 1.0)
        assert O.t_comm(pat, O.DOUBLE_SPLIT, M, N, K, n, B, B * f) <= \
            O.t_comm(pat, O.DOUBLE, M, N, K, n, B, B * f) * (1 + 1e-12)


def test_alltoall_closed_form_matches_brute_force_link_loads():
    # the one-round closed form against the per-link loads of every flow
    rng = random.Random(13)
    for _ in range(60):
        n = rng.choice([2, 4, 6, 8, 12, 16])
        M, K = n * rng.randint(1, 64) * 8, rng.randint(1, 64) * 64
        fwd, bwd = rng.uniform(1e9, 500e9), rng.uniform(1e9, 500e9)
        chunk = M * K * 2 / n
        want = O.alltoall_link_time(n, chunk, fwd, bwd)
        assert O.t_comm(O.AG, O.ALLTOALL, M, 1, K, n, fwd, bwd) == pytest.approx(want, rel=1e-13)
        assert O.t_comm(O.AG, O.ALLTOALL, M, 1, K, n, fwd, bwd, tau=2e-6) == pytest.approx(want + 2e-6, rel=1e-13)


def test_alltoall_is_about_half_the_single_ring_across_numa():
    # Section III-A: on the 8-GPU cross-NUMA topology the single ring reaches
    # (8/7) B_QPI and the AlltoAll pattern B_QPI / 2, whatever the (faster)
    # links inside a domain carry
    B = 40e9
    S = 8 * 8 * 1024 * 1024 * 2.0
    for intra in (B, 200e9, 1e12):
        t = O.t_comm(O.AG, O.ALLTOALL, 8 * 1024, 1, 8 * 1024, 8, intra, B)
        assert S / t == pytest.approx(B / 2, rel=1e-12)
    ring = O.t_comm(O.AG, O.SINGLE, 8 * 1024, 1, 8 * 1024, 8, B, B)
    assert ring / t == pytest.approx((1 / 2) / (8 / 7), rel=1e-12)


def test_alltoall_refuses_reducescatter_and_odd_n():
    with pytest.raises(ValueError):
        O.t_comm(O.RS, O.ALLTOALL, 64, 64, 64, 8, 1e9, 1e9)
    with pytest.raises(ValueError):
        O.t_comm(O.AG, O.ALLTOALL, 60, 64, 64, 3, 1e9, 1e9)
    with pytest.raises(ValueError):
        O.schedule(O.AG, O.ALLTOALL, 5, 0)


# ---- single ring with per-hop rates (Section III-A, cross-NUMA ring)
def test_hop_ring_uniform_rates_are_serialized_steps():
    for n in (2, 3, 8, 16):
        for r in range(n):
            got = O.ring_arrival_times(n, r, 3e6, [60e9] * n)
            assert got == pytest.approx([s * 3e6 / 60e9 for s in range(1, n)], rel=1e-13)
            # d sub-collectives run back to back: the same last arrival
            got4 = O.ring_arrival_times(n, r, 3e6 / 4, [60e9] * n, d=4)
            assert got4 == pytest.approx([t * 3e6 / 4 / 60e9 for t in range(1, 4 * (n - 1) + 1)], rel=1e-13)


def test_hop_ring_by_hand_n4():
    # hops 0->1, 1->2, 2->3 take 1 unit, hop 3->0 takes 4. Rank 0, right after
    # the slow hop, gets a chunk every 4 units; rank 3, furthest downstream,
    # gets its first three over fast hops.
    hops = [1.0, 1.0, 1.0, 0.25]
    want = {0: [4, 8, 12], 1: [1, 5, 9], 2: [1, 2, 6], 3: [1, 2, 3]}
    for r, w in want.items():
        assert O.ring_arrival_times(4, r, 1.0, hops) == pytest.approx(w, abs=1e-15)


def test_hop_ring_matches_event_simulation():
    rng = random.Random(17)
    for _ in range(150):
        n = rng.choice([1, 2, 3, 4, 5, 8, 12])
        hops = [rng.uniform(1e9, 100e9) for _ in range(n)]
        sim = O.simulate_timed_ring_allgather(n, 2e6, hops)
        for r in range(n):
            got = O.ring_arrival_times(n, r, 2e6, hops)
            assert [c for _, c in sim[r]] == O.schedule("ag", "single", n, r)[1:]
            assert got == pytest.approx([t for t, _ in sim[r]], rel=1e-13)


def test_cross_numa_ring_reaches_8_over_7_of_the_slow_link():
    # Section III-A, Fig. 5(a): 8 ranks, only hops 3->4 and 7->0 cross the
    # NUMA boundary (rate B); whatever the faster hops run at, the last
    # arrival anywhere is 7 chunks over B, an effective (8/7) B, and the
    # ranks right after the slow hops finish last
    rng = random.Random(19)
    B, m = 20e9, 4e6
    for _ in range(40):
        hops = [rng.uniform(B, 20 * B) for _ in range(8)]
        hops[3] = hops[7] = B
        last = [O.ring_arrival_times(8, r, m, hops)[-1] for r in range(8)]
        assert max(last) == pytest.approx(7 * m / B, rel=1e-13)
        assert last[0] == pytest.approx(7 * m / B, rel=1e-13) and last[4] == pytest.approx(7 * m / B, rel=1e-13)
        assert 8 * m / max(last) == pytest.approx(8 / 7 * B, rel=1e-13)


def test_hop_ring_busiest_hop_bounds_the_collective():
    # every hop carries d (n-1) pieces of m/d one after another, so the rank
    # after the slowest hop cannot finish before (n-1) m / B_min; arrivals at
    # a rank are in order
    rng = random.Random(23)
    for _ in range(60):
        n = rng.choice([2, 4, 8])
        hops = [rng.uniform(1e9, 100e9) for _ in range(n)]
        slow = min(range(n), key=lambda q: hops[q])
        for d in (1, 2, 4, 8):
            t = O.ring_arrival_times(n, (slow + 1) % n, 8e6 / d, hops, d=d)
            assert t[-1] >= (n - 1) * 8e6 / hops[slow] * (1 - 1e-12)
            for r in range(n):
                a = O.ring_arrival_times(n, r, 8e6 / d, hops, d=d)
                assert all(x < y for x, y in zip(a, a[1:]))
