"""Host-only checks of the C ABI (no GPU): the library loads and exports every
function declared in include/compass.h; the host calls (schedule, models,
selector, calibration) agree with the oracle — integers exactly, times to
1e-12 relative."""
import ctypes
import math
import os
import random
import re

import pytest

import oracle as O
from paper_2609_10549_amd import compass as C

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "compass.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(compass_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = C.lib()
    names = declared_functions()
    assert len(names) >= 14
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(C._SIGS), "binding and header disagree"


def test_every_header_constant_has_the_same_value_in_the_binding():
    text = open(os.path.join(ROOT, "include", "compass.h")).read()
    defs = dict(re.findall(r"^#define COMPASS_([A-Z0-9_]+)\s+(-?\d+)\b", text, flags=re.M))
    assert len(defs) >= 24
    for name, value in defs.items():
        assert getattr(C, name) == int(value), name
    opts = {k: v for k, v in defs.items() if k.startswith("OPT_")}
    assert len(set(opts.values())) == len(opts), "two options share a key"


def test_struct_sizes_match_c_layout():
    assert ctypes.sizeof(C.compass_links) == 40
    assert ctypes.sizeof(C.compass_problem) == 4 * 7 + 4 + 8 * 8
    assert ctypes.sizeof(C.compass_calib) == 6 * 8 + 8
    assert ctypes.sizeof(C.compass_choice) == 3 * 4 + 4 + 7 * 8


@pytest.mark.parametrize("pattern", ["ag", "rs"])
@pytest.mark.parametrize("ring", ["single", "double", "double_split"])
def test_schedule_bit_exact_vs_oracle(pattern, ring):
    for n in [1, 2, 3, 4, 5, 8, 16, 32]:
        for r in range(n):
            assert C.compass_schedule(pattern, ring, n, r) == O.schedule(pattern, ring, n, r)


def test_alltoall_schedule_bit_exact_vs_oracle():
    for n in [2, 4, 6, 8, 16, 32]:
        for r in range(n):
            assert C.compass_schedule("ag", "alltoall", n, r) == O.schedule("ag", "alltoall", n, r)
    with pytest.raises(C.CompassError) as e:
        C.compass_schedule("rs", "alltoall", 8, 0)
    assert e.value.code == C.ERR_UNSUPPORTED
    with pytest.raises(C.CompassError):
        C.compass_schedule("ag", "alltoall", 5, 0)


def test_model_t_comm_matches_oracle_for_every_ring():
    rng = random.Random(7)
    for _ in range(300):
        ring = rng.choice(["single", "double", "double_split", "alltoall"])
        pat = "ag" if ring == "alltoall" else rng.choice(["ag", "rs"])
        n = rng.choice([2, 4, 8, 16])
        M, N, K = 2 * n * rng.randint(1, 64) * 8, rng.randint(1, 64) * 64, rng.randint(1, 64) * 64
        fwd, bwd, tau = rng.uniform(1e9, 500e9), rng.uniform(1e9, 500e9), rng.uniform(0, 2e-5)
        w = C.compass_workload(pattern=C.PATTERNS[pat], M=M, N=N, K=K, n=n)
        t = C.compass_topology(ring=C.RINGS[ring], fwd_Bps=fwd, bwd_Bps=bwd, step_latency_s=tau)
        assert _rel(C.compass_model_t_comm(w, t), O.t_comm(pat, ring, M, N, K, n, fwd, bwd, tau)) < 1e-12
    w = C.compass_workload(pattern=C.PATTERNS["rs"], M=64, N=64, K=64, n=8)
    t = C.compass_topology(ring=C.RINGS["alltoall"], fwd_Bps=1e9, bwd_Bps=1e9, step_latency_s=0)
    assert C.compass_model_t_comm(w, t) < 0                      # AllGather only
    w.pattern, t.bwd_Bps = C.PATTERNS["ag"], 0.0
    assert C.compass_model_t_comm(w, t) < 0                      # needs the cross-domain rate
    t.ring = 9
    assert C.compass_model_t_comm(w, t) < 0


def test_ring_arrival_times_match_oracle():
    rng = random.Random(29)
    for _ in range(200):
        n = rng.choice([1, 2, 3, 4, 8, 16, 32])
        d = rng.choice([1, 2, 4, 16])
        hops = [rng.uniform(1e8, 500e9) for _ in range(n)]
        b = rng.uniform(0, 64e6)
        for r in {0, n - 1, rng.randrange(n)}:
            got = C.compass_ring_arrival_times(n, r, b, hops, d)
            ref = O.ring_arrival_times(n, r, b, hops, d)
            assert len(got) == len(ref) == d * (n - 1)
            assert all(_rel(x, y) < 1e-13 or x == y for x, y in zip(got, ref))
    for args in ((0, 0, 1.0, [1e9], 1), (4, 4, 1.0, [1e9] * 4, 1), (4, 0, 1.0, [1e9] * 4, 0),
                 (4, 0, 1.0, [1e9, 0.0, 1e9, 1e9], 1), (4, 0, -1.0, [1e9] * 4, 1),
                 (4, 0, 1.0, [1e9, float("nan"), 1e9, 1e9], 1)):
        with pytest.raises(C.CompassError):
            C.compass_ring_arrival_times(*args)


def test_partition_layout_bit_exact_vs_oracle():
    rng = random.Random(31)
    checked = 0
    for _ in range(400):
        ring = rng.choice(["single", "double", "double_split"])
        pat = rng.choice(["ag", "rs"])
        n = rng.choice([1, 2, 3, 4, 8, 16])
        base = n * (2 if ring != "single" else 1)
        sub = rng.choice([0, 1, 2, 3, 4, 8])
        if base * max(sub, 1) > 64:
            continue
        M = base * rng.choice([1, 3, 8, 64, 128, 512, 1024, 1536])
        fwd, bwd = rng.choice([(0.0, 0.0), (200e9, 50e9), (50e9, 200e9), (1e9, 3e9)])
        r = rng.randrange(n)
        ref = O.partition_layout(pat, ring, n, r, M, fwd, bwd, max(sub, 1))
        if min(ref[2]) < 1:
            with pytest.raises(C.CompassError):
                C.compass_partition_layout(pat, ring, n, r, M, C.links(fwd, bwd, sub_chunks=sub))
            continue
        got = C.compass_partition_layout(pat, ring, n, r, M, C.links(fwd, bwd, sub_chunks=sub))
        assert got == (ref[0], ref[1], ref[2]), (pat, ring, n, r, M, sub, fwd, bwd)
        checked += 1
    assert checked > 250


def test_sub_chunk_refusals_before_enqueue():
    lib = C.lib()
    for ring, kw, want in ((C.RING_ALLTOALL, dict(sub_chunks=2), C.ERR_UNSUPPORTED),
                           (C.RING_SINGLE, dict(sub_chunks=2, hop_Bps=[1e9, 1e9]), C.ERR_UNSUPPORTED),
                           (C.RING_DOUBLE, dict(sub_chunks=17), C.ERR_UNSUPPORTED),   # 4 x 17 > 64
                           (C.RING_SINGLE, dict(sub_chunks=-1), C.ERR_INVALID),
                           (C.RING_SINGLE, dict(sub_chunks=16), C.ERR_INVALID)):      # 8 rows, 16 pieces
        st, keep = _fake_problem(C.AG_GEMM, 16, 64, 64, 2, ring=ring)
        lk = C.links(1e9, 1e9, **kw)
        assert lib.compass_ag_gemm(ctypes.byref(st), ctypes.byref(lk), None) == want, (ring, kw)
    st, keep = _fake_problem(C.GEMM_RS, 64, 64, 64, 2)
    lk = C.links(1e9, 1e9, sub_chunks=2)
    assert lib.compass_decomp_gemm(ctypes.byref(st), 2, ctypes.byref(lk), None) == C.ERR_UNSUPPORTED


def test_hop_rates_refused_off_the_single_ring_or_out_of_range():
    lib = C.lib()
    for ring in (C.RING_DOUBLE, C.RING_DOUBLE_SPLIT, C.RING_ALLTOALL):
        st, keep = _fake_problem(C.AG_GEMM, 64, 64, 64, 2, ring=ring)
        lk = C.links(1e9, 1e9, hop_Bps=[1e9, 1e9])
        assert lib.compass_ag_gemm(ctypes.byref(st), ctypes.byref(lk), None) == C.ERR_UNSUPPORTED
    for pattern, call in ((C.AG_GEMM, lib.compass_ag_gemm), (C.GEMM_RS, lib.compass_gemm_rs)):
        st, keep = _fake_problem(pattern, 64, 64, 64, 2)
        for hops in ([1e9, 5e7], [1e9, float("inf")], [0.0, 1e9]):
            lk = C.links(1e9, hop_Bps=hops)
            assert call(ctypes.byref(st), ctypes.byref(lk), None) == C.ERR_INVALID


def test_pick_strategy_refuses_alltoall():
    w = C.compass_workload(pattern=C.PATTERNS["ag"], M=1024, N=64, K=64, n=8)
    t = C.compass_topology(ring=C.RINGS["alltoall"], fwd_Bps=1e9, bwd_Bps=1e9, step_latency_s=0)
    c = C.compass_calib(comp_a=0, comp_b=1e-12, alpha_decomp=1, beta_decomp=0.1, d_max=16)
    with pytest.raises(C.CompassError) as e:
        C.compass_pick_strategy(w, t, c)
    assert e.value.code == C.ERR_UNSUPPORTED


def test_schedule_errors():
    with pytest.raises(C.CompassError) as e:
        C.compass_schedule("ag", "single", 4, 4)
    assert e.value.code == C.ERR_INVALID
    with pytest.raises(C.CompassError):
        C.compass_schedule("ag", "single", 33, 0)
    assert "rank" in C.compass_last_error()


def _rel(a, b):
    return abs(a - b) / max(abs(b), 1e-300)


def test_model_functions_match_oracle():
    rng = random.Random(1)
    for _ in range(200):
        Tc, Tm = rng.uniform(0.1, 10), rng.uniform(0.1, 10)
        d = rng.choice([1, 2, 4, 8, 16])
        a, b = rng.uniform(0.5, 1.5), rng.uniform(0, 0.3)
        assert _rel(C.compass_model_t_decomp(Tc, Tm, d, a, b), O.t_decomp(Tc, Tm, d, a, b)) < 1e-12
        n = rng.choice([2, 4, 8])
        pat = rng.choice(["ag", "rs"])
        M, N, K = 1024 * n, rng.choice([2048, 4096]), rng.choice([4096, 8192])
        w = C.compass_workload(pattern=C.PATTERNS[pat], M=M, N=N, K=K, n=n)
        af, bf = rng.uniform(0, 1e-4), rng.uniform(0, 1e-12)
        step = Tm / (n - 1)
        ref = O.t_fusion([Tc / n] * n, [0.0] + [step] * (n - 1), af, bf, O.fusion_m(pat, M, N, K))
        assert _rel(C.compass_model_t_fusion(w, Tc, step, af, bf), ref) < 1e-12


def _pick_both(pat, ring, M, N, K, n, fwd, bwd, tau, cal):
    w = C.compass_workload(pattern=C.PATTERNS[pat], M=M, N=N, K=K, n=n)
    t = C.compass_topology(ring=C.RINGS[ring], fwd_Bps=fwd, bwd_Bps=bwd, step_latency_s=tau)
    c = C.compass_calib(**cal)
    got = C.compass_pick_strategy(w, t, c)
    ref = O.pick_strategy(pat, ring, M, N, K, n, fwd, bwd, tau, cal["comp_a"], cal["comp_b"],
                          cal["alpha_decomp"], cal["beta_decomp"], cal["alpha_fusion"], cal["beta_fusion"],
                          d_max=cal["d_max"], literal=bool(cal["literal_eq5"]))
    return got, ref


def test_pick_strategy_matches_oracle_over_table4():
    rng = random.Random(4)
    wl = O.table4_workloads()
    strategies = set()
    for i, (pat, M, N, K, n) in enumerate(wl):
        ring = ("single", "double", "double_split")[i % 3]
        fwd = rng.uniform(5e9, 400e9)
        bwd = fwd / rng.choice([1.0, 4.0])
        cal = dict(comp_a=rng.uniform(0, 2e-5), comp_b=1.0 / rng.uniform(3e14, 2e15),
                   alpha_decomp=rng.uniform(0.7, 1.2), beta_decomp=rng.uniform(0.0, 0.15),
                   alpha_fusion=rng.uniform(0, 5e-5), beta_fusion=rng.uniform(0, 1e-13),
                   d_max=16, literal_eq5=i % 4 == 1)
        got, ref = _pick_both(pat, ring, M, N, K, n, fwd, bwd, rng.uniform(0, 2e-5), cal)
        assert got.d_star == ref["d_star"] and got.d_cand == ref["d_cand"]
        assert got.strategy == (C.INTRA_FUSION if ref["strategy"] == "intra_fusion" else C.INTER_DECOM)
        for k, kk in [("t_comp", "t_comp"), ("t_comm", "t_comm"), ("lambda_", "lam"), ("t_fusion", "t_fusion"),
                      ("t_decomp", "t_decomp"), ("t_decomp1", "t_decomp1"), ("t_star", "t_star")]:
            assert _rel(getattr(got, k), ref[kk]) < 1e-12, k
        strategies.add(got.strategy)
    assert strategies == {C.INTRA_FUSION, C.INTER_DECOM}   # both branches exercised


def test_pick_strategy_rejects_bad_inputs():
    w = C.compass_workload(pattern=0, M=1001, N=64, K=64, n=8)   # M % n != 0
    t = C.compass_topology(ring=0, fwd_Bps=1e9, bwd_Bps=1e9, step_latency_s=0)
    c = C.compass_calib(comp_a=0, comp_b=1e-12, alpha_decomp=1, beta_decomp=0.1, d_max=16)
    with pytest.raises(C.CompassError):
        C.compass_pick_strategy(w, t, c)
    w.M = 1024
    t.fwd_Bps = 0
    with pytest.raises(C.CompassError):
        C.compass_pick_strategy(w, t, c)


def test_calibrate_matches_oracle_fits():
    rng = random.Random(8)
    samples, xs0, ys0, xs1, ys1, xs2, ys2 = [], [], [], [], [], [], []
    for i in range(30):
        n = rng.choice([4, 8])
        pat = rng.choice(["ag", "rs"])
        M, N, K = 1024 * n, rng.choice([2048, 4096]), rng.choice([2048, 8192])
        w = C.compass_workload(pattern=C.PATTERNS[pat], M=M, N=N, K=K, n=n)
        kind = i % 3
        Tc, Tm = rng.uniform(1e-4, 1e-3), rng.uniform(1e-4, 1e-3)
        d = rng.choice([2, 4, 8, 16])
        t = rng.uniform(2e-4, 3e-3)
        samples.append(C.compass_sample(kind=kind, w=w, d=d, t_meas=t, t_comp=Tc, t_comm=Tm))
        if kind == 0:
            xs0.append(2.0 * M * N * K)
            ys0.append(t)
        elif kind == 1:
            xs1.append(d)
            ys1.append(O.eta_observed(t, Tc, Tm, d))
        else:
            xs2.append(O.fusion_m(pat, M, N, K))
            ys2.append(O.fusion_overhead_observed(t, [Tc / n] * n, [0.0] + [Tm / (n - 1)] * (n - 1)))
    cal = C.compass_calibrate(samples, C.compass_calib(d_max=16))
    a0, b0 = O.fit_line(xs0, ys0)
    a1, b1 = O.fit_line(xs1, ys1)
    a2, b2 = O.fit_line(xs2, ys2)
    for got, ref in [(cal.comp_a, a0), (cal.comp_b, b0), (cal.alpha_decomp, a1), (cal.beta_decomp, b1),
                     (cal.alpha_fusion, a2), (cal.beta_fusion, b2)]:
        assert math.isclose(got, ref, rel_tol=1e-9, abs_tol=1e-18)


def test_calibrate_keeps_fields_without_data():
    cal = C.compass_calib(comp_a=1.0, comp_b=2.0, alpha_decomp=3.0, beta_decomp=4.0,
                          alpha_fusion=5.0, beta_fusion=6.0, d_max=16)
    C.compass_calibrate([], cal)
    assert (cal.comp_a, cal.beta_fusion) == (1.0, 6.0)


# ------------------------------------------------------------ argument validation (host only)
def _fake_problem(pattern, M, N, K, n, rank=0, ring=C.RING_SINGLE):
    """A problem whose buffers are placeholder addresses: every call below
    must be refused by the host-side checks, before anything is enqueued."""
    fake = 0x100000
    srcs = (ctypes.c_void_p * max(n, 1))(*([fake] * max(n, 1)))
    st = C.compass_problem(pattern=pattern, M=M, N=N, K=K, n=n, rank=rank, ring=ring, W=fake, C=fake,
                           shard_src=srcs, gathered=fake, A=fake, partial_src=srcs, partial_stage=fake,
                           send_dst=None)
    return st, srcs


@pytest.mark.parametrize("pattern", [C.AG_GEMM, C.GEMM_RS])
def test_degenerate_and_oversized_problems_are_refused_before_enqueue(pattern):
    lib = C.lib()
    lk = C.links(0.0, 0.0)
    call = lib.compass_ag_gemm if pattern == C.AG_GEMM else lib.compass_gemm_rs
    cases = [
        ((0, 64, 64, 2), C.ERR_INVALID),          # empty M
        ((64, 0, 64, 2), C.ERR_INVALID),          # empty N
        ((64, 64, 0, 2), C.ERR_INVALID),          # empty K
        ((66, 64, 64, 4), C.ERR_INVALID),         # M not divisible by the partition count
        ((64, 60, 64, 2), C.ERR_INVALID),         # N not a multiple of 8
        ((64, 64, 60, 2), C.ERR_INVALID),         # K not a multiple of 8
        ((64, 64, 64, 0), C.ERR_INVALID),         # no ranks
        ((128, 64, 64, 33), C.ERR_INVALID),       # more ranks than the flag masks hold
        ((65664, 64, 64, 2), C.ERR_UNSUPPORTED),     # M beyond the 65536 rows of the tile table
        ((64, 64, 2097160, 2), C.ERR_UNSUPPORTED),   # K so deep a 256-row tile spans over 1 GiB of A
    ]
    if pattern == C.GEMM_RS:   # N so wide a 256-row tile spans over 1 GiB of the fp32 partial
        cases.append(((64, 1048584, 64, 2), C.ERR_UNSUPPORTED))
    for (M, N, K, n), want in cases:
        st, keep = _fake_problem(pattern, M, N, K, n)
        assert call(ctypes.byref(st), ctypes.byref(lk), None) == want, (M, N, K, n)
        assert lib.compass_decomp_gemm(ctypes.byref(st), 1, ctypes.byref(lk), None) == want, (M, N, K, n)
    # rank out of range, unknown ring, missing buffers, bad links
    st, keep = _fake_problem(pattern, 64, 64, 64, 2, rank=2)
    assert call(ctypes.byref(st), ctypes.byref(lk), None) == C.ERR_INVALID
    st, keep = _fake_problem(pattern, 64, 64, 64, 2, ring=7)
    assert call(ctypes.byref(st), ctypes.byref(lk), None) == C.ERR_INVALID
    st, keep = _fake_problem(pattern, 64, 64, 64, 2)
    st.W = None
    assert call(ctypes.byref(st), ctypes.byref(lk), None) == C.ERR_INVALID
    st, keep = _fake_problem(pattern, 64, 64, 64, 2)
    for bad in (C.links(5e7, 5e7), C.links(float("nan")), C.links(0.0, 0.0, slice_bytes=1024),
                C.links(0.0, 0.0, engines_per_ring=-1)):
        assert call(ctypes.byref(st), ctypes.byref(bad), None) == C.ERR_INVALID
    assert call(None, ctypes.byref(lk), None) == C.ERR_INVALID
    assert call(ctypes.byref(st), None, None) == C.ERR_INVALID
    # InterDecom degree: a power of two dividing the rows of a partition
    st, keep = _fake_problem(pattern, 64, 64, 64, 2)
    for d in (0, 3, 64):
        assert lib.compass_decomp_gemm(ctypes.byref(st), d, ctypes.byref(lk), None) == C.ERR_INVALID
    # the wrong entry point for the pattern
    other = lib.compass_gemm_rs if pattern == C.AG_GEMM else lib.compass_ag_gemm
    assert other(ctypes.byref(st), ctypes.byref(lk), None) == C.ERR_INVALID
    assert "" != C.lib().compass_last_error().decode()


def test_alltoall_pattern_refusals_before_enqueue():
    lib = C.lib()
    lk = C.links(0.0, 0.0)
    st, keep = _fake_problem(C.GEMM_RS, 64, 64, 64, 2, ring=C.RING_ALLTOALL)
    assert lib.compass_gemm_rs(ctypes.byref(st), ctypes.byref(lk), None) == C.ERR_UNSUPPORTED
    st, keep = _fake_problem(C.AG_GEMM, 96, 64, 64, 3, ring=C.RING_ALLTOALL)    # odd n
    assert lib.compass_ag_gemm(ctypes.byref(st), ctypes.byref(lk), None) == C.ERR_INVALID
    st, keep = _fake_problem(C.AG_GEMM, 64, 64, 64, 2, ring=C.RING_ALLTOALL)
    assert lib.compass_decomp_gemm(ctypes.byref(st), 2, ctypes.byref(lk), None) == C.ERR_UNSUPPORTED


def test_plain_gemm_refuses_degenerate_shapes():
    lib = C.lib()
    fake = ctypes.c_void_p(0x100000)
    for M, N, K in ((0, 8, 8), (8, 0, 8), (8, 8, 0), (8, 12, 8), (8, 8, 12)):
        assert lib.compass_gemm(M, N, K, fake, fake, fake, None, None) == C.ERR_INVALID
    assert lib.compass_gemm(8, 8, 8, None, fake, fake, None, None) == C.ERR_INVALID
    assert lib.compass_gemm(65664, 64, 64, fake, fake, fake, None, None) == C.ERR_UNSUPPORTED      # M
    assert lib.compass_gemm(64, 64, 2097160, fake, fake, fake, None, None) == C.ERR_UNSUPPORTED    # K
    for it in (0, -1, 1 << 23):
        a, b = ctypes.c_double(), ctypes.c_double()
        assert lib.compass_probe_mfma(it, ctypes.byref(a), ctypes.byref(b)) == C.ERR_INVALID


def test_binding_checks_shapes_element_sizes_and_contiguity():
    # the binding rejects operands whose extents differ from what M, N, K and
    # n imply before any library call (host tensors suffice: nothing runs)
    torch = pytest.importorskip("torch")
    M, N, K, n = 64, 32, 16, 4
    i16 = lambda *s: torch.zeros(s, dtype=torch.int16)  # noqa: E731
    f32 = lambda *s: torch.zeros(s, dtype=torch.float32)  # noqa: E731
    sh = [i16(M // n, K) for _ in range(n)]
    C.ag_problem(sh, i16(M, K), i16(N, K), i16(M, N), 0, "single")
    with pytest.raises(ValueError, match=r"shards\[3\]"):
        C.ag_problem(sh[:3] + [i16(M // n, K + 8)], i16(M, K), i16(N, K), i16(M, N), 0, "single")
    with pytest.raises(ValueError, match="element size"):
        C.ag_problem(sh, i16(M, K), i16(N, K), f32(M, N), 0, "single")
    with pytest.raises(ValueError, match="contiguous"):
        C.ag_problem(sh, i16(M, K), i16(K, N).t(), i16(M, N), 0, "single")
    with pytest.raises(ValueError, match="split"):
        C.ag_problem(sh[:3], i16(M, K), i16(N, K), i16(M, N), 0, "single")
    parts = [f32(M // n, N) for _ in range(n)]
    sends = [None] + [i16(M // n, N) for _ in range(n - 1)]
    C.rs_problem(i16(M, K), i16(N, K), parts, f32(M, N), i16(M, N), sends, 0, "single")
    with pytest.raises(ValueError, match=r"partial_src\[1\]"):
        C.rs_problem(i16(M, K), i16(N, K), [parts[0], i16(M // n, N)] + parts[2:], f32(M, N), i16(M, N), sends, 0,
                     "single")
    with pytest.raises(ValueError, match="partial_stage"):
        C.rs_problem(i16(M, K), i16(N, K), parts, i16(M, N), i16(M, N), sends, 0, "single")
    with pytest.raises(ValueError, match=r"send_dst\[2\]"):
        C.rs_problem(i16(M, K), i16(N, K), parts, f32(M, N), i16(M, N), sends[:2] + [i16(M // n, N - 8)] + sends[3:],
                     0, "single")
    with pytest.raises(ValueError, match="entries"):
        C.rs_problem(i16(M, K), i16(N, K), parts, f32(M, N), i16(M, N), sends[:2], 0, "single")


def test_tail_split_options_are_validated_without_a_gpu():
    # host-side options: set and refused without touching the device
    lib = C.lib()
    good = [(C.OPT_TAIL_MIN_K, 0), (C.OPT_TAIL_MIN_K, 8192), (C.OPT_TAIL_MIN_K_128, 4096),
            (C.OPT_TAIL_MIN_K_128, 0), (C.OPT_TAIL_SLICE_K, 1024), (C.OPT_TAIL_SLICE_K, 2048),
            (C.OPT_TAIL_GROUPS, 1), (C.OPT_TAIL_GROUPS, 2)]
    for k, v in good:
        assert lib.compass_set_option(k, v) == C.OK, (k, v)
    bad = [(C.OPT_TAIL_MIN_K, -1), (C.OPT_TAIL_MIN_K, (1 << 21) + 1), (C.OPT_TAIL_MIN_K_128, -5),
           (C.OPT_TAIL_SLICE_K, 0), (C.OPT_TAIL_SLICE_K, 1000), (C.OPT_TAIL_GROUPS, 0), (C.OPT_TAIL_GROUPS, 9)]
    for k, v in bad:
        assert lib.compass_set_option(k, v) == C.ERR_INVALID, (k, v)
    # back to the defaults
    for k, v in [(C.OPT_TAIL_MIN_K, 8192), (C.OPT_TAIL_MIN_K_128, 0), (C.OPT_TAIL_SLICE_K, 2048),
                 (C.OPT_TAIL_GROUPS, 2)]:
        assert lib.compass_set_option(k, v) == C.OK
