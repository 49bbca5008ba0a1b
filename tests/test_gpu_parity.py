"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Bars: bf16 outputs within 5e-3 normwise relative error; integer-valued inputs
(every fp32 partial sum exact) bit-exact against the oracle's exact result
rounded to bf16 (nearest-even); schedules and index work bit-exact."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import oracle as O  # noqa: E402
from paper_2609_10549_amd import compass as C  # noqa: E402
from synth import make_ag_inputs, make_int_ag_inputs, make_int_rs_inputs, make_rs_inputs  # noqa: E402
from tests.gpu_helpers import TOL, AGCase, RSCase, host_bits, host_f64, rel_err, dev_bits  # noqa: E402

FAST = C.links(200e9, 200e9)   # emulated link rates for functional tests


def _say(*a):
    print(*a, flush=True)


@pytest.fixture(autouse=True)
def _sync_after():
    yield
    C.compass_sync()


# ------------------------------------------------------------ plain GEMM
@pytest.mark.parametrize("M,N,K", [(256, 256, 64), (300, 264, 200), (777, 520, 1032), (64, 8, 8), (1, 16, 8)])
def test_gemm_integer_exact(M, N, K):
    _say("gemm int", M, N, K)
    inp = make_int_ag_inputs(M, N, K, 1, seed=M + N + K)
    A = dev_bits(inp["shards"][0])
    W = dev_bits(inp["W"])
    Cm = torch.zeros((M, N), dtype=torch.int16, device="cuda")
    C.compass_gemm(A, W, Cm)
    torch.cuda.synchronize()
    ref = O.ag_gemm([O.bf16_to_f64(inp["shards"][0])], O.bf16_to_f64(inp["W"]))
    assert np.array_equal(host_bits(Cm), O.f64_to_bf16_rne(ref))


@pytest.mark.parametrize("M,N,K", [(512, 1024, 512), (1000, 776, 4104)])
def test_gemm_random(M, N, K):
    _say("gemm rand", M, N, K)
    inp = make_ag_inputs(M, N, K, 1, seed=5, dist_a=("normal", 1.0), dist_w=("normal", 0.02))
    A = dev_bits(inp["shards"][0])
    W = dev_bits(inp["W"])
    Cm = torch.zeros((M, N), dtype=torch.int16, device="cuda")
    C.compass_gemm(A, W, Cm)
    torch.cuda.synchronize()
    ref = O.ag_gemm([O.bf16_to_f64(inp["shards"][0])], O.bf16_to_f64(inp["W"]))
    assert rel_err(host_f64(Cm), ref) < TOL


def test_gemm_with_partial_integer_exact():
    M, N, K = 520, 264, 136
    inp = make_int_rs_inputs(M, N, K, 1, seed=3)
    A, W = dev_bits(inp["A"]), dev_bits(inp["W"])
    P = torch.from_numpy(inp["P_in"][0]).cuda()
    Cm = torch.zeros((M, N), dtype=torch.int16, device="cuda")
    C.compass_gemm(A, W, Cm, P)
    torch.cuda.synchronize()
    ref = O.gemm_rs(O.bf16_to_f64(inp["A"]), O.bf16_to_f64(inp["W"]), [inp["P_in"][0].astype(np.float64)], 1)
    assert np.array_equal(host_bits(Cm), O.f64_to_bf16_rne(ref))


# ------------------------------------------------------------ split K (few tiles, deep K)
@pytest.mark.parametrize("with_p", [False, True])
def test_split_k_integer_exact(with_p):
    # 2 x 5 tiles of 128 x 128 against 512 workgroup slots: K = 8192 is split
    M, N, K = 256, 520, 8192
    _say("split-k int", with_p)
    if with_p:
        inp = make_int_rs_inputs(M, N, K, 1, seed=61)
        A, W = dev_bits(inp["A"]), dev_bits(inp["W"])
        P = torch.from_numpy(inp["P_in"][0]).cuda()
        ref = O.gemm_rs(O.bf16_to_f64(inp["A"]), O.bf16_to_f64(inp["W"]), [inp["P_in"][0].astype(np.float64)], 1)
    else:
        inp = make_int_ag_inputs(M, N, K, 1, seed=60)
        A, W = dev_bits(inp["shards"][0]), dev_bits(inp["W"])
        P = None
        ref = O.ag_gemm([O.bf16_to_f64(inp["shards"][0])], O.bf16_to_f64(inp["W"]))
    for rep in range(2):   # the tile counters must be back at zero for the second call
        Cm = torch.zeros((M, N), dtype=torch.int16, device="cuda")
        C.compass_gemm(A, W, Cm, P)
        torch.cuda.synchronize()
        assert np.array_equal(host_bits(Cm), O.f64_to_bf16_rne(ref)), rep


def test_split_k_random_close_to_unsplit():
    M, N, K = 384, 776, 6144
    inp = make_ag_inputs(M, N, K, 1, seed=62, dist_a=("normal", 1.0), dist_w=("normal", 0.02))
    A, W = dev_bits(inp["shards"][0]), dev_bits(inp["W"])
    ref = O.ag_gemm([O.bf16_to_f64(inp["shards"][0])], O.bf16_to_f64(inp["W"]))
    out = {}
    try:
        for sched in (7, 3):   # with and without split K
            C.compass_set_option(C.OPT_SCHED, sched)
            Cm = torch.zeros((M, N), dtype=torch.int16, device="cuda")
            C.compass_gemm(A, W, Cm)
            torch.cuda.synchronize()
            out[sched] = host_f64(Cm)
            assert rel_err(out[sched], ref) < TOL, sched
    finally:
        C.compass_set_option(C.OPT_SCHED, 7)
    # both round the same fp32 sums up to ordering: at most one bf16 ulp apart
    assert rel_err(out[7], out[3]) < 2.0 ** -7


@pytest.mark.parametrize("K,slices", [(2560, 5), (3072, 6), (3584, 7), (4096, 8)])
@pytest.mark.parametrize("partial", [False, True])
def test_split_k_five_to_eight_slices_integer_exact(K, slices, partial):
    # a 256 x 256 plain GEMM is four 128 x 128 tiles on 512 workgroup slots:
    # K splits into as many 512-deep slices as it holds, up to 8, so these
    # depths reach the completing slice's instances for 5 to 8 slices (with
    # the fp32 partial: the ReduceScatter variant's); the tile trace counts
    # the slices
    M, N = 256, 256
    inp = make_int_rs_inputs(M, N, K, 1, seed=70 + slices)
    A, W = dev_bits(inp["A"]), dev_bits(inp["W"])
    prod = O.ag_gemm([O.bf16_to_f64(inp["A"])], O.bf16_to_f64(inp["W"]))
    P = None
    if partial:
        P = torch.from_numpy(np.ascontiguousarray(inp["P_in"][0], dtype=np.float32)).cuda()
        prod = prod + inp["P_in"][0].astype(np.float64)
    ref = O.f64_to_bf16_rne(prod)
    Cm = torch.full((M, N), 0x7FC0, dtype=torch.int16, device="cuda")
    _say("split k slices", slices, partial)
    C.compass_set_option(C.OPT_TILE_TRACE, 1024)
    try:
        C.compass_gemm(A, W, Cm, P)
        torch.cuda.synchronize()
        rec = C.compass_tile_trace(1024)
    finally:
        C.compass_set_option(C.OPT_TILE_TRACE, 0)
    assert len(rec) == 4 * slices
    assert np.array_equal(host_bits(Cm), ref)


def test_decomp_d16_split_integer_exact():
    # sub-GEMMs of 64 rows: one row tile each, K split
    n, d = 8, 16
    M, N, K = 1024, 264, 2048
    inp = make_int_ag_inputs(M, N, K, n, seed=63)
    ref = O.f64_to_bf16_rne(O.decomp_ag([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"]), d))
    case = AGCase(inp, 3, "single")
    _say("decomp d16 split")
    C.compass_decomp_gemm(case.problem, d, FAST)
    C.compass_sync()
    assert np.array_equal(host_bits(case.C), ref)


# ------------------------------------------------------------ fused AllGather+GEMM
@pytest.mark.parametrize("ring", ["single", "double"])
@pytest.mark.parametrize("n", [1, 2, 4, 8, 32])   # 1: nothing to gather; 32 double: 64 partitions, the most
def test_ag_gemm_integer_exact_all_ranks(ring, n):
    M, N, K = 64 * n * (2 if ring == "double" else 1) + 0, 264, 200
    inp = make_int_ag_inputs(M, N, K, n, seed=10 + n)
    ref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"])))
    for r in range(n):
        _say("ag int", ring, n, r, M, N, K)
        case = AGCase(inp, r, ring)
        C.compass_ag_gemm(case.problem, FAST)
        C.compass_sync()
        assert np.array_equal(host_bits(case.C), ref), f"rank {r}"


@pytest.mark.parametrize("rank,ring", [(3, "double"), (6, "single")])
def test_ag_gemm_tail_split_integer_exact(rank, ring):
    # two waves of 256 x 256 tiles at K = 8192: the fused AllGather takes the
    # larger tile, and the tiles of the last two arriving partitions split K
    # (4 slices of 2048, summed in slice order); NaN-filled output, paced 4:1
    n = 8
    M, N, K = 8192, 4096 + 8, 8192
    inp = make_int_ag_inputs(M, N, K, n, seed=31 + rank)
    ref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"])))
    _say("ag tail split", rank, ring, M, N, K)
    case = AGCase(inp, rank, ring)
    case.C.fill_(0x7FC0)
    C.compass_set_option(C.OPT_TILE_TRACE, 8192)
    try:
        C.compass_ag_gemm(case.problem, C.links(400e9, 100e9))
        C.compass_sync()
        rec = C.compass_tile_trace(8192)
    finally:
        C.compass_set_option(C.OPT_TILE_TRACE, 0)
    # 32 x 17 tiles of 256 x 256; the last two row-tile groups (one
    # partition each) split K: double ring, 512-row partitions, 2 x 2 x 17
    # tiles in 4 slices; single ring, 1024-row partitions, 2 x 4 x 17 tiles
    # in 3 slices (the 256 workgroups over a group's 68 tiles). The head:
    # the rank's own chunk, 4 row tiles x 17 = 68 tiles, in 3 slices (the
    # 256 workgroups over 68 tiles)
    extra = 68 * 3 if ring == "double" else 136 * 2
    assert len(rec) == 32 * 17 + extra + 68 * 2
    assert np.array_equal(host_bits(case.C), ref)
    # links unpaced (the engines' ceiling): the transfer is far shorter than
    # the GEMM (estimated comp / comm ratio above 2), so no tile splits
    case.C.fill_(0x7FC0)
    C.compass_set_option(C.OPT_TILE_TRACE, 8192)
    try:
        C.compass_ag_gemm(case.problem, C.links(0.0, 0.0))
        C.compass_sync()
        rec = C.compass_tile_trace(8192)
    finally:
        C.compass_set_option(C.OPT_TILE_TRACE, 0)
    assert len(rec) == 32 * 17
    assert np.array_equal(host_bits(case.C), ref)


def test_ag_gemm_tail_split_128_tiles_option_integer_exact():
    # the tail (and head) split for 128 x 128 tiles (off by default): the fc1
    # shape, the last row-tile group (8 row tiles, the last ring step's two
    # partitions) in 4 K slices of 1024, NaN-filled output
    M, N, K, n = 8192, 2048, 4096, 8
    inp = make_int_ag_inputs(M, N, K, n, seed=41)
    ref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"])))
    _say("ag tail split 128", M, N, K)
    case = AGCase(inp, 2, "double")
    case.C.fill_(0x7FC0)
    try:
        C.compass_set_option(C.OPT_TAIL_MIN_K_128, 4096)
        C.compass_set_option(C.OPT_TAIL_SLICE_K, 1024)
        C.compass_set_option(C.OPT_TAIL_GROUPS, 1)
        C.compass_set_option(C.OPT_TILE_TRACE, 8192)
        C.compass_ag_gemm(case.problem, C.links(200e9, 200e9))
        C.compass_sync()
        rec = C.compass_tile_trace(8192)
    finally:
        C.compass_set_option(C.OPT_TILE_TRACE, 0)
        C.compass_set_option(C.OPT_TAIL_MIN_K_128, 0)
        C.compass_set_option(C.OPT_TAIL_SLICE_K, 2048)
        C.compass_set_option(C.OPT_TAIL_GROUPS, 2)
    # 64 x 16 tiles of 128 x 128; the last group's 8 x 16 tiles in 4 slices,
    # and (the head split, under the same depth gate) the rank's own chunk,
    # one group of 8 x 16 tiles, in 4 slices too
    assert len(rec) == 64 * 16 + 8 * 16 * 3 + 8 * 16 * 3
    assert np.array_equal(host_bits(case.C), ref)


def test_ag_gemm_config1_all_ranks():
    # AllGather-GEMM, TP=2: shards 256x512 U[-1,1], B 512x1024, single ring
    inp = make_ag_inputs(512, 1024, 512, 2, seed=1, dist_a=("uniform", -1.0, 1.0), dist_w=("uniform", -1.0, 1.0))
    for r in range(2):
        _say("config1 rank", r)
        case = AGCase(inp, r, "single")
        C.compass_ag_gemm(case.problem, FAST)
        C.compass_sync()
        assert rel_err(host_f64(case.C), case.reference()) < TOL


@pytest.mark.parametrize("ring", ["single", "double"])
def test_ag_gemm_ragged_multi_tile_pinned_sources(ring):
    # several row tiles per partition, a ragged N and K, remote shards in pinned host memory
    n = 4
    M, N, K = 2048, 776, 1032
    inp = make_ag_inputs(M, N, K, n, seed=77)
    case = AGCase(inp, 1, ring, pinned_remote=True, local_in_place=False)
    _say("ag ragged pinned", ring)
    C.compass_ag_gemm(case.problem, C.links(50e9, 50e9, slice_bytes=1 << 20))
    C.compass_sync()
    assert rel_err(host_f64(case.C), case.reference()) < TOL
    # the gathered buffer holds every shard at its rows, byte for byte
    assert np.array_equal(host_bits(case.gathered), np.vstack(inp["shards"]))


def test_ag_gemm_nan_poison():
    # remote rows start as NaN; a tile read before its partition's flag would
    # carry NaN into C
    n = 8
    M, N, K = 4096, 512, 512
    inp = make_ag_inputs(M, N, K, n, seed=8)
    case = AGCase(inp, 3, "double")
    rows = M // n
    for it in range(3):
        for q in range(n):
            if q != 3:
                case.gathered[q * rows:(q + 1) * rows] = 0x7FC0   # bf16 quiet NaN
        torch.cuda.synchronize()
        _say("nan poison iteration", it)
        C.compass_ag_gemm(case.problem, C.links(20e9, 20e9, slice_bytes=1 << 20))
        C.compass_sync()
        got = host_f64(case.C)
        assert not np.isnan(got).any()
        assert rel_err(got, case.reference()) < TOL


# ------------------------------------------------------------ fused GEMM+ReduceScatter
@pytest.mark.parametrize("ring", ["single", "double"])
@pytest.mark.parametrize("n", [1, 2, 4, 8, 32])   # 32 double: a 128-row tile spans 2 of 64 partitions
def test_gemm_rs_integer_exact(ring, n):
    M, N, K = 128 * n, 264, 136
    inp = make_int_rs_inputs(M, N, K, n, seed=20 + n)
    ref = O.f64_to_bf16_rne(O.gemm_rs(O.bf16_to_f64(inp["A"]), O.bf16_to_f64(inp["W"]),
                                      [p.astype(np.float64) for p in inp["P_in"]], n))
    rows = M // n
    for r in sorted({0, n - 1, n // 2}):
        _say("rs int", ring, n, r)
        case = RSCase(inp, r, ring)
        C.compass_gemm_rs(case.problem, FAST)
        C.compass_sync()
        got = host_bits(case.C)
        assert np.array_equal(got, ref), f"rank {r}"
        for q in range(n):
            if q != r:
                assert np.array_equal(host_bits(case.send[q]), ref[q * rows:(q + 1) * rows]), f"send {q}"


@pytest.mark.parametrize("ring,source", [("single", "device"), ("double", "device"), ("single", "misaligned"),
                                         ("double", "misaligned"), ("single", "pinned")])
def test_gemm_rs_first_step_partial_sources_integer_exact(ring, source):
    # the first ring step's partials (resident from the start): read in place
    # from device memory (rows on tile boundaries), or staged into the landing
    # buffer when a source is not 16-byte aligned or lies in pinned host
    # memory; the landing buffer starts as NaN, so a partial read from the
    # wrong place shows
    n = 4
    M, N, K = 1024, 264, 136
    inp = make_int_rs_inputs(M, N, K, n, seed=98)
    ref = O.f64_to_bf16_rne(O.gemm_rs(O.bf16_to_f64(inp["A"]), O.bf16_to_f64(inp["W"]),
                                      [p.astype(np.float64) for p in inp["P_in"]], n))
    rows = M // n
    r = 2
    _say("rs first-step partials", ring, source)
    case = RSCase(inp, r, ring, pinned_remote=source == "pinned")
    keep = None
    if source == "misaligned":
        # every partial one float into a larger buffer: 4-byte but not 16-byte aligned
        keep = [torch.empty(rows * N + 4, dtype=torch.float32, device="cuda") for _ in range(n)]
        for c in range(n):
            keep[c][1:1 + rows * N].copy_(case.partials[c].reshape(-1))
        case.partials = [keep[c][1:1 + rows * N].view(rows, N) for c in range(n)]
        case.problem = C.rs_problem(case.A, case.W, case.partials, case.stage, case.C, case.send, r, ring)
    case.stage.fill_(float("nan"))
    torch.cuda.synchronize()
    C.compass_gemm_rs(case.problem, C.links(40e9, 10e9, slice_bytes=1 << 18))
    C.compass_sync()
    assert np.array_equal(host_bits(case.C), ref)
    for q in range(n):
        if q != r:
            assert np.array_equal(host_bits(case.send[q]), ref[q * rows:(q + 1) * rows]), f"send {q}"


@pytest.mark.parametrize("ring", ["single", "double"])
def test_gemm_rs_pinned_host_partials_and_sends_integer_exact(ring):
    # every remote buffer of the ReduceScatter in pinned host memory: the
    # incoming partials (the first step's staged, the others copied by the
    # engines across PCIe) and every chunk sent on
    n = 4
    M, N, K = 1024, 264, 136
    inp = make_int_rs_inputs(M, N, K, n, seed=99)
    ref = O.f64_to_bf16_rne(O.gemm_rs(O.bf16_to_f64(inp["A"]), O.bf16_to_f64(inp["W"]),
                                      [p.astype(np.float64) for p in inp["P_in"]], n))
    rows = M // n
    r = 1
    _say("rs pinned partials and sends", ring)
    case = RSCase(inp, r, ring, pinned_remote=True)
    case.send = [None if q == r else torch.zeros((rows, N), dtype=torch.int16, pin_memory=True) for q in range(n)]
    case.problem = C.rs_problem(case.A, case.W, case.partials, case.stage, case.C, case.send, r, ring)
    C.compass_gemm_rs(case.problem, C.links(40e9, 10e9, slice_bytes=1 << 18))
    C.compass_sync()
    assert np.array_equal(host_bits(case.C), ref)
    for q in range(n):
        if q != r:
            assert np.array_equal(case.send[q].numpy().view(np.uint16), ref[q * rows:(q + 1) * rows]), f"send {q}"


def test_gemm_rs_random_ragged_no_sends():
    n = 4
    M, N, K = 1024, 776, 1032
    inp = make_rs_inputs(M, N, K, n, seed=31)
    case = RSCase(inp, 2, "single", sends=False)
    _say("rs ragged")
    C.compass_gemm_rs(case.problem, FAST)
    C.compass_sync()
    assert rel_err(host_f64(case.C), case.reference()) < TOL


# ------------------------------------------------------------ InterDecom
@pytest.mark.parametrize("ring", ["single", "double"])
@pytest.mark.parametrize("d", [1, 2, 4, 8])
def test_decomp_ag_integer_exact(ring, d):
    n = 4
    M, N, K = 1024, 264, 136
    inp = make_int_ag_inputs(M, N, K, n, seed=40 + d)
    ref = O.f64_to_bf16_rne(O.decomp_ag([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"]), d))
    case = AGCase(inp, 1, ring)
    _say("decomp ag", ring, d)
    C.compass_decomp_gemm(case.problem, d, FAST)
    C.compass_sync()
    assert np.array_equal(host_bits(case.C), ref)


@pytest.mark.parametrize("ring", ["single", "double"])
@pytest.mark.parametrize("d", [1, 2, 4])
def test_decomp_rs_integer_exact(d, ring):
    # double ring, d > 1: the resident partitions' partials are staged piece by piece
    n = 4
    M, N, K = 1024, 264, 136
    inp = make_int_rs_inputs(M, N, K, n, seed=50 + d)
    ref = O.f64_to_bf16_rne(O.decomp_rs(O.bf16_to_f64(inp["A"]), O.bf16_to_f64(inp["W"]),
                                        [p.astype(np.float64) for p in inp["P_in"]], n, d))
    case = RSCase(inp, 0, ring)
    _say("decomp rs", d, ring)
    C.compass_decomp_gemm(case.problem, d, FAST)
    C.compass_sync()
    got = host_bits(case.C)
    assert np.array_equal(got, ref)
    rows = M // n
    for q in range(1, n):
        assert np.array_equal(host_bits(case.send[q]), ref[q * rows:(q + 1) * rows])


def test_decomp_rejects_bad_degree():
    inp = make_int_ag_inputs(512, 64, 64, 4, seed=1)
    case = AGCase(inp, 0, "single")
    with pytest.raises(C.CompassError) as e:
        C.compass_decomp_gemm(case.problem, 3, FAST)
    assert e.value.code == C.ERR_INVALID


# ------------------------------------------------------------ measurement companions
def test_transfer_moves_every_shard():
    n = 8
    M, N, K = 2048, 256, 512
    inp = make_ag_inputs(M, N, K, n, seed=60)
    case = AGCase(inp, 5, "double")
    _say("transfer ag")
    C.compass_transfer(case.problem, FAST)
    C.compass_sync()
    assert np.array_equal(host_bits(case.gathered), np.vstack(inp["shards"]))


def test_sequential_ag_and_rs():
    n = 4
    inp = make_ag_inputs(1024, 264, 200, n, seed=61)
    case = AGCase(inp, 2, "double")
    _say("sequential ag")
    C.compass_sequential(case.problem, FAST)
    C.compass_sync()
    assert rel_err(host_f64(case.C), case.reference()) < TOL
    rinp = make_rs_inputs(1024, 264, 200, n, seed=62)
    rcase = RSCase(rinp, 1, "single")
    # the sequential ReduceScatter's epilogue reads the staged partials as they
    # are at launch: stage them with a transfer first
    C.compass_transfer(rcase.problem, FAST)
    C.compass_sync()
    _say("sequential rs")
    C.compass_sequential(rcase.problem, FAST)
    C.compass_sync()
    assert rel_err(host_f64(rcase.C), rcase.reference()) < TOL


# ------------------------------------------------------------ failure handling
def test_never_arriving_partition_times_out_then_recovers():
    n = 4
    inp = make_ag_inputs(1024, 256, 256, n, seed=70)
    case = AGCase(inp, 0, "single")
    C.compass_set_option(C.OPT_SPIN_LIMIT, 20000)
    C.compass_set_option(C.OPT_DROP_FLAG, 2)
    try:
        _say("timeout case")
        C.compass_ag_gemm(case.problem, FAST)
        with pytest.raises(C.CompassError) as e:
            C.compass_sync()
        assert e.value.code == C.ERR_TIMEOUT
    finally:
        C.compass_set_option(C.OPT_DROP_FLAG, -1)
        C.compass_set_option(C.OPT_SPIN_LIMIT, 4 << 20)
    _say("recovery case")
    C.compass_ag_gemm(case.problem, FAST)
    C.compass_sync()
    assert rel_err(host_f64(case.C), case.reference()) < TOL


def test_invalid_shapes_rejected_before_enqueue():
    inp = make_int_ag_inputs(96, 64, 64, 4, seed=1)
    case = AGCase(inp, 0, "single")
    st = case.problem.st
    st.K = 60   # not a multiple of 8
    with pytest.raises(C.CompassError) as e:
        C.compass_ag_gemm(case.problem, FAST)
    assert e.value.code == C.ERR_INVALID
    st.K = 64
    st.rank = 7
    with pytest.raises(C.CompassError):
        C.compass_ag_gemm(case.problem, FAST)


# ------------------------------------------------------------ both tile configurations
@pytest.fixture
def tile_cfg(request):
    C.compass_set_option(C.OPT_TILE, request.param)
    yield request.param
    C.compass_set_option(C.OPT_TILE, 0)


@pytest.mark.parametrize("tile_cfg", [1, 2], indirect=True)
def test_tile_configs_integer_exact(tile_cfg):
    # plain, fused AllGather, fused ReduceScatter and InterDecom under one tile shape
    _say("tile cfg", tile_cfg)
    M, N, K = 1600, 520, 328
    inp = make_int_ag_inputs(M, N, K, 1, seed=90)
    A, W = dev_bits(inp["shards"][0]), dev_bits(inp["W"])
    Cm = torch.zeros((M, N), dtype=torch.int16, device="cuda")
    C.compass_gemm(A, W, Cm)
    torch.cuda.synchronize()
    ref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(inp["shards"][0])], O.bf16_to_f64(inp["W"])))
    assert np.array_equal(host_bits(Cm), ref)
    n = 8
    ag = make_int_ag_inputs(2048, 264, 200, n, seed=91)
    agref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(s) for s in ag["shards"]], O.bf16_to_f64(ag["W"])))
    for ring in ["single", "double"]:
        case = AGCase(ag, 5, ring)
        C.compass_ag_gemm(case.problem, FAST)
        C.compass_sync()
        assert np.array_equal(host_bits(case.C), agref), ring
        case = AGCase(ag, 2, ring)
        C.compass_decomp_gemm(case.problem, 4, FAST)
        C.compass_sync()
        assert np.array_equal(host_bits(case.C), agref), ring
    rs = make_int_rs_inputs(2048, 264, 136, n, seed=92)
    rsref = O.f64_to_bf16_rne(O.gemm_rs(O.bf16_to_f64(rs["A"]), O.bf16_to_f64(rs["W"]),
                                        [p.astype(np.float64) for p in rs["P_in"]], n))
    for ring in ["single", "double"]:
        case = RSCase(rs, 3, ring)
        C.compass_gemm_rs(case.problem, FAST)
        C.compass_sync()
        assert np.array_equal(host_bits(case.C), rsref), ring
        rows = 2048 // n
        for q in range(n):
            if q != 3:
                assert np.array_equal(host_bits(case.send[q]), rsref[q * rows:(q + 1) * rows])


# ------------------------------------------------------------ per-launch kernel timing
def test_kernel_times_one_per_launch():
    _say("kernel times")
    M, N, K = 1024, 512, 256
    inp = make_int_ag_inputs(M, N, K, 1, seed=93)
    A, W = dev_bits(inp["shards"][0]), dev_bits(inp["W"])
    Cm = torch.zeros((M, N), dtype=torch.int16, device="cuda")
    with pytest.raises(C.CompassError):
        C.compass_kernel_times()          # not enabled
    C.compass_set_option(C.OPT_KERNEL_TIMING, 1)
    try:
        C.compass_gemm(A, W, Cm)
        C.compass_gemm(A, W, Cm)
        ag = make_int_ag_inputs(2048, 264, 200, 8, seed=94)
        case = AGCase(ag, 1, "double")
        C.compass_decomp_gemm(case.problem, 4, FAST)
        C.compass_sync()
        t = C.compass_kernel_times()
        assert len(t) == 2 + 4
        assert all(0.0 < x < 1e6 for x in t)
        assert C.compass_kernel_times() == []   # reading resets
    finally:
        C.compass_set_option(C.OPT_KERNEL_TIMING, 0)


# ------------------------------------------------------------ matrix-core probe
def test_probe_mfma_reports_a_plausible_rate_and_clock():
    _say("matrix-core probe")
    with pytest.raises(C.CompassError):
        C.compass_probe_mfma(0)
    C.compass_probe_mfma(256)
    tf, ghz = C.compass_probe_mfma(8192)
    # bounded by the nominal bf16 peak at the maximum clock (2.4 GHz)
    assert 100.0 < tf < 2516.6 * 1.02, tf
    assert 0.5 < ghz < 2.5, ghz


# ------------------------------------------------------------ paced links and the tile trace
def test_pacing_headroom_and_an_unreachable_rate():
    # the headroom option's range; a rate no group of engines can carry (tiny
    # items at 1 TB/s per ring) runs one engine per item and lands every
    # partition, not far behind the unpaced transfer; any headroom delivers
    for bad in (-1, 101):
        with pytest.raises(C.CompassError):
            C.compass_set_option(C.OPT_PACE_HEADROOM, bad)
    n = 8
    M, N, K = 4096, 64, 1024
    inp = make_ag_inputs(M, N, K, n, seed=65)
    case = AGCase(inp, 5, "double")
    fast, unpaced = C.links(1e12, 1e12), C.links(0.0, 0.0)

    def best(lk):
        C.compass_transfer(case.problem, lk)   # warm
        C.compass_sync()
        t = []
        for _ in range(3):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            C.compass_transfer(case.problem, lk)
            b.record()
            b.synchronize()
            C.compass_sync()
            t.append(a.elapsed_time(b) * 1e-3)
        return min(t)

    try:
        for h in (0, 5, 100):
            C.compass_set_option(C.OPT_PACE_HEADROOM, h)
            rows = M // n   # clear the remote rows (the local shard stays in place)
            case.gathered.zero_()
            case.gathered[5 * rows:6 * rows] = dev_bits(inp["shards"][5])
            t_fast = best(fast)
            assert np.array_equal(host_bits(case.gathered), np.vstack(inp["shards"])), h
        t_unpaced = best(unpaced)
        _say("unreachable rate", t_fast, "unpaced", t_unpaced)
        assert t_fast < 2.0 * t_unpaced + 1e-3
    finally:
        C.compass_set_option(C.OPT_PACE_HEADROOM, 5)


def test_paced_link_never_beats_its_rate():
    # 7 items of 512 KiB per ring direction at 20 GB/s: the last flag is due
    # after 7 * 512 KiB / rate, and a paced link publishes none earlier
    n = 8
    M, N, K = 4096, 64, 1024
    inp = make_ag_inputs(M, N, K, n, seed=64)
    case = AGCase(inp, 2, "double")
    rate = 20e9
    lk = C.links(rate, rate)
    C.compass_transfer(case.problem, lk)   # warm
    C.compass_sync()
    per_ring = (n - 1) * (M // (2 * n)) * K * 2
    times = []
    for _ in range(3):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        C.compass_transfer(case.problem, lk)
        b.record()
        b.synchronize()
        C.compass_sync()
        times.append(a.elapsed_time(b) * 1e-3)
    _say("paced transfer", times, per_ring / rate)
    assert min(times) >= 0.98 * per_ring / rate      # no call beats the rate
    # and pacing is not grossly slow (the best of three, so that one late
    # wake-up of the host pacer thread does not decide)
    assert min(times) < 3.0 * per_ring / rate + 2e-3
    assert np.array_equal(host_bits(case.gathered), np.vstack(inp["shards"]))


def test_tile_trace_records_every_work_item():
    M, N, K = 512, 384, 4096          # 4 x 3 tiles of 128 x 128, K split
    inp = make_int_ag_inputs(M, N, K, 1, seed=65)
    A, W = dev_bits(inp["shards"][0]), dev_bits(inp["W"])
    Cm = torch.zeros((M, N), dtype=torch.int16, device="cuda")
    C.compass_set_option(C.OPT_TILE_TRACE, 4096)
    try:
        C.compass_gemm(A, W, Cm)
        rec = C.compass_tile_trace(4096)
    finally:
        C.compass_set_option(C.OPT_TILE_TRACE, 0)
    assert len(rec) >= 12 and len(rec) % 12 == 0          # tiles x K slices
    assert sorted(rec[:, 0].tolist()) == list(range(len(rec)))
    t = rec[:, 4:8].astype(np.int64)
    d = (t[:, 1:] - t[:, :-1]) % (1 << 32)                  # ticket <= gate <= loop <= end
    assert (d < (1 << 31)).all()
    ref = O.ag_gemm([O.bf16_to_f64(inp["shards"][0])], O.bf16_to_f64(inp["W"]))
    assert np.array_equal(host_bits(Cm), O.f64_to_bf16_rne(ref))


# ------------------------------------------------------------ double ring split by link rate
SPLIT_4_TO_1 = C.links(200e9, 50e9)


def test_ag_gemm_proportional_double_ring_integer_exact():
    # 1024 rows per chunk at 4 : 1 -> 208 rows on the backward ring, 816 forward
    n = 4
    M, N, K = 4096, 264, 200
    inp = make_int_ag_inputs(M, N, K, n, seed=81)
    ref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"])))
    for r in range(n):
        for lk in (SPLIT_4_TO_1, C.links(0.0, 0.0)):   # unpaced: halves
            _say("ag split", r, lk.fwd_Bps)
            case = AGCase(inp, r, "double_split")
            C.compass_ag_gemm(case.problem, lk)
            C.compass_sync()
            assert np.array_equal(host_bits(case.C), ref), f"rank {r}"
            assert np.array_equal(host_bits(case.gathered), np.vstack(inp["shards"]))


def test_gemm_rs_proportional_double_ring_integer_exact():
    n = 4
    M, N, K = 1024, 264, 136
    inp = make_int_rs_inputs(M, N, K, n, seed=82)
    ref = O.f64_to_bf16_rne(O.gemm_rs(O.bf16_to_f64(inp["A"]), O.bf16_to_f64(inp["W"]),
                                      [p.astype(np.float64) for p in inp["P_in"]], n))
    rows = M // n
    for r in range(n):
        _say("rs split", r)
        case = RSCase(inp, r, "double_split")
        C.compass_gemm_rs(case.problem, SPLIT_4_TO_1)
        C.compass_sync()
        assert np.array_equal(host_bits(case.C), ref), f"rank {r}"
        for q in range(n):
            if q != r:
                assert np.array_equal(host_bits(case.send[q]), ref[q * rows:(q + 1) * rows]), f"send {q}"


@pytest.mark.parametrize("pattern", ["ag", "rs"])
@pytest.mark.parametrize("d", [1, 2, 4])
def test_decomp_proportional_double_ring_integer_exact(pattern, d):
    n = 4
    if pattern == "ag":
        inp = make_int_ag_inputs(2048, 136, 200, n, seed=83)
        ref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"])))
        case = AGCase(inp, 1, "double_split")
    else:
        inp = make_int_rs_inputs(2048, 136, 136, n, seed=84)
        ref = O.f64_to_bf16_rne(O.gemm_rs(O.bf16_to_f64(inp["A"]), O.bf16_to_f64(inp["W"]),
                                          [p.astype(np.float64) for p in inp["P_in"]], n))
        case = RSCase(inp, 1, "double_split")
    _say("decomp split", pattern, d)
    C.compass_decomp_gemm(case.problem, d, SPLIT_4_TO_1)
    C.compass_sync()
    assert np.array_equal(host_bits(case.C), ref)


def test_proportional_split_shortens_a_4_to_1_transfer():
    # 7 steps of one 4 MiB chunk: halves wait 7 x 2 MiB on the 50 GB/s ring
    # (~294 us); the split finishes both rings after 7 x 4 MiB / 250 GB/s (~117 us)
    n = 8
    inp = make_ag_inputs(4096, 64, 4096, n, seed=85)
    t = {}
    for ring in ("double", "double_split"):
        case = AGCase(inp, 0, ring)
        C.compass_transfer(case.problem, SPLIT_4_TO_1)
        C.compass_sync()
        times = []
        for _ in range(3):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            C.compass_transfer(case.problem, SPLIT_4_TO_1)
            b.record()
            b.synchronize()
            C.compass_sync()
            times.append(a.elapsed_time(b) * 1e-3)
        t[ring] = min(times)
    _say("transfer halves / split", t)
    assert t["double_split"] < 0.75 * t["double"]


# ------------------------------------------------------------ AlltoAll pattern (Section III-A)
NUMA = C.links(200e9, 40e9)    # own-domain links, shared cross-domain link


@pytest.mark.parametrize("n", [2, 4, 8])
@pytest.mark.parametrize("paced", [True, False])
def test_ag_gemm_alltoall_integer_exact_all_ranks(n, paced):
    M, N, K = 64 * n, 264, 200
    inp = make_int_ag_inputs(M, N, K, n, seed=90 + n)
    ref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"])))
    for r in range(n):
        _say("ag alltoall int", n, r, paced)
        case = AGCase(inp, r, "alltoall")
        C.compass_ag_gemm(case.problem, NUMA if paced else C.links(0.0, 0.0))
        C.compass_sync()
        assert np.array_equal(host_bits(case.C), ref), f"rank {r}"
        assert np.array_equal(host_bits(case.gathered), np.vstack(inp["shards"]))


def test_alltoall_sequential_and_transfer():
    n = 8
    inp = make_ag_inputs(1024, 520, 1032, n, seed=93)
    case = AGCase(inp, 5, "alltoall")
    _say("alltoall sequential")
    C.compass_sequential(case.problem, NUMA)
    C.compass_sync()
    assert rel_err(host_f64(case.C), case.reference()) < TOL
    case = AGCase(inp, 3, "alltoall")
    C.compass_transfer(case.problem, NUMA)
    C.compass_sync()
    assert np.array_equal(host_bits(case.gathered), np.vstack(inp["shards"]))


def test_alltoall_transfer_is_about_half_the_single_ring_across_numa():
    # n = 8, 4 MiB chunks, cross-domain rate B = 40 GB/s: the single ring
    # takes 7 steps at B (~734 us); under AlltoAll the 16 flows into a
    # domain share B and land after 16 x 4 MiB / B (~1678 us), and none
    # earlier
    n = 8
    inp = make_ag_inputs(4096, 64, 4096, n, seed=94)
    chunk = 4096 // n * 4096 * 2
    B = 40e9
    t = {}
    for ring, lk in (("single", C.links(B, B)), ("alltoall", C.links(200e9, B))):
        case = AGCase(inp, 0, ring)
        C.compass_transfer(case.problem, lk)
        C.compass_sync()
        times = []
        for _ in range(3):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            C.compass_transfer(case.problem, lk)
            b.record()
            b.synchronize()
            C.compass_sync()
            times.append(a.elapsed_time(b) * 1e-3)
        t[ring] = min(times)
        assert np.array_equal(host_bits(case.gathered), np.vstack(inp["shards"]))
    _say("single ring / alltoall", t)
    assert t["alltoall"] >= 0.98 * 16 * chunk / B
    assert t["single"] >= 0.98 * 7 * chunk / B
    assert 0.3 < t["single"] / t["alltoall"] < 0.6     # model: (1/2) / (8/7) = 0.4375


# ------------------------------------------------------------ single ring with per-hop rates (Section III-A)
def _cross_numa_hops(n, slow, fast):
    # hops n/2-1 -> n/2 and n-1 -> 0 cross the NUMA boundary
    return [slow if q in (n // 2 - 1, n - 1) else fast for q in range(n)]


@pytest.mark.parametrize("n", [2, 4, 8])
def test_ag_gemm_hop_ring_integer_exact_all_ranks(n):
    M, N, K = 64 * n, 264, 200
    inp = make_int_ag_inputs(M, N, K, n, seed=110 + n)
    ref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"])))
    lk = C.links(100e9, hop_Bps=_cross_numa_hops(n, 10e9, 100e9))
    for r in range(n):
        _say("ag hop ring int", n, r)
        case = AGCase(inp, r, "single")
        C.compass_ag_gemm(case.problem, lk)
        C.compass_sync()
        assert np.array_equal(host_bits(case.C), ref), f"rank {r}"
        for d in (2, 4):
            case.C.zero_()
            C.compass_decomp_gemm(case.problem, d, lk)
            C.compass_sync()
            assert np.array_equal(host_bits(case.C), ref), f"rank {r} d {d}"


@pytest.mark.parametrize("n", [4, 8])
def test_gemm_rs_hop_ring_integer_exact_all_ranks(n):
    M, N, K = 64 * n, 136, 128
    inp = make_int_rs_inputs(M, N, K, n, seed=120 + n)
    ref = O.f64_to_bf16_rne(O.gemm_rs(O.bf16_to_f64(inp["A"]), O.bf16_to_f64(inp["W"]),
                                      [p.astype(np.float64) for p in inp["P_in"]], n))
    lk = C.links(100e9, hop_Bps=_cross_numa_hops(n, 10e9, 100e9))
    prow = M // n
    for r in range(n):
        _say("rs hop ring int", n, r)
        case = RSCase(inp, r, "single")
        C.compass_gemm_rs(case.problem, lk)
        C.compass_sync()
        got = host_bits(case.C)
        assert np.array_equal(got, ref), f"rank {r}"
        for q, snd in enumerate(case.send):
            if snd is not None:
                assert np.array_equal(host_bits(snd), ref[q * prow:(q + 1) * prow]), (r, q)


def test_hop_ring_transfer_follows_the_per_rank_arrival_times():
    # n = 8, 4 MiB chunks, hops 3->4 and 7->0 at 20 GB/s, the rest at 200 GB/s:
    # rank 0 (after a slow hop) waits 7 x 4 MiB / 20 GB/s; rank 3, three fast
    # hops downstream of one, finishes after 4 slow and 3 fast chunk times
    n = 8
    inp = make_ag_inputs(4096, 64, 4096, n, seed=125)
    chunk = 4096 // n * 4096 * 2
    hops = _cross_numa_hops(n, 20e9, 200e9)
    lk = C.links(200e9, hop_Bps=hops)
    t = {}
    for r in (0, 3):
        case = AGCase(inp, r, "single")
        C.compass_transfer(case.problem, lk)
        C.compass_sync()
        times = []
        for _ in range(3):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            C.compass_transfer(case.problem, lk)
            b.record()
            b.synchronize()
            C.compass_sync()
            times.append(a.elapsed_time(b) * 1e-3)
        t[r] = min(times)
        want = O.ring_arrival_times(n, r, chunk, hops)[-1]
        _say("hop ring rank", r, "transfer", t[r], "due", want)
        assert t[r] >= 0.98 * want
        assert t[r] < 1.25 * want + 1e-3
        assert np.array_equal(host_bits(case.gathered), np.vstack(inp["shards"]))
    assert t[3] < 0.8 * t[0]


@pytest.mark.parametrize("ring", ["alltoall", "single_hops"])
def test_ag_gemm_ragged_multi_tile_pinned_sources_numa_links(ring):
    # several row tiles per chunk, a ragged N and K, remote shards in pinned
    # host memory, over the two cross-NUMA link patterns
    n = 4
    M, N, K = 2048, 776, 1032
    inp = make_ag_inputs(M, N, K, n, seed=131)
    if ring == "alltoall":
        case, lk = AGCase(inp, 2, "alltoall", pinned_remote=True, local_in_place=False), C.links(50e9, 20e9)
    else:
        case = AGCase(inp, 2, "single", pinned_remote=True, local_in_place=False)
        lk = C.links(50e9, hop_Bps=_cross_numa_hops(n, 20e9, 50e9))
    _say("ag ragged pinned", ring)
    C.compass_ag_gemm(case.problem, lk)
    C.compass_sync()
    assert rel_err(host_f64(case.C), case.reference()) < TOL
    assert np.array_equal(host_bits(case.gathered), np.vstack(inp["shards"]))


@pytest.mark.parametrize("d", [2, 4])
def test_decomp_rs_hop_ring_integer_exact(d):
    n = 8
    M, N, K = 128 * n, 136, 256
    inp = make_int_rs_inputs(M, N, K, n, seed=140 + d)
    ref = O.f64_to_bf16_rne(O.gemm_rs(O.bf16_to_f64(inp["A"]), O.bf16_to_f64(inp["W"]),
                                      [p.astype(np.float64) for p in inp["P_in"]], n))
    lk = C.links(100e9, hop_Bps=_cross_numa_hops(n, 10e9, 100e9))
    prow = M // n
    for r in (0, 3):
        _say("rs decomp hop ring", d, r)
        case = RSCase(inp, r, "single")
        C.compass_decomp_gemm(case.problem, d, lk)
        C.compass_sync()
        assert np.array_equal(host_bits(case.C), ref), f"rank {r}"
        for q, snd in enumerate(case.send):
            if snd is not None:
                assert np.array_equal(host_bits(snd), ref[q * prow:(q + 1) * prow]), (r, q)


# ------------------------------------------------------------ sub-chunk arrival flags
@pytest.mark.parametrize("ring", ["single", "double", "double_split"])
@pytest.mark.parametrize("sub", [2, 4])
def test_ag_gemm_sub_chunks_integer_exact_all_ranks(ring, sub):
    n = 8
    M, N, K = 64 * 2 * n, 264, 200
    inp = make_int_ag_inputs(M, N, K, n, seed=150 + sub)
    ref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"])))
    for lk in (C.links(200e9, 50e9, sub_chunks=sub), C.links(0.0, 0.0, sub_chunks=sub)):
        for r in range(n):
            _say("ag sub-chunks int", ring, sub, r, lk.fwd_Bps)
            case = AGCase(inp, r, ring)
            C.compass_ag_gemm(case.problem, lk)
            C.compass_sync()
            assert np.array_equal(host_bits(case.C), ref), f"rank {r}"


@pytest.mark.parametrize("ring", ["single", "double", "double_split"])
@pytest.mark.parametrize("sub", [2, 4])
def test_gemm_rs_sub_chunks_integer_exact(ring, sub):
    n = 8
    M, N, K = 128 * n, 264, 136
    inp = make_int_rs_inputs(M, N, K, n, seed=160 + sub)
    ref = O.f64_to_bf16_rne(O.gemm_rs(O.bf16_to_f64(inp["A"]), O.bf16_to_f64(inp["W"]),
                                      [p.astype(np.float64) for p in inp["P_in"]], n))
    rows = M // n
    for lk in (C.links(200e9, 50e9, sub_chunks=sub), C.links(0.0, 0.0, sub_chunks=sub)):
        for r in (0, 5):
            _say("rs sub-chunks int", ring, sub, r, lk.fwd_Bps)
            case = RSCase(inp, r, ring)
            C.compass_gemm_rs(case.problem, lk)
            C.compass_sync()
            assert np.array_equal(host_bits(case.C), ref), f"rank {r}"
            for q in range(n):
                if q != r:
                    assert np.array_equal(host_bits(case.send[q]), ref[q * rows:(q + 1) * rows]), f"send {q}"


def test_sub_chunks_sequential_transfer_and_decomp_d1():
    n = 4
    inp = make_int_ag_inputs(512, 136, 264, n, seed=171)
    ref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"])))
    lk = C.links(100e9, 100e9, sub_chunks=4)
    for call in ("sequential", "decomp1", "transfer"):
        _say("sub-chunks", call)
        case = AGCase(inp, 1, "double")
        if call == "sequential":
            C.compass_sequential(case.problem, lk)
        elif call == "decomp1":
            C.compass_decomp_gemm(case.problem, 1, lk)
        else:
            C.compass_transfer(case.problem, lk)
        C.compass_sync()
        assert np.array_equal(host_bits(case.gathered), np.vstack(inp["shards"]))
        if call != "transfer":
            assert np.array_equal(host_bits(case.C), ref)
    rin = make_int_rs_inputs(512, 136, 264, n, seed=172)
    rref = O.f64_to_bf16_rne(O.gemm_rs(O.bf16_to_f64(rin["A"]), O.bf16_to_f64(rin["W"]),
                                       [p.astype(np.float64) for p in rin["P_in"]], n))
    case = RSCase(rin, 2, "single")
    # the unfused ReduceScatter's epilogue reads the staged partials as they
    # are at launch: stage them with a transfer first
    C.compass_transfer(case.problem, lk)
    C.compass_sync()
    C.compass_sequential(case.problem, lk)
    C.compass_sync()
    assert np.array_equal(host_bits(case.C), rref)


# ------------------------------------------------------------ unpaced directions sharing the copy engines
@pytest.fixture
def pool_depth(request):
    C.compass_set_option(C.OPT_POOL, request.param)
    yield request.param
    C.compass_set_option(C.OPT_POOL, 4)


UNPACED = C.links(0.0, 0.0, slice_bytes=64 << 10)   # small slices: several per item


@pytest.mark.parametrize("pool_depth", [0, 1, 4], indirect=True)
@pytest.mark.parametrize("ring", ["double", "double_split"])
def test_pooled_ag_gemm_integer_exact_all_ranks(pool_depth, ring):
    for bad in (-1, 9):
        with pytest.raises(C.CompassError):
            C.compass_set_option(C.OPT_POOL, bad)
    n = 8
    inp = make_int_ag_inputs(2048, 264, 328, n, seed=181)
    ref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"])))
    for rank in range(n):
        _say("pooled ag", pool_depth, ring, rank)
        case = AGCase(inp, rank, ring, pinned_remote=rank % 2 == 1)
        C.compass_ag_gemm(case.problem, UNPACED)
        C.compass_sync()
        assert np.array_equal(host_bits(case.C), ref), rank
    for d in (2, 4):
        case = AGCase(inp, 3, ring)
        C.compass_decomp_gemm(case.problem, d, UNPACED)
        C.compass_sync()
        assert np.array_equal(host_bits(case.C), ref), d


@pytest.mark.parametrize("pool_depth", [0, 1, 4], indirect=True)
@pytest.mark.parametrize("ring", ["single", "double"])
def test_pooled_gemm_rs_with_sends_integer_exact(pool_depth, ring):
    # the incoming partials and the gated outgoing sums in one pooled job:
    # every chunk sum and every sent chunk bit-exact, on every rank, fused and
    # through InterDecom; then the unfused operator and the transfer alone
    n = 8
    rin = make_int_rs_inputs(2048, 264, 136, n, seed=182)
    rref = O.f64_to_bf16_rne(O.gemm_rs(O.bf16_to_f64(rin["A"]), O.bf16_to_f64(rin["W"]),
                                       [p.astype(np.float64) for p in rin["P_in"]], n))
    rows = 2048 // n

    def check(case, tag):
        assert np.array_equal(host_bits(case.C), rref), tag
        for q in range(n):
            if q != case.rank:
                assert np.array_equal(host_bits(case.send[q]), rref[q * rows:(q + 1) * rows]), (tag, q)

    for rank in range(n):
        _say("pooled rs", pool_depth, ring, rank)
        case = RSCase(rin, rank, ring)
        C.compass_gemm_rs(case.problem, UNPACED)
        C.compass_sync()
        check(case, ("fused", rank))
    for d in (2, 4):
        case = RSCase(rin, 5, ring)
        C.compass_decomp_gemm(case.problem, d, UNPACED)
        C.compass_sync()
        check(case, ("decomp", d))
    case = RSCase(rin, 6, ring)
    C.compass_transfer(case.problem, UNPACED)   # stages the partials for the unfused epilogue
    C.compass_sync()
    C.compass_sequential(case.problem, UNPACED)
    C.compass_sync()
    check(case, "sequential")


@pytest.mark.parametrize("pool_depth", [0, 4], indirect=True)
def test_copy_side_timeout_then_recovers(pool_depth):
    # a copy-side wait bound of 1 us: the ReduceScatter's copy side gives up
    # between its first copies and their landing (or at a chunk-done gate),
    # lets the copies it issued land, and the kernel then times out on the
    # partials whose flags never come. compass_sync reports the timeout; the
    # next call, with the bounds restored, is bit-exact, sends included
    n = 4
    rin = make_int_rs_inputs(1024, 264, 136, n, seed=190)
    rref = O.f64_to_bf16_rne(O.gemm_rs(O.bf16_to_f64(rin["A"]), O.bf16_to_f64(rin["W"]),
                                       [p.astype(np.float64) for p in rin["P_in"]], n))
    rows = 1024 // n
    C.compass_set_option(C.OPT_SPIN_LIMIT, 20000)
    C.compass_set_option(C.OPT_HOST_TIMEOUT, 1)
    try:
        _say("copy-side timeout case", pool_depth)
        case = RSCase(rin, 1, "double")
        C.compass_gemm_rs(case.problem, UNPACED)
        with pytest.raises(C.CompassError) as e:
            C.compass_sync()
        assert e.value.code == C.ERR_TIMEOUT
    finally:
        C.compass_set_option(C.OPT_HOST_TIMEOUT, 5_000_000)
        C.compass_set_option(C.OPT_SPIN_LIMIT, 4 << 20)
    _say("copy-side recovery case", pool_depth)
    case = RSCase(rin, 1, "double")
    C.compass_gemm_rs(case.problem, UNPACED)
    C.compass_sync()
    assert np.array_equal(host_bits(case.C), rref)
    for q in range(n):
        if q != 1:
            assert np.array_equal(host_bits(case.send[q]), rref[q * rows:(q + 1) * rows]), q


# ------------------------------------------------------------ operands beyond 1 / 2 GiB
def test_gemm_rs_two_gib_partial_integer_exact():
    # Table IV's largest ReduceScatter output, one TP = 4 rank's share (M =
    # 32768 tokens, hidden 16384): a 2 GiB fp32 landing buffer and a 1 GiB
    # output; row offsets of the partial pass 2^31 bytes
    n = 4
    M, N, K = 32768, 16384, 1024
    _say("rs 2 GiB partial", M, N, K)
    inp = make_int_rs_inputs(M, N, K, n, seed=2048)
    case = RSCase(inp, 1, "single")
    case.C.fill_(0x7FC0)
    C.compass_gemm_rs(case.problem, C.links(0.0, 0.0))
    C.compass_sync()
    ref = O.f64_to_bf16_rne(case.reference())
    assert np.array_equal(host_bits(case.C), ref)
    rows = M // n
    for q in range(n):
        if q != 1:
            assert torch.equal(case.send[q], case.C[q * rows:(q + 1) * rows]), q


def test_ag_gemm_gathered_above_one_gib_integer_exact():
    # a gathered A of 32768 x 20480 bf16 (1.34 GB) over a paced double ring
    n = 8
    M, N, K = 32768, 264, 20480
    _say("ag gathered above 1 GiB", M, N, K)
    inp = make_int_ag_inputs(M, N, K, n, seed=2049)
    case = AGCase(inp, 6, "double")
    case.C.fill_(0x7FC0)
    C.compass_ag_gemm(case.problem, C.links(200e9, 50e9))
    C.compass_sync()
    ref = O.f64_to_bf16_rne(O.ag_gemm([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"])))
    assert np.array_equal(host_bits(case.C), ref)
