"""Parity at the full sizes of the evaluation workloads, in the launch
configuration the benchmark times: fused operators on device-resident remote
data, links unpaced at the copy engines' ceiling (configuration 5: its 4 : 1
paced ring directions). The GPU computes the whole output; the oracle
computes sampled rows (the first and last row of every partition plus seeded
random rows), which cover every column tile, one row at a time through its
own gather / GEMM / ReduceScatter code."""
from __future__ import annotations

import functools

import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_10549_amd import compass as C
from synth import make_config_inputs
from tests.gpu_helpers import TOL, AGCase, RSCase, host_f64, rel_err

pytestmark = pytest.mark.gpu

UNPACED = C.links(0.0, 0.0)
LINKS_4_TO_1 = C.links(200e9, 50e9)


def _say(*a):
    print(*a, flush=True)


@functools.lru_cache(maxsize=2)
def inputs(idx: int, pattern: str | None = None) -> dict:
    return make_config_inputs(idx, pattern)


def sample_rows(M: int, parts: int, seed: int, extra: int = 2) -> np.ndarray:
    rng = np.random.default_rng(seed)
    prow = M // parts
    rows = []
    for q in range(parts):
        lo = q * prow
        rows += [lo, lo + prow - 1] + list(rng.integers(lo, lo + prow, size=extra))
    return np.unique(np.array(rows, dtype=np.int64))


def device_rows(t: torch.Tensor, rows: np.ndarray) -> np.ndarray:
    return host_f64(t.index_select(0, torch.from_numpy(rows).cuda()))


def ag_rows_reference(inp: dict, rows: np.ndarray) -> np.ndarray:
    A = np.vstack(inp["shards"])[rows]
    return O.ag_gemm([O.bf16_to_f64(A)], O.bf16_to_f64(inp["W"]))


def rs_rows_reference(inp: dict, rows: np.ndarray) -> np.ndarray:
    n, M = inp["n"], inp["M"]
    prow = M // n
    P = np.stack([inp["P_in"][r // prow][r % prow] for r in rows]).astype(np.float64)
    return O.gemm_rs(O.bf16_to_f64(inp["A"][rows]), O.bf16_to_f64(inp["W"]), [P], 1)


def split_boundary_rows(inp: dict, frac_bwd: float) -> np.ndarray:
    """Rows on both sides of the candidate boundaries of a rate-proportional
    split of every chunk (the exact share, and its roundings to 8 and to 128
    rows)."""
    rows = inp["M"] // inp["n"]
    x = rows * frac_bwd
    cands = {int(x), int(round(x / 8.0)) * 8, int(x // 128) * 128, -(-int(x) // 128) * 128}
    return np.array(sorted({c * rows + h + o for c in range(inp["n"]) for h in cands for o in (-1, 0)
                            if 0 < h < rows}), dtype=np.int64)


def check_ag(case: AGCase, inp: dict, parts: int, seed: int, extra_rows=None):
    torch.cuda.synchronize()
    assert np.array_equal(case.gathered.cpu().numpy().view(np.uint16), np.vstack(inp["shards"]))
    rows = sample_rows(inp["M"], parts, seed)
    if extra_rows is not None:
        rows = np.unique(np.concatenate([rows, extra_rows]))
    got = device_rows(case.C, rows)
    assert np.isfinite(got).all()
    err = rel_err(got, ag_rows_reference(inp, rows))
    _say("rows", len(rows), "normwise rel. error", err)
    assert err < TOL


def check_rs(case: RSCase, inp: dict, parts: int, seed: int, extra_rows=None):
    torch.cuda.synchronize()
    rows = sample_rows(inp["M"], parts, seed)
    if extra_rows is not None:
        rows = np.unique(np.concatenate([rows, extra_rows]))
    got = device_rows(case.C, rows)
    assert np.isfinite(got).all()
    err = rel_err(got, rs_rows_reference(inp, rows))
    _say("rows", len(rows), "normwise rel. error", err)
    assert err < TOL
    # every chunk sum sent onward equals the stored one
    prow = inp["M"] // inp["n"]
    for q, s in enumerate(case.send):
        if s is None:
            continue
        assert torch.equal(s, case.C[q * prow:(q + 1) * prow]), q


def test_config2_fused_allgather_full_size():
    inp = inputs(2)
    case = AGCase(inp, 0, "double")
    _say("config 2: fused AllGather", inp["M"], inp["N"], inp["K"])
    C.compass_ag_gemm(case.problem, UNPACED)
    C.compass_sync()
    check_ag(case, inp, 2 * inp["n"], seed=201)


def test_config3_fused_reducescatter_full_size():
    inp = inputs(3)
    case = RSCase(inp, 0, "single")
    _say("config 3: fused ReduceScatter", inp["M"], inp["N"], inp["K"])
    C.compass_gemm_rs(case.problem, UNPACED)
    C.compass_sync()
    check_rs(case, inp, inp["n"], seed=301)


@pytest.mark.parametrize("d", [0, 1, 2, 4, 8, 16])
def test_config4_interdecom_full_size(d):
    # d = 0: the fused operator on the same workload
    inp = inputs(4)
    case = AGCase(inp, 0, "single")
    _say("config 4: d =", d)
    if d == 0:
        C.compass_ag_gemm(case.problem, UNPACED)
    else:
        C.compass_decomp_gemm(case.problem, d, UNPACED)
    C.compass_sync()
    check_ag(case, inp, inp["n"], seed=400 + d)


@pytest.mark.parametrize("pattern", ["ag", "rs"])
def test_config5_double_ring_4_to_1_full_size(pattern):
    inp = inputs(5, pattern)
    _say("config 5:", pattern, inp["M"], inp["N"], inp["K"])
    if pattern == "ag":
        case = AGCase(inp, 0, "double")
        C.compass_ag_gemm(case.problem, LINKS_4_TO_1)
        C.compass_sync()
        check_ag(case, inp, 2 * inp["n"], seed=501)
    else:
        case = RSCase(inp, 0, "double")
        C.compass_gemm_rs(case.problem, LINKS_4_TO_1)
        C.compass_sync()
        check_rs(case, inp, 2 * inp["n"], seed=502)


def test_config5_reducescatter_unpaced_takes_256_tiles():
    # Unpaced links make the GPT-3 ReduceScatter computation-dominated
    # (estimated lambda > 1), where the operator takes 256 x 256 tiles: the
    # tile trace holds one record per output tile, 32 x 48 of them.
    inp = inputs(5, "rs")
    case = RSCase(inp, 0, "double")
    _say("config 5: rs unpaced, tile trace")
    C.compass_set_option(C.OPT_TILE_TRACE, 8192)
    try:
        C.compass_gemm_rs(case.problem, UNPACED)
        C.compass_sync()
        rec = C.compass_tile_trace(8192)
    finally:
        C.compass_set_option(C.OPT_TILE_TRACE, 0)
    assert len(rec) == (inp["M"] // 256) * (inp["N"] // 256)
    check_rs(case, inp, 2 * inp["n"], seed=503)


@pytest.mark.parametrize("pattern", ["ag", "rs"])
def test_config5_proportional_double_ring_4_to_1_full_size(pattern):
    # the same workload with each chunk's rows split 1 : 4 between the rings
    inp = inputs(5, pattern)
    _say("config 5 split:", pattern)
    if pattern == "ag":
        case = AGCase(inp, 0, "double_split")
        C.compass_ag_gemm(case.problem, LINKS_4_TO_1)
        C.compass_sync()
        check_ag(case, inp, 2 * inp["n"], seed=511, extra_rows=split_boundary_rows(inp, 0.2))
    else:
        case = RSCase(inp, 0, "double_split")
        C.compass_gemm_rs(case.problem, LINKS_4_TO_1)
        C.compass_sync()
        check_rs(case, inp, 2 * inp["n"], seed=512, extra_rows=split_boundary_rows(inp, 0.2))


@pytest.mark.parametrize("ring", ["alltoall", "single_hops"])
def test_config2_cross_numa_links_full_size(ring):
    # the fc1 workload over the cross-NUMA link patterns: AlltoAll (own
    # domain 200 GB/s, 50 GB/s shared across) and the single ring with hops
    # 3 -> 4 and 7 -> 0 at 50 GB/s, the rest at 200 GB/s (rank 3)
    inp = inputs(2)
    _say("config 2 cross-NUMA:", ring)
    if ring == "alltoall":
        case, lk = AGCase(inp, 0, "alltoall"), C.links(200e9, 50e9)
    else:
        hops = [50e9 if q in (3, 7) else 200e9 for q in range(inp["n"])]
        case, lk = AGCase(inp, 3, "single"), C.links(200e9, hop_Bps=hops)
    C.compass_ag_gemm(case.problem, lk)
    C.compass_sync()
    check_ag(case, inp, inp["n"], seed=521)


@pytest.mark.parametrize("pattern", ["ag", "rs"])
def test_config2_config3_sub_chunk_flags_full_size(pattern):
    # the benchmark's two operators with four arrival flags per partition
    # (128-row pieces for the AllGather's 512-row partitions)
    lk = C.links(0.0, 0.0, sub_chunks=4)
    if pattern == "ag":
        inp = inputs(2)
        case = AGCase(inp, 0, "double")
        _say("config 2 sub-chunks")
        C.compass_ag_gemm(case.problem, lk)
        C.compass_sync()
        check_ag(case, inp, 8 * inp["n"], seed=531)
    else:
        inp = inputs(3)
        case = RSCase(inp, 0, "single")
        _say("config 3 sub-chunks")
        C.compass_gemm_rs(case.problem, lk)
        C.compass_sync()
        check_rs(case, inp, 4 * inp["n"], seed=532)
