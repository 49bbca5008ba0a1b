"""Pins of the oracle's GEMM parts against definitions independent of it:
a pure-Python triple loop, integer-exact inputs, IEEE bf16 facts, and the
invariants the method must keep (tile order and decomposition degree do not
change the result)."""
import itertools
import random

import numpy as np
import pytest

import oracle as O
from synth import bf16_bits, make_ag_inputs, make_int_ag_inputs, make_int_rs_inputs, make_rs_inputs


def brute_matmul(A, Bt):
    """C[i][j] = sum_k A[i][k] * Bt[j][k] with Python floats."""
    M, K = len(A), len(A[0])
    N = len(Bt)
    return [[sum(A[i][k] * Bt[j][k] for k in range(K)) for j in range(N)] for i in range(M)]


def test_bf16_decode_ieee_facts():
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0000, 0x8000, 0x4049, 0x7F7F], dtype=np.uint16)
    got = O.bf16_to_f64(bits)
    want = [1.0, -2.0, 1.0 + 2.0 ** -7, 0.0, -0.0, 3.140625, (2 - 2.0 ** -7) * 2.0 ** 127]
    assert list(got) == want


@pytest.mark.parametrize("x,bits", [
    (1.0, 0x3F80), (1.0 + 2.0 ** -8, 0x3F80), (1.0 + 3 * 2.0 ** -8, 0x3F82),
    (257.0, 0x4380), (259.0, 0x4382), (-259.0, 0xC382), (1.0 + 2.0 ** -8 + 2.0 ** -20, 0x3F81),
    (0.0, 0x0000), (-3.0, 0xC040),
])
def test_bf16_round_nearest_even(x, bits):
    assert int(O.f64_to_bf16_rne(np.array([x]))[0]) == bits


def test_generator_bits_round_trip():
    x = np.array([1.0, -2.5, 0.15625, 1024.0])
    assert list(O.bf16_to_f64(bf16_bits(x))) == list(x)


@pytest.mark.parametrize("n", [2, 4])
def test_ag_gemm_matches_triple_loop(n):
    rng = random.Random(7 + n)
    M, K, N = 8, 16, 8
    shards = [[[rng.uniform(-1, 1) for _ in range(K)] for _ in range(M // n)] for _ in range(n)]
    W = [[rng.uniform(-1, 1) for _ in range(K)] for _ in range(N)]
    A = [row for s in shards for row in s]          # rank order = row order
    ref = brute_matmul(A, W)
    got = O.ag_gemm([np.array(s) for s in shards], np.array(W))
    assert np.max(np.abs(got - np.array(ref))) < 1e-12


def test_ag_gemm_shard_order_matters():
    # a transposed operand or swapped shard order must be caught
    inp = make_int_ag_inputs(8, 6, 16, 2, seed=3)
    sh = [O.bf16_to_f64(s) for s in inp["shards"]]
    W = O.bf16_to_f64(inp["W"])
    good = O.ag_gemm(sh, W)
    assert not np.array_equal(good, O.ag_gemm(sh[::-1], W))
    ref = brute_matmul(np.vstack(sh).tolist(), W.tolist())
    assert np.array_equal(good, np.array(ref))


def test_ag_gemm_integer_exact():
    inp = make_int_ag_inputs(24, 16, 32, 4, seed=11)
    sh = [O.bf16_to_f64(s) for s in inp["shards"]]
    W = O.bf16_to_f64(inp["W"])
    got = O.ag_gemm(sh, W)
    ref = np.array(brute_matmul(np.vstack(sh).tolist(), W.tolist()))
    assert np.array_equal(got, ref)
    assert np.all(got == np.round(got))


@pytest.mark.parametrize("n", [2, 4])
def test_gemm_rs_matches_triple_loop(n):
    inp = make_int_rs_inputs(8, 12, 16, n, seed=5)
    A = O.bf16_to_f64(inp["A"])
    W = O.bf16_to_f64(inp["W"])
    P = [p.astype(np.float64) for p in inp["P_in"]]
    got = O.gemm_rs(A, W, P, n)
    prod = brute_matmul(A.tolist(), W.tolist())
    rows = 8 // n
    for c in range(n):
        for i in range(rows):
            for j in range(12):
                assert got[c * rows + i, j] == prod[c * rows + i][j] + P[c][i, j]


@pytest.mark.parametrize("d", [1, 2, 4, 8])
def test_decomp_ag_equals_fused_integer(d):
    inp = make_int_ag_inputs(64, 24, 32, 4, seed=21)
    sh = [O.bf16_to_f64(s) for s in inp["shards"]]
    W = O.bf16_to_f64(inp["W"])
    assert np.array_equal(O.decomp_ag(sh, W, d), O.ag_gemm(sh, W))


@pytest.mark.parametrize("d", [2, 4, 16])
def test_decomp_ag_equals_fused_random(d):
    inp = make_ag_inputs(128, 40, 48, 4, seed=22)
    sh = [O.bf16_to_f64(s) for s in inp["shards"]]
    W = O.bf16_to_f64(inp["W"])
    a, b = O.decomp_ag(sh, W, d), O.ag_gemm(sh, W)
    assert np.linalg.norm(a - b) / np.linalg.norm(b) < 1e-12


@pytest.mark.parametrize("d", [1, 2, 4])
def test_decomp_rs_equals_fused(d):
    inp = make_int_rs_inputs(32, 20, 24, 4, seed=23)
    A = O.bf16_to_f64(inp["A"])
    W = O.bf16_to_f64(inp["W"])
    P = [p.astype(np.float64) for p in inp["P_in"]]
    assert np.array_equal(O.decomp_rs(A, W, P, 4, d), O.gemm_rs(A, W, P, 4))


def test_decomp_rejects_uneven():
    inp = make_int_ag_inputs(24, 8, 16, 4, seed=1)
    with pytest.raises(ValueError):
        O.decomp_ag([O.bf16_to_f64(s) for s in inp["shards"]], O.bf16_to_f64(inp["W"]), 4)


def test_tile_order_independence():
    inp = make_int_ag_inputs(40, 28, 32, 4, seed=9)   # ragged 40x28 with 16x8 tiles
    sh = [O.bf16_to_f64(s) for s in inp["shards"]]
    W = O.bf16_to_f64(inp["W"])
    full = O.ag_gemm(sh, W)
    tiles = 3 * 4
    rng = random.Random(3)
    orders = [list(range(tiles)), list(reversed(range(tiles)))]
    for _ in range(5):
        o = list(range(tiles))
        rng.shuffle(o)
        orders.append(o)
    for o in orders:
        assert np.array_equal(O.tile_ordered_ag(sh, W, o, 16, 8), full)


def test_tile_ordered_missing_tile_shows():
    inp = make_int_ag_inputs(32, 16, 16, 2, seed=9)
    sh = [O.bf16_to_f64(s) for s in inp["shards"]]
    W = O.bf16_to_f64(inp["W"])
    C = O.tile_ordered_ag(sh, W, [0, 1, 2], 16, 8)   # tile 3 never computed
    assert np.isnan(C).any()


def test_tile_ordered_rs_schedules():
    inp = make_int_rs_inputs(32, 16, 16, 4, seed=10)
    A = O.bf16_to_f64(inp["A"])
    W = O.bf16_to_f64(inp["W"])
    P = [p.astype(np.float64) for p in inp["P_in"]]
    full = O.gemm_rs(A, W, P, 4)
    for r in range(4):
        sched = O.schedule("rs", "single", 4, r)
        order = [c * 2 + j for c in sched for j in range(2)]  # one row tile per chunk, 2 col tiles
        assert np.array_equal(O.tile_ordered_rs(A, W, P, 4, order, 8, 8), full)


def test_rs_random_normwise():
    inp = make_rs_inputs(64, 32, 48, 4, seed=12)
    A = O.bf16_to_f64(inp["A"])
    W = O.bf16_to_f64(inp["W"])
    P = [p.astype(np.float64) for p in inp["P_in"]]
    out = O.gemm_rs(A, W, P, 4)
    ref = np.array(brute_matmul(A.tolist(), W.tolist())) + np.vstack(P)
    assert np.linalg.norm(out - ref) / np.linalg.norm(ref) < 1e-13
