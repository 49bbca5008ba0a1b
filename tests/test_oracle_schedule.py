"""Pins of the ring schedules: permutation, local-first / local-last rules of
Section II-B and III-B, agreement with an independent message-passing ring
simulation (Section III-A, Fig. 5), and the ReduceScatter semantics."""
import numpy as np
import pytest

import oracle as O
from synth import make_int_rs_inputs


@pytest.mark.parametrize("pattern", ["ag", "rs"])
@pytest.mark.parametrize("ring", ["single", "double"])
@pytest.mark.parametrize("n", [1, 2, 3, 4, 8])
def test_schedule_is_permutation(pattern, ring, n):
    size = n if ring == "single" else 2 * n
    for r in range(n):
        s = O.schedule(pattern, ring, n, r)
        assert sorted(s) == list(range(size))


@pytest.mark.parametrize("n", [2, 4, 8])
def test_ag_local_first_rs_local_last(n):
    for r in range(n):
        assert O.schedule("ag", "single", n, r)[0] == r
        assert O.schedule("ag", "double", n, r)[:2] == [2 * r, 2 * r + 1]
        assert O.schedule("rs", "single", n, r)[-1] == r
        assert sorted(O.schedule("rs", "double", n, r)[-2:]) == [2 * r, 2 * r + 1]


@pytest.mark.parametrize("ring", ["single", "double"])
@pytest.mark.parametrize("n", [2, 3, 4, 8])
def test_ag_schedule_equals_simulated_arrivals(ring, n):
    held = O.simulate_ring_allgather(n, ring)
    for q in range(n):
        assert held[q] == O.schedule("ag", ring, n, q)
        assert sorted(held[q]) == list(range(n if ring == "single" else 2 * n))


def test_four_gpu_double_ring_example():
    # Section III-B, Fig. 6: 4 GPUs, 4 chunks -> 8 partitions; each GPU starts
    # on its local data; the backward ring carries even partitions and the
    # forward ring odd partitions, in opposite directions.
    n = 4
    for r in range(n):
        s = O.schedule("ag", "double", n, r)
        assert len(s) == 8 and s[:2] == [2 * r, 2 * r + 1]
        for step in range(1, n):
            fwd, bwd = s[2 * step], s[2 * step + 1]
            assert fwd % 2 == 1 and fwd // 2 == (r - step) % n   # came from r-1 side
            assert bwd % 2 == 0 and bwd // 2 == (r + step) % n   # came from r+1 side


def test_single_ring_arrivals_n4():
    # on a forward ring, rank 0 receives the chunk of rank 3 first, then 2, 1
    held = O.simulate_ring_allgather(4, "single")
    assert held[0] == [0, 3, 2, 1]
    assert held[2] == [2, 1, 0, 3]


@pytest.mark.parametrize("ring", ["single", "double"])
@pytest.mark.parametrize("n", [2, 4])
def test_ring_reduce_scatter_equals_direct_sum(ring, n):
    M, N = 8 * n, 6
    partials = []
    for q in range(n):
        inp = make_int_rs_inputs(M, N, 4, n, seed=40 + q)
        partials.append(np.vstack(inp["P_in"]).astype(np.float64))
    result, order = O.simulate_ring_reduce_scatter(partials, ring)
    total = sum(partials)
    rows = M // n
    for q in range(n):
        assert np.array_equal(result[q], total[q * rows:(q + 1) * rows])
        assert order[q] == O.schedule("rs", ring, n, q)


def test_rs_local_chunk_only_completes_at_owner():
    n = 4
    partials = [np.full((8, 2), float(q + 1)) for q in range(n)]
    result, _ = O.simulate_ring_reduce_scatter(partials, "single")
    for q in range(n):
        assert np.all(result[q] == 10.0)


@pytest.mark.parametrize("n", [2, 4, 6, 8, 16])
def test_alltoall_schedule_own_domain_first(n):
    # own chunk, then every chunk of the own NUMA domain (direct links), then
    # every chunk of the other domain (shared cross-domain link)
    h = n // 2
    for r in range(n):
        s = O.schedule("ag", "alltoall", n, r)
        assert sorted(s) == list(range(n)) and s[0] == r
        assert {q // h for q in s[1:h]} <= {r // h}
        assert {q // h for q in s[h:]} == {1 - r // h}


# ---- partition layout: sub-chunk flags and the rate-proportional split
@pytest.mark.parametrize("pattern", ["ag", "rs"])
@pytest.mark.parametrize("ring", ["single", "double", "double_split"])
def test_partition_layout_tiles_the_rows_in_order(pattern, ring):
    for n, M, sub, fwd, bwd in [(2, 64, 1, 0, 0), (4, 4096, 2, 200e9, 50e9), (8, 8192, 4, 50e9, 200e9),
                                (8, 2048, 3, 1e9, 1e9), (3, 96, 2, 0, 0), (1, 40, 4, 0, 0)]:
        for r in range(n):
            order, row0, cnt = O.partition_layout(pattern, ring, n, r, M, fwd, bwd, sub)
            P = len(row0)
            assert sorted(order) == list(range(P))
            # consecutive ids cover [0, M) without gaps or overlaps, none empty
            assert row0[0] == 0 and all(c > 0 for c in cnt)
            assert all(row0[q] + cnt[q] == row0[q + 1] for q in range(P - 1)) and row0[-1] + cnt[-1] == M
            # the pieces of one base partition follow one another in the order
            base = O.schedule(pattern, ring, n, r)
            assert [q // sub for q in order] == [b for b in base for _ in range(sub)]


def test_partition_layout_reduces_to_chunks_and_halves():
    # Section III-B: a single ring moves whole chunks; the double ring splits
    # each chunk into a backward (first) and a forward (second) half
    o, r0, c = O.partition_layout("ag", "single", 4, 1, 4096)
    assert r0 == [0, 1024, 2048, 3072] and c == [1024] * 4 and o == O.schedule("ag", "single", 4, 1)
    o, r0, c = O.partition_layout("ag", "double", 4, 1, 4096)
    assert r0 == [0, 512, 1024, 1536, 2048, 2560, 3072, 3584] and c == [512] * 8
    # the proportional split at equal or unpaced rates is the paper's halves
    for f, b in [(1e9, 1e9), (0, 0), (0, 50e9)]:
        assert O.partition_layout("rs", "double_split", 4, 2, 4096, f, b) == \
            O.partition_layout("rs", "double", 4, 2, 4096)


def test_proportional_split_by_hand_and_by_brute_force():
    # 4 : 1 on 1024-row chunks: 204.8 rows is the rate share; of 128 and 256,
    # 128 gives the shorter step (max(640, 1120) against max(1280, 960))
    assert O.backward_rows(1024, 200e9, 50e9, "double_split") == 128
    assert O.partition_layout("ag", "double_split", 8, 0, 8192, 200e9, 50e9)[2][:2] == [128, 896]
    rng = np.random.default_rng(5)
    for _ in range(300):
        rows = int(rng.choice([16, 40, 64, 200, 512, 1024, 1536, 3072, 6000]))
        f, b = float(rng.uniform(1e9, 400e9)), float(rng.uniform(1e9, 400e9))
        h = O.backward_rows(rows, f, b, "double_split")
        fb = b / (f + b)
        G = 128 if rows >= 1024 else 8
        lo = min(G, rows // 2)
        cands = [x for x in range(0, rows + 1, G) if lo <= x <= rows - lo] + [lo, rows - lo]
        best = min(max(x / fb, (rows - x) / (1 - fb)) for x in cands)
        # no multiple of G (nor either bound) in range has a shorter step
        assert max(h / fb, (rows - h) / (1 - fb)) <= best * (1 + 1e-12)
        assert lo <= h <= rows - lo
