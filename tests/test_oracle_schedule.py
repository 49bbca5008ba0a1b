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
