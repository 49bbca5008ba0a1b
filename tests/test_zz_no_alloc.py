"""compass_gemm_noalloc, the plain GEMM for callers that cannot allocate,
against compass_gemm through the C ABI: two calls in a row, the second on a
smaller input, so the shared scratch's ticket queues must start each launch
cleared. Integer-valued inputs (every fp32 partial sum exact) must give the
same bits as compass_gemm and as the oracle's exact product rounded once;
seeded normal inputs must stay within 5e-3 normwise of the fp64 oracle (the
two entry points may sum K in different slice orders)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle as O
from paper_2609_10549_amd import compass as C
from synth import make_ag_inputs, make_int_ag_inputs, make_int_rs_inputs

BF16_NAN = 0x7FC0

# (M, N, K): a 256 x 256-tile shape with ragged edges, then a smaller
# 128 x 128-tile one; the GPT-3 AllGather shape, then a small one
PAIRS = [((1544, 1048, 520), (264, 136, 200)), ((8192, 6144, 12288), (520, 264, 136))]


def _gemm(fn, A, W, P, M, N):
    import torch
    Cm = torch.full((M, N), BF16_NAN, dtype=torch.int16, device="cuda")
    fn(A, W, Cm, P)
    torch.cuda.synchronize()
    return Cm.cpu().numpy().view(np.uint16)


def _dev(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


@pytest.mark.gpu
@pytest.mark.parametrize("pair", range(len(PAIRS)))
@pytest.mark.parametrize("partial", [False, True])
def test_noalloc_gemm_equals_compass_gemm_two_calls(pair, partial):
    import torch
    for call, (M, N, K) in enumerate(PAIRS[pair]):
        print(f"no-alloc GEMM call {call}: M={M} N={N} K={K} partial={partial}", flush=True)
        seed = 500 + 10 * pair + call
        if partial:
            inp = make_int_rs_inputs(M, N, K, 1, seed=seed)
            A, W = _dev(inp["A"]), _dev(inp["W"])
            P = torch.from_numpy(inp["P_in"][0]).cuda()
            ref = O.gemm_rs(O.bf16_to_f64(inp["A"]), O.bf16_to_f64(inp["W"]), [inp["P_in"][0].astype(np.float64)], 1)
        else:
            inp = make_int_ag_inputs(M, N, K, 1, seed=seed)
            A, W = _dev(inp["shards"][0]), _dev(inp["W"])
            P = None
            ref = O.ag_gemm([O.bf16_to_f64(inp["shards"][0])], O.bf16_to_f64(inp["W"]))
        got = _gemm(C.compass_gemm_noalloc, A, W, P, M, N)
        want = _gemm(C.compass_gemm, A, W, P, M, N)
        assert np.array_equal(got, want), (call, int((got != want).sum()))
        assert np.array_equal(got, O.f64_to_bf16_rne(ref)), call
        del A, W, P
        torch.cuda.empty_cache()


@pytest.mark.gpu
def test_noalloc_gemm_seeded_inputs_two_calls():
    for call, (M, N, K) in enumerate(((2056, 1032, 1544), (136, 264, 72))):
        print(f"no-alloc GEMM seeded call {call}: M={M} N={N} K={K}", flush=True)
        inp = make_ag_inputs(M, N, K, 1, seed=600 + call)
        A, W = _dev(inp["shards"][0]), _dev(inp["W"])
        ref = O.ag_gemm([O.bf16_to_f64(inp["shards"][0])], O.bf16_to_f64(inp["W"]))
        for fn in (C.compass_gemm_noalloc, C.compass_gemm):
            got = O.bf16_to_f64(_gemm(fn, A, W, None, M, N))
            assert np.isfinite(got).all()
            err = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
            assert err < 5e-3, (fn.__name__, call, err)


def test_noalloc_gemm_rejects_sizes_before_touching_the_device():
    # validation precedes any device call, so this runs without a GPU
    lib = C.lib()
    assert lib.compass_gemm_noalloc(65537, 64, 64, 16, 16, 16, None, None) == C.ERR_UNSUPPORTED
    assert lib.compass_gemm_noalloc(64, 64, 60, 16, 16, 16, None, None) == C.ERR_INVALID
    assert lib.compass_gemm_noalloc(64, 64, 64, None, 16, 16, None, None) == C.ERR_INVALID
    # a 256-row tile spanning over 1 GiB of A (K) or of the fp32 partial (N)
    assert lib.compass_gemm_noalloc(64, 64, 2097160, 16, 16, 16, None, None) == C.ERR_UNSUPPORTED
    assert lib.compass_gemm_noalloc(64, 1048584, 64, 16, 16, 16, 16, None) == C.ERR_UNSUPPORTED
