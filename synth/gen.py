"""Seeded input generators for the fused AllGather-GEMM / GEMM-ReduceScatter
workloads (tensor-parallel MLP shapes, Section II-A; Table IV grid).

Layout conventions shared by every consumer:

* Activations are row-major bf16 bit patterns (numpy uint16). An AllGather
  input is a list of ``n`` row shards, shard ``q`` holding rows
  ``[q*M/n, (q+1)*M/n)`` of the gathered matrix.
* The weight is stored as ``W`` with shape ``(N, K)`` (row-major, K
  contiguous: the usual Linear-layer layout). The GEMM operand ``B`` of
  ``C = A @ B`` is ``W`` transposed.
* ReduceScatter incoming partial sums are fp32 arrays, one ``(M/n, N)``
  array per row chunk.

Random streams come from ``numpy.random.Generator(PCG64)`` seeded through
``SeedSequence(seed).spawn``; each tensor has its own child stream.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "CONFIGS", "bf16_bits", "config_shapes", "make_ag_inputs", "make_rs_inputs",
    "make_int_ag_inputs", "make_int_rs_inputs", "make_config_inputs", "make_int_config_inputs",
]


def bf16_bits(x) -> np.ndarray:
    """Encode real values as bf16 bit patterns (uint16).

    The values go to float32 first (numpy's round-to-nearest-even), then the
    float32 pattern is rounded to its upper 16 bits, again to nearest-even.
    This only fixes which bf16 values the inputs take; both consumers read
    the same bits.
    """
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    bias = 0x7FFF + ((u >> 16) & 1)
    return ((u + bias) >> 16).astype(np.uint16)


def _draw(rng: np.random.Generator, shape, dist: tuple) -> np.ndarray:
    kind = dist[0]
    if kind == "uniform":
        lo, hi = dist[1], dist[2]
        return rng.uniform(lo, hi, size=shape)
    if kind == "normal":
        return rng.normal(0.0, dist[1], size=shape)
    if kind == "int":
        lo, hi = dist[1], dist[2]
        return rng.integers(lo, hi + 1, size=shape).astype(np.float64)
    raise ValueError(f"unknown distribution {dist!r}")


def _streams(seed: int, count: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(count)]


def make_ag_inputs(M: int, N: int, K: int, n: int, seed: int,
                   dist_a=("normal", 1.0), dist_w=("normal", 0.02)) -> dict:
    """AllGather-GEMM inputs: ``n`` bf16 shards of ``(M/n, K)`` and ``W (N, K)``."""
    if M % n:
        raise ValueError("M must be divisible by n")
    rs = _streams(seed, n + 1)
    shards = [bf16_bits(_draw(rs[q], (M // n, K), dist_a)) for q in range(n)]
    W = bf16_bits(_draw(rs[n], (N, K), dist_w))
    return {"pattern": "ag", "M": M, "N": N, "K": K, "n": n, "seed": seed,
            "shards": shards, "W": W}


def make_rs_inputs(M: int, N: int, K: int, n: int, seed: int,
                   dist_a=("normal", 1.0), dist_w=("normal", 0.02),
                   dist_p=("normal", 1.0)) -> dict:
    """GEMM-ReduceScatter inputs: bf16 ``A (M, K)``, ``W (N, K)`` and ``n``
    fp32 incoming partials of ``(M/n, N)``."""
    if M % n:
        raise ValueError("M must be divisible by n")
    rs = _streams(seed, n + 2)
    A = bf16_bits(_draw(rs[0], (M, K), dist_a))
    W = bf16_bits(_draw(rs[1], (N, K), dist_w))
    P = [np.ascontiguousarray(_draw(rs[2 + c], (M // n, N), dist_p).astype(np.float32))
         for c in range(n)]
    return {"pattern": "rs", "M": M, "N": N, "K": K, "n": n, "seed": seed,
            "A": A, "W": W, "P_in": P}


def make_int_ag_inputs(M, N, K, n, seed, lo=-4, hi=4) -> dict:
    """AllGather-GEMM inputs whose values are small integers, so that every
    fp32 partial sum of the product is exact."""
    return make_ag_inputs(M, N, K, n, seed, ("int", lo, hi), ("int", lo, hi))


def make_int_rs_inputs(M, N, K, n, seed, lo=-4, hi=4) -> dict:
    """GEMM-ReduceScatter inputs with small-integer values (partials too)."""
    return make_rs_inputs(M, N, K, n, seed, ("int", lo, hi), ("int", lo, hi),
                          ("int", -64, 64))


# The five evaluation workloads, sized as one tensor-parallel rank's share.
CONFIGS = {
    1: dict(name="ag_tp2_small", pattern="ag", M=512, N=1024, K=512, n=2, ring="single",
            seed=1, dist_a=("uniform", -1.0, 1.0), dist_w=("uniform", -1.0, 1.0)),
    2: dict(name="ag_tp8_mlp_fc1", pattern="ag", M=8192, N=2048, K=4096, n=8, ring="double",
            seed=2, dist_a=("normal", 1.0), dist_w=("normal", 0.02)),
    3: dict(name="rs_tp8_mlp_fc2", pattern="rs", M=8192, N=4096, K=2048, n=8, ring="single",
            seed=3, dist_a=("normal", 1.0), dist_w=("normal", 0.02), dist_p=("normal", 1.0)),
    4: dict(name="ag_tp8_qkv_decomp", pattern="ag", M=4096, N=3072, K=8192, n=8, ring="single",
            seed=4, dist_a=("normal", 1.0), dist_w=("normal", 0.02), d_list=(1, 2, 4, 8, 16)),
    5: dict(name="gpt3_175b_tp8_double_ring", pattern="ag+rs", ring="double", n=8, seed=5,
            ag=dict(M=8192, N=6144, K=12288), rs=dict(M=8192, N=12288, K=6144),
            dist=("normal", 1.0), rate_ratio=4.0),
}


def config_shapes(idx: int) -> list:
    """List of (pattern, M, N, K, n) tuples for a configuration."""
    c = CONFIGS[idx]
    if idx == 5:
        return [("ag", c["ag"]["M"], c["ag"]["N"], c["ag"]["K"], c["n"]),
                ("rs", c["rs"]["M"], c["rs"]["N"], c["rs"]["K"], c["n"])]
    return [(c["pattern"], c["M"], c["N"], c["K"], c["n"])]


def make_config_inputs(idx: int, pattern: str | None = None) -> dict:
    """Full-size inputs of configuration ``idx`` (for config 5 pass the
    pattern, ``"ag"`` or ``"rs"``)."""
    c = CONFIGS[idx]
    if idx == 5:
        sh = c[pattern]
        d = c["dist"]
        if pattern == "ag":
            return make_ag_inputs(sh["M"], sh["N"], sh["K"], c["n"], c["seed"], d, d)
        return make_rs_inputs(sh["M"], sh["N"], sh["K"], c["n"], c["seed"] + 100, d, d, d)
    if c["pattern"] == "ag":
        return make_ag_inputs(c["M"], c["N"], c["K"], c["n"], c["seed"], c["dist_a"], c["dist_w"])
    return make_rs_inputs(c["M"], c["N"], c["K"], c["n"], c["seed"], c["dist_a"],
                          c["dist_w"], c["dist_p"])


def make_int_config_inputs(idx: int, pattern: str | None = None) -> dict:
    """Configuration ``idx`` at its full shape with small-integer values
    (activations and weights in [-4, 4], partials in [-64, 64]): every fp32
    partial sum of the product is exact (|sum| <= 16 K + 64 < 2**24 for
    K <= 12288), so a correct GEMM's bf16 output is the exact result rounded
    once. Seeds differ from the seeded-normal inputs of the same shape."""
    c = CONFIGS[idx]
    if idx == 5:
        sh = c[pattern]
        M, N, K, pat = sh["M"], sh["N"], sh["K"], pattern
    else:
        M, N, K, pat = c["M"], c["N"], c["K"], c["pattern"]
    seed = 1000 + 10 * idx + (1 if pat == "rs" else 0)
    if pat == "ag":
        return make_int_ag_inputs(M, N, K, c["n"], seed)
    return make_int_rs_inputs(M, N, K, c["n"], seed)
