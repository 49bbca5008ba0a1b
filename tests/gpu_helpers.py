"""Helpers for the GPU tests: move synth inputs to the device, build problem
descriptions, compare against the oracle."""
from __future__ import annotations

import numpy as np
import torch

import oracle as O
from paper_2609_10549_amd import compass as C

TOL = 5e-3   # normwise relative error bound for bf16 outputs


def dev_bits(bits: np.ndarray, pinned: bool = False) -> torch.Tensor:
    """uint16 bf16 patterns -> int16 tensor on the GPU (or pinned host)."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    if pinned:
        return t.pin_memory()
    return t.cuda()


def dev_f32(x: np.ndarray, pinned: bool = False) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.pin_memory() if pinned else t.cuda()


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def host_f64(t: torch.Tensor) -> np.ndarray:
    return O.bf16_to_f64(host_bits(t))


def rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))


class AGCase:
    """Device buffers of one AllGather+GEMM instance."""

    def __init__(self, inp: dict, rank: int, ring: str, pinned_remote: bool = False, local_in_place: bool = True):
        M, N, K, n = inp["M"], inp["N"], inp["K"], inp["n"]
        self.inp, self.rank, self.ring = inp, rank, ring
        self.gathered = torch.zeros((M, K), dtype=torch.int16, device="cuda")
        self.W = dev_bits(inp["W"])
        self.C = torch.zeros((M, N), dtype=torch.int16, device="cuda")
        rows = M // n
        self.shards = []
        for q, s in enumerate(inp["shards"]):
            if q == rank:
                if local_in_place:
                    self.gathered[q * rows:(q + 1) * rows] = dev_bits(s)
                    self.shards.append(self.gathered[q * rows:(q + 1) * rows])
                else:
                    self.shards.append(dev_bits(s))
            else:
                self.shards.append(dev_bits(s, pinned=pinned_remote))
        self.problem = C.ag_problem(self.shards, self.gathered, self.W, self.C, rank, ring)

    def reference(self) -> np.ndarray:
        sh = [O.bf16_to_f64(s) for s in self.inp["shards"]]
        return O.ag_gemm(sh, O.bf16_to_f64(self.inp["W"]))


class RSCase:
    """Device buffers of one GEMM+ReduceScatter instance."""

    def __init__(self, inp: dict, rank: int, ring: str, sends: bool = True, pinned_remote: bool = False):
        M, N, K, n = inp["M"], inp["N"], inp["K"], inp["n"]
        self.inp, self.rank, self.ring = inp, rank, ring
        self.A = dev_bits(inp["A"])
        self.W = dev_bits(inp["W"])
        self.C = torch.zeros((M, N), dtype=torch.int16, device="cuda")
        self.stage = torch.zeros((M, N), dtype=torch.float32, device="cuda")
        self.partials = [dev_f32(p, pinned=pinned_remote) for p in inp["P_in"]]
        rows = M // n
        self.send = None
        if sends:
            self.send = [None if q == rank else torch.zeros((rows, N), dtype=torch.int16, device="cuda")
                         for q in range(n)]
        self.problem = C.rs_problem(self.A, self.W, self.partials, self.stage, self.C, self.send, rank, ring)

    def reference(self) -> np.ndarray:
        P = [p.astype(np.float64) for p in self.inp["P_in"]]
        return O.gemm_rs(O.bf16_to_f64(self.inp["A"]), O.bf16_to_f64(self.inp["W"]), P, self.inp["n"])
