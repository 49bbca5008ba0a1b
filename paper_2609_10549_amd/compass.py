"""ctypes binding of libcompass.so (include/compass.h).

Argument marshalling only: every entry point forwards to the C ABI of the
same name. Tensors are passed by their device (or pinned host) addresses;
there is no Python or PyTorch implementation of any step behind these
functions, and a missing library raises instead of falling back.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
# COMPASS_LIBRARY selects another build of the same library (the host
# sanitizer build, libcompass_san.so, in CPU-only test runs)
LIB_PATH = os.environ.get("COMPASS_LIBRARY") or os.path.join(_HERE, "libcompass.so")

OK = 0
ERR_INVALID = -1
ERR_UNSUPPORTED = -2
ERR_HIP = -3
ERR_TIMEOUT = -4
ERR_IN_FLIGHT = -5

AG_GEMM = 0
GEMM_RS = 1
RING_SINGLE = 0
RING_DOUBLE = 1
INTRA_FUSION = 0
INTER_DECOM = 1

OPT_SPIN_LIMIT = 1
OPT_HOST_TIMEOUT = 2
OPT_GRID = 3
OPT_DROP_FLAG = 4
OPT_TILE = 5
OPT_ENGINE_MASK = 6
OPT_KERNEL_TIMING = 7
OPT_TILE_TRACE = 8
OPT_SCHED = 9
OPT_POOL = 10
OPT_PACE_HEADROOM = 12
OPT_TAIL_MIN_K = 13
OPT_TAIL_MIN_K_128 = 14
OPT_TAIL_SLICE_K = 15
OPT_TAIL_GROUPS = 16
OPT_HEAD_SPLIT = 17

PATTERNS = {"ag": AG_GEMM, "rs": GEMM_RS}
RING_DOUBLE_SPLIT = 2
RING_ALLTOALL = 3
RINGS = {"single": RING_SINGLE, "double": RING_DOUBLE, "double_split": RING_DOUBLE_SPLIT,
         "alltoall": RING_ALLTOALL}


class CompassError(RuntimeError):
    def __init__(self, code: int, where: str, msg: str):
        super().__init__(f"{where} failed ({code}): {msg}")
        self.code = code


class compass_links(ctypes.Structure):
    _fields_ = [("fwd_Bps", ctypes.c_double), ("bwd_Bps", ctypes.c_double),
                ("slice_bytes", ctypes.c_size_t), ("engines_per_ring", ctypes.c_int),
                ("sub_chunks", ctypes.c_int), ("hop_Bps", ctypes.POINTER(ctypes.c_double))]


class compass_problem(ctypes.Structure):
    _fields_ = [("pattern", ctypes.c_int), ("M", ctypes.c_int), ("N", ctypes.c_int), ("K", ctypes.c_int),
                ("n", ctypes.c_int), ("rank", ctypes.c_int), ("ring", ctypes.c_int),
                ("W", ctypes.c_void_p), ("C", ctypes.c_void_p),
                ("shard_src", ctypes.POINTER(ctypes.c_void_p)), ("gathered", ctypes.c_void_p),
                ("A", ctypes.c_void_p), ("partial_src", ctypes.POINTER(ctypes.c_void_p)),
                ("partial_stage", ctypes.c_void_p), ("send_dst", ctypes.POINTER(ctypes.c_void_p))]


class compass_workload(ctypes.Structure):
    _fields_ = [("pattern", ctypes.c_int), ("M", ctypes.c_int), ("N", ctypes.c_int), ("K", ctypes.c_int),
                ("n", ctypes.c_int)]


class compass_topology(ctypes.Structure):
    _fields_ = [("ring", ctypes.c_int), ("fwd_Bps", ctypes.c_double), ("bwd_Bps", ctypes.c_double),
                ("step_latency_s", ctypes.c_double)]


class compass_calib(ctypes.Structure):
    _fields_ = [("comp_a", ctypes.c_double), ("comp_b", ctypes.c_double),
                ("alpha_decomp", ctypes.c_double), ("beta_decomp", ctypes.c_double),
                ("alpha_fusion", ctypes.c_double), ("beta_fusion", ctypes.c_double),
                ("d_max", ctypes.c_int), ("literal_eq5", ctypes.c_int)]


class compass_choice(ctypes.Structure):
    _fields_ = [("strategy", ctypes.c_int), ("d_star", ctypes.c_int), ("d_cand", ctypes.c_int),
                ("t_star", ctypes.c_double), ("lambda_", ctypes.c_double),
                ("t_comp", ctypes.c_double), ("t_comm", ctypes.c_double),
                ("t_fusion", ctypes.c_double), ("t_decomp", ctypes.c_double),
                ("t_decomp1", ctypes.c_double)]


class compass_sample(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("w", compass_workload), ("d", ctypes.c_int),
                ("t_meas", ctypes.c_double), ("t_comp", ctypes.c_double), ("t_comm", ctypes.c_double)]


_lib = None

# name -> (restype, argtypes)
_SIGS = {
    "compass_schedule": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                        ctypes.POINTER(ctypes.c_int32), ctypes.c_int]),
    "compass_ag_gemm": (ctypes.c_int, [ctypes.POINTER(compass_problem), ctypes.POINTER(compass_links), ctypes.c_void_p]),
    "compass_gemm_rs": (ctypes.c_int, [ctypes.POINTER(compass_problem), ctypes.POINTER(compass_links), ctypes.c_void_p]),
    "compass_decomp_gemm": (ctypes.c_int, [ctypes.POINTER(compass_problem), ctypes.c_int,
                                           ctypes.POINTER(compass_links), ctypes.c_void_p]),
    "compass_gemm": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "compass_gemm_noalloc": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "compass_transfer": (ctypes.c_int, [ctypes.POINTER(compass_problem), ctypes.POINTER(compass_links), ctypes.c_void_p]),
    "compass_sequential": (ctypes.c_int, [ctypes.POINTER(compass_problem), ctypes.POINTER(compass_links), ctypes.c_void_p]),
    "compass_sync": (ctypes.c_int, []),
    "compass_kernel_times": (ctypes.c_int, [ctypes.POINTER(ctypes.c_double), ctypes.c_int]),
    "compass_tile_trace": (ctypes.c_int, [ctypes.POINTER(ctypes.c_uint32), ctypes.c_int]),
    "compass_probe_mfma": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    "compass_set_option": (ctypes.c_int, [ctypes.c_int, ctypes.c_longlong]),
    "compass_pick_strategy": (ctypes.c_int, [ctypes.POINTER(compass_workload), ctypes.POINTER(compass_topology),
                                             ctypes.POINTER(compass_calib), ctypes.POINTER(compass_choice)]),
    "compass_partition_layout": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                                ctypes.POINTER(compass_links), ctypes.POINTER(ctypes.c_int32),
                                                ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32),
                                                ctypes.c_int]),
    "compass_ring_arrival_times": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                                  ctypes.POINTER(ctypes.c_double), ctypes.c_int,
                                                  ctypes.POINTER(ctypes.c_double), ctypes.c_int]),
    "compass_model_t_comm": (ctypes.c_double, [ctypes.POINTER(compass_workload), ctypes.POINTER(compass_topology)]),
    "compass_model_t_decomp": (ctypes.c_double, [ctypes.c_double, ctypes.c_double, ctypes.c_int,
                                                 ctypes.c_double, ctypes.c_double]),
    "compass_model_t_fusion": (ctypes.c_double, [ctypes.POINTER(compass_workload), ctypes.c_double, ctypes.c_double,
                                                 ctypes.c_double, ctypes.c_double]),
    "compass_calibrate": (ctypes.c_int, [ctypes.POINTER(compass_sample), ctypes.c_int, ctypes.POINTER(compass_calib)]),
    "compass_last_error": (ctypes.c_char_p, []),
    "compass_version": (ctypes.c_char_p, []),
}


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_10549_amd.build`")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(h, name)
            f.restype = res
            f.argtypes = args
        _lib = h
    return _lib


def _check(rc: int, where: str) -> int:
    if rc < 0:
        raise CompassError(rc, where, lib().compass_last_error().decode())
    return rc


def _addr(x) -> int | None:
    """Device / pinned-host address of a tensor (or an int address, or None)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _ptr_array(items: Sequence) -> ctypes.Array:
    arr = (ctypes.c_void_p * len(items))()
    for i, x in enumerate(items):
        arr[i] = _addr(x)
    return arr


class Problem:
    """A compass_problem plus the pointer arrays it references (kept alive)."""

    def __init__(self, st: compass_problem, keep: list):
        self.st = st
        self._keep = keep


def _shape_of(x):
    return tuple(int(v) for v in x.shape)


def _need(x, what: str, shape: tuple, elsize: int) -> None:
    """Raise ValueError unless tensor x is contiguous with the given shape and
    element size (the library takes raw addresses and derives every extent
    from M, N, K and n, so a mismatch would send its copies and loads outside
    the tensor). Plain int addresses are the caller's responsibility."""
    if x is None or isinstance(x, int):
        return
    if _shape_of(x) != tuple(shape):
        raise ValueError(f"{what}: shape {_shape_of(x)}, expected {tuple(shape)}")
    if x.element_size() != elsize:
        raise ValueError(f"{what}: element size {x.element_size()} bytes, expected {elsize}")
    if not x.is_contiguous():
        raise ValueError(f"{what}: must be contiguous")


def ag_problem(shards: Sequence, gathered, W, C, rank: int, ring: str | int = "double") -> Problem:
    """AllGather+GEMM operands: n shards (M/n x K bf16), gathered (M x K),
    W (N x K), C (M x N). Tensors hold bf16 values (dtype bfloat16 or int16)."""
    n = len(shards)
    M, K = gathered.shape
    N = W.shape[0]
    if n < 1 or M % n:
        raise ValueError(f"M = {M} rows must split into n = {n} shards")
    _need(gathered, "gathered", (M, K), 2)
    _need(W, "W", (N, K), 2)
    _need(C, "C", (M, N), 2)
    for q, sh in enumerate(shards):
        _need(sh, f"shards[{q}]", (M // n, K), 2)
    arr = _ptr_array(shards)
    st = compass_problem(pattern=AG_GEMM, M=M, N=N, K=K, n=n, rank=rank,
                         ring=RINGS.get(ring, ring), W=_addr(W), C=_addr(C),
                         shard_src=arr, gathered=_addr(gathered))
    return Problem(st, [arr])


def rs_problem(A, W, partial_src: Sequence, partial_stage, C, send_dst: Sequence | None,
               rank: int, ring: str | int = "single") -> Problem:
    """GEMM+ReduceScatter operands: A (M x K), W (N x K), n fp32 partials
    (M/n x N), an M x N fp32 landing buffer, C (M x N), optional n send
    destinations (entry `rank` may be None)."""
    n = len(partial_src)
    M, K = A.shape
    N = W.shape[0]
    if n < 1 or M % n:
        raise ValueError(f"M = {M} rows must split into n = {n} chunks")
    _need(A, "A", (M, K), 2)
    _need(W, "W", (N, K), 2)
    _need(C, "C", (M, N), 2)
    _need(partial_stage, "partial_stage", (M, N), 4)
    for q, p in enumerate(partial_src):
        _need(p, f"partial_src[{q}]", (M // n, N), 4)
    if send_dst is not None:
        if len(send_dst) != n:
            raise ValueError(f"send_dst: {len(send_dst)} entries, expected {n}")
        for q, x in enumerate(send_dst):
            _need(x, f"send_dst[{q}]", (M // n, N), 2)
    parr = _ptr_array(partial_src)
    sarr = None
    if send_dst is not None:
        sarr = _ptr_array([0 if x is None else x for x in send_dst])
    st = compass_problem(pattern=GEMM_RS, M=M, N=N, K=K, n=n, rank=rank,
                         ring=RINGS.get(ring, ring), W=_addr(W), C=_addr(C), A=_addr(A),
                         partial_src=parr, partial_stage=_addr(partial_stage),
                         send_dst=sarr)
    return Problem(st, [parr, sarr])


def links(fwd_Bps: float = 0.0, bwd_Bps: float | None = None, slice_bytes: int = 0,
          engines_per_ring: int = 0, hop_Bps: Sequence[float] | None = None,
          sub_chunks: int = 0) -> compass_links:
    lk = compass_links(fwd_Bps=fwd_Bps, bwd_Bps=fwd_Bps if bwd_Bps is None else bwd_Bps,
                       slice_bytes=slice_bytes, engines_per_ring=engines_per_ring, sub_chunks=sub_chunks)
    if hop_Bps is not None:
        arr = (ctypes.c_double * len(hop_Bps))(*hop_Bps)
        lk.hop_Bps = arr
        lk._hops = arr   # kept alive with the struct
    return lk


def _lk(lk) -> compass_links:
    return links() if lk is None else lk


# ------------------------------------------------------------------ calls
def compass_schedule(pattern, ring, n: int, rank: int) -> list:
    cap = 2 * max(n, 1)
    out = (ctypes.c_int32 * cap)()
    k = _check(lib().compass_schedule(PATTERNS.get(pattern, pattern), RINGS.get(ring, ring), n, rank, out, cap),
               "compass_schedule")
    return list(out[:k])


def compass_ag_gemm(problem: Problem, lk: compass_links | None = None, stream=None) -> None:
    _check(lib().compass_ag_gemm(ctypes.byref(problem.st), ctypes.byref(_lk(lk)), _stream(stream)), "compass_ag_gemm")


def compass_gemm_rs(problem: Problem, lk: compass_links | None = None, stream=None) -> None:
    _check(lib().compass_gemm_rs(ctypes.byref(problem.st), ctypes.byref(_lk(lk)), _stream(stream)), "compass_gemm_rs")


def compass_decomp_gemm(problem: Problem, d: int, lk: compass_links | None = None, stream=None) -> None:
    _check(lib().compass_decomp_gemm(ctypes.byref(problem.st), d, ctypes.byref(_lk(lk)), _stream(stream)),
           "compass_decomp_gemm")


def compass_gemm(A, W, C, P=None, stream=None) -> None:
    M, K = A.shape
    N = W.shape[0]
    _need(A, "A", (M, K), 2)
    _need(W, "W", (N, K), 2)
    _need(C, "C", (M, N), 2)
    _need(P, "P", (M, N), 4)
    _check(lib().compass_gemm(M, N, K, _addr(A), _addr(W), _addr(C), _addr(P), _stream(stream)), "compass_gemm")


def compass_gemm_noalloc(A, W, C, P=None, stream=None) -> None:
    M, K = A.shape
    N = W.shape[0]
    _need(A, "A", (M, K), 2)
    _need(W, "W", (N, K), 2)
    _need(C, "C", (M, N), 2)
    _need(P, "P", (M, N), 4)
    _check(lib().compass_gemm_noalloc(M, N, K, _addr(A), _addr(W), _addr(C), _addr(P), _stream(stream)),
           "compass_gemm_noalloc")


def compass_transfer(problem: Problem, lk: compass_links | None = None, stream=None) -> None:
    _check(lib().compass_transfer(ctypes.byref(problem.st), ctypes.byref(_lk(lk)), _stream(stream)), "compass_transfer")


def compass_sequential(problem: Problem, lk: compass_links | None = None, stream=None) -> None:
    _check(lib().compass_sequential(ctypes.byref(problem.st), ctypes.byref(_lk(lk)), _stream(stream)),
           "compass_sequential")


def compass_sync() -> None:
    _check(lib().compass_sync(), "compass_sync")


def compass_kernel_times(cap: int = 512) -> list:
    out = (ctypes.c_double * cap)()
    k = _check(lib().compass_kernel_times(out, cap), "compass_kernel_times")
    return list(out[:k])


def compass_tile_trace(cap: int = 1 << 16):
    """Tile records (numpy uint32, shape (k, 8)) of the GEMM launches since the
    previous call; see the header for the fields."""
    import numpy as np
    out = np.zeros((cap, 8), dtype=np.uint32)
    k = _check(lib().compass_tile_trace(out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)), cap),
               "compass_tile_trace")
    return out[:k]


def compass_probe_mfma(iters: int = 16384) -> tuple:
    """(bf16 TFLOP/s, shader clock GHz) of the matrix-core probe; see the header."""
    tf, ghz = ctypes.c_double(), ctypes.c_double()
    _check(lib().compass_probe_mfma(iters, ctypes.byref(tf), ctypes.byref(ghz)), "compass_probe_mfma")
    return tf.value, ghz.value


def compass_set_option(key: int, value: int) -> None:
    _check(lib().compass_set_option(key, value), "compass_set_option")


def compass_pick_strategy(workload: compass_workload, topology: compass_topology,
                          calib: compass_calib) -> compass_choice:
    out = compass_choice()
    _check(lib().compass_pick_strategy(ctypes.byref(workload), ctypes.byref(topology), ctypes.byref(calib),
                                       ctypes.byref(out)), "compass_pick_strategy")
    return out


def compass_partition_layout(pattern, ring, n: int, rank: int, M: int, lk: compass_links | None = None):
    """(order, row0, rows) of the partitions of one rank; see the header."""
    cap = 64
    order, row0, rows = (ctypes.c_int32 * cap)(), (ctypes.c_int32 * cap)(), (ctypes.c_int32 * cap)()
    k = _check(lib().compass_partition_layout(PATTERNS.get(pattern, pattern), RINGS.get(ring, ring), n, rank, M,
                                              ctypes.byref(_lk(lk)), order, row0, rows, cap),
               "compass_partition_layout")
    return list(order[:k]), list(row0[:k]), list(rows[:k])


def compass_ring_arrival_times(n: int, rank: int, piece_bytes: float, hop_Bps: Sequence[float],
                               d: int = 1) -> list:
    hops = (ctypes.c_double * max(n, 1))(*list(hop_Bps)[:max(n, 1)])
    cap = max(1, d * max(n - 1, 0))
    out = (ctypes.c_double * cap)()
    k = _check(lib().compass_ring_arrival_times(n, rank, piece_bytes, hops, d, out, cap),
               "compass_ring_arrival_times")
    return list(out[:k])


def compass_model_t_comm(workload: compass_workload, topology: compass_topology) -> float:
    return lib().compass_model_t_comm(ctypes.byref(workload), ctypes.byref(topology))


def compass_model_t_decomp(t_comp: float, t_comm: float, d: int, alpha: float, beta: float) -> float:
    return lib().compass_model_t_decomp(t_comp, t_comm, d, alpha, beta)


def compass_model_t_fusion(workload: compass_workload, t_comp: float, t_comm_step: float,
                           alpha_f: float, beta_f: float) -> float:
    return lib().compass_model_t_fusion(ctypes.byref(workload), t_comp, t_comm_step, alpha_f, beta_f)


def compass_calibrate(samples: Sequence[compass_sample], calib: compass_calib) -> compass_calib:
    arr = (compass_sample * len(samples))(*samples)
    _check(lib().compass_calibrate(arr, len(samples), ctypes.byref(calib)), "compass_calibrate")
    return calib


def compass_last_error() -> str:
    return lib().compass_last_error().decode()


def compass_version() -> str:
    return lib().compass_version().decode()
