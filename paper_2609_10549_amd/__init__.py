"""MI355X implementation of the Compass hot path (arXiv 2609.10549).

One tensor-parallel rank's share of fused AllGather+GEMM and
GEMM+ReduceScatter (TA-IntraFusion), the d-way InterDecom operator, and the
analytic strategy selector, behind the C ABI of include/compass.h. The Python
module `compass` is a thin ctypes binding of that library.
"""
from . import compass  # noqa: F401
from .compass import (  # noqa: F401
    compass_ag_gemm,
    compass_calibrate,
    compass_decomp_gemm,
    compass_gemm,
    compass_gemm_rs,
    compass_kernel_times,
    compass_tile_trace,
    compass_probe_mfma,
    compass_last_error,
    compass_model_t_comm,
    compass_partition_layout,
    compass_ring_arrival_times,
    compass_model_t_decomp,
    compass_model_t_fusion,
    compass_pick_strategy,
    compass_schedule,
    compass_sequential,
    compass_set_option,
    compass_sync,
    compass_transfer,
    compass_version,
)
