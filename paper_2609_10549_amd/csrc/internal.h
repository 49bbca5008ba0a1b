// Internal declarations shared by the host-side translation units.
#pragma once
#include <stdint.h>

#include "compass.h"

namespace compass {

constexpr int kMaxRanks = 32;

int set_error(int code, const char *fmt, ...);
const char *last_error();

int schedule_fill(int pattern, int ring, int n, int rank, int32_t *out, int cap);
int pick(const compass_workload *w, const compass_topology *t, const compass_calib *cal, compass_choice *out);
int calibrate(const compass_sample *s, int count, compass_calib *inout);
double model_t_comm(const compass_workload &w, const compass_topology &t);
int ring_arrivals(int n, int rank, double piece_bytes, const double *hop_Bps, int d, double *out, int cap);
double model_t_decomp(double tc, double tm, int d, double alpha, double beta);
double model_t_fusion(const compass_workload &w, double tc, double tm_step, double af, double bf);

// runtime (GPU side)
int op_ag_gemm(const compass_problem *p, const compass_links *l, void *stream);
int op_gemm_rs(const compass_problem *p, const compass_links *l, void *stream);
int op_decomp(const compass_problem *p, int d, const compass_links *l, void *stream);
int op_gemm(int M, int N, int K, const void *A, const void *W, void *C, const float *P, void *stream);
int op_gemm_noalloc(int M, int N, int K, const void *A, const void *W, void *C, const float *P, void *stream);
int op_transfer(const compass_problem *p, const compass_links *l, void *stream);
int op_partition_layout(int pattern, int ring, int n, int rank, int M, const compass_links *l, int32_t *order,
                        int32_t *row0, int32_t *rows, int cap);
int op_sequential(const compass_problem *p, const compass_links *l, void *stream);
int op_sync();
int op_set_option(int key, long long value);
int op_kernel_times(double *us, int cap);
int op_tile_trace(uint32_t *out, int cap);
int op_probe_mfma(int iters, double *tflops, double *sclk_ghz);

}  // namespace compass
