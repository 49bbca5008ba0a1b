// extern "C" entry points declared in compass.h.
#include "compass.h"
#include "internal.h"

using namespace compass;

extern "C" {

int compass_schedule(int pattern, int ring, int n, int rank, int32_t *out, int cap) {
    return schedule_fill(pattern, ring, n, rank, out, cap);
}

int compass_ag_gemm(const compass_problem *p, const compass_links *links, void *stream) {
    return op_ag_gemm(p, links, stream);
}

int compass_gemm_rs(const compass_problem *p, const compass_links *links, void *stream) {
    return op_gemm_rs(p, links, stream);
}

int compass_decomp_gemm(const compass_problem *p, int d, const compass_links *links, void *stream) {
    return op_decomp(p, d, links, stream);
}

int compass_gemm(int M, int N, int K, const void *A, const void *W, void *C, const float *P, void *stream) {
    return op_gemm(M, N, K, A, W, C, P, stream);
}

int compass_gemm_noalloc(int M, int N, int K, const void *A, const void *W, void *C, const float *P, void *stream) {
    return op_gemm_noalloc(M, N, K, A, W, C, P, stream);
}

int compass_transfer(const compass_problem *p, const compass_links *links, void *stream) {
    return op_transfer(p, links, stream);
}

int compass_sequential(const compass_problem *p, const compass_links *links, void *stream) {
    return op_sequential(p, links, stream);
}

int compass_sync(void) { return op_sync(); }

int compass_set_option(int key, long long value) { return op_set_option(key, value); }

int compass_kernel_times(double *us, int cap) { return op_kernel_times(us, cap); }

int compass_tile_trace(uint32_t *records, int cap) { return op_tile_trace(records, cap); }

int compass_probe_mfma(int iters, double *tflops, double *sclk_ghz) {
    return op_probe_mfma(iters, tflops, sclk_ghz);
}

int compass_pick_strategy(const compass_workload *w, const compass_topology *t, const compass_calib *cal,
                          compass_choice *out) {
    return pick(w, t, cal, out);
}

int compass_partition_layout(int pattern, int ring, int n, int rank, int M, const compass_links *l, int32_t *order,
                             int32_t *row0, int32_t *rows, int cap) {
    return op_partition_layout(pattern, ring, n, rank, M, l, order, row0, rows, cap);
}

int compass_ring_arrival_times(int n, int rank, double piece_bytes, const double *hop_Bps, int d, double *out,
                               int cap) {
    return ring_arrivals(n, rank, piece_bytes, hop_Bps, d, out, cap);
}

double compass_model_t_comm(const compass_workload *w, const compass_topology *t) {
    if (!w || !t || w->n < 1) return -1.0;
    const int r = t->ring;
    if (r != COMPASS_RING_SINGLE && r != COMPASS_RING_DOUBLE && r != COMPASS_RING_DOUBLE_SPLIT &&
        r != COMPASS_RING_ALLTOALL)
        return -1.0;
    if (r == COMPASS_RING_ALLTOALL && (w->pattern != COMPASS_AG_GEMM || w->n % 2)) return -1.0;
    if (!(t->fwd_Bps > 0) || (r != COMPASS_RING_SINGLE && !(t->bwd_Bps > 0))) return -1.0;
    return model_t_comm(*w, *t);
}

double compass_model_t_decomp(double t_comp, double t_comm, int d, double alpha, double beta) {
    return model_t_decomp(t_comp, t_comm, d, alpha, beta);
}

double compass_model_t_fusion(const compass_workload *w, double t_comp, double t_comm_step, double alpha_f,
                              double beta_f) {
    if (!w || w->n < 1) return -1.0;
    return model_t_fusion(*w, t_comp, t_comm_step, alpha_f, beta_f);
}

int compass_calibrate(const compass_sample *s, int count, compass_calib *inout) { return calibrate(s, count, inout); }

const char *compass_last_error(void) { return last_error(); }

const char *compass_version(void) { return "compass-mi355x 0.1 (gfx950)"; }

}  // extern "C"
