// Host-side parts of the Compass hot path that need no GPU: ring schedules
// (Section III-A/B), the InterDecom and IntraFusion time models (Eq. 2-8),
// the strategy selector (Algorithm 1) and the calibration fits
// (Section IV-C). Everything is fp64 and O(1) per call.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "compass.h"
#include "internal.h"

namespace compass {

int schedule_fill(int pattern, int ring, int n, int rank, int32_t *out, int cap) {
    if (n < 1 || n > kMaxRanks || rank < 0 || rank >= n)
        return set_error(COMPASS_ERR_INVALID, "schedule: need 1 <= n <= 32 and 0 <= rank < n");
    if (pattern != COMPASS_AG_GEMM && pattern != COMPASS_GEMM_RS)
        return set_error(COMPASS_ERR_INVALID, "schedule: unknown pattern");
    if (ring != COMPASS_RING_SINGLE && ring != COMPASS_RING_DOUBLE && ring != COMPASS_RING_DOUBLE_SPLIT &&
        ring != COMPASS_RING_ALLTOALL)
        return set_error(COMPASS_ERR_INVALID, "schedule: unknown ring");
    const bool one = ring == COMPASS_RING_SINGLE || ring == COMPASS_RING_ALLTOALL;
    const int len = one ? n : 2 * n;
    if (!out || cap < len) return set_error(COMPASS_ERR_INVALID, "schedule: output too small");
    auto md = [n](int x) { return ((x % n) + n) % n; };
    int k = 0;
    if (ring == COMPASS_RING_ALLTOALL) {
        if (pattern != COMPASS_AG_GEMM) return set_error(COMPASS_ERR_UNSUPPORTED, "schedule: AlltoAll is AllGather only");
        if (n % 2) return set_error(COMPASS_ERR_INVALID, "schedule: AlltoAll needs an even n");
        // own chunk, the own domain's peers from r + 1, then the other domain's
        const int h = n / 2, d0 = rank / h * h;
        out[k++] = rank;
        for (int i = 1; i < h; ++i) out[k++] = d0 + (rank - d0 + i) % h;
        for (int i = 0; i < h; ++i) out[k++] = (d0 + h) % n + i;
        return k;
    }
    if (pattern == COMPASS_AG_GEMM) {
        if (ring == COMPASS_RING_SINGLE) {
            // step s holds the chunk that travelled s hops on the forward ring
            for (int s = 0; s < n; ++s) out[k++] = md(rank - s);
        } else {
            out[k++] = 2 * rank;          // local halves first
            out[k++] = 2 * rank + 1;
            for (int s = 1; s < n; ++s) {
                out[k++] = 2 * md(rank - s) + 1;  // odd half, forward ring
                out[k++] = 2 * md(rank + s);      // even half, backward ring
            }
        }
    } else {
        if (ring == COMPASS_RING_SINGLE) {
            for (int s = 0; s < n; ++s) out[k++] = md(rank - 1 - s);
        } else {
            for (int s = 0; s < n; ++s) {
                out[k++] = 2 * md(rank - 1 - s) + 1;
                out[k++] = 2 * md(rank + 1 + s);
            }
        }
    }
    return k;
}

// Bytes one ring link carries per step (incoming, outgoing). AllGather moves
// the M x K bf16 input; ReduceScatter receives M x N fp32 partials and sends
// M x N bf16 sums. A single ring moves m/n per step, the double ring m/(2n)
// per ring (Section III-A).
static void step_bytes(const compass_workload &w, int ring, double *in, double *out) {
    const double div = ring == COMPASS_RING_SINGLE ? w.n : 2.0 * w.n;
    if (w.pattern == COMPASS_AG_GEMM) {
        *in = (double)w.M * w.K * 2.0 / div;
        *out = 0.0;
    } else {
        *in = (double)w.M * w.N * 4.0 / div;
        *out = (double)w.M * w.N * 2.0 / div;
    }
}

double model_t_comm(const compass_workload &w, const compass_topology &t) {
    double in, out;
    if (t.ring == COMPASS_RING_ALLTOALL) {
        // every chunk at once: the own domain's over their own links, the other
        // domain's (n/2)^2 flows sharing the cross-domain link
        step_bytes(w, COMPASS_RING_SINGLE, &in, &out);
        const double h = w.n / 2.0;
        const double intra = w.n > 2 ? in / t.fwd_Bps : 0.0;   // n = 2: no peer inside a domain
        return std::fmax(intra, h * h * in / t.bwd_Bps) + t.step_latency_s;
    }
    if (t.ring == COMPASS_RING_DOUBLE_SPLIT) {
        // the step's whole chunk over both rings, each carrying its rate's share
        step_bytes(w, COMPASS_RING_SINGLE, &in, &out);
        const double both = t.fwd_Bps + t.bwd_Bps;
        return (w.n - 1) * (std::fmax(in, out) / both + t.step_latency_s);
    }
    step_bytes(w, t.ring, &in, &out);
    double step = 0.0;
    const int rings = t.ring == COMPASS_RING_SINGLE ? 1 : 2;
    for (int i = 0; i < rings; ++i) {
        const double r = i == 0 ? t.fwd_Bps : t.bwd_Bps;
        step = std::fmax(step, std::fmax(in / r, out / r));
    }
    return (w.n - 1) * (step + t.step_latency_s);
}

int ring_arrivals(int n, int rank, double piece_bytes, const double *hop_Bps, int d, double *out, int cap) {
    if (!hop_Bps || !out) return set_error(COMPASS_ERR_INVALID, "ring_arrival_times: NULL argument");
    if (n < 1 || n > kMaxRanks || rank < 0 || rank >= n || d < 1)
        return set_error(COMPASS_ERR_INVALID, "ring_arrival_times: need 1 <= n <= %d, 0 <= rank < n, d >= 1", kMaxRanks);
    if (!(piece_bytes >= 0) || !std::isfinite(piece_bytes))
        return set_error(COMPASS_ERR_INVALID, "ring_arrival_times: bad piece size");
    for (int q = 0; q < n; ++q)
        if (!(hop_Bps[q] > 0) || !std::isfinite(hop_Bps[q]))
            return set_error(COMPASS_ERR_INVALID, "ring_arrival_times: hop %d rate must be positive", q);
    const long total = (long)d * (n - 1);
    if (cap < total) return set_error(COMPASS_ERR_INVALID, "ring_arrival_times: output too small");
    // into[q]: when the hop into rank q delivered its last piece;
    // has[q]: when rank q holds the piece it forwards at the next step
    double into[kMaxRanks] = {}, has[kMaxRanks], nxt[kMaxRanks];
    int k = 0;
    for (int j = 0; j < d; ++j) {
        for (int q = 0; q < n; ++q) has[q] = 0.0;   // every rank's own piece of sub-collective j
        for (int st = 1; st < n; ++st) {
            for (int q = 0; q < n; ++q) {
                const int from = (q + n - 1) % n;
                nxt[q] = std::fmax(has[from], into[q]) + piece_bytes / hop_Bps[from];
            }
            for (int q = 0; q < n; ++q) into[q] = has[q] = nxt[q];
            out[k++] = nxt[rank];
        }
    }
    return k;
}

double model_t_comp(const compass_workload &w, const compass_calib &c) {
    return c.comp_a + c.comp_b * (2.0 * w.M * (double)w.N * w.K);
}

double model_t_decomp(double tc, double tm, int d, double alpha, double beta) {
    // Eq. 2 with Eq. 3: (d-1) stages of max(Tc, Tm)/d scaled by eta(d), plus
    // the non-overlapped Tc/d + Tm/d.
    const double stage = std::fmax(tc / d, tm / d);
    return (d - 1) * stage * (alpha + beta * d) + tc / d + tm / d;
}

int p2_round(double x) {
    // nearest power of two in log2; ties to the smaller power; < 1 -> 1
    if (!(x > 1.0)) return 1;
    const double lg = std::log2(x);
    const double k = std::floor(lg);
    const double frac = lg - k;
    const int e = (int)k + (frac > 0.5 ? 1 : 0);
    if (e >= 30) return 1 << 30;
    return 1 << e;
}

double d_stationary(double lam, double alpha, double beta, int literal) {
    if (beta <= 0.0) return INFINITY;
    const double r = literal ? 1.0 / lam : std::fmin(lam, 1.0 / lam);
    const double num = 1.0 - alpha + r;
    if (num <= 0.0) return 0.0;
    return std::sqrt(num / beta);
}

double model_t_fusion(const compass_workload &w, double tc, double tm_step, double af, double bf) {
    // Eq. 7: chunk 1 exposes its computation; chunks 2..n overlap their
    // computation (Tc/n each) with one ring step of communication; Eq. 8 adds
    // n-1 synchronisation overheads alpha_f + beta_f * m.
    const int n = w.n;
    const double c = tc / n;
    double body = 0.0;
    for (int i = 1; i < n; ++i) body += std::fmax(c, tm_step);
    const double m = w.pattern == COMPASS_AG_GEMM ? (double)w.M * w.K : (double)w.M * w.N;
    return body + c + (n - 1) * (af + bf * m);
}

// Degree of ODP-InterDecom (Section IV-C) for base times tc, tm: the
// stationary point of Eq. 2 in d rounded to a power of two (Eq. 5), capped at
// d_max and at the largest power of two that splits a chunk's rows evenly,
// kept only when its predicted time beats the undecomposed operator (Eq. 4).
struct Degree {
    int cand, best;         // Eq. 5 candidate, chosen degree
    double t_best, t_one;   // Eq. 2 at the chosen degree and at d = 1
};

static Degree optimal_degree(double tc, double tm, int chunk_rows, const compass_calib &cal) {
    int feasible = 1;
    while (feasible * 2 <= cal.d_max && chunk_rows % (feasible * 2) == 0) feasible *= 2;
    const double x = d_stationary(tc / tm, cal.alpha_decomp, cal.beta_decomp, cal.literal_eq5);
    Degree g;
    g.cand = std::isinf(x) ? feasible : std::min(std::max(p2_round(x), 1), feasible);
    g.t_one = model_t_decomp(tc, tm, 1, cal.alpha_decomp, cal.beta_decomp);
    const double t_cand = model_t_decomp(tc, tm, g.cand, cal.alpha_decomp, cal.beta_decomp);
    g.best = t_cand < g.t_one ? g.cand : 1;
    g.t_best = g.best == g.cand ? t_cand : g.t_one;
    return g;
}

// Strategy selection of Section V (the problem of Eq. 6, solved in O(1) by
// the selection algorithm, Algorithm 1): predict the operator time of
// ODP-InterDecom at its degree (Eq. 2-5) and of TA-IntraFusion (Eq. 7-8,
// chunk computation Tc / n against one ring step of communication), both from
// the calibrated base times, and take the lower; a tie goes to InterDecom.
int pick(const compass_workload *w, const compass_topology *t, const compass_calib *cal,
         compass_choice *out) {
    if (!w || !t || !cal || !out) return set_error(COMPASS_ERR_INVALID, "pick_strategy: null argument");
    if (w->n < 1 || w->M < 1 || w->N < 1 || w->K < 1 || w->M % w->n)
        return set_error(COMPASS_ERR_INVALID, "pick_strategy: bad workload");
    if (w->pattern != COMPASS_AG_GEMM && w->pattern != COMPASS_GEMM_RS)
        return set_error(COMPASS_ERR_INVALID, "pick_strategy: unknown pattern");
    if (t->ring == COMPASS_RING_ALLTOALL)
        return set_error(COMPASS_ERR_UNSUPPORTED, "pick_strategy: the models are for rings");
    if (t->ring != COMPASS_RING_SINGLE && t->ring != COMPASS_RING_DOUBLE && t->ring != COMPASS_RING_DOUBLE_SPLIT)
        return set_error(COMPASS_ERR_INVALID, "pick_strategy: unknown ring");
    if (!(t->fwd_Bps > 0) || (t->ring != COMPASS_RING_SINGLE && !(t->bwd_Bps > 0)))
        return set_error(COMPASS_ERR_INVALID, "pick_strategy: link rates must be positive");
    if (cal->d_max < 1) return set_error(COMPASS_ERR_INVALID, "pick_strategy: d_max < 1");
    const double tc = model_t_comp(*w, *cal);
    const double tm = model_t_comm(*w, *t);
    if (!(tc > 0) || !(tm > 0)) return set_error(COMPASS_ERR_INVALID, "pick_strategy: non-positive base time");
    const Degree dg = optimal_degree(tc, tm, w->M / w->n, *cal);
    const double step = w->n > 1 ? tm / (w->n - 1) : 0.0;
    const double tfus = model_t_fusion(*w, tc, step, cal->alpha_fusion, cal->beta_fusion);
    out->strategy = tfus < dg.t_best ? COMPASS_INTRA_FUSION : COMPASS_INTER_DECOM;
    out->t_star = std::fmin(tfus, dg.t_best);
    out->d_star = dg.best;
    out->d_cand = dg.cand;
    out->lambda = tc / tm;
    out->t_comp = tc;
    out->t_comm = tm;
    out->t_fusion = tfus;
    out->t_decomp = dg.t_best;
    out->t_decomp1 = dg.t_one;
    return COMPASS_OK;
}

// Least squares y ~ a + b x; false when fewer than two distinct x.
static bool fit_line(const std::vector<double> &x, const std::vector<double> &y, double *a, double *b) {
    const size_t n = x.size();
    if (n < 2) return false;
    double mx = 0, my = 0;
    for (size_t i = 0; i < n; ++i) { mx += x[i]; my += y[i]; }
    mx /= n; my /= n;
    double sxx = 0, sxy = 0;
    for (size_t i = 0; i < n; ++i) { sxx += (x[i] - mx) * (x[i] - mx); sxy += (x[i] - mx) * (y[i] - my); }
    if (!(sxx > 0)) return false;
    *b = sxy / sxx;
    *a = my - *b * mx;
    return true;
}

int calibrate(const compass_sample *s, int count, compass_calib *c) {
    if (!c || count < 0 || (count > 0 && !s)) return set_error(COMPASS_ERR_INVALID, "calibrate: bad arguments");
    std::vector<double> x0, y0, x1, y1, x2, y2;
    for (int i = 0; i < count; ++i) {
        const compass_sample &q = s[i];
        if (q.w.n < 1) return set_error(COMPASS_ERR_INVALID, "calibrate: sample with n < 1");
        if (q.kind == 0) {
            x0.push_back(2.0 * q.w.M * (double)q.w.N * q.w.K);
            y0.push_back(q.t_meas);
        } else if (q.kind == 1) {
            if (q.d < 2) continue;
            // invert Eq. 2 for the overhead factor at this point
            const double d = q.d;
            const double e = (q.t_meas - (q.t_comp + q.t_comm) / d) * d /
                             ((d - 1) * std::fmax(q.t_comp, q.t_comm));
            x1.push_back(d);
            y1.push_back(e);
        } else if (q.kind == 2) {
            if (q.w.n < 2) continue;
            // invert Eq. 7 for the per-synchronisation overhead
            const int n = q.w.n;
            const double cc = q.t_comp / n, ms = q.t_comm / (n - 1);
            double base = cc;
            for (int k = 1; k < n; ++k) base += std::fmax(cc, ms);
            const double o = (q.t_meas - base) / (n - 1);
            const double m = q.w.pattern == COMPASS_AG_GEMM ? (double)q.w.M * q.w.K : (double)q.w.M * q.w.N;
            x2.push_back(m);
            y2.push_back(o);
        } else {
            return set_error(COMPASS_ERR_INVALID, "calibrate: unknown sample kind");
        }
    }
    double a, b;
    if (fit_line(x0, y0, &a, &b)) { c->comp_a = a; c->comp_b = b; }
    if (fit_line(x1, y1, &a, &b)) { c->alpha_decomp = a; c->beta_decomp = b; }
    if (fit_line(x2, y2, &a, &b)) { c->alpha_fusion = a; c->beta_fusion = b; }
    return COMPASS_OK;
}

}  // namespace compass
