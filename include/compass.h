/*
 * compass.h — C ABI of the MI355X implementation of the Compass hot path.
 *
 * Compass (arXiv 2609.10549) hides tensor-parallel communication behind GEMM
 * work in two ways: IntraFusion, one fused operator whose output tiles run in
 * the order their input chunks arrive over a single or double ring
 * (Section III), and InterDecom, d pipelined sub-operators (Section II-B,
 * Section IV). An analytic model picks the degree d and the strategy
 * (Section IV-C, Section V, Algorithm 1).
 *
 * This library implements one tensor-parallel rank's share of both operators
 * on a single GPU. The other ranks are emulated: their shards / partial sums
 * live in separate device allocations or in pinned host memory, and SDMA copy
 * engines move them into this rank's buffers at configurable per-ring link
 * rates, publishing per-partition arrival flags that the GEMM kernel polls.
 *
 * Conventions
 *   - bf16 data is passed as raw 16-bit patterns (uint16); fp32 as float.
 *   - Every matrix is row-major and densely packed (leading dimension = its
 *     column count).
 *   - The GEMM computes C = A * B with B = W^T, where W is N x K (the Linear
 *     weight layout: K contiguous for both operands). Products accumulate in
 *     fp32; C is rounded once to bf16, nearest-even.
 *   - "device" pointers are HIP device allocations of the current device;
 *     "pinned host" pointers come from hipHostMalloc. Every buffer is owned by
 *     the caller; the library keeps only a small control block per device
 *     (flags, counters, copy-engine state), allocated on first use.
 *   - Calls are stream-ordered on the stream passed in (a hipStream_t; NULL is
 *     the default stream). Operations of this library must not overlap on one
 *     device: they share the control block. Issue them from one host thread.
 *   - Every entry point returns COMPASS_OK (0) or a negative status; the
 *     message of the last failure on the calling thread is returned by
 *     compass_last_error(). Argument checks happen before anything is
 *     enqueued. A kernel-side wait that exceeds its bound is reported as
 *     COMPASS_ERR_TIMEOUT by the next call or by compass_sync().
 */
#ifndef COMPASS_H
#define COMPASS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define COMPASS_OK               0
#define COMPASS_ERR_INVALID     -1  /* bad argument (shape, pointer, rank...) */
#define COMPASS_ERR_UNSUPPORTED -2  /* valid but outside what is implemented  */
#define COMPASS_ERR_HIP         -3  /* HIP / HSA runtime call failed          */
#define COMPASS_ERR_TIMEOUT     -4  /* a bounded wait (flag, copy) expired    */
#define COMPASS_ERR_IN_FLIGHT   -5  /* copies of a failed job were still running
                                       when the copy side gave up waiting for
                                       them: they may still write caller
                                       buffers, so every later call is refused
                                       with this status (the process must not
                                       free or reuse those buffers)          */

/* ---- enumerations ------------------------------------------------------ */
#define COMPASS_AG_GEMM   0  /* AllGather + GEMM      (Section II-A, Fig. 1) */
#define COMPASS_GEMM_RS   1  /* GEMM + ReduceScatter  (Section II-A, Fig. 1) */

#define COMPASS_RING_SINGLE 0  /* one ring, n-1 steps of m/n (Section III-A) */
#define COMPASS_RING_DOUBLE 1  /* two counter-rotating rings, each chunk split
                                  into a forward and a backward half
                                  (Section III-A, Fig. 5(b); III-B, Fig. 6) */
#define COMPASS_RING_DOUBLE_SPLIT 2  /* not the paper's design, an extension of it
                                  for unequal directions: the double ring with
                                  each chunk's rows split in proportion to the
                                  two link rates (backward share first, rounded
                                  to a multiple of 128 rows for chunks of at
                                  least 1024 rows, else of 8, toward the shorter
                                  step), so that both directions finish every
                                  step together, nearly;
                                  the schedule is COMPASS_RING_DOUBLE's. With a
                                  rate <= 0 (unpaced) the split is in halves.
                                  InterDecom sub-operators split each piece
                                  the same way. Model: a step carries m/n over
                                  both rings at B_fwd + B_bwd. */
#define COMPASS_RING_ALLTOALL 3  /* not a ring: the direct-push AlltoAll pattern the
                                  paper compares its rings against (Section III-A),
                                  AllGather only, n even, fused operator, transfer
                                  and unfused baseline (InterDecom and the selector
                                  return COMPASS_ERR_UNSUPPORTED). Ranks [0, n/2)
                                  and [n/2, n) are two NUMA domains. Every peer of
                                  this rank's domain pushes its chunk at the same
                                  time over a link of its own at fwd_Bps; the n/2
                                  peers of the other domain push at the same time
                                  over the cross-domain link of bwd_Bps, which the
                                  (n/2)^2 flows into this domain share equally, so
                                  their chunks land together after
                                  (n/2)^2 (m/n) / bwd_Bps (effective B/2 at n = 8,
                                  against the single ring's 8/7 B over the same
                                  link). Order: own chunk, the own domain's peers
                                  in rank order from r + 1, then the other domain's
                                  in rank order. */

#define COMPASS_INTRA_FUSION 0  /* TA-IntraFusion  (Algorithm 1) */
#define COMPASS_INTER_DECOM  1  /* ODP-InterDecom  (Algorithm 1) */

/* ---- ring schedule (Section III-A, III-B) -------------------------------
 * Writes the order in which rank `rank` of an n-rank ring processes the
 * chunks (single ring: chunk ids 0..n-1) or partitions (double ring:
 * partition p = 2c + h, h = 0 for the first row half of chunk c, carried by
 * the backward ring, h = 1 for the second half, forward ring).
 *   AllGather:      local data first, then arrivals step by step; under the
 *                   double ring the forward-ring partition precedes the
 *                   backward-ring one within a step.
 *   ReduceScatter:  textbook ring order (r-1-s) mod n, local chunk last.
 *   COMPASS_RING_ALLTOALL (AllGather, even n): chunk ids in the order given
 *                   with the constant; other patterns or an odd n return
 *                   COMPASS_ERR_UNSUPPORTED / COMPASS_ERR_INVALID.
 * `out` receives `cap` >= n (single ring, AlltoAll) or 2n (double ring)
 * int32 entries.
 * Returns the number of entries written, or a negative status.
 * Host only; needs no GPU. */
int compass_schedule(int pattern, int ring, int n, int rank, int32_t *out, int cap);

/* ---- emulated links -----------------------------------------------------
 * Rates are the emulated per-direction link bandwidths of the two rings
 * (bytes per second). A single ring uses fwd_Bps only.
 *
 * Paced (rate >= 1e8): the link delivers one item (a partition, or a chunk
 * sum sent onward) at a time at that rate; an item is due when the link has
 * finished the previous one (or its data became ready, if later) plus
 * bytes / rate. Its arrival flag is never published before the due time.
 * The copy goes out whole on a group of the ring direction's SDMA engines,
 * ahead of its due time by its predicted latency; if the engines cannot
 * keep up, items arrive late (the achieved rate is what transfer timings
 * measure).
 * Unpaced (rate <= 0): copies go out as fast as the engines take them, in
 * slices round-robin over the engines; flags publish when the data landed.
 * With more than one active direction the directions share every engine
 * (COMPASS_OPT_POOL). Rates in (0, 1e8) are rejected.
 *
 * slice_bytes: largest single copy (0: library default, 2 MiB, or 3 MiB for
 * unpaced directions sharing the engines; else >= 4 KiB). engines_per_ring:
 * SDMA engines per ring direction (0: library default, all usable engines
 * split over the active directions; not used when they share the engines).
 *
 * hop_Bps (single ring only; NULL: every hop at fwd_Bps): n rates, hop q
 * carrying rank q -> q+1 mod n, each >= 1e8 (paced), for a ring whose hops
 * differ, as on the cross-NUMA ring of Section III-A. The ring then has no
 * step barrier: item s reaches this rank at the time
 * compass_ring_arrival_times gives (store and forward, one item per hop at
 * a time, the emulated ranks forwarding as soon as they hold an item). The
 * incoming items take the rate of the hop into this rank, the ReduceScatter
 * sums sent onward that of the hop out of it. The caller owns the array; it
 * is read during the call only. Another ring with hop_Bps set returns
 * COMPASS_ERR_UNSUPPORTED.
 *
 * sub_chunks (0 or 1: one arrival flag per partition): s >= 2 splits every
 * partition's rows into s pieces of consecutive rows (piece t: rows
 * [cnt t / s, cnt (t+1) / s) of the partition's cnt rows), each moved as an
 * item of its own, in row order, with an arrival flag of its own, so tiles
 * start on the first piece before the rest of the partition lands, and
 * under ReduceScatter each piece's sum is sent on as soon as its tiles are
 * done. Fused operators, transfer and unfused baseline; needs the single or
 * double ring without hop_Bps, s times the partition count at most 64, and
 * a row for every piece (else COMPASS_ERR_UNSUPPORTED / _INVALID);
 * compass_decomp_gemm with d > 1 returns COMPASS_ERR_UNSUPPORTED. */
typedef struct compass_links {
    double fwd_Bps;
    double bwd_Bps;
    size_t slice_bytes;
    int    engines_per_ring;
    int    sub_chunks;
    const double *hop_Bps;
} compass_links;

/* Partition layout of rank `rank` (host only, no GPU): the P partitions the
 * operators move and gate on (n or 2n base partitions times sub_chunks),
 * from pattern, ring, n, M and the link parameters that shape it (the rate
 * split of COMPASS_RING_DOUBLE_SPLIT, sub_chunks). order[i] is the partition
 * at schedule position i (each base partition's pieces in row order);
 * partition q holds global rows [row0[q], row0[q] + rows[q]) for InterDecom
 * degree 1. Returns P, or a negative status (the operators' checks on
 * these arguments, a NULL pointer, cap < P). */
int compass_partition_layout(int pattern, int ring, int n, int rank, int M, const compass_links *l,
                             int32_t *order, int32_t *row0, int32_t *rows, int cap);

/* ---- one operator instance ----------------------------------------------
 * Describes the rank-local share of one AllGather+GEMM or GEMM+ReduceScatter.
 * The emulated rank r owns row chunk r, rows [r*M/n, (r+1)*M/n).
 *
 * Requirements: 1 <= n <= 32, 0 <= rank < n, M % n == 0 (and M % (2n) == 0
 * for the double ring), K % 8 == 0, N % 8 == 0, and the size limits below.
 * Every range a copy engine reads or writes (a shard, a partial, a send
 * chunk, their rows of gathered / partial_stage / C) must lie inside the
 * allocation that holds its first byte, as the HSA runtime reports it:
 * otherwise COMPASS_ERR_INVALID, before anything is enqueued.
 *
 * AllGather + GEMM (pattern COMPASS_AG_GEMM):
 *   shard_src[q], q = 0..n-1: (M/n) x K bf16 shard of rank q. shard_src[rank]
 *     is device memory; if it is not already the rank's rows of `gathered`
 *     it is copied there (on the stream) before the operator starts. The
 *     others are device memory or pinned host memory; they are read by copy
 *     engines only.
 *   gathered: device, M x K bf16, receives every shard at its row chunk.
 *   W: device, N x K bf16.  C: device, M x N bf16 output, C = gathered * W^T.
 *
 * GEMM + ReduceScatter (pattern COMPASS_GEMM_RS):
 *   A: device, M x K bf16 (this rank's full input); W: device, N x K bf16.
 *   partial_src[c], c = 0..n-1: (M/n) x N fp32 incoming partial sum of row
 *     chunk c (device or pinned host). The partial of the rank's first
 *     ReduceScatter step (a true ring has none there) is treated as resident:
 *     in device memory, with the resident rows on tile boundaries (the usual
 *     case), the GEMM's epilogue reads it from partial_src directly (d = 1,
 *     fused and sequential); otherwise, unless partial_src of that chunk
 *     already points at its rows of partial_stage, it is copied there (on
 *     the stream) before the operator starts; either way the caller keeps it
 *     unchanged until the call's work on the stream is done. The other n-1
 *     arrive over the emulated link in ring order.
 *   partial_stage: device, M x N fp32 landing buffer (chunk c at its rows).
 *   C: device, M x N bf16: row chunk c = bf16(A[chunk c] * W^T + partial c).
 *   send_dst: NULL, or n pointers; for every chunk c != rank, send_dst[c]
 *     (device or pinned host, (M/n) x N bf16) receives chunk c of C as soon
 *     as all of its tiles are stored — the emulated send to the next rank.
 *
 * Unused fields of the other pattern may be NULL. Size limits: K and N
 * multiples of 8; M at most 65536 (the row-tile table); the kernel addresses
 * a tile's operands with 32-bit offsets from the tile's first row of A and
 * of the partial (its first column of W), so a 256-row tile may span at most
 * 1 GiB of each: K <= 2^21 and, for the ReduceScatter, N <= 2^20 (InterDecom
 * with d > 1: the row pieces a tile covers, a chunk apart, within the same
 * 1 GiB). Operands may exceed 4 GiB. Beyond these: COMPASS_ERR_UNSUPPORTED. */
typedef struct compass_problem {
    int pattern;
    int M, N, K;
    int n, rank, ring;
    const void *W;
    void *C;
    /* AllGather + GEMM */
    const void *const *shard_src;
    void *gathered;
    /* GEMM + ReduceScatter */
    const void *A;
    const float *const *partial_src;
    float *partial_stage;
    void *const *send_dst;
} compass_problem;

/* ---- TA-IntraFusion: fused AllGather + GEMM (Section III-B, Fig. 6) ------
 * One persistent bf16 MFMA GEMM kernel takes output tiles in ring-arrival
 * order (compass_schedule) and waits on each partition's arrival flag before
 * reading its rows; copy engines deliver the remote shards at the link
 * rates. Returns once everything is enqueued; the kernel ends after every
 * partition arrived and every tile is stored. */
int compass_ag_gemm(const compass_problem *p, const compass_links *links, void *stream);

/* ---- TA-IntraFusion: fused GEMM + ReduceScatter (Section III-B) ----------
 * Tiles run in ReduceScatter order (local chunk last). The main loop never
 * waits; the epilogue of a tile waits for its chunk's incoming partial, adds
 * it in fp32 and stores bf16. When the last tile of a non-local chunk is
 * stored, that chunk is sent to send_dst. A final wait on the stream covers
 * the sends. */
int compass_gemm_rs(const compass_problem *p, const compass_links *links, void *stream);

/* ---- ODP-InterDecom with degree d (Section II-B Fig. 2(c); Section IV) ---
 * d sub-operators: sub-operator j owns row piece j, rows
 * [j*M/(n d), (j+1)*M/(n d)) of every chunk. AllGather: its pieces are
 * gathered over the ring (ring order, paced), then a GEMM over those M/d
 * rows writes them at their global positions; the copy engines run ahead,
 * so gathering piece j+1 overlaps GEMM j. ReduceScatter: sub-GEMM j's
 * epilogue waits for piece j of each chunk's partial. d must be a power of
 * two dividing M/n (M/(2n) for the double ring); d = 1 is the sequential
 * operator. */
int compass_decomp_gemm(const compass_problem *p, int d, const compass_links *links, void *stream);

/* ---- measurement companions ----------------------------------------------
 * compass_gemm: the same GEMM kernel with nothing to wait for (T_gemm).
 *   A: device M x K bf16, W: device N x K bf16, C: device M x N bf16,
 *   P: NULL or device M x N fp32 added before rounding. Same size limits as
 *   a compass_problem (K, N multiples of 8; M at most 65536; a 256-row tile
 *   of A, W and P within 1 GiB, i.e. K <= 2^21 and, with P, N <= 2^20).
 * compass_transfer: exactly the copies the fused operator of `p` issues, at
 *   the same pacing, with no GEMM (T_xfer); a one-workgroup kernel on the
 *   stream starts the copies and ends when the last one landed.
 * compass_sequential: the unfused operator (T_unfused). AllGather: all
 *   copies, then the GEMM (identical to compass_decomp_gemm with d = 1).
 *   ReduceScatter: the GEMM first (its epilogue reads partial_stage as it is
 *   at launch), then the incoming and outgoing copies. */
int compass_gemm(int M, int N, int K, const void *A, const void *W, void *C,
                 const float *P, void *stream);
int compass_transfer(const compass_problem *p, const compass_links *links, void *stream);
int compass_sequential(const compass_problem *p, const compass_links *links, void *stream);

/* ---- compass_gemm for callers that cannot allocate ------------------------
 * For code under HIP graph capture, tight serving loops and harnesses that
 * forbid allocation: the plain GEMM of compass_gemm (same arguments, layout,
 * limits and result: C = A W^T (+ P), fp32 accumulation, one bf16 rounding)
 * without any allocation, library initialisation or copy-side state. Its
 * only scratch, the persistent scheduler's ticket queues and exit counter
 * (256 bytes), lives in a device array of the library's code object, held
 * by each GPU until the process ends; the first call on a device resolves
 * its address. The launch never splits K, so shapes with few output tiles
 * run slower than compass_gemm (which splits K into a workspace). The call
 * enqueues a scratch-clearing kernel and the GEMM on `stream`. Calls that
 * overlap on one GPU (concurrent streams) race on the shared scratch; issue
 * them on one stream. Errors: COMPASS_ERR_INVALID for a bad shape or NULL
 * operand, COMPASS_ERR_UNSUPPORTED beyond the size limits (M above the
 * 65536 rows of the tile table, K above 2^21, N above 2^20 with P)
 * or on a device other than gfx950, COMPASS_ERR_HIP when a launch fails;
 * all before anything is enqueued except the last. */
int compass_gemm_noalloc(int M, int N, int K, const void *A, const void *W, void *C,
                         const float *P, void *stream);

/* Wait until the copy side of every enqueued operator has finished and the
 * device is idle; return the pending asynchronous status (COMPASS_OK or
 * COMPASS_ERR_TIMEOUT) and clear it. COMPASS_ERR_IN_FLIGHT (not cleared) when
 * a failed job's copies did not land within the host-side bound. */
int compass_sync(void);

/* ---- tuning / test options -------------------------------------------- */
#define COMPASS_OPT_SPIN_LIMIT   1  /* max polls of one kernel-side wait (default ~2 s) */
#define COMPASS_OPT_HOST_TIMEOUT 2  /* host-side wait bound, microseconds (default 5 s) */
#define COMPASS_OPT_GRID         3  /* persistent grid size; 0 = one workgroup per CU */
#define COMPASS_OPT_DROP_FLAG    4  /* test only: index of an AllGather partition whose
                                       copy and flag are never issued; -1 = none */
#define COMPASS_OPT_TILE         5  /* GEMM tile: 0 = chosen per operator, 1 = 256 x 256
                                       (one workgroup per CU), 2 = 128 x 128 (two) */
#define COMPASS_OPT_ENGINE_MASK  6  /* bit i set: SDMA engine i may carry emulated link
                                       traffic; 0 = every engine that accepts a copy */
#define COMPASS_OPT_KERNEL_TIMING 7 /* 1: record HIP events on the launch stream around
                                       every GEMM kernel (up to 512 between reads) */
#define COMPASS_OPT_TILE_TRACE   8  /* > 0: record one timing record per work item (an
                                       output tile, or one K slice of a split tile) of
                                       every GEMM launch, up to this many records
                                       (a device buffer of value * 32 bytes); 0 = off */
#define COMPASS_OPT_SCHED        9  /* work dealing, bit mask (default 7): 1 = gated
                                       operators deal one row-tile group per XCD queue,
                                       2 = their first tickets go one per CU, 4 = GEMMs
                                       that do not gate (plain, InterDecom, unfused) with
                                       fewer tiles than half the workgroup slots split K
                                       (fp32 partial tiles in a library workspace of
                                       CUs x 256 KiB, summed in slice order) */
#define COMPASS_OPT_POOL        10  /* operators whose copies all stay in device memory
                                       (not the AlltoAll pattern): > 0 = every ring
                                       direction, incoming and outgoing, shares every copy
                                       engine, each engine with at most this many copies
                                       queued; an engine with room takes the next slice of
                                       the ready item with the earliest due time (unpaced:
                                       due at once, transfer order; paced: when its link,
                                       carrying one item at a time at its rate, would have
                                       delivered it), and a paced item's flag waits for its
                                       due time; slices of 2 MiB paced, 3 MiB unpaced,
                                       unless the links set slice_bytes; 0 = the engines
                                       split per direction in proportion to their bytes
                                       (default 4: queued copies hide the copy side's
                                       reaction time; at most 8). Copies to or from host
                                       memory always keep a job per direction. */
#define COMPASS_OPT_PACE_HEADROOM 12 /* paced links: the engines of a direction form groups
                                       of k per item, the widest k whose groups carry the
                                       link rate with this many per cent to spare (0..100,
                                       default 5); wider groups land each item sooner */
#define COMPASS_OPT_TAIL_MIN_K   13 /* fused AllGather with 256 x 256 tiles: from this K
                                       on, the tiles of the last COMPASS_OPT_TAIL_GROUPS
                                       row-tile groups of the ready order (the last
                                       arrivals) split K into at most 4 slices, each at
                                       least COMPASS_OPT_TAIL_SLICE_K deep, as many as the
                                       workgroup slots over one group's tiles; fp32
                                       partial tiles in the split-K workspace (default
                                       8192; 0 = never; at most 2^21); only while the
                                       operator's estimated comp / comm ratio (the GEMM
                                       at 1 PFLOP/s against the slower direction's
                                       transfer) is below 2 */
#define COMPASS_OPT_TAIL_MIN_K_128 14 /* the same for 128 x 128 tiles (default 0 = never) */
#define COMPASS_OPT_TAIL_SLICE_K 15 /* least K depth of a tail slice, a positive multiple
                                       of 64 (default 2048) */
#define COMPASS_OPT_TAIL_GROUPS  16 /* row-tile groups the tail split covers, 1..8
                                       (default 2); none when the launch has fewer than
                                       twice as many groups */
#define COMPASS_OPT_HEAD_SPLIT  17 /* fused AllGather under the tail split's conditions
                                       (256 x 256 tiles, K from COMPASS_OPT_TAIL_MIN_K,
                                       estimated comp / comm ratio below 2): 1 = the tiles
                                       of the leading row-tile groups whose partitions are
                                       all resident (the rank's own chunk) split K into at
                                       most 4 slices, as many as the workgroup slots over
                                       their tiles, so that the work available before the
                                       first remote partition lands occupies more CUs;
                                       0 = off (default 1) */
int compass_set_option(int key, long long value);

/* Durations in microseconds of the GEMM kernels launched since the previous
 * call (launch order), measured with HIP events recorded on their stream
 * right before and after each launch; waits for those events. Needs
 * COMPASS_OPT_KERNEL_TIMING = 1. Writes at most `cap` values and returns the
 * number written, or a negative status. */
int compass_kernel_times(double *us, int cap);

/* Tile records of the GEMM launches since the previous call (tracing aid for
 * the overlap analysis; needs COMPASS_OPT_TILE_TRACE > 0). Synchronizes the
 * device, copies at most `cap` records of 8 uint32 each into host memory
 * `records` (caller-owned, 32 * cap bytes) and returns the number copied, or
 * a negative status. Records are in launch order, one block per launch with
 * one record per work item (a tile, or one K slice of a split tile), indexed
 * by the item's position in the launch's ready order: [0] position, [1] row
 * tile << 16 | column tile,
 * [2] HW_ID and [3] XCC_ID of the workgroup that ran it, [4..7] the GPU's
 * 100 MHz real-time counter (low 32 bits) when the workgroup took the ticket,
 * passed the arrival gate (ReduceScatter: the epilogue's gate, so [5] comes
 * after [6]), left the main loop and finished the epilogue. */
int compass_tile_trace(uint32_t *records, int cap);

/* Matrix-core probe (roofline context: the bf16 peak the chip sustains under
 * load, against the nominal one at the maximum clock). Launches one
 * workgroup of 8 waves per CU on the null stream; every wave issues `iters`
 * rounds of 8 independent v_mfma_f32_32x32x16_bf16 (no memory traffic) and
 * reads the shader-clock and 100 MHz real-time counters around them.
 * Synchronizes. On success writes the achieved bf16 TFLOP/s over the
 * kernel's event time to *tflops and the mean shader clock during the loop,
 * GHz, to *sclk_ghz. iters must lie in [1, 2^22] (about 1 ms per 4096);
 * COMPASS_ERR_INVALID otherwise or on a null pointer. The library allocates
 * a small result buffer on the first call and keeps it. */
int compass_probe_mfma(int iters, double *tflops, double *sclk_ghz);

/* ---- analytic model and selector (Section IV, Section V, Algorithm 1) ---- */
typedef struct compass_workload {   /* W of Eq. 1 / Eq. 6 */
    int pattern;                    /* COMPASS_AG_GEMM or COMPASS_GEMM_RS     */
    int M, N, K, n;
} compass_workload;

typedef struct compass_topology {   /* T of Eq. 1 / Eq. 6 */
    int    ring;                    /* COMPASS_RING_*                         */
    double fwd_Bps, bwd_Bps;        /* per-direction link rates, bytes/s      */
    double step_latency_s;          /* fixed cost of one ring step            */
} compass_topology;

typedef struct compass_calib {
    double comp_a, comp_b;          /* T_comp = comp_a + comp_b * 2MNK        */
    double alpha_decomp, beta_decomp; /* Eq. 3 */
    double alpha_fusion, beta_fusion; /* Eq. 8 */
    int    d_max;                   /* largest degree considered (Table IV: 16) */
    int    literal_eq5;             /* 1: Eq. 5 exactly as printed (1/lambda);
                                       0: min(lambda, 1/lambda), the minimiser
                                       in both the compute- and the
                                       communication-bound regime            */
} compass_calib;

typedef struct compass_choice {     /* (S*, T*) of Algorithm 1, with details  */
    int    strategy;                /* COMPASS_INTRA_FUSION / _INTER_DECOM    */
    int    d_star, d_cand;          /* Eq. 4 and Eq. 5                        */
    double t_star;                  /* min(T_fusion, T_decomp(d*))            */
    double lambda;                  /* T_comp / T_comm                        */
    double t_comp, t_comm;
    double t_fusion;                /* Eq. 7 + Eq. 8                          */
    double t_decomp;                /* Eq. 2 at d*                            */
    double t_decomp1;               /* Eq. 2 at d = 1 (T_comp + T_comm)       */
} compass_choice;

/* Algorithm 1. T_comp is linear in 2MNK; T_comm is n-1 ring steps, each the
 * slowest active ring's per-link bytes over its rate plus step_latency_s
 * (AllGather moves the M x K bf16 input; ReduceScatter receives M x N fp32
 * partials and sends M x N bf16 sums on the opposite link direction).
 * d* is additionally limited to powers of two that split every chunk (double
 * ring: every half-chunk) evenly. Host only, O(1); needs no GPU. */
int compass_pick_strategy(const compass_workload *w, const compass_topology *t,
                          const compass_calib *cal, compass_choice *out);

/* T_comm of the whole collective under topology t, in seconds (host only):
 * single / double ring as compass_pick_strategy computes it (n - 1 steps);
 * COMPASS_RING_DOUBLE_SPLIT: n - 1 steps of the whole chunk at
 * fwd_Bps + bwd_Bps; COMPASS_RING_ALLTOALL (AllGather, even n): one round,
 * max((m/n) / fwd_Bps, (n/2)^2 (m/n) / bwd_Bps) + step_latency_s (the first
 * term only for n > 2).
 * Returns a negative value for a NULL argument, an unknown ring, n < 1 or a
 * rate the ring needs that is not positive. */
double compass_model_t_comm(const compass_workload *w, const compass_topology *t);

/* Arrival times at `rank` of a single ring with per-hop rates (seconds
 * from the start; the emulator's due times under compass_links.hop_Bps):
 * hop q carries rank q -> q+1 mod n at hop_Bps[q]; every hop carries one
 * piece of piece_bytes at a time; a rank forwards a piece once it holds it.
 * d >= 1 sub-collectives (InterDecom) run one after another on the same
 * hops. out[j*(n-1) + s-1] = arrival of step s (1..n-1) of sub-collective j.
 * Returns d*(n-1), or a negative status (NULL pointers, n outside
 * [1, 32], rank outside [0, n), d < 1, cap too small, a rate that is not
 * positive and finite, piece_bytes < 0). Host only (Section III-A). */
int compass_ring_arrival_times(int n, int rank, double piece_bytes, const double *hop_Bps, int d,
                               double *out, int cap);

/* Eq. 2 and Eq. 7-8 evaluated directly (host only). */
double compass_model_t_decomp(double t_comp, double t_comm, int d, double alpha, double beta);
double compass_model_t_fusion(const compass_workload *w, double t_comp, double t_comm_step,
                              double alpha_f, double beta_f);

/* ---- calibration (Section IV-C: offline linear regression) --------------
 * Each sample is one measurement:
 *   kind 0  GEMM alone:        t_meas of the plain GEMM on workload w
 *   kind 1  InterDecom:        t_meas at degree d, with t_comp / t_comm the
 *                              measured GEMM-alone and transfer-alone times
 *   kind 2  IntraFusion:       t_meas of the fused operator, with t_comp /
 *                              t_comm as above (t_comm = all n-1 steps)
 * compass_calibrate fits comp_a/comp_b by least squares over kind-0 samples,
 * alpha/beta_decomp over the per-sample overhead factors implied by Eq. 2
 * (kind 1, d >= 2), and alpha/beta_fusion over the per-synchronisation
 * overheads implied by Eq. 7 against Eq. 8's volume m (kind 2). Fields with
 * fewer than two distinct abscissae stay as passed in. Host only. */
typedef struct compass_sample {
    int kind;
    compass_workload w;
    int d;
    double t_meas, t_comp, t_comm;
} compass_sample;
int compass_calibrate(const compass_sample *s, int count, compass_calib *inout);

/* Message of the last failing call on this thread ("" if none). */
const char *compass_last_error(void);

/* Library version string. */
const char *compass_version(void);

#ifdef __cplusplus
}
#endif
#endif /* COMPASS_H */
