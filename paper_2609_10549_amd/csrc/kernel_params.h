// Launch parameters shared by the host runtime and the gfx950 kernels.
#pragma once
#include <stdint.h>

namespace compass {

constexpr int kThreads = 256;        // 4 waves of 64, 2 x 2 over the tile
constexpr int kProbeThreads = 512;   // matrix-core probe: 8 waves per workgroup
constexpr int kMaxRowTiles = 512;    // row tiles per launch
constexpr int kMaxParts = 64;        // partitions per launch (2 n, n <= 32)
constexpr int kMaxFlags = 2048;      // arrival / done flag slots
constexpr int kFinalFlag0 = kMaxFlags - 8;  // end-of-job flags
constexpr int kMaxJoin = 80;
constexpr int kMaxQueues = 8;        // ticket queues (one per XCD)
constexpr int kCtrlExit = kMaxQueues;       // ctrl word: exit counter
constexpr int kTraceWords = 8;       // words per tile-trace record
constexpr int kCuSlots = 8 * 256;    // ctrl words: per (XCC, SE/SH/CU id) slot claims
constexpr int kMaxSplitTiles = 512;  // tiles of a split-K launch (one counter each)
constexpr int kMaxSplit = 16;        // K slices per tile
constexpr uint64_t kTileSpanMax = 1ull << 30;   // bytes of A, W or P one tile may span

// Tile configurations of the GEMM kernel.
enum TileCfg : int {
    kTile256 = 0,   // 256 x 256 output tile, 128 KiB LDS, one workgroup per CU
    kTile128 = 1,   // 128 x 128 output tile, 64 KiB LDS, two workgroups per CU
};
inline int tile_rows(int cfg) { return cfg == kTile256 ? 256 : 128; }
inline int tile_cols(int cfg) { return cfg == kTile256 ? 256 : 128; }
inline int tile_wg_per_cu(int cfg) { return cfg == kTile256 ? 1 : 2; }

// Where a tile waits for its partitions' arrival flags.
enum GateMode : int {
    kGateNone = 0,       // everything resident
    kGateMain = 1,       // before the first A load (AllGather)
    kGateEpilogue = 2,   // before adding the incoming partial (ReduceScatter)
};

struct GemmParams {
    const uint16_t *A;   // bf16, rows addressed through the row map below
    const uint16_t *W;   // bf16, N x K
    uint16_t *C;         // bf16 output, rows addressed through the row map
    const float *P;      // fp32 partial added before rounding (or null)
    // aliased partial rows: the partial of (mapped) rows [palt_lo[i],
    // palt_hi[i]) is read from palt[i] + (row - palt_lo[i]) * ldp instead of
    // P (each range a whole number of tiles; empty when lo == hi)
    const float *palt[2];
    int palt_lo[2], palt_hi[2];
    // extents in bytes; a tile's buffer loads (and, with a partial, its
    // stores of C) are bounded by them, from a base at the tile's first row
    // of A, P and C (its first column of W), with 32-bit offsets from there
    // (the host keeps each tile's span of A, W and P below kTileSpanMax; C's
    // rows are half as wide as P's)
    uint64_t a_bytes;
    uint64_t w_bytes;
    uint64_t p_bytes;
    uint64_t c_bytes;
    int M, N, K;         // logical rows of this launch, columns, depth
    int lda, ldw, ldc, ldp;
    int tiles_m, tiles_n;
    // logical row i -> physical row (i / piece) * pstride + poff + i % piece;
    // piece == 0 means the identity map
    int piece, pstride, poff;
    // tile distribution: queue v = blockIdx % nq takes super-blocks
    // v, v + nq, ... of q_size consecutive positions of the ready order;
    // positions walk group_m row tiles before the next column tile
    int nq, q_size, group_m;
    int grid;
    // first-ticket spreading: the second workgroup on a CU (by HW_ID) takes
    // its first ticket only once `spread_wait` tickets of its queue are gone
    // (or after ~10 us), so the first tickets land one per CU; 0 = off.
    // `cu_slots` are claim words tagged with `launch_seq`.
    int spread_wait;
    uint32_t launch_seq;
    uint32_t *cu_slots;
    // split K. Head: the first head_tiles tile positions split into
    // head_split slices of head_kslice (work position u * head_split + j:
    // tile u, slice j), workspace tiles [u * head_split, + head_split),
    // counter u. Then whole tiles up to tile position split_from. From
    // split_from on (the tail), tile position t = split_from + u, slice j,
    // K range [j kslice, (j + 1) kslice), workspace tiles
    // head_tiles * head_split + u * ksplit + j, counter head_tiles + u.
    // Every slice stores its fp32 partial tile in the workspace; the slice
    // that completes its tile's count sums the partials in slice order and
    // runs the epilogue. ksplit == 1: no tail split (kslice = K);
    // split_from == 0: every tile after the head split (needs head_tiles ==
    // 0); head_tiles == 0: no head split.
    int ksplit, kslice, split_from;
    int head_tiles, head_split, head_kslice;
    uint32_t *split_cnt;
    float *split_ws;
    // gating: flag index of partition p is flag_base + p. Arrival flags live
    // in pinned host memory (written by the copy-side threads); the first
    // workgroup that needs a partition in an epoch (`leader`) polls it and
    // copies it into `mirror` (device memory), which the others poll.
    uint32_t *flags;
    uint32_t *mirror;
    uint32_t *leader;
    int gate;                // GateMode
    int flag_base;
    int nparts;              // partitions used by this launch
    uint64_t resident_mask;  // partitions present before the launch (no wait)
    uint64_t send_mask;      // partitions whose completion is signalled
    uint32_t epoch;
    uint32_t spin_limit;
    // ReduceScatter chunk-done tracking (done_host null: off)
    uint32_t *done_cnt;      // device counters, indexed like flags
    uint32_t *done_host;     // host-visible done flags, indexed like flags
    // control
    uint32_t *ctrl;          // [0, nq) tickets, [kCtrlExit] exit counter
    uint32_t *start_word;    // host-visible; written with epoch at start (or null)
    uint32_t *err_word;      // host-visible error word
    // optional tile trace: record (trace_base + position) gets kTraceWords
    // words: position, row tile << 16 | column tile, HW_ID, XCC_ID, and the
    // 100 MHz real-time counter (low 32 bits) at ticket, after the gate, after
    // the main loop and after the epilogue
    uint32_t *tile_trace;
    uint32_t trace_base, trace_cap;
    uint16_t rt_order[kMaxRowTiles];   // ready order of the row tiles
    uint8_t rt_lo[kMaxRowTiles];       // partitions [lo, hi] a row tile depends on
    uint8_t rt_hi[kMaxRowTiles];
    uint32_t done_expect[kMaxParts];   // tiles per partition to count (0: none)
};

struct JoinParams {
    uint32_t *flags;
    uint32_t *start_word;   // written with epoch first (or null)
    uint32_t *err_word;
    uint32_t epoch;
    uint32_t spin_limit;
    int count;
    uint16_t idx[kMaxJoin];
};

// Work items (tickets) of a launch: the head's slices, the whole tiles,
// the tail's slices.
__host__ __device__ inline int work_items(const GemmParams &p) {
    const int tiles = p.tiles_m * p.tiles_n;
    return p.head_tiles * p.head_split + (p.split_from - p.head_tiles) + (tiles - p.split_from) * p.ksplit;
}

// One work item: the tile at position `tpos` of the ready order and, when
// its K is split (`split`), slice `slice` of `ns`, covering K from
// slice * ksl (at most ksl deep), counted by split counter `uc`, its
// partial at workspace tile wsf + slice (the tile's slices at [wsf,
// wsf + ns)). An unsplit tile runs its whole K (slice 0 of 1).
struct WorkItem {
    int tpos, slice, ns, uc, wsf, ksl;
    bool split;
};

// Work position -> work item: positions [0, head_tiles * head_split) are
// the head's slices (tile u = pos / head_split), then the whole tiles up to
// tile position split_from, then the tail's slices (ksplit per tile).
__host__ __device__ inline WorkItem decode_item(const GemmParams &p, int pos) {
    const int head_items = p.head_tiles * p.head_split;
    WorkItem w;
    w.slice = 0;
    w.ns = 1;
    w.uc = 0;
    w.wsf = 0;
    w.ksl = p.K;
    w.split = false;
    if (pos < head_items) {
        w.uc = pos / p.head_split;
        w.slice = pos - w.uc * p.head_split;
        w.tpos = w.uc;
        w.split = true;
        w.ns = p.head_split;
        w.wsf = w.uc * p.head_split;
        w.ksl = p.head_kslice;
    } else {
        const int q = pos - head_items + p.head_tiles;   // position in the unsplit-head order
        if (p.ksplit > 1 && q >= p.split_from) {
            const int u = (q - p.split_from) / p.ksplit;
            w.slice = q - p.split_from - u * p.ksplit;
            w.tpos = p.split_from + u;
            w.split = true;
            w.ns = p.ksplit;
            w.uc = p.head_tiles + u;
            w.wsf = head_items + u * p.ksplit;
            w.ksl = p.kslice;
        } else {
            w.tpos = q;
        }
    }
    return w;
}

// Tile position -> (row-tile ordinal in rt_order, column tile): positions
// walk group_m row tiles (fewer in a last, partial group) before the next
// column tile.
__host__ __device__ inline void tile_of(const GemmParams &p, int tpos, int *ti, int *tn) {
    const int gsz = p.group_m * p.tiles_n;
    const int grp = tpos / gsz;
    const int rin = tpos - grp * gsz;
    const int left = p.tiles_m - grp * p.group_m;
    const int rows_here = p.group_m < left ? p.group_m : left;
    *ti = grp * p.group_m + rin % rows_here;
    *tn = rin / rows_here;
}

}  // namespace compass
