// gfx950 kernels of the Compass hot path.
//
// gemm_kernel<BM, BN, RS, WT>: persistent bf16 GEMM, C = A * W^T with fp32
// accumulation on the CDNA4 matrix cores (v_mfma_f32_32x32x16_bf16) and one
// bf16 round-to-nearest-even store. Workgroups take BM x BN output tiles from
// atomic ticket queues in the order the host chose (ring-arrival order for
// TA-IntraFusion, Section III-B), and, depending on the gate mode, wait on the
// per-partition arrival flags published for the copy engines before reading A
// (AllGather) or before adding the incoming partial sum (ReduceScatter).
//
// Tile distribution: the ready order of tiles is cut into super-blocks; queue
// v (one per XCD: workgroups are dispatched round-robin over the 8 XCDs, so
// workgroup b serves queue b % 8) takes super-blocks v, v + 8, ...; inside
// the order, positions walk a group of row tiles before moving to the next
// column tile, so the tiles one XCD holds at a time share A rows and W rows
// in that XCD's L2.
//
// Data path per tile: 4 waves split the tile 2 x 2; each wave holds
// (BM/2) x (BN/2) fp32 accumulators as 32 x 32 MFMA blocks. A and W stream
// through two LDS stages of K = 64 (rows of 128 bytes, whole cache lines per
// load: the texture path's cost grows with the lines a load touches) with
// buffer_load ... lds (no register staging; out-of-range rows or K columns
// read as zero through the buffer bound). The one barrier per stage sits
// before its last substep: by then every wave has read that stage's
// fragments, so the next-but-one stage's loads may overwrite it, and the next
// stage's first fragments are read while the last substep computes. Loads of
// stage s + 1 go out in the last substep of stage s - 1 (A) and the first of
// stage s (W). Fragment reads of the next substep are issued between the
// current one's MFMAs; scheduling barriers keep the compiler from sinking
// them to their use. The 16-byte chunks of LDS row r are XOR-permuted with
// (r >> 1) & 7, so a 32-row fragment read hits distinct banks.
//
// join_kernel: one wave that (optionally) marks the start of a transfer job
// and waits for a list of flags, putting the end of the copy side onto the
// stream.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernel_params.h"

namespace compass {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

#define LDS_AS(p) ((__attribute__((address_space(3))) void *)(p))

// Buffer loads of a tile go through a resource based at the tile's first
// row (A, the partial) or first column (W), bounded by the bytes left in the
// operand, at most kTileSpanMax; offsets are relative to that base. An
// out-of-range row or column takes an offset at or beyond the bound:
// kOOBRow = 2^31 for a row, kOOBCol = 2^30 for a K column. A valid row offset
// plus a valid column offset stays below the 2^30 bound (the host checks the
// tile's span), a valid one plus an out-of-range one reaches it, and two
// out-of-range ones sum to 3 * 2^30, below 2^32, so no sum wraps.
constexpr uint32_t kOOBRow = 0x80000000u;
constexpr uint32_t kOOBCol = 0x40000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const void *base, uint64_t total, uint64_t off) {
    const uint64_t left = total > off ? total - off : 0;
    const uint32_t bound = (uint32_t)(left < kTileSpanMax ? left : kTileSpanMax);
    return __builtin_amdgcn_make_buffer_rsrc((void *)((const char *)base + off), (short)0, (int)bound, 0x00020000);
}

__device__ __forceinline__ uint32_t ld_flag(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__device__ __forceinline__ uint32_t ld_dev(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Poll *w until it reaches epoch; false on the bound or a raised error word.
__device__ __forceinline__ bool poll_epoch(const uint32_t *w, bool host, uint32_t epoch, uint32_t limit,
                                           uint32_t *err, int sleep_code) {
    uint32_t polls = 0;
    while ((int32_t)((host ? ld_flag(w) : ld_dev(w)) - epoch) < 0) {
        if (++polls > limit) {
            __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
            return false;
        }
        if ((polls & 255u) == 0 && ld_flag(err) != 0) return false;
        if (sleep_code == 4) __builtin_amdgcn_s_sleep(4);
        else __builtin_amdgcn_s_sleep(16);
    }
    return true;
}

// Wait of wave 0 for every partition in `mask` (bit q: partition q, at most
// 64): lane q handles partition q, so the flags are polled in parallel. Per
// partition and epoch one workgroup (the first to claim `leader`) polls the
// host-memory arrival flag and forwards it to `mirror` in device memory;
// every other workgroup polls the mirror. A system-scope acquire follows, so
// that the rows the copy engines wrote are read from memory, not from stale
// cache lines. True when every partition arrived (false: bound or error).
__device__ bool wait_flags(const GemmParams &p, uint64_t mask, int lane) {
    bool ok = true;
    if ((mask >> lane) & 1ull) {
        const int f = p.flag_base + lane;
        if ((int32_t)(ld_dev(&p.mirror[f]) - p.epoch) < 0) {
            uint32_t cur = ld_dev(&p.leader[f]);
            bool lead = false;
            while ((int32_t)(cur - p.epoch) < 0) {
                uint32_t expect = cur;
                if (__hip_atomic_compare_exchange_strong(&p.leader[f], &expect, p.epoch, __ATOMIC_RELAXED,
                                                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
                    lead = true;
                    break;
                }
                cur = expect;
            }
            if (lead) {
                ok = poll_epoch(&p.flags[f], true, p.epoch, p.spin_limit, p.err_word, 16);
                if (ok) __hip_atomic_store(&p.mirror[f], p.epoch, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
            } else {
                ok = poll_epoch(&p.mirror[f], false, p.epoch, p.spin_limit, p.err_word, 4);
            }
        }
    }
    const bool all_ok = __ballot(!ok) == 0ull;
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
    return all_ok;
}

__device__ __forceinline__ uint32_t rtc32() { return (uint32_t)__builtin_amdgcn_s_memrealtime(); }

__device__ __forceinline__ uint32_t hw_id() {
    uint32_t v;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(v));
    return v;
}

__device__ __forceinline__ uint32_t xcc_id() {
    uint32_t v;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
    return v;
}

// Order of this workgroup among the workgroups of this launch on its CU
// (0 for the first): a claim word per (XCC, SE, SH, CU) holds
// launch_seq << 8 | count.
__device__ uint32_t claim_cu_slot(const GemmParams &p) {
    const uint32_t key = ((xcc_id() & 7u) << 8) | ((hw_id() >> 8) & 0xFFu);
    uint32_t *w = p.cu_slots + key;
    const uint32_t tag = p.launch_seq & 0xFFFFFFu;
    uint32_t cur = ld_dev(w);
    for (;;) {
        const bool same = (cur >> 8) == tag;
        const uint32_t want = same ? cur + 1u : ((tag << 8) | 1u);
        uint32_t expect = cur;
        if (__hip_atomic_compare_exchange_strong(w, &expect, want, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT))
            return same ? (cur & 0xFFu) : 0u;
        cur = expect;
    }
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const __bf16 a = (__bf16)lo, b = (__bf16)hi;   // round to nearest even
    return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

__device__ __forceinline__ int map_row(const GemmParams &p, int i) {
    if (p.piece == 0) return i;
    const int q = i / p.piece;
    return q * p.pstride + p.poff + (i - q * p.piece);
}

__device__ __forceinline__ uint64_t range_mask(int lo, int hi) {
    const uint64_t upto = hi >= 63 ? ~0ull : ((2ull << hi) - 1ull);
    return upto & ~((1ull << lo) - 1ull);
}

// Position in the ready order of local ticket c of queue v.
__device__ __forceinline__ int ticket_position(const GemmParams &p, int v, uint32_t c) {
    const int k = (int)(c / (uint32_t)p.q_size);
    const int i = (int)(c - (uint32_t)k * (uint32_t)p.q_size);
    return (v + p.nq * k) * p.q_size + i;
}

// s_waitcnt vmcnt(VM) lgkmcnt(0), expcnt untouched (gfx9 encoding)
template <int VM>
__device__ __forceinline__ void wait_vm_lgkm0() {
    static_assert(VM >= 0 && VM < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4));
}

// Workgroup barrier with no memory fence: the caller has already waited for
// the LDS traffic that must be complete (s_waitcnt), and the scheduling
// barriers keep the compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// CNT global -> LDS loads (16 bytes per lane, 1 KiB per wave and load) of one
// operand into the 1 KiB blocks (q0 + j) * 4 + wave of `lds`.
template <int CNT>
__device__ __forceinline__ void load_blocks(__amdgpu_buffer_rsrc_t rsrc, char *lds, const uint32_t *off, int q0,
                                            uint32_t kc2, int wave) {
#pragma unroll
    for (int j = 0; j < CNT; ++j)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, LDS_AS(lds + ((q0 + j) * 4 + wave) * 1024), 16,
                                                 off[q0 + j] + kc2, 0, 0, 0);
}

// Fragments of MFMA substep kk of the stage in (sA, sW): ROWB-byte rows,
// 16-byte chunk c of row r stored at chunk c ^ swz.
template <int FM, int FN, int ROWB>
__device__ __forceinline__ void read_frags(const char *sA, const char *sW, int r, int swz, int kk, int hi, int wm0,
                                           int wn0, bf16x8 (&a)[FM], bf16x8 (&b)[FN]) {
    const int coff = ((2 * kk + hi) ^ swz) << 4;
#pragma unroll
    for (int mi = 0; mi < FM; ++mi)
        a[mi] = *reinterpret_cast<const bf16x8 *>(sA + (wm0 + mi * 32 + r) * ROWB + coff);
#pragma unroll
    for (int ni = 0; ni < FN; ++ni)
        b[ni] = *reinterpret_cast<const bf16x8 *>(sW + (wn0 + ni * 32 + r) * ROWB + coff);
}

// MFMAs [I0, I0 + CNT) of a substep (block i: acc[i / FM][i % FM]).
template <int I0, int CNT, int FM, int FN>
__device__ __forceinline__ void mfma_range(f32x16 (&acc)[FN][FM], const bf16x8 (&a)[FM], const bf16x8 (&b)[FN]) {
#pragma unroll
    for (int i = I0; i < I0 + CNT; ++i)
        acc[i / FM][i % FM] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[i / FM], a[i % FM], acc[i / FM][i % FM], 0, 0, 0);
}

// Scheduling groups for the CNT MFMAs just emitted: one instruction of class
// MASK (NX in all) after each MFMA, the rest after the last; then a barrier
// that nothing is scheduled across.
template <int CNT, int MASK, int NX>
__device__ __forceinline__ void interleave() {
#pragma unroll
    for (int i = 0; i < CNT - 1; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (i < NX) __builtin_amdgcn_sched_group_barrier(MASK, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if constexpr (NX > CNT - 1) __builtin_amdgcn_sched_group_barrier(MASK, NX - (CNT - 1), 0);
    __builtin_amdgcn_sched_barrier(0);
}

constexpr int kDsRead = 0x100, kVmemRead = 0x020;

constexpr int kBK = 64;   // K depth of one LDS stage

// ---- the pipeline: two LDS stages of K = 64, barrier before the last substep
// Stage s on (cA, cW), substep-0 fragments in (a0, b0). Substep 0 issues the
// W loads of stage s + 1 into (nA, nW) (its A loads went out in stage s - 1);
// substep 3 waits for all of stage s + 1, joins the barrier, reads stage
// s + 1's first fragments and issues the A loads of stage s + 2 into
// (cA, cW), which no wave reads any more.
template <int BM, int BN, int FM, int FN>
__device__ __forceinline__ void stage2e(char *cA, char *cW, char *nA, char *nW, f32x16 (&acc)[FN][FM],
                                        bf16x8 (&a0)[FM], bf16x8 (&b0)[FN], bf16x8 (&a1)[FM], bf16x8 (&b1)[FN],
                                        __amdgpu_buffer_rsrc_t rA, __amdgpu_buffer_rsrc_t rW, const uint32_t *offA,
                                        const uint32_t *offW, uint32_t kc2_next, uint32_t kc2_next2, int r, int swz,
                                        int hi, int wm0, int wn0, int wave) {
    constexpr int NM = FM * FN, H = NM / 2, ND = FM + FN;
    constexpr int L = BM / 32;   // loads per wave and operand per stage
    // substep 0
    read_frags<FM, FN, 128>(cA, cW, r, swz, 1, hi, wm0, wn0, a1, b1);
    mfma_range<0, H, FM, FN>(acc, a0, b0);
    interleave<H, kDsRead, ND>();
    load_blocks<L>(rW, nW, offW, 0, kc2_next, wave);
    mfma_range<H, NM - H, FM, FN>(acc, a0, b0);
    interleave<NM - H, kVmemRead, L>();
    // substep 1
    read_frags<FM, FN, 128>(cA, cW, r, swz, 2, hi, wm0, wn0, a0, b0);
    mfma_range<0, H, FM, FN>(acc, a1, b1);
    interleave<H, kDsRead, ND>();
    mfma_range<H, NM - H, FM, FN>(acc, a1, b1);
    interleave<NM - H, kVmemRead, 0>();
    // substep 2
    read_frags<FM, FN, 128>(cA, cW, r, swz, 3, hi, wm0, wn0, a1, b1);
    mfma_range<0, H, FM, FN>(acc, a0, b0);
    interleave<H, kDsRead, ND>();
    mfma_range<H, NM - H, FM, FN>(acc, a0, b0);
    interleave<NM - H, kVmemRead, 0>();
    // substep 3
    wait_vm_lgkm0<0>();
    lds_barrier();
    read_frags<FM, FN, 128>(nA, nW, r, swz, 0, hi, wm0, wn0, a0, b0);
    mfma_range<0, H, FM, FN>(acc, a1, b1);
    interleave<H, kDsRead, ND>();
    load_blocks<L>(rA, cA, offA, 0, kc2_next2, wave);
    mfma_range<H, NM - H, FM, FN>(acc, a1, b1);
    interleave<NM - H, kVmemRead, L>();
}

// RS = false: optional main-loop gate (AllGather), plain store.
// RS = true: optional epilogue gate, fp32 partial add, chunk-done signalling;
// WT = true (a launch whose finished chunks the copy engines send on): the
// partial-add epilogue stores every tile with system-scope write-through.
template <int BM, int BN, bool RS, bool WT = false>
__global__ __launch_bounds__(kThreads, BM == 256 ? 1 : 2)
void gemm_kernel(const GemmParams p) {
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int FM = WM / 32, FN = WN / 32;
    constexpr int NOFF = BM / 32;   // loads per wave, operand and stage
    static_assert(BM == BN && BM * 128 >= 16384, "square tiles; stage buffers hold the epilogue patches");
    __shared__ __attribute__((aligned(1024))) char sA0[BM * 128];
    __shared__ __attribute__((aligned(1024))) char sA1[BM * 128];
    __shared__ __attribute__((aligned(1024))) char sW0[BN * 128];
    __shared__ __attribute__((aligned(1024))) char sW1[BN * 128];
    __shared__ int s_pos;
    __shared__ int s_ok;
    __shared__ int s_last;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm0 = (wave >> 1) * WM;
    const int wn0 = (wave & 1) * WN;
    const int total = work_items(p);
    const int v = p.nq > 1 ? (int)(blockIdx.x % (uint32_t)p.nq) : 0;


    // loader geometry: load q of this wave covers tile rows 32 q + 8 wave +
    // (lane >> 3), 128 bytes (K = 64) each; the lane loads the logical chunk
    // that the permutation (row >> 1) & 7 puts at its physical chunk lane & 7
    const int lrow0 = 8 * wave + (lane >> 3);
    const int cchunk = (lane & 7) ^ ((4 * wave + (lane >> 4)) & 7);
    const int r = lane & 31;                       // fragment row
    const int hi = lane >> 5;                      // fragment K half
    const int swz = (r >> 1) & 7;

    uint64_t known = 0;   // partitions already acquired by this workgroup
    bool failed = false;

    if (tid == 0) {
        if (p.spread_wait > 0 && claim_cu_slot(p) > 0) {
            // bounded: a scheduling preference, never a dependency
            const uint32_t t_end = rtc32() + 1000u;   // 10 us of the 100 MHz counter
            while ((int)ld_dev(&p.ctrl[v]) < p.spread_wait && (int32_t)(rtc32() - t_end) < 0)
                __builtin_amdgcn_s_sleep(2);
        }
        const uint32_t c = __hip_atomic_fetch_add(&p.ctrl[v], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int pos = ticket_position(p, v, c);
        if (pos == 0 && p.start_word)
            __hip_atomic_store(p.start_word, p.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        s_pos = pos;
    }
    __syncthreads();
    int pos = s_pos;

    while (pos < total) {
        // work position -> (tile position, K slice); `split`: this tile's K
        // is split into `ns` slices, counted by split_cnt[uc], its partials
        // at workspace tiles [wsf, wsf + ns)
        const WorkItem wi = decode_item(p, pos);
        const bool split = wi.split;
        const int tpos = wi.tpos, slice = wi.slice, ns = wi.ns, uc = wi.uc, wsf = wi.wsf, ksl = wi.ksl;
        const int kb = split ? slice * ksl : 0;
        const int ke = split ? min(p.K, kb + ksl) : p.K;
        // tile position -> (row-tile ordinal, column tile): group_m rows at a time
        int ti, tn;
        tile_of(p, tpos, &ti, &tn);
        const int rt = p.rt_order[ti];
        const int m0 = rt * BM;
        const int n0 = tn * BN;
        const uint64_t touch = range_mask(p.rt_lo[rt], p.rt_hi[rt]);
        const uint64_t need = touch & ~p.resident_mask & ~known;
        const bool traced = p.tile_trace && p.trace_base + (uint32_t)pos < p.trace_cap;
        uint32_t t_tick = 0, t_gate = 0, t_loop = 0;
        if (traced && tid == 0) t_tick = rtc32();

        if (!RS && p.gate == kGateMain && need) {
            if (wave == 0) {
                const bool ok = wait_flags(p, need, lane);
                if (lane == 0) s_ok = ok;
            }
            __syncthreads();
            if (!s_ok) failed = true;
            known |= need;
        }
        if (!RS && traced && tid == 0) t_gate = rtc32();

        f32x16 acc[FN][FM];
#pragma unroll
        for (int ni = 0; ni < FN; ++ni)
#pragma unroll
            for (int mi = 0; mi < FM; ++mi)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[ni][mi][e] = 0.0f;

        {   // a timed-out tile still runs (its loads stay in bounds); only its
            // stores are dropped
            // A from the tile's first (mapped) row, W from its first column
            const int row0 = map_row(p, m0);
            const __amdgpu_buffer_rsrc_t rA = tile_rsrc(p.A, p.a_bytes, (uint64_t)row0 * (uint64_t)p.lda * 2u);
            const __amdgpu_buffer_rsrc_t rW = tile_rsrc(p.W, p.w_bytes, (uint64_t)n0 * (uint64_t)p.ldw * 2u);
            uint32_t offA[NOFF], offW[NOFF];
#pragma unroll
            for (int q = 0; q < NOFF; ++q) {
                const int ia = m0 + 32 * q + lrow0;
                offA[q] = ia < p.M ? (uint32_t)(map_row(p, ia) - row0) * (uint32_t)p.lda * 2u : kOOBRow;
                const int iw = n0 + 32 * q + lrow0;
                offW[q] = iw < p.N ? (uint32_t)(iw - n0) * (uint32_t)p.ldw * 2u : kOOBRow;
            }
            auto kcol = [&](int st) -> uint32_t {   // byte offset of this lane's K chunk in stage st
                const int kc = kb + st * kBK + cchunk * 8;
                return kc < ke ? (uint32_t)kc * 2u : kOOBCol;
            };
            // an even stage count keeps the unrolled loop free of early exits
            // (padding stages read only out-of-range columns, i.e. zeros)
            const int KT = (((ke - kb + kBK - 1) / kBK) + 1) & ~1;
            // prologue: stage 0 and the A half of stage 1 in flight; stage 0
            // landed, its first fragments read
            load_blocks<NOFF>(rA, sA0, offA, 0, kcol(0), wave);
            load_blocks<NOFF>(rW, sW0, offW, 0, kcol(0), wave);
            load_blocks<NOFF>(rA, sA1, offA, 0, kcol(1), wave);
            wait_vm_lgkm0<NOFF>();
            lds_barrier();
            bf16x8 a0[FM], b0[FN], a1[FM], b1[FN];
            read_frags<FM, FN, 128>(sA0, sW0, r, swz, 0, hi, wm0, wn0, a0, b0);
            for (int st = 0; st < KT; st += 2) {
                stage2e<BM, BN, FM, FN>(sA0, sW0, sA1, sW1, acc, a0, b0, a1, b1, rA, rW, offA, offW, kcol(st + 1),
                                        kcol(st + 2), r, swz, hi, wm0, wn0, wave);
                stage2e<BM, BN, FM, FN>(sA1, sW1, sA0, sW0, acc, a0, b0, a1, b1, rA, rW, offA, offW, kcol(st + 2),
                                        kcol(st + 3), r, swz, hi, wm0, wn0, wave);
            }
            // the loads issued past the end (zeros) land before the buffers
            // are reused
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
        }

        if (traced && tid == 0) t_loop = rtc32();
        // fetch the next ticket while the epilogue runs
        if (tid == 0) {
            const uint32_t c = __hip_atomic_fetch_add(&p.ctrl[v], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_pos = ticket_position(p, v, c);
        }

        // Each 32 x 32 fp32 block of the accumulators goes through a per-wave
        // 4 KiB LDS patch (rows of 128 bytes, 16-byte chunks XOR-permuted by
        // row & 7) and comes back row-contiguous: 8 lanes per row hold 128
        // contiguous bytes. `emit(tile row, tile column, 4 values)`.
        char *patch = sA0 + wave * 4096;
        auto through_patch = [&](auto &&emit) {
            const int rr = lane >> 3;          // read-back row within 8
            const int rc = lane & 7;           // read-back chunk (4 floats)
#pragma unroll
            for (int mi = 0; mi < FM; ++mi) {
#pragma unroll
                for (int ni = 0; ni < FN; ++ni) {
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int cc = 2 * g + hi;
                        f32x4 v4 = {acc[ni][mi][4 * g + 0], acc[ni][mi][4 * g + 1],
                                    acc[ni][mi][4 * g + 2], acc[ni][mi][4 * g + 3]};
                        *reinterpret_cast<f32x4 *>(patch + r * 128 + ((cc ^ (r & 7)) << 4)) = v4;
                    }
                    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): patch written
#pragma unroll
                    for (int it = 0; it < 4; ++it) {
                        const int row = rr + 8 * it;
                        const f32x4 x = *reinterpret_cast<const f32x4 *>(patch + row * 128 + ((rc ^ (row & 7)) << 4));
                        emit(wm0 + mi * 32 + row, wn0 + ni * 32 + 4 * rc, x);
                    }
                    __builtin_amdgcn_s_waitcnt(0xC07F);   // patch read before reuse
                }
            }
        };
        const int mlim = failed ? 0 : p.M;   // a failed tile stores nothing
        // the tile's partial sum: from P, or, for the rows of an aliased
        // range (a whole number of tiles), from that range's own buffer
        const float *pbase = p.P;
        int plo = 0;
        uint64_t pbytes = p.p_bytes;
        if (RS) {
            const int pm0 = map_row(p, m0);
#pragma unroll
            for (int i = 0; i < 2; ++i)
                if (pm0 >= p.palt_lo[i] && pm0 < p.palt_hi[i]) {
                    pbase = p.palt[i];
                    plo = p.palt_lo[i];
                    pbytes = (uint64_t)(p.palt_hi[i] - plo) * (uint64_t)p.ldp * 4u;
                }
        }
        // a tile of a chunk that is sent on (ReduceScatter) stores with
        // system-scope write-through, so that no L2 write-back is needed
        // before the copy engines read it
        const bool wt = RS && p.done_host != nullptr && (touch & p.send_mask) != 0;
        // bf16 store of 4 values at tile (row, col), after adding the fp32
        // partial sum (ReduceScatter): 64 contiguous bytes of C per row
        auto store4 = [&](int row, int col, float v0, float v1, float v2, float v3, bool add_p) {
            const int m = m0 + row, n = n0 + col;
            if (m < mlim && n < p.N) {
                const int pm = map_row(p, m);
                if (add_p) {
                    const f32x4 pv = *reinterpret_cast<const f32x4 *>(pbase + (size_t)(pm - plo) * p.ldp + n);
                    v0 += pv[0]; v1 += pv[1]; v2 += pv[2]; v3 += pv[3];
                }
                const uint64_t o = (uint64_t)pack_bf16x2(v0, v1) | ((uint64_t)pack_bf16x2(v2, v3) << 32);
                uint64_t *dst = reinterpret_cast<uint64_t *>(p.C + (size_t)pm * p.ldc + n);
                if (wt)   // written through to memory: the copy engines read it
                    __hip_atomic_store(dst, o, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
                else
                    *dst = o;
            }
        };
        const bool has_p = RS && p.P != nullptr;

        // split K: every slice stores its partial tile (fp32, row-major);
        // the slice that completes the tile's count sums all of them in
        // slice order, so the result does not depend on which one was last
        bool finish = true;
        if (split) {
            float *ws = p.split_ws + (size_t)(wsf + slice) * (BM * BN);
            through_patch([&](int row, int col, f32x4 x) {
                *reinterpret_cast<f32x4 *>(ws + row * BN + col) = x;
            });
            // The workspace is uncached device memory: a store acknowledged
            // to the wave is in memory, visible to every XCD, and loads read
            // memory. So ordering needs no cache maintenance: each wave waits
            // for its stores, the barrier joins the waves, then the count.
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            if (tid == 0) {
                const uint32_t old = __hip_atomic_fetch_add(&p.split_cnt[uc], 1u, __ATOMIC_RELAXED,
                                                            __HIP_MEMORY_SCOPE_AGENT);
                const bool last = old + 1u == (uint32_t)ns;
                if (last) __hip_atomic_store(&p.split_cnt[uc], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                s_last = last;
            }
            __syncthreads();   // the partial loads below are issued after the count
            finish = s_last != 0;
        }

        if (RS && finish && p.gate == kGateEpilogue && need) {
            if (wave == 0) {
                const bool ok = !failed && wait_flags(p, need, lane);
                if (lane == 0) s_ok = ok;
            }
            __syncthreads();
            if (!s_ok) failed = true;
            known |= need;
        }
        if (RS && traced && tid == 0) t_gate = rtc32();

        if (finish) {
            if (split) {
                const float *ws0 = p.split_ws + (size_t)wsf * (BM * BN);
                // B elements of 4 per thread at a time, all their slices' loads
                // (and the partial sum's) in flight at once, then each summed in
                // slice order: the workspace is uncached, so every load costs a
                // memory round trip, and B x S of them overlap. With the slice
                // count a compile-time constant (EX) the loads carry no branch,
                // and the waits before the sums count them exactly; otherwise
                // S is an upper bound and slices from ns on are skipped.
                auto finish_split = [&](auto b_const, auto s_const, auto ex_const) {
                    constexpr int B = decltype(b_const)::value, S = decltype(s_const)::value;
                    constexpr bool EX = decltype(ex_const)::value;
                    constexpr int E = BM * BN / 4;
                    static_assert(E % (kThreads * B) == 0, "whole batches");
                    for (int e0 = tid; e0 < E; e0 += kThreads * B) {
                        f32x4 part[B][S];
                        f32x4 pv[B];
#pragma unroll
                        for (int b = 0; b < B; ++b) {
                            const int e = e0 + b * kThreads;
                            const int row = e / (BN / 4), col = (e - row * (BN / 4)) * 4;
#pragma unroll
                            for (int jj = 0; jj < S; ++jj)
                                if (EX || jj < ns)
                                    part[b][jj] = *reinterpret_cast<const f32x4 *>(ws0 + (size_t)jj * (BM * BN) +
                                                                                    row * BN + col);
                            pv[b] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                            const int m = m0 + row, n = n0 + col;
                            if (has_p && m < p.M && n < p.N)
                                pv[b] = *reinterpret_cast<const f32x4 *>(pbase + (size_t)(map_row(p, m) - plo) * p.ldp +
                                                                         n);
                        }
#pragma unroll
                        for (int b = 0; b < B; ++b) {
                            const int e = e0 + b * kThreads;
                            const int row = e / (BN / 4), col = (e - row * (BN / 4)) * 4;
                            f32x4 sum = part[b][0];
#pragma unroll
                            for (int jj = 1; jj < S; ++jj)
                                if (EX || jj < ns) {
                                    sum[0] += part[b][jj][0]; sum[1] += part[b][jj][1];
                                    sum[2] += part[b][jj][2]; sum[3] += part[b][jj][3];
                                }
                            store4(row, col, sum[0] + pv[b][0], sum[1] + pv[b][1], sum[2] + pv[b][2],
                                   sum[3] + pv[b][3], false);
                        }
                    }
                };
                // The host splits a tile into 2 to 8 slices (more only through
                // kMaxSplit): each count has its own branch-free instance. Batches
                // of 4 elements (2 from 5 slices on, and in the ReduceScatter
                // variant, whose partial-sum epilogue leaves fewer registers) keep
                // the loads within the registers the main loop leaves, with no
                // spills.
                constexpr int BL = RS ? 2 : 4;
                using yes = std::true_type;
                using no = std::false_type;
                using std::integral_constant;
                switch (ns) {
                case 2: finish_split(integral_constant<int, BL>{}, integral_constant<int, 2>{}, yes{}); break;
                case 3: finish_split(integral_constant<int, BL>{}, integral_constant<int, 3>{}, yes{}); break;
                case 4: finish_split(integral_constant<int, BL>{}, integral_constant<int, 4>{}, yes{}); break;
                case 5: finish_split(integral_constant<int, 2>{}, integral_constant<int, 5>{}, yes{}); break;
                case 6: finish_split(integral_constant<int, 2>{}, integral_constant<int, 6>{}, yes{}); break;
                case 7: finish_split(integral_constant<int, 2>{}, integral_constant<int, 7>{}, yes{}); break;
                case 8: finish_split(integral_constant<int, 2>{}, integral_constant<int, 8>{}, yes{}); break;
                default:
                    finish_split(integral_constant<int, BL / 2>{}, integral_constant<int, kMaxSplit>{}, no{});
                }
            } else if (has_p) {
                // as through_patch, with each 32 x 32 block's fp32 partial
                // brought into LDS by buffer_load ... lds two blocks ahead of
                // its use, into three 4 KiB buffers per wave, one in each of
                // the freed stage buffers sA1, sW0 and sW1. C goes out through
                // buffer stores that the buffer bound drops for rows or
                // columns outside C (or all of a failed tile), so every block
                // issues the same memory operations and the wait for a
                // block's partial lets the two later blocks' loads and the
                // stores in between stay in flight (with one block ahead, or
                // with stores skipped by a branch, it waited for all of them:
                // the epilogue took 17 us per 256 x 256 tile at any number of
                // workgroups, against 7 us without a partial)
                constexpr int NB = FM * FN;
                constexpr int NSLOT = 3, AHEAD = NSLOT - 1;
                const int prow0 = map_row(p, m0);
                const __amdgpu_buffer_rsrc_t rP =
                    tile_rsrc(pbase, pbytes, (uint64_t)(prow0 - plo) * (uint64_t)p.ldp * 4u);
                const int rr = lane >> 3, rc = lane & 7;
                char *const pslot[NSLOT] = {sA1 + wave * 4096, sW0 + wave * 4096, sW1 + wave * 4096};
                const __amdgpu_buffer_rsrc_t rC =
                    tile_rsrc(p.C, p.c_bytes, (uint64_t)prow0 * (uint64_t)p.ldc * 2u);
                auto store_c = [&](int row, int col, float v0, float v1, float v2, float v3) {
                    const int m = m0 + row, n = n0 + col;
                    const uint32_t off = (m < mlim && n < p.N)
                                             ? ((uint32_t)(map_row(p, m) - prow0) * (uint32_t)p.ldc + (uint32_t)n) * 2u
                                             : kOOBRow;
                    const u32x2 o = {pack_bf16x2(v0, v1), pack_bf16x2(v2, v3)};
                    // (a per-tile choice would be a branch around each store,
                    // which the compiler cannot count)
                    if constexpr (WT)   // sc0 sc1: written through to memory, the copy engines read it
                        __builtin_amdgcn_raw_buffer_store_b64(o, rC, off, 0, 17);
                    else
                        __builtin_amdgcn_raw_buffer_store_b64(o, rC, off, 0, 0);
                };
                auto load_p = [&](int blk, char *dst) {
                    const int mi = blk / FN, ni = blk % FN;
                    const int n = n0 + wn0 + ni * 32 + 4 * rc;
#pragma unroll
                    for (int it = 0; it < 4; ++it) {
                        const int m = m0 + wm0 + mi * 32 + rr + 8 * it;
                        const uint32_t off = (m < p.M && n < p.N)
                                                 ? ((uint32_t)(map_row(p, m) - prow0) * (uint32_t)p.ldp + (uint32_t)n) * 4u
                                                 : kOOBRow;
                        __builtin_amdgcn_raw_ptr_buffer_load_lds(rP, LDS_AS(dst + it * 1024), 16, off, 0, 0, 0);
                    }
                };
#pragma unroll
                for (int blk = 0; blk < AHEAD && blk < NB; ++blk) load_p(blk, pslot[blk]);
#pragma unroll
                for (int blk = 0; blk < NB; ++blk) {
                    char *pcur = pslot[blk % NSLOT];
                    // into the slot of block blk - 1, whose reads ended the last iteration
                    if (blk + AHEAD < NB) load_p(blk + AHEAD, pslot[(blk + AHEAD) % NSLOT]);
                    const int mi = blk / FN, ni = blk % FN;
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int cc = 2 * g + hi;
                        f32x4 v4 = {acc[ni][mi][4 * g + 0], acc[ni][mi][4 * g + 1],
                                    acc[ni][mi][4 * g + 2], acc[ni][mi][4 * g + 3]};
                        *reinterpret_cast<f32x4 *>(patch + r * 128 + ((cc ^ (r & 7)) << 4)) = v4;
                    }
                    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): patch written
#pragma unroll
                    for (int it = 0; it < 4; ++it) {
                        const int row = rr + 8 * it;
                        const f32x4 x = *reinterpret_cast<const f32x4 *>(patch + row * 128 + ((rc ^ (row & 7)) << 4));
                        const f32x4 pv = *reinterpret_cast<const f32x4 *>(pcur + row * 128 + rc * 16);
                        store_c(wm0 + mi * 32 + row, wn0 + ni * 32 + 4 * rc, x[0] + pv[0], x[1] + pv[1],
                                x[2] + pv[2], x[3] + pv[3]);
                    }
                    __builtin_amdgcn_s_waitcnt(0xC07F);   // patch and partial read before reuse
                }
            } else {
                through_patch([&](int row, int col, f32x4 x) { store4(row, col, x[0], x[1], x[2], x[3], has_p); });
            }
        }

        if (wt) __builtin_amdgcn_s_waitcnt(0);   // write-through stores acknowledged
        __syncthreads();   // stores issued and complete; LDS free for the next tile
        if (RS && finish && p.done_host && !failed && tid == 0) {
            uint64_t dm = touch & p.send_mask;
            if (dm) {
                while (dm) {
                    const int q = __builtin_ctzll(dm);
                    const uint32_t old = __hip_atomic_fetch_add(&p.done_cnt[p.flag_base + q], 1u,
                                                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (old + 1u == p.done_expect[q])
                        __hip_atomic_store(&p.done_host[p.flag_base + q], p.epoch, __ATOMIC_RELEASE,
                                           __HIP_MEMORY_SCOPE_SYSTEM);
                    dm &= dm - 1;
                }
            }
        }
        if (traced && tid == 0) {
            uint4 *rec = reinterpret_cast<uint4 *>(p.tile_trace + (size_t)(p.trace_base + (uint32_t)pos) * kTraceWords);
            rec[0] = make_uint4((uint32_t)pos, ((uint32_t)rt << 16) | (uint32_t)tn, hw_id(), xcc_id());
            rec[1] = make_uint4(t_tick, t_gate, t_loop, rtc32());
        }
        pos = s_pos;
    }

    // exit: the last workgroup out resets the shared counters
    __syncthreads();
    if (tid == 0) {
        const uint32_t old = __hip_atomic_fetch_add(&p.ctrl[kCtrlExit], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (old == (uint32_t)p.grid - 1u) {
            if (RS && p.done_host)
                for (int q = 0; q < p.nparts; ++q)
                    __hip_atomic_store(&p.done_cnt[p.flag_base + q], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            for (int q = 0; q < p.nq; ++q)
                __hip_atomic_store(&p.ctrl[q], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&p.ctrl[kCtrlExit], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

__global__ __launch_bounds__(64) void join_kernel(const JoinParams j) {
    if (threadIdx.x != 0) return;
    if (j.start_word) __hip_atomic_store(j.start_word, j.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    for (int i = 0; i < j.count; ++i) {
        const uint32_t *f = j.flags + j.idx[i];
        uint32_t polls = 0;
        while ((int32_t)(ld_flag(f) - j.epoch) < 0) {
            if (++polls > j.spin_limit) {
                __hip_atomic_fetch_or(j.err_word, 2u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
                return;
            }
            if ((polls & 255u) == 0 && ld_flag(j.err_word) != 0) return;
            __builtin_amdgcn_s_sleep(8);
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
}

// Matrix-core probe: every wave issues `iters` rounds of 8 independent
// v_mfma_f32_32x32x16_bf16 and reads the shader-clock counter (s_memtime)
// and the 100 MHz real-time counter before and after them; out[3 w ..] gets
// wave w's two deltas and a value that keeps the products live. The 96 KiB
// LDS reservation leaves room for one workgroup (8 waves, two per SIMD) per
// CU, so a grid of one workgroup per CU runs all waves at once.
__global__ __launch_bounds__(kProbeThreads) void mfma_probe_kernel(uint64_t *out, int iters) {
    __shared__ float reserve[24 * 1024];
    const int tid = threadIdx.x;
    bf16x8 a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = (__bf16)(0.001f * (float)((tid + i) & 15));
        b[i] = (__bf16)(0.002f * (float)(i + 1));
    }
    f32x16 acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[j][e] = 0.0f;
    const uint64_t t0 = __builtin_amdgcn_s_memtime();
    const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
    }
    const uint64_t t1 = __builtin_amdgcn_s_memtime();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
    float sum = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) sum += acc[j][e];
    // one exchange through the reservation keeps it allocated
    reserve[tid] = sum;
    __syncthreads();
    const float other = reserve[tid ^ 64];
    const size_t w = (size_t)blockIdx.x * (kProbeThreads / 64) + (tid >> 6);
    if ((tid & 63) == 0) {
        out[3 * w + 0] = t1 - t0;
        out[3 * w + 1] = r1 - r0;
        out[3 * w + 2] = (uint64_t)__builtin_bit_cast(uint32_t, sum + other);
    }
}

hipError_t launch_mfma_probe(uint64_t *out, int grid, int iters, hipStream_t stream) {
    hipLaunchKernelGGL(mfma_probe_kernel, dim3(grid), dim3(kProbeThreads), 0, stream, out, iters);
    return hipGetLastError();
}

hipError_t launch_gemm(const GemmParams &p, int cfg, bool rs, hipStream_t stream) {
    if (cfg == kTile256) {
        if (rs && p.done_host)
            hipLaunchKernelGGL((gemm_kernel<256, 256, true, true>), dim3(p.grid), dim3(kThreads), 0, stream, p);
        else if (rs)
            hipLaunchKernelGGL((gemm_kernel<256, 256, true>), dim3(p.grid), dim3(kThreads), 0, stream, p);
        else
            hipLaunchKernelGGL((gemm_kernel<256, 256, false>), dim3(p.grid), dim3(kThreads), 0, stream, p);
    } else {
        if (rs && p.done_host)
            hipLaunchKernelGGL((gemm_kernel<128, 128, true, true>), dim3(p.grid), dim3(kThreads), 0, stream, p);
        else if (rs)
            hipLaunchKernelGGL((gemm_kernel<128, 128, true>), dim3(p.grid), dim3(kThreads), 0, stream, p);
        else
            hipLaunchKernelGGL((gemm_kernel<128, 128, false>), dim3(p.grid), dim3(kThreads), 0, stream, p);
    }
    return hipGetLastError();
}

hipError_t launch_join(const JoinParams &j, hipStream_t stream) {
    hipLaunchKernelGGL(join_kernel, dim3(1), dim3(64), 0, stream, j);
    return hipGetLastError();
}

}  // namespace compass
