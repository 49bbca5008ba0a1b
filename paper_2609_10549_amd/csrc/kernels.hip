// gfx950 kernels of the Compass hot path.
//
// gemm_kernel<BM, BN, RS>: persistent bf16 GEMM, C = A * W^T with fp32
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
// Data path per tile: A and W stream through LDS in K-steps of 64, double
// buffered; global -> LDS moves use buffer_load ... lds (no register staging;
// out-of-range rows or K columns read as zero through the buffer bound). The
// 4 waves split the tile 2 x 2; each wave holds (BM/2) x (BN/2) fp32
// accumulators as 32 x 32 MFMA blocks. LDS rows are 128 bytes; the 16-byte
// chunks of row r are XOR-permuted with (r >> 1) & 7 so that a fragment read
// (32 rows, one chunk) hits distinct banks.
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

#define LDS_AS(p) ((__attribute__((address_space(3))) void *)(p))

constexpr uint32_t kOOB = 0x80000000u;   // byte offset beyond every buffer bound

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

// Thread-0 wait for every partition in `mask`. Per partition and epoch one
// workgroup (the first to claim `leader`) polls the host-memory arrival flag
// and forwards it to `mirror` in device memory; every other workgroup polls
// the mirror. A system-scope acquire follows, so that the rows the copy
// engines wrote are read from memory, not from stale cache lines.
__device__ bool wait_flags(const GemmParams &p, uint64_t mask) {
    while (mask) {
        const int f = p.flag_base + __builtin_ctzll(mask);
        mask &= mask - 1;
        if ((int32_t)(ld_dev(&p.mirror[f]) - p.epoch) >= 0) continue;
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
            if (!poll_epoch(&p.flags[f], true, p.epoch, p.spin_limit, p.err_word, 16)) return false;
            __hip_atomic_store(&p.mirror[f], p.epoch, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            if (!poll_epoch(&p.mirror[f], false, p.epoch, p.spin_limit, p.err_word, 4)) return false;
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
    return true;
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

// Issue one K-stage (64 columns) of an R-row operand into LDS. Load q of a
// wave fills LDS bytes [(4q + wave) KiB, +1 KiB): rows 32q + 8 wave + lane/8,
// physical chunk lane % 8, which holds logical chunk `cchunk` (the XOR
// permutation; one value per lane). `row_off` is each load's row start in
// bytes, kOOB past the last row.
template <int R>
__device__ __forceinline__ void load_stage(__amdgpu_buffer_rsrc_t rsrc, char *lds, const uint32_t *row_off,
                                           int cchunk, int k0, int K, int wave) {
    const int kc = k0 + cchunk * 8;
    const bool kin = kc < K;
#pragma unroll
    for (int q = 0; q < R / 32; ++q) {
        const uint32_t off = (row_off[q] == kOOB || !kin) ? kOOB : row_off[q] + (uint32_t)kc * 2u;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, LDS_AS(lds + (q * 4 + wave) * 1024), 16, off, 0, 0, 0);
    }
}

template <int FM, int FN>
__device__ __forceinline__ void read_frags(const char *sA, const char *sW, int r, int swz, int kk, int hi,
                                           int wm0, int wn0, bf16x8 (&a)[FM], bf16x8 (&b)[FN]) {
    const int coff = ((2 * kk + hi) ^ swz) << 4;
#pragma unroll
    for (int mi = 0; mi < FM; ++mi)
        a[mi] = *reinterpret_cast<const bf16x8 *>(sA + (wm0 + mi * 32 + r) * 128 + coff);
#pragma unroll
    for (int ni = 0; ni < FN; ++ni)
        b[ni] = *reinterpret_cast<const bf16x8 *>(sW + (wn0 + ni * 32 + r) * 128 + coff);
}

// One K-stage (4 MFMA K-substeps of 16) on the LDS buffers sA/sW. Fragments
// of substep kk+1 are read from LDS while the MFMAs of kk run (two register
// sets), and the next stage's global->LDS loads (into dA/dW, when `load`) are
// spread over the substeps; scheduling groups interleave the three streams.
template <int BM, int BN, int FM, int FN>
__device__ __forceinline__ void compute_stage(const char *sA, const char *sW, int lane, int wm0, int wn0,
                                              f32x16 (&acc)[FN][FM], bool load, __amdgpu_buffer_rsrc_t rA,
                                              __amdgpu_buffer_rsrc_t rW, char *dA, char *dW,
                                              const uint32_t *offA, const uint32_t *offW, int cchunk, int k0n,
                                              int K, int wave) {
    constexpr int LA = BM / 32, LW = BN / 32;           // global loads per wave per stage
    constexpr int LAK = LA / 4, LWK = LW / 4;           // ... per substep
    const int r = lane & 31;
    const int swz = (r >> 1) & 7;
    const int hi = lane >> 5;
    const int kc = k0n + cchunk * 8;
    const bool kin = kc < K;
    bf16x8 a[2][FM], b[2][FN];
    read_frags<FM, FN>(sA, sW, r, swz, 0, hi, wm0, wn0, a[0], b[0]);
#pragma unroll
    for (int kk = 0; kk < kTileK / 16; ++kk) {
        const int cur = kk & 1;
        if (kk + 1 < kTileK / 16) read_frags<FM, FN>(sA, sW, r, swz, kk + 1, hi, wm0, wn0, a[cur ^ 1], b[cur ^ 1]);
        if (load) {
#pragma unroll
            for (int j = 0; j < LAK; ++j) {
                const int q = kk * LAK + j;
                const uint32_t off = (offA[q] == kOOB || !kin) ? kOOB : offA[q] + (uint32_t)kc * 2u;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, LDS_AS(dA + (q * 4 + wave) * 1024), 16, off, 0, 0, 0);
            }
#pragma unroll
            for (int j = 0; j < LWK; ++j) {
                const int q = kk * LWK + j;
                const uint32_t off = (offW[q] == kOOB || !kin) ? kOOB : offW[q] + (uint32_t)kc * 2u;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rW, LDS_AS(dW + (q * 4 + wave) * 1024), 16, off, 0, 0, 0);
            }
        }
#pragma unroll
        for (int ni = 0; ni < FN; ++ni)
#pragma unroll
            for (int mi = 0; mi < FM; ++mi)
                acc[ni][mi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[cur][ni], a[cur][mi], acc[ni][mi], 0, 0, 0);
        // per substep: FM*FN MFMAs, FM+FN LDS reads (next substep), LAK+LWK
        // global loads; alternate MFMA with reads and loads
        constexpr int NM = FM * FN, ND = FM + FN, NV = LAK + LWK;
#pragma unroll
        for (int i = 0; i < NM; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
            if (i < ND) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // LDS read
            if (i < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
        }
    }
}

// RS = false: optional main-loop gate (AllGather), plain store.
// RS = true: optional epilogue gate, fp32 partial add, chunk-done signalling.
template <int BM, int BN, bool RS>
__global__ __launch_bounds__(kThreads, BM == 256 ? 1 : 2)
void gemm_kernel(const GemmParams p) {
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int FM = WM / 32, FN = WN / 32;
    __shared__ __attribute__((aligned(1024))) char sA0[BM * 128];
    __shared__ __attribute__((aligned(1024))) char sA1[BM * 128];
    __shared__ __attribute__((aligned(1024))) char sW0[BN * 128];
    __shared__ __attribute__((aligned(1024))) char sW1[BN * 128];
    __shared__ int s_pos;
    __shared__ int s_ok;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm0 = (wave >> 1) * WM;
    const int wn0 = (wave & 1) * WN;
    const int total = p.tiles_m * p.tiles_n;
    const int KT2 = (((p.K + kTileK - 1) / kTileK) + 1) & ~1;
    const int v = p.nq > 1 ? (int)(blockIdx.x % (uint32_t)p.nq) : 0;

    const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc((void *)p.A, (short)0, (int)p.a_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t rW = __builtin_amdgcn_make_buffer_rsrc((void *)p.W, (short)0, (int)p.w_bytes, 0x00020000);

    // loader geometry: row of load q is 32 q + lrow0; logical chunk of the lane
    const int lrow0 = 8 * wave + (lane >> 3);
    const int cchunk = (lane & 7) ^ ((4 * wave + (lane >> 4)) & 7);

    uint64_t known = 0;   // partitions already acquired by this workgroup
    bool failed = false;

    if (tid == 0) {
        const uint32_t c = __hip_atomic_fetch_add(&p.ctrl[v], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int pos = ticket_position(p, v, c);
        if (pos == 0 && p.start_word)
            __hip_atomic_store(p.start_word, p.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        s_pos = pos;
    }
    __syncthreads();
    int pos = s_pos;

    while (pos < total) {
        // position -> (row-tile ordinal, column tile): group_m rows at a time
        const int gsz = p.group_m * p.tiles_n;
        const int grp = pos / gsz;
        const int rin = pos - grp * gsz;
        const int rows_here = min(p.group_m, p.tiles_m - grp * p.group_m);
        const int ti = grp * p.group_m + rin % rows_here;
        const int tn = rin / rows_here;
        const int rt = p.rt_order[ti];
        const int m0 = rt * BM;
        const int n0 = tn * BN;
        const uint64_t touch = range_mask(p.rt_lo[rt], p.rt_hi[rt]);
        const uint64_t need = touch & ~p.resident_mask & ~known;

        if (!RS && p.gate == kGateMain && need) {
            if (tid == 0) s_ok = wait_flags(p, need);
            __syncthreads();
            if (!s_ok) failed = true;
            known |= need;
        }

        f32x16 acc[FN][FM];
#pragma unroll
        for (int ni = 0; ni < FN; ++ni)
#pragma unroll
            for (int mi = 0; mi < FM; ++mi)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[ni][mi][e] = 0.0f;

        {   // a timed-out tile still runs (its loads stay in bounds); only its
            // stores are dropped
            uint32_t offA[BM / 32], offW[BN / 32];
#pragma unroll
            for (int q = 0; q < BM / 32; ++q) {
                const int ia = m0 + 32 * q + lrow0;
                offA[q] = ia < p.M ? (uint32_t)map_row(p, ia) * (uint32_t)p.lda * 2u : kOOB;
            }
#pragma unroll
            for (int q = 0; q < BN / 32; ++q) {
                const int iw = n0 + 32 * q + lrow0;
                offW[q] = iw < p.N ? (uint32_t)iw * (uint32_t)p.ldw * 2u : kOOB;
            }
            load_stage<BM>(rA, sA0, offA, cchunk, 0, p.K, wave);
            load_stage<BN>(rW, sW0, offW, cchunk, 0, p.K, wave);
            // An even number of K-steps keeps the loop free of early exits (the
            // accumulators then stay in place); a padding step reads only
            // out-of-range columns, i.e. zeros.
            for (int kt = 0; kt < KT2; kt += 2) {
                __builtin_amdgcn_s_waitcnt(0);
                __syncthreads();
                compute_stage<BM, BN, FM, FN>(sA0, sW0, lane, wm0, wn0, acc, true, rA, rW, sA1, sW1, offA, offW,
                                              cchunk, (kt + 1) * kTileK, p.K, wave);
                __builtin_amdgcn_s_waitcnt(0);
                __syncthreads();
                compute_stage<BM, BN, FM, FN>(sA1, sW1, lane, wm0, wn0, acc, kt + 2 < KT2, rA, rW, sA0, sW0, offA,
                                              offW, cchunk, (kt + 2) * kTileK, p.K, wave);
            }
        }

        // fetch the next ticket while the epilogue runs
        if (tid == 0) {
            const uint32_t c = __hip_atomic_fetch_add(&p.ctrl[v], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_pos = ticket_position(p, v, c);
        }

        if (RS && p.gate == kGateEpilogue && need) {
            if (tid == 0) s_ok = failed ? 0 : wait_flags(p, need);
            __syncthreads();
            if (!s_ok) failed = true;
            known |= need;
        }

        if (!RS) {
            const int r = lane & 31;
            const int hi = lane >> 5;
            const int mlim = failed ? 0 : p.M;   // a failed tile stores nothing
#pragma unroll
            for (int mi = 0; mi < FM; ++mi) {
                const int m = m0 + wm0 + mi * 32 + r;
                if (m >= mlim) continue;
                uint16_t *crow = p.C + (size_t)map_row(p, m) * p.ldc;
#pragma unroll
                for (int ni = 0; ni < FN; ++ni) {
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int n = n0 + wn0 + ni * 32 + 8 * g + 4 * hi;
                        if (n >= p.N) continue;
                        uint2 o;
                        o.x = pack_bf16x2(acc[ni][mi][4 * g + 0], acc[ni][mi][4 * g + 1]);
                        o.y = pack_bf16x2(acc[ni][mi][4 * g + 2], acc[ni][mi][4 * g + 3]);
                        *reinterpret_cast<uint2 *>(crow + n) = o;
                    }
                }
            }
        } else {
            // Each 32 x 32 fp32 block goes through a per-wave 4 KiB LDS patch
            // (rows of 128 bytes, 16-byte chunks XOR-permuted by row & 7) and
            // comes back row-contiguous: 8 lanes per row add 128 contiguous
            // bytes of the partial sum and store 64 contiguous bytes of C.
            char *patch = sA0 + wave * 4096;
            const int r = lane & 31;
            const int hi = lane >> 5;
            const int rr = lane >> 3;          // read-back row within 8
            const int rc = lane & 7;           // read-back chunk (4 floats)
            const int mlim = failed ? 0 : p.M;
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
                        const int m = m0 + wm0 + mi * 32 + row;
                        const int n = n0 + wn0 + ni * 32 + 4 * rc;
                        if (m < mlim && n < p.N) {
                            const int pm = map_row(p, m);
                            float v0 = x[0], v1 = x[1], v2 = x[2], v3 = x[3];
                            if (p.P) {
                                const f32x4 pv = *reinterpret_cast<const f32x4 *>(p.P + (size_t)pm * p.ldp + n);
                                v0 += pv[0]; v1 += pv[1]; v2 += pv[2]; v3 += pv[3];
                            }
                            uint2 o;
                            o.x = pack_bf16x2(v0, v1);
                            o.y = pack_bf16x2(v2, v3);
                            *reinterpret_cast<uint2 *>(p.C + (size_t)pm * p.ldc + n) = o;
                        }
                    }
                    __builtin_amdgcn_s_waitcnt(0xC07F);   // patch read before reuse
                }
            }
        }

        __syncthreads();   // stores issued and complete; LDS free for the next tile
        if (RS && p.done_host && !failed && tid == 0) {
            uint64_t dm = touch & p.send_mask;
            if (dm) {
                __threadfence_system();   // tile data written back before counting
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

hipError_t launch_gemm(const GemmParams &p, int cfg, bool rs, hipStream_t stream) {
    if (cfg == kTile256) {
        if (rs) hipLaunchKernelGGL((gemm_kernel<256, 256, true>), dim3(p.grid), dim3(kThreads), 0, stream, p);
        else hipLaunchKernelGGL((gemm_kernel<256, 256, false>), dim3(p.grid), dim3(kThreads), 0, stream, p);
    } else {
        if (rs) hipLaunchKernelGGL((gemm_kernel<128, 128, true>), dim3(p.grid), dim3(kThreads), 0, stream, p);
        else hipLaunchKernelGGL((gemm_kernel<128, 128, false>), dim3(p.grid), dim3(kThreads), 0, stream, p);
    }
    return hipGetLastError();
}

hipError_t launch_join(const JoinParams &j, hipStream_t stream) {
    hipLaunchKernelGGL(join_kernel, dim3(1), dim3(64), 0, stream, j);
    return hipGetLastError();
}

}  // namespace compass
