// compass_gemm_noalloc: the plain GEMM of compass_gemm for callers that
// cannot allocate device memory (code under HIP graph capture, tight serving
// loops, harnesses that forbid allocation).
//
// The persistent GEMM kernel needs a little scratch: the ticket queues it
// takes its tiles from and the exit counter whose last workgroup resets
// them. compass_gemm keeps them in the library's control block, allocated
// when the library initialises (with the copy-side state, signals and the
// split-K workspace). Here they live in `scratch`, a file-scope device array
// of the code object (each GPU holds its own copy, for the life of the
// process), so a call allocates nothing: no hipMalloc, no hipFree, no
// library initialisation. The launch never splits K (that would need a
// partial-tile workspace), so every tile runs its whole K range.
//
// Host code never passes the array's name to a kernel: the first call on a
// device resolves the array's device address with hipGetSymbolAddress, with
// that device current, and keeps it per device; kernels take that pointer.
// Every call on a GPU shares that GPU's array: a small kernel clears the
// ticket words before each GEMM launch (the GEMM's last workgroup also
// resets them), and calls that overlap on one GPU (concurrent streams)
// race on them.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <mutex>

#include "compass.h"
#include "internal.h"
#include "kernel_params.h"

namespace compass {

hipError_t launch_gemm(const GemmParams &p, int cfg, bool rs, hipStream_t stream);

// words [0, kMaxQueues): ticket queues; [kCtrlExit]: exit counter
constexpr int kScratchWords = 64;
static_assert(kCtrlExit < kScratchWords, "scratch holds the ticket queues and the exit counter");
static __device__ __align__(256) uint32_t scratch[kScratchWords];

__global__ __launch_bounds__(64) void clear_scratch_kernel(uint32_t *s) {
    if (threadIdx.x < (unsigned)kScratchWords) s[threadIdx.x] = 0u;
}

namespace {

constexpr int kMaxDevices = 64;

struct DeviceScratch {
    bool ready = false;
    uint32_t *ptr = nullptr;   // device address of `scratch` on this device
    int num_cu = 0;
};

DeviceScratch g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

int hip_error(hipError_t e, const char *what) {
    return set_error(COMPASS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// The scratch address and CU count of the current device, resolved on the
// first call on that device.
int current_scratch(DeviceScratch *out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_error(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return set_error(COMPASS_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    DeviceScratch &d = g_scratch[dev];
    if (!d.ready) {
        hipDeviceProp_t prop;
        if ((e = hipGetDeviceProperties(&prop, dev)) != hipSuccess) return hip_error(e, "hipGetDeviceProperties");
        if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
            return set_error(COMPASS_ERR_UNSUPPORTED, "device %d is %s, this library is built for gfx950", dev,
                             prop.gcnArchName);
        void *p = nullptr;
        if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess)
            return hip_error(e, "hipGetSymbolAddress(scratch)");
        if (!p) return set_error(COMPASS_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
        d.ptr = static_cast<uint32_t *>(p);
        d.num_cu = prop.multiProcessorCount;
        d.ready = true;
    }
    *out = d;
    return COMPASS_OK;
}

}  // namespace

int op_gemm_noalloc(int M, int N, int K, const void *A, const void *W, void *C, const float *P, void *stream) {
    if (M < 1 || N < 1 || K < 1 || K % 8 || N % 8)
        return set_error(COMPASS_ERR_INVALID, "need positive M, N, K with K, N multiples of 8");
    if (!A || !W || !C) return set_error(COMPASS_ERR_INVALID, "A, W and C are required");
    if ((M + 127) / 128 > kMaxRowTiles)
        return set_error(COMPASS_ERR_UNSUPPORTED, "M = %d above the %d rows of the tile table", M, kMaxRowTiles * 128);
    // the kernel addresses a tile's operands with 32-bit offsets from the
    // tile's first row (column of W): a 256-row tile spans at most
    // kTileSpanMax bytes of each
    if (256ull * (uint64_t)K * 2 > kTileSpanMax || (P && 256ull * (uint64_t)N * 4 > kTileSpanMax))
        return set_error(COMPASS_ERR_UNSUPPORTED, "K = %d, N = %d: a 256-row tile would span more than 1 GiB of A, W "
                                                  "or the partial", K, N);
    DeviceScratch d;
    int rc = current_scratch(&d);
    if (rc != COMPASS_OK) return rc;

    GemmParams g;
    std::memset(&g, 0, sizeof g);
    // the larger tile when it still fills every CU (as compass_gemm)
    const long t256 = (long)((M + 255) / 256) * ((N + 255) / 256);
    const int cfg = t256 >= d.num_cu ? kTile256 : kTile128;
    const int bm = tile_rows(cfg), bn = tile_cols(cfg);
    g.A = (const uint16_t *)A;
    g.W = (const uint16_t *)W;
    g.C = (uint16_t *)C;
    g.P = P;
    g.M = M;
    g.N = N;
    g.K = K;
    g.lda = K;
    g.ldw = K;
    g.ldc = N;
    g.ldp = N;
    g.a_bytes = (uint64_t)M * (uint64_t)K * 2;
    g.w_bytes = (uint64_t)N * (uint64_t)K * 2;
    g.p_bytes = P ? (uint64_t)M * (uint64_t)N * 4 : 0u;
    g.c_bytes = (uint64_t)M * (uint64_t)N * 2;
    g.tiles_m = (M + bm - 1) / bm;
    g.tiles_n = (N + bn - 1) / bn;
    const int total = g.tiles_m * g.tiles_n;
    g.grid = std::max(1, std::min(total, d.num_cu * tile_wg_per_cu(cfg)));
    g.nq = g.grid >= kMaxQueues ? kMaxQueues : 1;
    g.q_size = std::max(1, g.grid / g.nq);
    g.group_m = cfg == kTile256 ? 4 : 8;
    g.ksplit = 1;
    g.kslice = K;
    g.gate = kGateNone;
    g.ctrl = d.ptr;   // the scratch array's device address, never its name
    for (int t = 0; t < g.tiles_m; ++t) g.rt_order[t] = (uint16_t)t;

    hipStream_t s = (hipStream_t)stream;
    hipLaunchKernelGGL(clear_scratch_kernel, dim3(1), dim3(64), 0, s, d.ptr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_error(e, "scratch clear launch");
    e = launch_gemm(g, cfg, P != nullptr, s);
    if (e != hipSuccess) return hip_error(e, "GEMM launch");
    return COMPASS_OK;
}

}  // namespace compass
