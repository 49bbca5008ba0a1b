// Host runtime of the Compass hot path on one MI355X.
//
// Emulated links (the push-based DMA ring transfers of Section III-B): each
// ring direction is served by a pacer thread that owns a set of SDMA engines
// (HSA async copies forced onto SDMA, so no compute unit is taken from the
// GEMM). A job is an ordered list of partition transfers; the pacer issues
// them in slices no earlier than their paced times (rate = the emulated link
// bandwidth), and after the last slice of a partition it appends a 4-byte
// copy of the call's epoch into that partition's arrival flag, dependent on
// the partition's slices. The GEMM kernel polls those flags (fine-grained
// device memory) with system-scope acquire loads.
//
// Operators (Section III-B TA-IntraFusion, Section II-B / IV InterDecom) are
// built from one persistent GEMM launch (or d launches) plus these jobs. Row
// tiles are ordered by the ring schedule; each tile waits for the partitions
// its rows touch (AllGather: before reading A; ReduceScatter: before adding
// the incoming partial). ReduceScatter tiles count per-partition completions;
// the last tile of a partition raises a host-visible done flag that gates the
// outgoing copy of that partition.
#include <hip/hip_runtime.h>
#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>
#include <immintrin.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "compass.h"
#include "internal.h"
#include "kernel_params.h"

namespace compass {

hipError_t launch_gemm(const GemmParams &p, bool rs, hipStream_t stream);
hipError_t launch_join(const JoinParams &j, hipStream_t stream);

// ---------------------------------------------------------------- errors
static thread_local std::string t_err;

int set_error(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_err = buf;
    return code;
}

const char *last_error() { return t_err.c_str(); }

static double now_s() {
    return std::chrono::duration<double>(std::chrono::steady_clock::now().time_since_epoch()).count();
}

// ---------------------------------------------------------------- state
constexpr int kRoles = 4;            // in-fwd, in-bwd, out-fwd, out-bwd
constexpr int kSignals = 512;        // completion signals per pacer
constexpr int kEpochSlots = 256;
constexpr size_t kDefaultSlice = 4u << 20;
// host_words layout (pinned, coherent host memory)
constexpr int kHwStart = 0, kHwErr = 1, kHwDone = 64, kHwEpoch = kHwDone + kMaxFlags;
constexpr int kHwWords = kHwEpoch + kEpochSlots;
// ctrl layout (device memory)
constexpr int kCtrlDone = 64;
constexpr int kCtrlWords = kCtrlDone + kMaxFlags;

struct Item {
    void *dst;
    const void *src;
    size_t bytes;
    hsa_agent_t dst_agent, src_agent;
    int flag;   // arrival flag to publish after the item, -1: none
    int gate;   // host done flag to wait for before the item, -1: none
};

struct Job {
    std::vector<Item> items;
    std::vector<uint32_t> engines;   // SDMA engine id bits
    double rate = 0;                 // bytes / s, <= 0: unpaced
    size_t slice = kDefaultSlice;
    uint32_t epoch = 0;
    bool wait_start = true;
    int final_flag = -1;             // flag published after every item landed
};

struct Ctx;

struct Pacer {
    Ctx *ctx = nullptr;
    std::thread th;
    std::mutex mu;
    std::condition_variable cv;
    std::deque<Job> q;
    std::atomic<int> pending{0};
    std::atomic<bool> stop{false};
    hsa_signal_t sig[kSignals];
    int sig_next = 0;
    void loop();
    void execute(Job &job);
    hsa_signal_t take_signal();
};

struct Ctx {
    bool ready = false;
    int device = -1;
    int num_cu = 0;
    hsa_agent_t gpu{}, cpu{};
    std::vector<uint32_t> engines;   // SDMA engines usable device->device
    uint32_t *flags = nullptr;       // fine-grained device memory
    uint32_t *ctrl = nullptr;        // device memory
    uint32_t *hw = nullptr;          // pinned host words
    uint32_t epoch = 0;
    Pacer pacer[kRoles];
    std::atomic<int> async_err{0};
    uint32_t spin_limit = 4u << 20;  // kernel polls (about 0.5 us each)
    double host_timeout = 5.0;       // seconds
    int grid_override = 0;
    int drop_flag = -1;
    struct Range { uintptr_t lo, hi; hsa_agent_t owner; };
    std::vector<Range> ranges;       // pointer -> owning agent cache
    ~Ctx();
};

static Ctx g_ctx;
static std::mutex g_init_mu;

Ctx::~Ctx() {
    if (!ready) return;
    for (auto &p : pacer) {
        p.stop.store(true);
        p.cv.notify_all();
    }
    for (auto &p : pacer)
        if (p.th.joinable()) p.th.join();
}

static hsa_status_t agent_cb(hsa_agent_t a, void *data) {
    auto *v = static_cast<std::vector<hsa_agent_t> *>(data);
    v->push_back(a);
    return HSA_STATUS_SUCCESS;
}

static int hip_fail(hipError_t e, const char *what) {
    return set_error(COMPASS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

static int ensure_init() {
    std::lock_guard<std::mutex> lk(g_init_mu);
    Ctx &c = g_ctx;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (c.ready) {
        if (dev != c.device) return set_error(COMPASS_ERR_UNSUPPORTED, "library bound to device %d, current is %d", c.device, dev);
        return COMPASS_OK;
    }
    hipDeviceProp_t prop;
    if ((e = hipGetDeviceProperties(&prop, dev)) != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return set_error(COMPASS_ERR_UNSUPPORTED, "device %d is %s, this library is built for gfx950", dev, prop.gcnArchName);
    c.device = dev;
    c.num_cu = prop.multiProcessorCount;
    if (hsa_init() != HSA_STATUS_SUCCESS) return set_error(COMPASS_ERR_HIP, "hsa_init failed");
    std::vector<hsa_agent_t> agents;
    hsa_iterate_agents(agent_cb, &agents);
    std::vector<hsa_agent_t> gpus;
    bool have_cpu = false;
    for (auto a : agents) {
        hsa_device_type_t t;
        hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &t);
        if (t == HSA_DEVICE_TYPE_GPU) gpus.push_back(a);
        if (t == HSA_DEVICE_TYPE_CPU && !have_cpu) { c.cpu = a; have_cpu = true; }
    }
    // match the HIP device by PCI location
    bool found = false;
    for (auto a : gpus) {
        uint32_t bdf = 0;
        hsa_agent_get_info(a, (hsa_agent_info_t)HSA_AMD_AGENT_INFO_BDFID, &bdf);
        const uint32_t want = ((uint32_t)prop.pciBusID << 8) | ((uint32_t)prop.pciDeviceID << 3);
        if ((bdf & 0xFFF8u) == (want & 0xFFF8u)) { c.gpu = a; found = true; break; }
    }
    if (!found && (int)gpus.size() > dev) { c.gpu = gpus[dev]; found = true; }
    if (!found || !have_cpu) return set_error(COMPASS_ERR_HIP, "could not find the HSA agents");
    if ((e = hipExtMallocWithFlags((void **)&c.flags, kMaxFlags * sizeof(uint32_t), hipDeviceMallocFinegrained)) != hipSuccess)
        return hip_fail(e, "flag allocation");
    if ((e = hipMalloc((void **)&c.ctrl, kCtrlWords * sizeof(uint32_t))) != hipSuccess) return hip_fail(e, "control allocation");
    if ((e = hipHostMalloc((void **)&c.hw, kHwWords * sizeof(uint32_t), hipHostMallocCoherent)) != hipSuccess)
        return hip_fail(e, "host word allocation");
    std::memset(c.hw, 0, kHwWords * sizeof(uint32_t));
    if ((e = hipMemset(c.flags, 0, kMaxFlags * sizeof(uint32_t))) != hipSuccess) return hip_fail(e, "flag clear");
    if ((e = hipMemset(c.ctrl, 0, kCtrlWords * sizeof(uint32_t))) != hipSuccess) return hip_fail(e, "control clear");
    if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(e, "init sync");
    for (auto &p : c.pacer) {
        p.ctx = &c;
        for (auto &s : p.sig)
            if (hsa_signal_create(0, 0, nullptr, &s) != HSA_STATUS_SUCCESS)
                return set_error(COMPASS_ERR_HIP, "hsa_signal_create failed");
    }
    // Usable SDMA engines: the runtime's availability mask only lists engines
    // no other client holds yet, so instead every engine is tried with a
    // 4-byte device-to-device copy forced onto it; engines the mask reports
    // free come first.
    {
        uint32_t avail = 0;
        if (hsa_amd_memory_copy_engine_status(c.gpu, c.gpu, &avail) != HSA_STATUS_SUCCESS) avail = 0;
        std::vector<uint32_t> ok_free, ok_busy;
        hsa_signal_t s = c.pacer[0].sig[0];
        for (int i = 0; i < 16; ++i) {
            const uint32_t id = 1u << i;
            hsa_signal_store_relaxed(s, 1);
            if (hsa_amd_memory_async_copy_on_engine(c.flags + kMaxFlags - 1, c.gpu, c.flags + kMaxFlags - 2, c.gpu,
                                                    sizeof(uint32_t), 0, nullptr, s, (hsa_amd_sdma_engine_id_t)id,
                                                    true) != HSA_STATUS_SUCCESS) {
                hsa_signal_store_relaxed(s, 0);
                continue;
            }
            const double t0 = now_s();
            bool done = true;
            while (hsa_signal_load_scacquire(s) > 0)
                if (now_s() - t0 > 1.0) { done = false; break; }
            if (!done) return set_error(COMPASS_ERR_HIP, "probe copy on SDMA engine %d did not complete", i);
            if (hsa_signal_load_scacquire(s) < 0) continue;
            (avail & id ? ok_free : ok_busy).push_back(id);
        }
        c.engines = ok_free;
        c.engines.insert(c.engines.end(), ok_busy.begin(), ok_busy.end());
        if (c.engines.empty()) return set_error(COMPASS_ERR_UNSUPPORTED, "no SDMA engine accepted a copy");
        if (std::getenv("COMPASS_VERBOSE"))
            std::fprintf(stderr, "compass: %zu SDMA engines usable (%zu reported free)\n", c.engines.size(), ok_free.size());
    }
    for (auto &p : c.pacer) p.th = std::thread([&p] { p.loop(); });
    c.ready = true;
    return COMPASS_OK;
}

// Owning agent of a pointer (device memory -> GPU, host memory -> CPU).
static int agent_of(const void *ptr, hsa_agent_t *out) {
    Ctx &c = g_ctx;
    const uintptr_t u = (uintptr_t)ptr;
    for (auto &r : c.ranges)
        if (u >= r.lo && u < r.hi) { *out = r.owner; return COMPASS_OK; }
    hsa_amd_pointer_info_t info;
    std::memset(&info, 0, sizeof info);
    info.size = sizeof info;
    if (hsa_amd_pointer_info(ptr, &info, nullptr, nullptr, nullptr) != HSA_STATUS_SUCCESS)
        return set_error(COMPASS_ERR_INVALID, "pointer %p is not known to the runtime", ptr);
    if (info.type == HSA_EXT_POINTER_TYPE_UNKNOWN)
        return set_error(COMPASS_ERR_INVALID, "pointer %p is neither device nor pinned host memory", ptr);
    hsa_device_type_t t = HSA_DEVICE_TYPE_CPU;
    hsa_agent_get_info(info.agentOwner, HSA_AGENT_INFO_DEVICE, &t);
    const hsa_agent_t owner = t == HSA_DEVICE_TYPE_GPU ? c.gpu : c.cpu;
    if (t == HSA_DEVICE_TYPE_GPU && info.agentOwner.handle != c.gpu.handle)
        return set_error(COMPASS_ERR_UNSUPPORTED, "pointer %p belongs to another GPU", ptr);
    const uintptr_t lo = (uintptr_t)(info.type == HSA_EXT_POINTER_TYPE_LOCKED ? info.hostBaseAddress : info.agentBaseAddress);
    if (c.ranges.size() > 256) c.ranges.clear();
    c.ranges.push_back({lo, lo + info.sizeInBytes, owner});
    *out = owner;
    return COMPASS_OK;
}

// ---------------------------------------------------------------- pacer
hsa_signal_t Pacer::take_signal() {
    hsa_signal_t s = sig[sig_next];
    sig_next = (sig_next + 1) % kSignals;
    // a slot is reused kSignals copies later; make sure that copy finished
    const double t0 = now_s();
    while (hsa_signal_load_scacquire(s) > 0) {
        if (now_s() - t0 > ctx->host_timeout) { ctx->async_err.store(COMPASS_ERR_TIMEOUT); break; }
        _mm_pause();
    }
    hsa_signal_store_relaxed(s, 1);
    return s;
}

void Pacer::loop() {
    double idle_since = now_s();
    while (!stop.load()) {
        if (pending.load(std::memory_order_acquire) == 0) {
            if (now_s() - idle_since > 0.05) {
                std::unique_lock<std::mutex> lk(mu);
                cv.wait_for(lk, std::chrono::milliseconds(20), [this] { return stop.load() || !q.empty(); });
            } else {
                _mm_pause();
            }
            continue;
        }
        Job job;
        {
            std::lock_guard<std::mutex> lk(mu);
            if (q.empty()) continue;
            job = std::move(q.front());
            q.pop_front();
        }
        execute(job);
        pending.fetch_sub(1, std::memory_order_acq_rel);
        idle_since = now_s();
    }
}

static bool spin_until_epoch(volatile uint32_t *w, uint32_t epoch, double timeout) {
    const double t0 = now_s();
    while ((int32_t)(__atomic_load_n(w, __ATOMIC_ACQUIRE) - epoch) < 0) {
        if (now_s() - t0 > timeout) return false;
        _mm_pause();
    }
    return true;
}

void Pacer::execute(Job &job) {
    Ctx &c = *ctx;
    if (job.items.empty() && job.final_flag < 0) return;
    if (job.wait_start && !spin_until_epoch(&c.hw[kHwStart], job.epoch, c.host_timeout)) {
        c.async_err.store(COMPASS_ERR_TIMEOUT);
        return;
    }
    const size_t E = job.engines.size();
    std::vector<hsa_signal_t> last(E);
    std::vector<bool> used(E, false);
    const uint32_t *epoch_src = &c.hw[kHwEpoch + job.epoch % kEpochSlots];
    double t_next = now_s();
    size_t rr = 0;
    for (const Item &it : job.items) {
        if (it.gate >= 0) {
            if (!spin_until_epoch(&c.hw[kHwDone + it.gate], job.epoch, c.host_timeout)) {
                c.async_err.store(COMPASS_ERR_TIMEOUT);
                return;
            }
            t_next = std::max(t_next, now_s());
        }
        std::vector<hsa_signal_t> deps;
        std::vector<bool> item_used(E, false);
        std::vector<hsa_signal_t> item_last(E);
        size_t off = 0;
        size_t e_last = 0;
        while (off < it.bytes) {
            const size_t len = std::min(job.slice, it.bytes - off);
            if (job.rate > 0) {
                while (now_s() < t_next) _mm_pause();
                t_next += (double)len / job.rate;
            }
            const size_t e = rr++ % E;
            hsa_signal_t s = take_signal();
            const hsa_status_t st = hsa_amd_memory_async_copy_on_engine(
                (char *)it.dst + off, it.dst_agent, (const char *)it.src + off, it.src_agent, len, 0, nullptr, s,
                (hsa_amd_sdma_engine_id_t)job.engines[e], true);
            if (st != HSA_STATUS_SUCCESS) {
                hsa_signal_store_relaxed(s, 0);
                c.async_err.store(COMPASS_ERR_HIP);
                return;
            }
            last[e] = s; used[e] = true;
            item_last[e] = s; item_used[e] = true;
            e_last = e;
            off += len;
        }
        if (it.flag >= 0) {
            for (size_t e = 0; e < E; ++e)
                if (item_used[e]) deps.push_back(item_last[e]);
            hsa_signal_t s = take_signal();
            const hsa_status_t st = hsa_amd_memory_async_copy_on_engine(
                c.flags + it.flag, c.gpu, epoch_src, c.cpu, sizeof(uint32_t), (uint32_t)deps.size(),
                deps.empty() ? nullptr : deps.data(), s, (hsa_amd_sdma_engine_id_t)job.engines[e_last], true);
            if (st != HSA_STATUS_SUCCESS) {
                hsa_signal_store_relaxed(s, 0);
                c.async_err.store(COMPASS_ERR_HIP);
                return;
            }
            last[e_last] = s;
        }
    }
    std::vector<hsa_signal_t> deps;
    for (size_t e = 0; e < E; ++e)
        if (used[e]) deps.push_back(last[e]);
    if (job.final_flag >= 0) {
        hsa_signal_t s = take_signal();
        const hsa_status_t st = hsa_amd_memory_async_copy_on_engine(
            c.flags + job.final_flag, c.gpu, epoch_src, c.cpu, sizeof(uint32_t), (uint32_t)deps.size(),
            deps.empty() ? nullptr : deps.data(), s, (hsa_amd_sdma_engine_id_t)job.engines[0], true);
        if (st != HSA_STATUS_SUCCESS) {
            hsa_signal_store_relaxed(s, 0);
            c.async_err.store(COMPASS_ERR_HIP);
            return;
        }
        deps.push_back(s);
    }
    // the job is over once its copies have landed
    const double t0 = now_s();
    for (auto s : deps)
        while (hsa_signal_load_scacquire(s) > 0) {
            if (now_s() - t0 > c.host_timeout) { c.async_err.store(COMPASS_ERR_TIMEOUT); return; }
            _mm_pause();
        }
}

static void submit(int role, Job &&job) {
    Pacer &p = g_ctx.pacer[role];
    p.pending.fetch_add(1);
    {
        std::lock_guard<std::mutex> lk(p.mu);
        p.q.push_back(std::move(job));
    }
    p.cv.notify_one();
}

static bool pacers_idle() {
    for (auto &p : g_ctx.pacer)
        if (p.pending.load() != 0) return false;
    return true;
}

// ---------------------------------------------------------------- helpers
static int take_async_error() {
    Ctx &c = g_ctx;
    const int a = c.async_err.exchange(0);
    const uint32_t k = __atomic_exchange_n(&c.hw[kHwErr], 0u, __ATOMIC_ACQ_REL);
    if (k != 0) return set_error(COMPASS_ERR_TIMEOUT, "a kernel-side wait exceeded its bound (code %u)", k);
    if (a == COMPASS_ERR_TIMEOUT) return set_error(COMPASS_ERR_TIMEOUT, "a copy-side wait exceeded its bound");
    if (a != 0) return set_error(a, "an asynchronous copy failed");
    return COMPASS_OK;
}

static uint32_t next_epoch() {
    Ctx &c = g_ctx;
    const uint32_t e = ++c.epoch;
    __atomic_store_n(&c.hw[kHwEpoch + e % kEpochSlots], e, __ATOMIC_RELEASE);
    return e;
}

static std::vector<uint32_t> engines_for(int role, int roles_active, int per_ring) {
    const auto &all = g_ctx.engines;
    const int n = (int)all.size();
    const int share = std::max(1, n / roles_active);
    int k = per_ring > 0 ? per_ring : std::min(share, roles_active > 2 ? 3 : 4);
    k = std::min(k, share);
    std::vector<uint32_t> out;
    for (int i = 0; i < k; ++i) out.push_back(all[(role * share + i) % n]);
    return out;
}

struct Geometry {
    int P;           // partitions
    int rows;        // rows per chunk
    int prow;        // rows per partition
    int32_t sched[2 * kMaxRanks];
    int pos[2 * kMaxRanks];   // position of each partition in the schedule
};

static int validate(const compass_problem *p, const compass_links *l, int want_pattern, Geometry *g) {
    if (!p) return set_error(COMPASS_ERR_INVALID, "problem is NULL");
    if (!l) return set_error(COMPASS_ERR_INVALID, "links is NULL");
    if (want_pattern >= 0 && p->pattern != want_pattern) return set_error(COMPASS_ERR_INVALID, "wrong pattern for this call");
    if (p->pattern != COMPASS_AG_GEMM && p->pattern != COMPASS_GEMM_RS) return set_error(COMPASS_ERR_INVALID, "unknown pattern");
    if (p->ring != COMPASS_RING_SINGLE && p->ring != COMPASS_RING_DOUBLE) return set_error(COMPASS_ERR_INVALID, "unknown ring");
    if (p->n < 1 || p->n > kMaxRanks || p->rank < 0 || p->rank >= p->n)
        return set_error(COMPASS_ERR_INVALID, "need 1 <= n <= %d and 0 <= rank < n", kMaxRanks);
    if (p->M < 1 || p->N < 1 || p->K < 1) return set_error(COMPASS_ERR_INVALID, "M, N, K must be positive");
    const int P = p->ring == COMPASS_RING_SINGLE ? p->n : 2 * p->n;
    if (p->M % P) return set_error(COMPASS_ERR_INVALID, "M must be divisible by %d", P);
    if (p->K % 8 || p->N % 8) return set_error(COMPASS_ERR_INVALID, "K and N must be multiples of 8");
    if ((p->M + kTileM - 1) / kTileM > kMaxRowTiles) return set_error(COMPASS_ERR_UNSUPPORTED, "M too large");
    if ((double)p->M * p->K * 2 >= 2147483648.0 || (double)p->N * p->K * 2 >= 2147483648.0 ||
        (double)p->M * p->N * 4 >= 2147483648.0)
        return set_error(COMPASS_ERR_UNSUPPORTED, "operand larger than 2 GiB");
    if (!p->W || !p->C) return set_error(COMPASS_ERR_INVALID, "W and C are required");
    if (p->pattern == COMPASS_AG_GEMM) {
        if (!p->shard_src || !p->gathered) return set_error(COMPASS_ERR_INVALID, "shard_src and gathered are required");
        for (int q = 0; q < p->n; ++q)
            if (!p->shard_src[q]) return set_error(COMPASS_ERR_INVALID, "shard_src[%d] is NULL", q);
    } else {
        if (!p->A || !p->partial_src || !p->partial_stage) return set_error(COMPASS_ERR_INVALID, "A, partial_src and partial_stage are required");
        for (int q = 0; q < p->n; ++q)
            if (!p->partial_src[q]) return set_error(COMPASS_ERR_INVALID, "partial_src[%d] is NULL", q);
        if (p->send_dst)
            for (int q = 0; q < p->n; ++q)
                if (q != p->rank && !p->send_dst[q]) return set_error(COMPASS_ERR_INVALID, "send_dst[%d] is NULL", q);
    }
    if (l->slice_bytes != 0 && l->slice_bytes < 4096) return set_error(COMPASS_ERR_INVALID, "slice_bytes below 4 KiB");
    if (l->engines_per_ring < 0) return set_error(COMPASS_ERR_INVALID, "engines_per_ring < 0");
    g->P = P;
    g->rows = p->M / p->n;
    g->prow = p->M / P;
    const int len = schedule_fill(p->pattern, p->ring, p->n, p->rank, g->sched, 2 * kMaxRanks);
    if (len != P) return len < 0 ? len : set_error(COMPASS_ERR_INVALID, "schedule failed");
    for (int i = 0; i < P; ++i) g->pos[g->sched[i]] = i;
    return COMPASS_OK;
}

static void init_params(GemmParams &g, uint32_t epoch) {
    std::memset(&g, 0, sizeof g);
    Ctx &c = g_ctx;
    g.flags = c.flags;
    g.ctrl = c.ctrl;
    g.done_cnt = c.ctrl + kCtrlDone;
    g.err_word = &c.hw[kHwErr];
    g.spin_limit = c.spin_limit;
    g.epoch = epoch;
}

static void set_shape(GemmParams &g, int M, int N, int K, const void *A, size_t a_rows, const void *W, void *C,
                      const float *P) {
    g.A = (const uint16_t *)A;
    g.W = (const uint16_t *)W;
    g.C = (uint16_t *)C;
    g.P = P;
    g.M = M; g.N = N; g.K = K;
    g.lda = K; g.ldw = K; g.ldc = N; g.ldp = N;
    g.a_bytes = (uint32_t)(a_rows * (size_t)K * 2);
    g.w_bytes = (uint32_t)((size_t)N * K * 2);
    g.tiles_m = (M + kTileM - 1) / kTileM;
    g.tiles_n = (N + kTileN - 1) / kTileN;
    const int total = g.tiles_m * g.tiles_n;
    const int cap = g_ctx.grid_override > 0 ? g_ctx.grid_override : g_ctx.num_cu;
    g.grid = std::max(1, std::min(total, cap));
    for (int t = 0; t < g.tiles_m; ++t) g.rt_order[t] = (uint16_t)t;
}

// Row tiles ordered by the schedule position of the last partition they
// touch; touch masks from the identity row map.
static void order_by_schedule(GemmParams &g, const Geometry &geo, int M) {
    std::vector<std::pair<int, int>> key;
    for (int t = 0; t < g.tiles_m; ++t) {
        const int r0 = t * kTileM, r1 = std::min(M, r0 + kTileM) - 1;
        const int p0 = r0 / geo.prow, p1 = r1 / geo.prow;
        uint64_t m = 0;
        int k = 0;
        for (int q = p0; q <= p1; ++q) { m |= 1ull << q; k = std::max(k, geo.pos[q]); }
        g.rt_touch[t] = m;
        key.push_back({k, t});
    }
    std::stable_sort(key.begin(), key.end());
    for (int i = 0; i < g.tiles_m; ++i) g.rt_order[i] = (uint16_t)key[i].second;
}

static hipError_t copy_if_needed(void *dst, const void *src, size_t bytes, hipStream_t s) {
    if (dst == src) return hipSuccess;
    return hipMemcpyAsync(dst, src, bytes, hipMemcpyDefault, s);
}

// Partition p's rows (identity map): chunk c = p (single) or p / 2 (double).
static inline int part_chunk(const compass_problem *p, int q) { return p->ring == COMPASS_RING_SINGLE ? q : q / 2; }
static inline int part_half(const compass_problem *p, int q) { return p->ring == COMPASS_RING_SINGLE ? 0 : q % 2; }
static inline bool part_fwd(const compass_problem *p, int q) { return p->ring == COMPASS_RING_SINGLE || (q % 2) == 1; }

static int make_item(Item *it, void *dst, const void *src, size_t bytes, int flag, int gate) {
    int rc;
    if ((rc = agent_of(dst, &it->dst_agent)) != COMPASS_OK) return rc;
    if ((rc = agent_of(src, &it->src_agent)) != COMPASS_OK) return rc;
    it->dst = dst;
    it->src = src;
    it->bytes = bytes;
    it->flag = flag;
    it->gate = gate;
    return COMPASS_OK;
}

static void fill_job(Job &j, const compass_links *l, bool fwd, uint32_t epoch, int role, int roles_active) {
    j.rate = fwd ? l->fwd_Bps : l->bwd_Bps;
    j.slice = l->slice_bytes ? l->slice_bytes : kDefaultSlice;
    j.epoch = epoch;
    j.engines = engines_for(role, roles_active, l->engines_per_ring);
}

// ---------------------------------------------------------------- AllGather jobs
// Items: the remote partitions in schedule order (the local ones are already
// in place); forward-ring partitions go to role 0, backward-ring to role 1.
// `d` > 1: InterDecom sub-gathers, piece j of every remote partition, j-major,
// with flags j * P + partition.
static int ag_jobs(const compass_problem *p, const Geometry &geo, const compass_links *l, uint32_t epoch, int d,
                   bool wait_start, Job *fwd, Job *bwd) {
    fill_job(*fwd, l, true, epoch, 0, 2);
    fill_job(*bwd, l, false, epoch, 1, 2);
    fwd->wait_start = bwd->wait_start = wait_start;
    const size_t K = (size_t)p->K;
    const int pc = geo.rows / d;                                     // chunk rows per sub-operator
    const int piece = p->ring == COMPASS_RING_SINGLE ? pc : pc / 2;  // rows per item
    for (int j = 0; j < d; ++j) {
        for (int s = 0; s < geo.P; ++s) {
            const int q = geo.sched[s];
            const int c = part_chunk(p, q), h = part_half(p, q);
            if (c == p->rank) continue;
            if (q == g_ctx.drop_flag && d == 1) continue;
            const size_t row_in_chunk = (size_t)j * pc + (size_t)h * piece;
            const size_t row = (size_t)c * geo.rows + row_in_chunk;
            Item it;
            const int rc = make_item(&it, (char *)p->gathered + row * K * 2,
                                     (const char *)p->shard_src[c] + row_in_chunk * K * 2, (size_t)piece * K * 2,
                                     j * geo.P + q, -1);
            if (rc != COMPASS_OK) return rc;
            (part_fwd(p, q) ? fwd : bwd)->items.push_back(it);
        }
    }
    return COMPASS_OK;
}

// ---------------------------------------------------------------- ReduceScatter jobs
// Incoming partials of every non-resident partition (schedule order) and,
// when send_dst is given, outgoing sums of every non-local partition, gated
// on its done flag (or ungated when `gate_out` is false).
static int rs_jobs(const compass_problem *p, const Geometry &geo, const compass_links *l, uint32_t epoch, int d,
                   uint64_t resident, bool gate_out, bool wait_start, Job jobs[4]) {
    for (int r = 0; r < 4; ++r) {
        fill_job(jobs[r], l, r % 2 == 0, epoch, r, 4);
        jobs[r].wait_start = wait_start;
    }
    const size_t N = (size_t)p->N;
    const int pc = geo.rows / d;
    const int piece = p->ring == COMPASS_RING_SINGLE ? pc : pc / 2;
    for (int j = 0; j < d; ++j) {
        for (int s = 0; s < geo.P; ++s) {
            const int q = geo.sched[s];
            if (resident & (1ull << q)) continue;
            const int c = part_chunk(p, q), h = part_half(p, q);
            const size_t row_in_chunk = (size_t)j * pc + (size_t)h * piece;
            const size_t row = (size_t)c * geo.rows + row_in_chunk;
            Item it;
            const int rc = make_item(&it, (char *)p->partial_stage + row * N * 4,
                                     (const char *)p->partial_src[c] + row_in_chunk * N * 4, (size_t)piece * N * 4,
                                     j * geo.P + q, -1);
            if (rc != COMPASS_OK) return rc;
            jobs[part_fwd(p, q) ? 0 : 1].items.push_back(it);
        }
        if (!p->send_dst) continue;
        for (int s = 0; s < geo.P; ++s) {
            const int q = geo.sched[s];
            const int c = part_chunk(p, q), h = part_half(p, q);
            if (c == p->rank) continue;
            const size_t row_in_chunk = (size_t)j * pc + (size_t)h * piece;
            const size_t row = (size_t)c * geo.rows + row_in_chunk;
            Item it;
            const int rc = make_item(&it, (char *)p->send_dst[c] + row_in_chunk * N * 2,
                                     (const char *)p->C + row * N * 2, (size_t)piece * N * 2, -1,
                                     gate_out ? j * geo.P + q : -1);
            if (rc != COMPASS_OK) return rc;
            jobs[part_fwd(p, q) ? 2 : 3].items.push_back(it);
        }
    }
    for (int r = 2; r < 4; ++r)
        if (!jobs[r].items.empty()) jobs[r].final_flag = kFinalFlag0 + r;
    return COMPASS_OK;
}

static uint64_t resident_mask(const compass_problem *p, const Geometry &geo) {
    if (p->pattern == COMPASS_AG_GEMM) {
        if (p->ring == COMPASS_RING_SINGLE) return 1ull << p->rank;
        return 3ull << (2 * p->rank);
    }
    if (p->ring == COMPASS_RING_SINGLE) return 1ull << geo.sched[0];
    return (1ull << geo.sched[0]) | (1ull << geo.sched[1]);
}

static uint64_t nonlocal_mask(const compass_problem *p, const Geometry &geo) {
    uint64_t m = 0;
    for (int q = 0; q < geo.P; ++q)
        if (part_chunk(p, q) != p->rank) m |= 1ull << q;
    return m;
}

static int stage_local_shard(const compass_problem *p, const Geometry &geo, hipStream_t s) {
    const size_t K = (size_t)p->K;
    void *dst = (char *)p->gathered + (size_t)p->rank * geo.rows * K * 2;
    const hipError_t e = copy_if_needed(dst, p->shard_src[p->rank], (size_t)geo.rows * K * 2, s);
    return e == hipSuccess ? COMPASS_OK : hip_fail(e, "local shard copy");
}

static int stage_resident_partials(const compass_problem *p, const Geometry &geo, uint64_t resident, hipStream_t s) {
    const size_t N = (size_t)p->N;
    for (int q = 0; q < geo.P; ++q) {
        if (!(resident & (1ull << q))) continue;
        const int c = part_chunk(p, q), h = part_half(p, q);
        const size_t row_in_chunk = (size_t)h * geo.prow;
        void *dst = (char *)p->partial_stage + ((size_t)c * geo.rows + row_in_chunk) * N * 4;
        const void *src = (const char *)p->partial_src[c] + row_in_chunk * N * 4;
        const hipError_t e = copy_if_needed(dst, src, (size_t)geo.prow * N * 4, s);
        if (e != hipSuccess) return hip_fail(e, "resident partial copy");
    }
    return COMPASS_OK;
}

static int launch(const GemmParams &g, bool rs, hipStream_t s) {
    const hipError_t e = launch_gemm(g, rs, s);
    return e == hipSuccess ? COMPASS_OK : hip_fail(e, "GEMM launch");
}

static int join(uint32_t epoch, const std::vector<int> &flags, bool write_start, hipStream_t s) {
    JoinParams j;
    std::memset(&j, 0, sizeof j);
    Ctx &c = g_ctx;
    j.flags = c.flags;
    j.start_word = write_start ? &c.hw[kHwStart] : nullptr;
    j.err_word = &c.hw[kHwErr];
    j.epoch = epoch;
    j.spin_limit = c.spin_limit;
    if ((int)flags.size() > kMaxJoin) return set_error(COMPASS_ERR_UNSUPPORTED, "too many flags to join");
    j.count = (int)flags.size();
    for (size_t i = 0; i < flags.size(); ++i) j.idx[i] = (uint16_t)flags[i];
    const hipError_t e = launch_join(j, s);
    return e == hipSuccess ? COMPASS_OK : hip_fail(e, "join launch");
}

static int begin(void) {
    int rc = ensure_init();
    if (rc != COMPASS_OK) return rc;
    return take_async_error();
}

// ---------------------------------------------------------------- operators
int op_ag_gemm(const compass_problem *p, const compass_links *l, void *stream) {
    Geometry geo;
    int rc = validate(p, l, COMPASS_AG_GEMM, &geo);
    if (rc != COMPASS_OK) return rc;
    if ((rc = begin()) != COMPASS_OK) return rc;
    hipStream_t s = (hipStream_t)stream;
    const uint32_t epoch = next_epoch();
    Job fwd, bwd;
    if ((rc = ag_jobs(p, geo, l, epoch, 1, true, &fwd, &bwd)) != COMPASS_OK) return rc;
    if ((rc = stage_local_shard(p, geo, s)) != COMPASS_OK) return rc;
    GemmParams g;
    init_params(g, epoch);
    set_shape(g, p->M, p->N, p->K, p->gathered, p->M, p->W, p->C, nullptr);
    order_by_schedule(g, geo, p->M);
    g.gate = kGateMain;
    g.nparts = geo.P;
    g.resident_mask = resident_mask(p, geo);
    g.start_word = &g_ctx.hw[kHwStart];
    submit(0, std::move(fwd));
    submit(1, std::move(bwd));
    return launch(g, false, s);
}

int op_gemm_rs(const compass_problem *p, const compass_links *l, void *stream) {
    Geometry geo;
    int rc = validate(p, l, COMPASS_GEMM_RS, &geo);
    if (rc != COMPASS_OK) return rc;
    if ((rc = begin()) != COMPASS_OK) return rc;
    hipStream_t s = (hipStream_t)stream;
    const uint32_t epoch = next_epoch();
    const uint64_t res = resident_mask(p, geo);
    Job jobs[4];
    if ((rc = rs_jobs(p, geo, l, epoch, 1, res, true, true, jobs)) != COMPASS_OK) return rc;
    if ((rc = stage_resident_partials(p, geo, res, s)) != COMPASS_OK) return rc;
    GemmParams g;
    init_params(g, epoch);
    set_shape(g, p->M, p->N, p->K, p->A, p->M, p->W, p->C, p->partial_stage);
    order_by_schedule(g, geo, p->M);
    g.gate = kGateEpilogue;
    g.nparts = geo.P;
    g.resident_mask = res;
    g.start_word = &g_ctx.hw[kHwStart];
    std::vector<int> finals;
    if (p->send_dst) {
        g.done_host = &g_ctx.hw[kHwDone];
        g.send_mask = nonlocal_mask(p, geo);
        for (int q = 0; q < geo.P; ++q) {
            if (!(g.send_mask & (1ull << q))) continue;
            uint32_t cnt = 0;
            for (int t = 0; t < g.tiles_m; ++t)
                if (g.rt_touch[t] & (1ull << q)) cnt += g.tiles_n;
            g.done_expect[q] = cnt;
        }
        for (int r = 2; r < 4; ++r)
            if (jobs[r].final_flag >= 0) finals.push_back(jobs[r].final_flag);
    }
    for (int r = 0; r < 4; ++r) submit(r, std::move(jobs[r]));
    if ((rc = launch(g, true, s)) != COMPASS_OK) return rc;
    if (!finals.empty()) return join(epoch, finals, false, s);
    return COMPASS_OK;
}

int op_decomp(const compass_problem *p, int d, const compass_links *l, void *stream) {
    Geometry geo;
    int rc = validate(p, l, -1, &geo);
    if (rc != COMPASS_OK) return rc;
    if (d < 1 || (d & (d - 1)) || geo.prow % d)
        return set_error(COMPASS_ERR_INVALID, "d must be a power of two dividing %d", geo.prow);
    if (d * geo.P > kFinalFlag0) return set_error(COMPASS_ERR_UNSUPPORTED, "d * partitions exceeds the flag slots");
    if ((rc = begin()) != COMPASS_OK) return rc;
    hipStream_t s = (hipStream_t)stream;
    const uint32_t epoch = next_epoch();
    const uint64_t res = resident_mask(p, geo);
    const uint64_t all = geo.P == 64 ? ~0ull : ((1ull << geo.P) - 1);
    const int piece = geo.rows / d;   // rows of a chunk per sub-operator
    std::vector<int> finals;
    Job ag_f, ag_b, rs[4];
    if (p->pattern == COMPASS_AG_GEMM) {
        if ((rc = ag_jobs(p, geo, l, epoch, d, true, &ag_f, &ag_b)) != COMPASS_OK) return rc;
        if ((rc = stage_local_shard(p, geo, s)) != COMPASS_OK) return rc;
    } else {
        if ((rc = rs_jobs(p, geo, l, epoch, d, res, true, true, rs)) != COMPASS_OK) return rc;
        if ((rc = stage_resident_partials(p, geo, res, s)) != COMPASS_OK) return rc;
        if (p->send_dst)
            for (int r = 2; r < 4; ++r)
                if (rs[r].final_flag >= 0) finals.push_back(rs[r].final_flag);
    }
    std::vector<GemmParams> launches(d);
    for (int j = 0; j < d; ++j) {
        GemmParams &g = launches[j];
        init_params(g, epoch);
        const bool ag = p->pattern == COMPASS_AG_GEMM;
        set_shape(g, p->M / d, p->N, p->K, ag ? p->gathered : p->A, p->M, p->W, p->C, ag ? nullptr : p->partial_stage);
        if (d > 1) {
            g.piece = piece;
            g.pstride = geo.rows;
            g.poff = j * piece;
        }
        g.gate = ag ? kGateMain : kGateEpilogue;
        g.flag_base = j * geo.P;
        g.nparts = geo.P;
        g.resident_mask = res;
        for (int t = 0; t < g.tiles_m; ++t) g.rt_touch[t] = all;   // a sub-operator needs its whole sub-collective
        if (j == 0) g.start_word = &g_ctx.hw[kHwStart];
        if (!ag && p->send_dst) {
            g.done_host = &g_ctx.hw[kHwDone];
            g.send_mask = nonlocal_mask(p, geo);
            for (int q = 0; q < geo.P; ++q)
                if (g.send_mask & (1ull << q)) g.done_expect[q] = (uint32_t)(g.tiles_m * g.tiles_n);
        }
    }
    if (p->pattern == COMPASS_AG_GEMM) {
        submit(0, std::move(ag_f));
        submit(1, std::move(ag_b));
    } else {
        for (int r = 0; r < 4; ++r) submit(r, std::move(rs[r]));
    }
    for (int j = 0; j < d; ++j)
        if ((rc = launch(launches[j], p->pattern == COMPASS_GEMM_RS, s)) != COMPASS_OK) return rc;
    if (!finals.empty()) return join(epoch, finals, false, s);
    return COMPASS_OK;
}

int op_gemm(int M, int N, int K, const void *A, const void *W, void *C, const float *P, void *stream) {
    if (M < 1 || N < 1 || K < 1 || K % 8 || N % 8) return set_error(COMPASS_ERR_INVALID, "need positive M, N, K with K, N multiples of 8");
    if (!A || !W || !C) return set_error(COMPASS_ERR_INVALID, "A, W and C are required");
    if ((M + kTileM - 1) / kTileM > kMaxRowTiles) return set_error(COMPASS_ERR_UNSUPPORTED, "M too large");
    if ((double)M * K * 2 >= 2147483648.0 || (double)N * K * 2 >= 2147483648.0 || (double)M * N * 4 >= 2147483648.0)
        return set_error(COMPASS_ERR_UNSUPPORTED, "operand larger than 2 GiB");
    int rc = begin();
    if (rc != COMPASS_OK) return rc;
    GemmParams g;
    init_params(g, g_ctx.epoch);
    set_shape(g, M, N, K, A, M, W, C, P);
    g.gate = kGateNone;
    return launch(g, P != nullptr, (hipStream_t)stream);
}

int op_transfer(const compass_problem *p, const compass_links *l, void *stream) {
    Geometry geo;
    int rc = validate(p, l, -1, &geo);
    if (rc != COMPASS_OK) return rc;
    if ((rc = begin()) != COMPASS_OK) return rc;
    hipStream_t s = (hipStream_t)stream;
    const uint32_t epoch = next_epoch();
    std::vector<int> wait;
    if (p->pattern == COMPASS_AG_GEMM) {
        Job f, b;
        if ((rc = ag_jobs(p, geo, l, epoch, 1, true, &f, &b)) != COMPASS_OK) return rc;
        for (auto &it : f.items) wait.push_back(it.flag);
        for (auto &it : b.items) wait.push_back(it.flag);
        if ((rc = join(epoch, wait, true, s)) != COMPASS_OK) return rc;
        submit(0, std::move(f));
        submit(1, std::move(b));
    } else {
        Job jobs[4];
        if ((rc = rs_jobs(p, geo, l, epoch, 1, resident_mask(p, geo), false, true, jobs)) != COMPASS_OK) return rc;
        for (int r = 0; r < 2; ++r)
            for (auto &it : jobs[r].items) wait.push_back(it.flag);
        for (int r = 2; r < 4; ++r)
            if (jobs[r].final_flag >= 0) wait.push_back(jobs[r].final_flag);
        if ((rc = join(epoch, wait, true, s)) != COMPASS_OK) return rc;
        for (int r = 0; r < 4; ++r) submit(r, std::move(jobs[r]));
    }
    return COMPASS_OK;
}

int op_sequential(const compass_problem *p, const compass_links *l, void *stream) {
    if (p && p->pattern == COMPASS_AG_GEMM) return op_decomp(p, 1, l, stream);
    Geometry geo;
    int rc = validate(p, l, COMPASS_GEMM_RS, &geo);
    if (rc != COMPASS_OK) return rc;
    if ((rc = begin()) != COMPASS_OK) return rc;
    hipStream_t s = (hipStream_t)stream;
    const uint32_t epoch = next_epoch();
    const uint64_t res = resident_mask(p, geo);
    Job jobs[4];
    if ((rc = rs_jobs(p, geo, l, epoch, 1, res, false, true, jobs)) != COMPASS_OK) return rc;
    if ((rc = stage_resident_partials(p, geo, res, s)) != COMPASS_OK) return rc;
    GemmParams g;
    init_params(g, epoch);
    set_shape(g, p->M, p->N, p->K, p->A, p->M, p->W, p->C, p->partial_stage);
    g.gate = kGateNone;
    if ((rc = launch(g, true, s)) != COMPASS_OK) return rc;
    std::vector<int> wait;
    for (int r = 0; r < 2; ++r)
        for (auto &it : jobs[r].items) wait.push_back(it.flag);
    for (int r = 2; r < 4; ++r)
        if (jobs[r].final_flag >= 0) wait.push_back(jobs[r].final_flag);
    if ((rc = join(epoch, wait, true, s)) != COMPASS_OK) return rc;
    for (int r = 0; r < 4; ++r) submit(r, std::move(jobs[r]));
    return COMPASS_OK;
}

int op_sync() {
    int rc = ensure_init();
    if (rc != COMPASS_OK) return rc;
    const double t0 = now_s();
    while (!pacers_idle()) {
        if (now_s() - t0 > g_ctx.host_timeout + 1.0) {
            g_ctx.async_err.store(COMPASS_ERR_TIMEOUT);
            break;
        }
        std::this_thread::yield();
    }
    const hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    return take_async_error();
}

int op_set_option(int key, long long v) {
    Ctx &c = g_ctx;
    switch (key) {
    case COMPASS_OPT_SPIN_LIMIT:
        if (v < 1 || v > 0xFFFFFFFFll) return set_error(COMPASS_ERR_INVALID, "spin limit out of range");
        c.spin_limit = (uint32_t)v;
        return COMPASS_OK;
    case COMPASS_OPT_HOST_TIMEOUT:
        if (v < 1) return set_error(COMPASS_ERR_INVALID, "host timeout must be positive");
        c.host_timeout = (double)v * 1e-6;
        return COMPASS_OK;
    case COMPASS_OPT_GRID:
        if (v < 0 || v > 65536) return set_error(COMPASS_ERR_INVALID, "grid out of range");
        c.grid_override = (int)v;
        return COMPASS_OK;
    case COMPASS_OPT_DROP_FLAG:
        if (v < -1 || v >= 2 * kMaxRanks) return set_error(COMPASS_ERR_INVALID, "drop flag out of range");
        c.drop_flag = (int)v;
        return COMPASS_OK;
    default:
        return set_error(COMPASS_ERR_INVALID, "unknown option %d", key);
    }
}

}  // namespace compass
