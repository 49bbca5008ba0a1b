// Host runtime of the Compass hot path on one MI355X.
//
// Emulated links (the push-based DMA ring transfers of Section III-B): each
// ring direction is served by a pacer thread that owns a set of SDMA engines
// (HSA async copies forced onto SDMA, so no compute unit is taken from the
// GEMM). A job is an ordered list of partition transfers; the pacer issues
// them in slices no earlier than their paced times (rate = the emulated link
// bandwidth), polls the slices' completion signals, and publishes a
// partition's arrival flag (a release store of the call's epoch into pinned
// host memory) once all of its slices have landed. Copies never depend on one
// another through signals: every completion signal is re-armed only after the
// copy it tracked has completed. Unpaced operators with several active
// directions instead run one pooled job on every engine (execute_pooled):
// the directions then share the engines slice by slice, in transfer order.
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
#include <execinfo.h>
#include <immintrin.h>
#include <signal.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cmath>
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

hipError_t launch_gemm(const GemmParams &p, int cfg, bool rs, hipStream_t stream);
hipError_t launch_join(const JoinParams &j, hipStream_t stream);
hipError_t launch_mfma_probe(uint64_t *out, int grid, int iters, hipStream_t stream);

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
constexpr int kSignals = 256;        // completion signals per pacer
constexpr size_t kDefaultSlice = 2u << 20;
constexpr int kDefaultPoolDepth = 4;
// slice of a pooled job when the links leave it to the library: fewer,
// larger copies carry more per engine (the fused fc2 ReduceScatter at 3 MiB
// against 2 MiB: kernel 259 against 298 us), and a 4 MiB AllGather
// partition is still two copies on two engines
constexpr size_t kPoolSlice = 3u << 20;
constexpr int kSchedFineQueues = 1, kSchedSpread = 2, kSchedSplitK = 4;
// split-K workspace: one fp32 partial tile per workgroup slot (the largest
// of 256 x 256 on one workgroup per CU and 128 x 128 on two)
constexpr int kMinSliceK = 512;      // K depth of a slice at least
constexpr int kSplitWsTiles = 3;     // workspace: this many 256 x 256 fp32 partial tiles per CU
constexpr int kTailMinK = 8192;      // fused AllGather: split the tail's K from this depth on
constexpr int kTailSliceK = 2048;    // ... into slices at least this deep, at most 4
constexpr double kTailMaxLambda = 2.0;   // ... when the estimated comp / comm ratio is below this
// host_words layout (pinned, coherent host memory): start word, error word,
// done flags (kernel -> copy side), arrival flags (copy side -> kernel)
constexpr int kHwStart = 0, kHwErr = 1, kHwDone = 64, kHwFlags = kHwDone + kMaxFlags;
constexpr int kHwWords = kHwFlags + kMaxFlags;
// ctrl layout (device memory): tickets, done counters, flag mirrors, leaders
constexpr int kCtrlDone = 64;
constexpr int kCtrlMirror = kCtrlDone + kMaxFlags;
constexpr int kCtrlLeader = kCtrlMirror + kMaxFlags;
constexpr int kCtrlCuSlot = kCtrlLeader + kMaxFlags;
constexpr int kCtrlSplit = kCtrlCuSlot + kCuSlots;
constexpr int kCtrlWords = kCtrlSplit + kMaxSplitTiles;

struct Item {
    void *dst;
    const void *src;
    size_t bytes;
    hsa_agent_t dst_agent, src_agent;
    int flag;   // arrival flag to publish after the item, -1: none
    int gate;   // host done flag to wait for before the item, -1: none
    double due_at = -1.0;   // paced, >= 0: due this long after the job started
    int seq = 0;            // position in the operator's transfer order (pooled jobs)
    // pooled jobs: the link the item travels on (its direction's role), that
    // link's rate (<= 0: unpaced) and the item's slice size
    int link = 0;
    double rate = 0.0;
    size_t slice = 0;
};

struct Job {
    std::vector<Item> items;
    std::vector<uint32_t> engines;   // SDMA engine id bits
    double rate = 0;                 // bytes / s, <= 0: unpaced
    size_t slice = kDefaultSlice;
    bool slice_default = true;       // the links left the slice to the library
    uint32_t epoch = 0;
    bool wait_start = true;
    bool concurrent = false;         // paced: every item on a link of its own
    int final_flag = -1;             // flag published after every item landed
    std::vector<int> more_finals;    // further such flags (a pooled job)
    int pool_depth = 0;              // > 0: unpaced directions sharing every engine,
                                     // at most this many copies queued per engine
};

struct Ctx;

struct Pacer {
    Ctx *ctx = nullptr;
    int role = 0;
    std::thread th;
    std::mutex mu;
    std::condition_variable cv;
    std::deque<Job> q;
    std::atomic<int> pending{0};
    std::atomic<bool> stop{false};
    hsa_signal_t sig[kSignals];
    int sig_next = 0;
    double lat_scale = 1.3;   // observed / modelled copy latency of paced items (biased late)
    void loop();
    void execute(Job &job);
    void execute_pooled(Job &job);
    bool take_signal(hsa_signal_t *out);
    bool quiesce();
};

struct Ctx {
    bool ready = false;
    int device = -1;
    int num_cu = 0;
    uint64_t *probe_out = nullptr;   // matrix-core probe results (3 words per wave)
    hsa_agent_t gpu{}, cpu{};
    std::vector<uint32_t> engines;   // SDMA engines usable device->device
    uint32_t *ctrl = nullptr;        // device memory
    uint32_t *hw = nullptr;          // pinned host words
    uint32_t epoch = 0;
    Pacer pacer[kRoles];
    std::atomic<int> async_err{0};
    std::atomic<bool> in_flight{false};   // a failed job's copies outlived the bound
    uint32_t spin_limit = 4u << 20;  // kernel polls (about 0.5 us each)
    double host_timeout = 5.0;       // seconds
    int grid_override = 0;
    int drop_flag = -1;
    int tile_override = 0;           // 0 auto, 1 256 x 256, 2 128 x 128
    int pool_depth = kDefaultPoolDepth;   // unpaced directions share the engines (0: split)
    double pace_headroom = 0.05;          // paced groups: throughput to spare over the link rate
    // fused AllGather tail split: K depth from which it applies (per tile
    // shape, 0: never), least slice depth, row-tile groups it covers
    int tail_min_k[2] = {kTailMinK, 0};   // [0] 256 x 256, [1] 128 x 128
    int tail_slice_k = kTailSliceK;
    int tail_groups = 2;
    bool head_split = true;               // fused AllGather: split the resident tiles' K (see set_head_split)
    // optional HIP events around every GEMM launch (kernel durations)
    bool timing = false;
    static constexpr int kTimed = 512;
    hipEvent_t ev_begin[kTimed] = {}, ev_end[kTimed] = {};
    int timed_count = 0;             // launches recorded since the last read
    uint32_t launch_seq = 0;         // tags the per-CU slot claims of a launch
    int sched = kSchedFineQueues | kSchedSpread | kSchedSplitK;
    float *split_ws = nullptr;       // device, split_ws_bytes
    size_t split_ws_bytes = 0;
    // optional per-tile trace records (device buffer of trace_cap records)
    uint32_t *tile_trace = nullptr;
    uint32_t trace_cap = 0, trace_used = 0;
    uint32_t engine_mask = 0;        // hardware engines allowed (0: all usable)
    // copy-side trace (COMPASS_TRACE=<file>): one line per event
    bool tracing = false;
    std::string trace_path;
    std::mutex trace_mu;
    std::vector<std::string> trace;
    struct Range { uintptr_t lo, hi; hsa_agent_t owner; };
    std::vector<Range> ranges;       // allocations looked up by the current call (owner, bounds)
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
    if (tracing && !trace.empty()) {
        if (FILE *f = std::fopen(trace_path.c_str(), "w")) {
            std::fputs("t_s,role,epoch,event,item,bytes\n", f);
            for (auto &l : trace) std::fputs(l.c_str(), f);
            std::fclose(f);
        }
    }
}

static void trace_event(int role, uint32_t epoch, const char *ev, int item, size_t bytes) {
    Ctx &c = g_ctx;
    if (!c.tracing) return;
    char buf[160];
    std::snprintf(buf, sizeof buf, "%.9f,%d,%u,%s,%d,%zu\n", now_s(), role, epoch, ev, item, bytes);
    std::lock_guard<std::mutex> lk(c.trace_mu);
    if (c.trace.size() < 2000000) c.trace.push_back(buf);
}

// COMPASS_DEBUG_SEGV=1: print the native backtrace of a thread that faults
// on the host, then fall back to the default action.
static void segv_handler(int sig) {
    void *frames[64];
    const int n = backtrace(frames, 64);
    static const char msg[] = "compass: host fault, native backtrace:\n";
    (void)!write(2, msg, sizeof msg - 1);
    backtrace_symbols_fd(frames, n, 2);
    signal(sig, SIG_DFL);
    raise(sig);
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
    if (std::getenv("COMPASS_DEBUG_SEGV")) {
        signal(SIGSEGV, segv_handler);
        signal(SIGBUS, segv_handler);
    }
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
    if ((e = hipMalloc((void **)&c.ctrl, kCtrlWords * sizeof(uint32_t))) != hipSuccess) return hip_fail(e, "control allocation");
    if ((e = hipHostMalloc((void **)&c.hw, kHwWords * sizeof(uint32_t), hipHostMallocCoherent)) != hipSuccess)
        return hip_fail(e, "host word allocation");
    std::memset(c.hw, 0, kHwWords * sizeof(uint32_t));
    if ((e = hipMemset(c.ctrl, 0, kCtrlWords * sizeof(uint32_t))) != hipSuccess) return hip_fail(e, "control clear");
    {
        // Uncached, so that partial tiles written on one XCD are read on
        // another without cache maintenance. Held until the process ends
        // (uncached memory is never freed once a kernel has read it).
        const size_t ws = (size_t)kSplitWsTiles * c.num_cu * std::max(256 * 256, 2 * 128 * 128) * sizeof(float);
        if ((e = hipExtMallocWithFlags((void **)&c.split_ws, ws, hipDeviceMallocUncached)) != hipSuccess)
            return hip_fail(e, "split-K workspace");
        c.split_ws_bytes = ws;
    }
    if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(e, "init sync");
    for (int r = 0; r < kRoles; ++r) c.pacer[r].role = r;
    if (const char *tp = std::getenv("COMPASS_TRACE")) {
        c.tracing = true;
        c.trace_path = tp;
    }
    // Completion signals are polled by the pacer threads, never waited on:
    // naming the GPU as their only consumer gives plain memory signals, with
    // no interrupt raised per copy (COMPASS_SIGNALS=interrupt restores
    // runtime-default signals).
    const char *sm = std::getenv("COMPASS_SIGNALS");
    const bool interrupt = sm && std::strcmp(sm, "interrupt") == 0;
    for (auto &p : c.pacer) {
        p.ctx = &c;
        for (auto &s : p.sig)
            if (hsa_signal_create(0, interrupt ? 0 : 1, interrupt ? nullptr : &c.gpu, &s) != HSA_STATUS_SUCCESS)
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
            if (hsa_amd_memory_async_copy_on_engine(c.ctrl + kCtrlWords - 1, c.gpu, c.ctrl + kCtrlWords - 2, c.gpu,
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
        // engines other clients hold are used only when fewer than four are free
        c.engines = ok_free;
        if (c.engines.size() < 4) c.engines.insert(c.engines.end(), ok_busy.begin(), ok_busy.end());
        if (c.engines.empty()) return set_error(COMPASS_ERR_UNSUPPORTED, "no SDMA engine accepted a copy");
        if (std::getenv("COMPASS_VERBOSE"))
            std::fprintf(stderr, "compass: %zu SDMA engines usable (%zu reported free)\n", c.engines.size(), ok_free.size());
    }
    for (auto &p : c.pacer) p.th = std::thread([&p] { p.loop(); });
    c.ready = true;
    return COMPASS_OK;
}

// The agent owning the allocation that holds `ptr` (device memory -> the
// GPU, host memory -> the CPU), and the end of that allocation (*end,
// optional).
static int agent_of(const void *ptr, hsa_agent_t *out, uintptr_t *end = nullptr) {
    Ctx &c = g_ctx;
    const uintptr_t u = (uintptr_t)ptr;
    for (auto &r : c.ranges)
        if (u >= r.lo && u < r.hi) {
            *out = r.owner;
            if (end) *end = r.hi;
            return COMPASS_OK;
        }
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
    if (end) *end = lo + info.sizeInBytes;
    return COMPASS_OK;
}

// ---------------------------------------------------------------- pacer
// The next completion signal, armed with 1 for a new copy. A slot comes
// round again kSignals copies later: if the copy it tracked has not landed
// within the host-side bound, the slot is left as it is (re-armed, the old
// copy's completion would count as the new copy's landing) and false is
// returned, so that the caller issues nothing and the job ends on the error.
bool Pacer::take_signal(hsa_signal_t *out) {
    hsa_signal_t s = sig[sig_next];
    const double t0 = now_s();
    while (hsa_signal_load_scacquire(s) > 0) {
        if (now_s() - t0 > ctx->host_timeout) {
            ctx->async_err.store(COMPASS_ERR_TIMEOUT);
            return false;
        }
        _mm_pause();
    }
    sig_next = (sig_next + 1) % kSignals;
    hsa_signal_store_relaxed(s, 1);
    *out = s;
    return true;
}

// Wait until every copy issued with this pacer's signals has completed
// (bounded: the host timeout, at least one second, since the timeout may be
// what ended the job). False when copies were still in flight at the bound.
bool Pacer::quiesce() {
    const double t0 = now_s(), bound = std::max(1.0, ctx->host_timeout);
    for (int i = 0; i < kSignals; ++i)
        while (hsa_signal_load_scacquire(sig[i]) > 0) {
            if (now_s() - t0 > bound) return false;
            _mm_pause();
        }
    return true;
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
        // a job that ended on an error may have left copies in flight: let them
        // land before the job counts as done, so that compass_sync() returns
        // with none of them still writing the caller's buffers
        // (copies that outlive the bound leave the library refusing every
        // later call: they may still write the caller's buffers)
        if (ctx->async_err.load() != 0 && !quiesce()) ctx->in_flight.store(true);
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

// ---- paced links
// Engine cost model for device-to-device SDMA copies measured on MI355X with
// every engine busy: a copy of s bytes occupies its engine for about
// kCopyFixed + s / kEngineBps. It sizes the engine groups and the lead time
// of paced items; the observed latencies correct it as items land.
constexpr double kCopyFixed = 10e-6;
constexpr double kEngineBps = 38e9;

// Engines per item for a paced job: the widest group (shortest item latency)
// whose E / k groups still carry the link rate with `headroom` to spare. If
// none does, the rate is out of reach, and the widest group that still moves
// 90 % of what single copies do (E at a time, paying the fixed cost of a
// copy least often): for small items that is one engine per item (all E
// engines on a 1 MiB item would carry a fraction of what single copies do),
// for large ones the whole set (a 22 MB item on one engine lands after
// ~590 us, on four after ~155 us, for 5 % less throughput). The first items
// of a job are issued at once and land one group latency after the start,
// so too narrow a group delays them all: at 268 GB/s with 22 MiB items, 10 %
// headroom left groups of 2 engines (≈ 310 µs per item) where 5 % allows 4
// (≈ 160 µs), and the fused GPT-3 AllGather took 1429 against 1144 µs.
static size_t group_width(double rate, size_t E, size_t item_bytes, double headroom) {
    auto carried = [&](size_t k) {
        const double lat = kCopyFixed + (double)item_bytes / ((double)k * kEngineBps);
        return (double)(E / k) * (double)item_bytes / lat;
    };
    for (size_t k = E; k >= 1; --k) {
        if (E % k) continue;
        if (carried(k) >= (1.0 + headroom) * rate) return k;
    }
    for (size_t k = E; k > 1; --k)
        if (E % k == 0 && carried(k) >= 0.9 * carried(1)) return k;
    return 1;
}

// One job.
//
// Paced (rate > 0): the emulated link carries one item at a time at `rate`,
// so item i is due at link_free + bytes / rate, where link_free is when the
// link finished the previous item (or when the item's gate opened, if
// later). The item goes out whole on one group of k engines (groups taken in
// turn), issued ahead of its due time by its predicted copy latency; its
// arrival flag is published at the due time or when its copies have landed,
// whichever is later. The kernel therefore never sees data before the link
// would have delivered it.
//
// Concurrent (paced): every item has a link of its own at `rate`, all of them
// starting with the job (or at the item's gate), so item i is due at
// start + bytes / rate and the link_free chain is not advanced.
//
// An item with a due time of its own (due_at >= 0, paced) is due that long
// after the job started, whatever the chain says (a ring whose hops differ).
//
// Unpaced (rate <= 0): slices go out round-robin over the engines as fast as
// they are taken; an item's flag is published when its slices have landed.
//
// Flags are release stores of the epoch into host memory. Copies carry no
// dependencies on one another; completion is observed here by polling.
void Pacer::execute(Job &job) {
    Ctx &c = *ctx;
    if (job.items.empty() && job.final_flag < 0) return;
    if (job.pool_depth > 0) {
        execute_pooled(job);
        return;
    }
    trace_event(role, job.epoch, "job_begin", -1, 0);
    if (job.wait_start && !spin_until_epoch(&c.hw[kHwStart], job.epoch, c.host_timeout)) {
        c.async_err.store(COMPASS_ERR_TIMEOUT);
        return;
    }
    trace_event(role, job.epoch, "start_seen", -1, 0);
    struct Pend {
        int flag;
        size_t first, count;   // its signals in `issued`
        double due;            // earliest publication time
        double issued_at, model;
        bool landed;
    };
    const size_t E = job.engines.size();
    const bool paced = job.rate > 0;
    size_t max_item = 0;
    for (auto &it : job.items) max_item = std::max(max_item, it.bytes);
    // concurrent items each take a group of their own where the engines allow
    const size_t k = !paced ? E
                     : job.concurrent ? std::max<size_t>(1, E / std::max<size_t>(1, job.items.size()))
                                      : group_width(job.rate, E, max_item, c.pace_headroom);
    const size_t groups = E / k;
    std::vector<hsa_signal_t> issued;
    std::vector<Pend> pend;
    double link_free = now_s();
    const double job_start = link_free;
    double last_progress = link_free;
    size_t rr = 0, idx = 0, off = 0, item_first = 0;
    bool gate_ok = false;
    double gate_time = 0;

    auto issue = [&](const Item &it, size_t o, size_t len, size_t e) -> bool {
        hsa_signal_t sg;
        if (!take_signal(&sg)) return false;
        const hsa_status_t st = hsa_amd_memory_async_copy_on_engine(
            (char *)it.dst + o, it.dst_agent, (const char *)it.src + o, it.src_agent, len, 0, nullptr, sg,
            (hsa_amd_sdma_engine_id_t)job.engines[e], true);
        if (st != HSA_STATUS_SUCCESS) {
            hsa_signal_store_relaxed(sg, 0);
            c.async_err.store(COMPASS_ERR_HIP);
            return false;
        }
        trace_event(role, job.epoch, "slice", __builtin_ctz(job.engines[e]), len);
        issued.push_back(sg);
        return true;
    };

    for (;;) {
        bool progress = false;
        const double now = now_s();
        for (size_t i = 0; i < pend.size();) {
            Pend &pd = pend[i];
            if (!pd.landed) {
                bool landed = true;
                for (size_t si = pd.first; si < pd.first + pd.count && landed; ++si)
                    landed = hsa_signal_load_scacquire(issued[si]) <= 0;
                if (landed) {
                    pd.landed = true;
                    trace_event(role, job.epoch, "item_landed", pd.flag, 0);
                    if (paced && pd.model > 0) {
                        // latency correction, biased late: an early item only waits for its due time
                        const double ratio = (now - pd.issued_at) / pd.model;
                        lat_scale = 0.7 * lat_scale + 0.3 * std::min(4.0, std::max(0.5, 1.15 * ratio));
                    }
                }
            }
            if (pd.landed && now >= pd.due) {
                __atomic_store_n(&c.hw[kHwFlags + pd.flag], job.epoch, __ATOMIC_RELEASE);
                trace_event(role, job.epoch, "flag", pd.flag, 0);
                pend.erase(pend.begin() + (long)i);
                progress = true;
            } else {
                ++i;
            }
        }
        if (idx < job.items.size()) {
            const Item &it = job.items[idx];
            if (it.gate >= 0 && !gate_ok &&
                (int32_t)(__atomic_load_n(&c.hw[kHwDone + it.gate], __ATOMIC_ACQUIRE) - job.epoch) >= 0) {
                gate_ok = true;
                gate_time = now_s();
                trace_event(role, job.epoch, "gate_open", it.gate, 0);
            }
            if (it.gate < 0 || gate_ok) {
                if (paced) {
                    const double start = std::max(link_free, it.gate >= 0 ? gate_time : 0.0);
                    const double due = it.due_at >= 0 ? job_start + it.due_at : start + (double)it.bytes / job.rate;
                    const double model = kCopyFixed + (double)it.bytes / ((double)k * kEngineBps);
                    if (now_s() >= due - model * lat_scale) {
                        const size_t first = issued.size();
                        const size_t g0 = (idx % groups) * k;
                        size_t per = (it.bytes + k - 1) / k;
                        per = std::min((per + 255) & ~(size_t)255, job.slice);
                        size_t o = 0, j = 0;
                        while (o < it.bytes) {
                            const size_t len = std::min(per, it.bytes - o);
                            if (!issue(it, o, len, g0 + (j++ % k))) return;
                            o += len;
                        }
                        if (it.flag >= 0) pend.push_back({it.flag, first, issued.size() - first, due, now_s(), model, false});
                        trace_event(role, job.epoch, "item_due_ns", it.flag, (size_t)std::max(0.0, (due - job_start) * 1e9));
                        if (!job.concurrent) link_free = due;
                        ++idx;
                        gate_ok = false;
                        progress = true;
                    }
                } else {
                    if (off == 0) item_first = issued.size();
                    if (off < it.bytes) {
                        const size_t len = std::min(job.slice, it.bytes - off);
                        if (!issue(it, off, len, rr++ % E)) return;
                        off += len;
                    }
                    if (off >= it.bytes) {
                        if (it.flag >= 0) pend.push_back({it.flag, item_first, issued.size() - item_first, 0.0, 0.0, 0.0, false});
                        ++idx;
                        off = 0;
                        gate_ok = false;
                    }
                    progress = true;
                }
            }
        } else if (pend.empty()) {
            break;
        }
        if (progress) {
            last_progress = now_s();
        } else {
            // waiting for a due time (paced) is not a stall
            double horizon = last_progress;
            if (paced) horizon = std::max(horizon, link_free + (double)max_item / job.rate);
            if (now_s() - horizon > c.host_timeout) {
                c.async_err.store(COMPASS_ERR_TIMEOUT);
                return;
            }
            _mm_pause();
        }
    }
    trace_event(role, job.epoch, "issued", -1, 0);
    // the job is over once every copy has landed
    const double t0 = now_s();
    for (auto sg : issued)
        while (hsa_signal_load_scacquire(sg) > 0) {
            if (now_s() - t0 > c.host_timeout) {
                c.async_err.store(COMPASS_ERR_TIMEOUT);
                return;
            }
            _mm_pause();
        }
    if (job.final_flag >= 0) __atomic_store_n(&c.hw[kHwFlags + job.final_flag], job.epoch, __ATOMIC_RELEASE);
    trace_event(role, job.epoch, "landed", -1, 0);
}

// Pooled (the directions of one operator sharing every engine): the job
// holds the items of every active ring direction in the operator's transfer
// order. Each engine keeps at most `pool_depth` copies queued; whenever one
// has room it takes the next slice of the ready item (gate open) with bytes
// left whose due time is earliest, the first in transfer order among equal
// ones. An item's flag is published when all of its slices have landed and
// its due time has passed.
//
// Due times: an unpaced item (rate <= 0) is due at once, so the engines
// serve the items in transfer order: an outgoing sum follows the incoming
// partial of its partition, a finished chunk's send goes out ahead of later
// arrivals, and no engine idles while either direction has ready work. A
// paced item is due when its link would have delivered it: its link carries
// one item at a time at the link's rate, so item i is due at
// max(due of the link's previous item, when its gate opened) + bytes / rate
// (an item with a due time of its own, a ring whose hops differ, keeps it).
// The copy engines move a paced item as early as their queues allow and the
// flag waits for the due time: the kernel sees exactly the link's arrival
// times, and no item lands late for lack of engines while another
// direction's engines idle (engines split per direction, the first items of
// the faster direction of a 4 : 1 ring landed 130 us after their due times).
// Items are cut into equal slices of at most their `slice` bytes.
void Pacer::execute_pooled(Job &job) {
    Ctx &c = *ctx;
    trace_event(role, job.epoch, "job_begin", -1, 0);
    if (job.wait_start && !spin_until_epoch(&c.hw[kHwStart], job.epoch, c.host_timeout)) {
        c.async_err.store(COMPASS_ERR_TIMEOUT);
        return;
    }
    const double job_start = now_s();
    trace_event(role, job.epoch, "start_seen", -1, 0);
    const size_t E = job.engines.size();
    const int depth = std::max(1, job.pool_depth);
    constexpr double kUnknown = -1.0;
    struct State {
        size_t off = 0, per = 0;
        int inflight = 0;
        bool ready = false, done = false;
        double opened = 0.0;      // when the gate opened (the job start if none)
        double due = kUnknown;    // earliest publication
    };
    struct Copy {
        hsa_signal_t sg;
        size_t item, eng, len;
    };
    std::vector<State> st(job.items.size());
    size_t remaining = 0;
    int links = 1;
    for (size_t i = 0; i < job.items.size(); ++i) {
        const Item &it = job.items[i];
        const size_t slice = it.slice ? it.slice : job.slice;
        const size_t k = std::max<size_t>(1, (it.bytes + slice - 1) / slice);
        st[i].per = std::max<size_t>(256, ((it.bytes + k - 1) / k + 255) & ~(size_t)255);
        st[i].ready = it.gate < 0;
        st[i].opened = job_start;
        links = std::max(links, it.link + 1);
        ++remaining;
    }
    // per link: when it has delivered its last item with a due time, and
    // the next item (in order) still without one
    std::vector<double> link_free(links, job_start);
    std::vector<size_t> next_due(links, 0);
    auto assign_dues = [&]() {
        for (int L = 0; L < links; ++L) {
            size_t &i = next_due[L];
            for (; i < job.items.size(); ++i) {
                const Item &it = job.items[i];
                if (it.link != L) continue;
                State &s = st[i];
                if (!s.ready) break;   // later items of this link wait for it
                if (it.due_at >= 0) {
                    s.due = job_start + it.due_at;
                } else if (it.rate > 0) {
                    s.due = std::max(link_free[L], s.opened) + (double)it.bytes / it.rate;
                    link_free[L] = s.due;
                } else {
                    s.due = 0.0;
                }
                if (it.flag >= 0 && s.due > 0) trace_event(role, job.epoch, "item_due_ns", it.flag,
                                                          (size_t)((s.due - job_start) * 1e9));
            }
        }
    };
    assign_dues();
    std::vector<Copy> fly;
    std::vector<int> load(E, 0);
    size_t rr = 0, first_open = 0;
    double last_progress = now_s();
    while (remaining > 0) {
        bool progress = false;
        for (size_t i = 0; i < fly.size();) {
            if (hsa_signal_load_scacquire(fly[i].sg) > 0) {
                ++i;
                continue;
            }
            --load[fly[i].eng];
            trace_event(role, job.epoch, "copy_done", __builtin_ctz(job.engines[fly[i].eng]), fly[i].len);
            State &s = st[fly[i].item];
            --s.inflight;
            fly[i] = fly.back();
            fly.pop_back();
            progress = true;
        }
        const double now = now_s();
        bool opened = false;
        for (size_t i = first_open; i < job.items.size(); ++i) {
            const Item &it = job.items[i];
            State &s = st[i];
            if (s.done) continue;
            if (!s.ready && (int32_t)(__atomic_load_n(&c.hw[kHwDone + it.gate], __ATOMIC_ACQUIRE) - job.epoch) >= 0) {
                s.ready = true;
                s.opened = now;
                opened = true;
                progress = true;
                trace_event(role, job.epoch, "gate_open", it.gate, 0);
            }
            if (s.ready && s.inflight == 0 && s.off >= it.bytes && s.due != kUnknown && now >= s.due) {
                if (it.flag >= 0) {
                    __atomic_store_n(&c.hw[kHwFlags + it.flag], job.epoch, __ATOMIC_RELEASE);
                    trace_event(role, job.epoch, "flag", it.flag, 0);
                }
                s.done = true;
                --remaining;
                progress = true;
            }
        }
        if (opened) assign_dues();
        while (first_open < job.items.size() && st[first_open].done) ++first_open;
        for (;;) {
            size_t e = E;
            for (size_t k = 0; k < E; ++k) {
                const size_t cand = (rr + k) % E;
                if (load[cand] < depth && (e == E || load[cand] < load[e])) e = cand;
            }
            if (e == E) break;
            size_t pick = job.items.size();
            for (size_t i = first_open; i < job.items.size(); ++i) {
                const State &s = st[i];
                if (!s.ready || s.due == kUnknown || s.off >= job.items[i].bytes) continue;
                if (pick == job.items.size() || s.due < st[pick].due) pick = i;
            }
            if (pick == job.items.size()) break;
            const Item &it = job.items[pick];
            State &s = st[pick];
            const size_t len = std::min(s.per, it.bytes - s.off);
            hsa_signal_t sg;
            if (!take_signal(&sg)) return;
            const hsa_status_t rc = hsa_amd_memory_async_copy_on_engine(
                (char *)it.dst + s.off, it.dst_agent, (const char *)it.src + s.off, it.src_agent, len, 0, nullptr, sg,
                (hsa_amd_sdma_engine_id_t)job.engines[e], true);
            if (rc != HSA_STATUS_SUCCESS) {
                hsa_signal_store_relaxed(sg, 0);
                c.async_err.store(COMPASS_ERR_HIP);
                return;
            }
            trace_event(role, job.epoch, "slice", __builtin_ctz(job.engines[e]), len);
            fly.push_back({sg, pick, e, len});
            ++load[e];
            ++s.inflight;
            s.off += len;
            rr = e + 1;
            progress = true;
        }
        if (progress) {
            last_progress = now_s();
        } else {
            // waiting for a due time is not a stall
            double horizon = last_progress;
            for (size_t i = first_open; i < job.items.size(); ++i)
                if (!st[i].done && st[i].due != kUnknown) horizon = std::max(horizon, st[i].due);
            if (now_s() - horizon > c.host_timeout) {
                c.async_err.store(COMPASS_ERR_TIMEOUT);
                return;
            }
            _mm_pause();
        }
    }
    trace_event(role, job.epoch, "issued", -1, 0);
    if (job.final_flag >= 0) __atomic_store_n(&c.hw[kHwFlags + job.final_flag], job.epoch, __ATOMIC_RELEASE);
    for (int f : job.more_finals) __atomic_store_n(&c.hw[kHwFlags + f], job.epoch, __ATOMIC_RELEASE);
    trace_event(role, job.epoch, "landed", -1, 0);
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
    if (c.in_flight.load())
        return set_error(COMPASS_ERR_IN_FLIGHT, "copies of a failed transfer job outlived the host-side bound and may "
                                                "still write the caller's buffers; the library refuses further calls");
    const int a = c.async_err.exchange(0);
    const uint32_t k = __atomic_exchange_n(&c.hw[kHwErr], 0u, __ATOMIC_ACQ_REL);
    if (k != 0) return set_error(COMPASS_ERR_TIMEOUT, "a kernel-side wait exceeded its bound (code %u)", k);
    if (a == COMPASS_ERR_TIMEOUT) return set_error(COMPASS_ERR_TIMEOUT, "a copy-side wait exceeded its bound");
    if (a != 0) return set_error(a, "an asynchronous copy failed");
    return COMPASS_OK;
}

static uint32_t next_epoch() { return ++g_ctx.epoch; }

// SDMA engines of one ring direction: the usable engines are split over the
// directions active in the operator in proportion to `weight` (`active`
// lists their roles): the bytes each carries, times its rate when the
// directions are paced at different rates (a link four times faster needs
// four times the copy throughput while it runs). Unequal shares go in whole
// pairs of engines, so that a paced direction can group its engines (a group
// width divides the count: 13 engines would leave only groups of 1 or 13),
// with every direction keeping at least one pair; equal-rate splits keep
// their plain proportional ranges.
static std::vector<uint32_t> engines_for(int role, const std::vector<int> &active, const std::vector<double> &weight,
                                         int per_ring, bool paired = false) {
    std::vector<uint32_t> all;
    for (uint32_t e : g_ctx.engines)
        if (g_ctx.engine_mask == 0 || (g_ctx.engine_mask & e)) all.push_back(e);
    if (all.empty()) all = g_ctx.engines;
    const int n = (int)all.size();
    const int na = std::max<int>(1, (int)active.size());
    double wsum = 0;
    for (int i = 0; i < na; ++i) wsum += weight[i];
    int first = 0, count = 1;
    if (paired && n >= 2 * na) {
        // largest-remainder apportionment of n / 2 pairs, at least one each
        const int units = n / 2;
        std::vector<int> cnt(na);
        std::vector<double> rem(na);
        int used = 0;
        for (int i = 0; i < na; ++i) {
            const double ideal = units * weight[i] / wsum;
            cnt[i] = std::max(1, (int)std::floor(ideal));
            rem[i] = ideal - std::floor(ideal);
            used += cnt[i];
        }
        while (used > units) {   // a forced pair came out of the largest share
            const int big = (int)(std::max_element(cnt.begin(), cnt.end()) - cnt.begin());
            --cnt[big];
            --used;
        }
        while (used < units) {
            const int r = (int)(std::max_element(rem.begin(), rem.end()) - rem.begin());
            ++cnt[r];
            rem[r] = -1.0;
            ++used;
        }
        for (int i = 0, acc = 0; i < na; ++i) {
            const int c = 2 * cnt[i] + (i == na - 1 ? n - 2 * units : 0);
            if (active[i] == role) {
                first = acc;
                count = c;
            }
            acc += c;
        }
    } else {
        double acc = 0;
        for (int i = 0; i < na; ++i) {
            const int lo = (int)((double)n * acc / wsum);
            acc += weight[i];
            const int hi = (int)((double)n * acc / wsum);
            if (active[i] == role) {
                first = lo;
                count = std::max(1, hi - lo);
            }
        }
    }
    if (per_ring > 0) count = std::min(count, per_ring);
    std::vector<uint32_t> out;
    for (int i = 0; i < count; ++i) out.push_back(all[(first + i) % n]);
    return out;
}

// Engine weights of the active directions: `bytes` (their relative traffic),
// times the direction's rate when all of them are paced and the two ring
// directions' rates differ (roles 0 and 2 run at the forward rate, 1 and 3
// at the backward one). Returns whether the rates entered.
static bool direction_weights(const std::vector<int> &active, const std::vector<int> &bytes, const compass_links *l,
                              std::vector<double> *out) {
    out->assign(bytes.begin(), bytes.end());
    const bool by_rate = l->fwd_Bps > 0 && l->bwd_Bps > 0 && l->fwd_Bps != l->bwd_Bps && !l->hop_Bps;
    if (!by_rate) return false;
    bool both = false;
    for (int r : active) both |= r % 2 == 1;
    if (!both) return false;
    for (size_t i = 0; i < active.size(); ++i) (*out)[i] *= active[i] % 2 == 0 ? l->fwd_Bps : l->bwd_Bps;
    return true;
}

// The paper's double ring in either split (two partitions per chunk).
static inline bool two_rings(const compass_problem *p) {
    return p->ring == COMPASS_RING_DOUBLE || p->ring == COMPASS_RING_DOUBLE_SPLIT;
}

// Partitions: the ring's base partitions (a chunk, or a chunk's part on one
// ring of the double ring), each split into `sub` pieces of consecutive rows
// with a copy and an arrival flag of their own (sub-chunk flags). Partition
// q is piece q % sub of base partition q / sub, so partition ids still grow
// with the row.
struct Geometry {
    int P;           // partitions, BP * sub
    int BP;          // base partitions: n (single ring) or 2n (double ring)
    int sub;         // pieces per base partition (1: one flag per base partition)
    int rows;        // rows per chunk
    int prow;        // rows per base partition (double ring: half a chunk)
    bool dbl;        // double ring (either split)
    double fb;       // double ring: share of a chunk's rows on the backward ring
    int32_t sched[2 * kMaxRanks];
    int pos[2 * kMaxRanks];   // position of each partition in the schedule
};

// Rows of the backward (first) part of a block of r rows of one chunk under
// the double ring: half of it, or (proportional split) the backward ring's
// share of the two rates, rounded to a multiple of G rows (G = 128, the
// smaller tile's height, for blocks of at least 1024 rows, so that no tile
// spans both parts; else 8), down or up, whichever gives the shorter step,
// and leaving at least G (or half the block, if smaller) to each ring.
static int half0(const Geometry &g, int r) {
    if (g.fb == 0.5) return r / 2;
    const int G = r >= 1024 ? 128 : 8;
    const int lo = std::min(G, r / 2);
    auto clampv = [&](int h) { return std::min(std::max(h, lo), r - lo); };
    const int dn = clampv((int)std::floor(r * g.fb / G) * G);
    const int up = clampv((int)std::ceil(r * g.fb / G) * G);
    // step time in units of 1 / (B_fwd + B_bwd): max(h / fb, (r - h) / (1 - fb))
    auto step = [&](int h) { return std::fmax(h / g.fb, (r - h) / (1.0 - g.fb)); };
    return step(up) < step(dn) ? up : dn;
}

// Rows [*off, *off + *cnt) of a block of r chunk rows that base partition
// half h carries (single ring: all of them).
static void base_rows(const Geometry &g, int r, int h, int *off, int *cnt) {
    if (!g.dbl) { *off = 0; *cnt = r; return; }
    const int h0 = half0(g, r);
    *off = h ? h0 : 0;
    *cnt = h ? r - h0 : h0;
}

// Piece t of `sub` of a base block of cnt rows: rows [cnt t / sub, cnt (t+1) / sub).
static inline int piece_lo(int cnt, int t, int sub) { return (int)((long)cnt * t / sub); }

// Partition holding global row r (the fused operators' arrival gates).
static int part_of_row(const Geometry &g, int r) {
    const int c = r / g.rows;
    const int in = r - c * g.rows;
    int h = 0;
    if (g.dbl) h = in < half0(g, g.rows) ? 0 : 1;
    const int b = g.dbl ? 2 * c + h : c;
    if (g.sub == 1) return b;
    int off, cnt;
    base_rows(g, g.rows, h, &off, &cnt);
    int t = g.sub - 1;
    while (t > 0 && piece_lo(cnt, t, g.sub) > in - off) --t;
    return b * g.sub + t;
}

// Rows of the smallest partition.
static int min_part_rows(const Geometry &g) {
    int m = g.rows;
    if (g.dbl) {
        const int h0 = half0(g, g.rows);
        m = std::min(h0, g.rows - h0);
    }
    return m / g.sub;
}

// The partition layout of one rank: pattern, ring, ranks, rows and the link
// parameters that shape it (the rate split of COMPASS_RING_DOUBLE_SPLIT,
// sub-chunk flags). Host only.
static int make_geometry(int pattern, int ring, int n, int rank, int M, const compass_links *l, Geometry *g) {
    if (pattern != COMPASS_AG_GEMM && pattern != COMPASS_GEMM_RS) return set_error(COMPASS_ERR_INVALID, "unknown pattern");
    if (ring != COMPASS_RING_SINGLE && ring != COMPASS_RING_DOUBLE && ring != COMPASS_RING_DOUBLE_SPLIT &&
        ring != COMPASS_RING_ALLTOALL)
        return set_error(COMPASS_ERR_INVALID, "unknown ring");
    if (n < 1 || n > kMaxRanks || rank < 0 || rank >= n)
        return set_error(COMPASS_ERR_INVALID, "need 1 <= n <= %d and 0 <= rank < n", kMaxRanks);
    if (ring == COMPASS_RING_ALLTOALL) {
        if (pattern != COMPASS_AG_GEMM) return set_error(COMPASS_ERR_UNSUPPORTED, "the AlltoAll pattern is AllGather only");
        if (n % 2) return set_error(COMPASS_ERR_INVALID, "the AlltoAll pattern needs an even n");
    }
    if (M < 1) return set_error(COMPASS_ERR_INVALID, "M, N, K must be positive");
    const bool dbl = ring == COMPASS_RING_DOUBLE || ring == COMPASS_RING_DOUBLE_SPLIT;
    const int BP = dbl ? 2 * n : n;
    if (l->sub_chunks < 0) return set_error(COMPASS_ERR_INVALID, "sub_chunks < 0");
    const int sub = l->sub_chunks > 1 ? l->sub_chunks : 1;
    if (sub > 1) {
        if (l->hop_Bps || ring == COMPASS_RING_ALLTOALL)
            return set_error(COMPASS_ERR_UNSUPPORTED, "sub-chunk flags need the single or double ring with uniform hops");
        if ((long)BP * sub > 2 * kMaxRanks)
            return set_error(COMPASS_ERR_UNSUPPORTED, "partitions x sub-chunks above %d", 2 * kMaxRanks);
    }
    if (M % BP) return set_error(COMPASS_ERR_INVALID, "M must be divisible by %d", BP);
    g->P = BP * sub;
    g->BP = BP;
    g->sub = sub;
    g->rows = M / n;
    g->prow = M / BP;
    g->dbl = dbl;
    g->fb = 0.5;
    if (ring == COMPASS_RING_DOUBLE_SPLIT && l->fwd_Bps > 0 && l->bwd_Bps > 0)
        g->fb = l->bwd_Bps / (l->fwd_Bps + l->bwd_Bps);
    if (min_part_rows(*g) < 1)
        return set_error(COMPASS_ERR_INVALID, "sub_chunks %d leaves a partition without rows", sub);
    int32_t base[2 * kMaxRanks];
    const int len = schedule_fill(pattern, ring, n, rank, base, 2 * kMaxRanks);
    if (len != BP) return len < 0 ? len : set_error(COMPASS_ERR_INVALID, "schedule failed");
    // each base partition's pieces in row order
    for (int i = 0; i < BP; ++i)
        for (int t = 0; t < sub; ++t) g->sched[i * sub + t] = base[i] * sub + t;
    for (int i = 0; i < g->P; ++i) g->pos[g->sched[i]] = i;
    return COMPASS_OK;
}

// Whether a tile whose rows span `span_rows` rows of A (and of the fp32
// partial, with_p) and 256 columns of W stays within the kernel's 32-bit
// buffer offsets from its base (kTileSpanMax bytes each).
static bool spans_fit(int K, int N, bool with_p, uint64_t span_rows) {
    return span_rows * (uint64_t)K * 2 <= kTileSpanMax && 256ull * (uint64_t)K * 2 <= kTileSpanMax &&
           (!with_p || span_rows * (uint64_t)N * 4 <= kTileSpanMax);
}

static int validate(const compass_problem *p, const compass_links *l, int want_pattern, Geometry *g) {
    if (!p) return set_error(COMPASS_ERR_INVALID, "problem is NULL");
    if (!l) return set_error(COMPASS_ERR_INVALID, "links is NULL");
    if (want_pattern >= 0 && p->pattern != want_pattern) return set_error(COMPASS_ERR_INVALID, "wrong pattern for this call");
    int rc = make_geometry(p->pattern, p->ring, p->n, p->rank, p->M, l, g);
    if (rc != COMPASS_OK) return rc;
    if (p->N < 1 || p->K < 1) return set_error(COMPASS_ERR_INVALID, "M, N, K must be positive");
    if (p->K % 8 || p->N % 8) return set_error(COMPASS_ERR_INVALID, "K and N must be multiples of 8");
    if ((p->M + 127) / 128 > kMaxRowTiles) return set_error(COMPASS_ERR_UNSUPPORTED, "M too large");
    if (!spans_fit(p->K, p->N, p->pattern == COMPASS_GEMM_RS, 256))
        return set_error(COMPASS_ERR_UNSUPPORTED, "K = %d, N = %d: a 256-row tile would span more than 1 GiB of A, W "
                                                  "or the partial", p->K, p->N);
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
    for (double r : {l->fwd_Bps, l->bwd_Bps})
        if (!std::isfinite(r) || (r > 0 && r < 1e8))
            return set_error(COMPASS_ERR_INVALID, "link rates must be <= 0 (unpaced) or at least 1e8 bytes/s");
    if (l->hop_Bps) {
        if (p->ring != COMPASS_RING_SINGLE) return set_error(COMPASS_ERR_UNSUPPORTED, "per-hop rates need the single ring");
        for (int q = 0; q < p->n; ++q)
            if (!std::isfinite(l->hop_Bps[q]) || l->hop_Bps[q] < 1e8)
                return set_error(COMPASS_ERR_INVALID, "hop %d: per-hop rates must be at least 1e8 bytes/s", q);
    }
    return COMPASS_OK;
}

static void init_params(GemmParams &g, uint32_t epoch) {
    std::memset(&g, 0, sizeof g);
    Ctx &c = g_ctx;
    g.flags = &c.hw[kHwFlags];
    g.mirror = c.ctrl + kCtrlMirror;
    g.leader = c.ctrl + kCtrlLeader;
    g.ctrl = c.ctrl;
    g.done_cnt = c.ctrl + kCtrlDone;
    g.cu_slots = c.ctrl + kCtrlCuSlot;
    g.split_cnt = c.ctrl + kCtrlSplit;
    g.split_ws = c.split_ws;
    g.ksplit = 1;
    g.err_word = &c.hw[kHwErr];
    g.spin_limit = c.spin_limit;
    g.epoch = epoch;
}

static int pick_tile(int M, int N, bool gated, int prow = 0, double lam_est = 0.0, bool rs = false) {
    if (g_ctx.tile_override == 1) return kTile256;
    if (g_ctx.tile_override == 2) return kTile128;
    // A plain GEMM takes the larger (faster) tile when it still fills every
    // CU. The fused AllGather needs several tiles per arriving partition; it
    // takes it when a partition spans whole 256-row tiles and the GEMM is at
    // least two waves of 256 x 256 tiles (the tiles of the last arrivals then
    // split K, see set_tail_split): on the GPT-3 AllGather (3 waves, 4 : 1
    // double ring, lambda ~ 1) 1156 us against 1361 us with 128 x 128 tiles,
    // whose main loop runs ~15 % slower per flop.
    // The fused ReduceScatter takes 256 x 256 only when computation dominates
    // (estimated lambda >= 1) over at least two waves: with one workgroup per
    // CU its chunks finish in bursts of a whole wave and the sends of the last
    // burst trail the kernel, which the faster GEMM repays only when the
    // transfer is the smaller part.
    const long t256 = (long)((M + 255) / 256) * ((N + 255) / 256);
    if (gated) {
        const bool whole = prow >= 256 && prow % 256 == 0;
        const long cu = g_ctx.num_cu;
        if (rs) return whole && t256 >= 2 * cu && lam_est >= 1.0 ? kTile256 : kTile128;
        return whole && t256 >= 2 * cu ? kTile256 : kTile128;
    }
    return t256 >= g_ctx.num_cu ? kTile256 : kTile128;
}

// Rough comp/comm ratio of a fused operator, used only to pick its tile: the
// GEMM at 1 PFLOP/s against the slower ring direction's bytes at its rate
// (unpaced: that direction's share of the copy engines at the engine model's
// rate; ReduceScatter incoming gets two thirds of a direction's engines).
static double lambda_estimate(const compass_problem *p, const Geometry &geo, const compass_links *l) {
    const double flops = 2.0 * p->M * (double)p->N * p->K;
    double step = p->pattern == COMPASS_AG_GEMM ? (double)geo.prow * p->K * 2 : (double)geo.prow * p->N * 4;
    const bool dbl = two_rings(p);
    double rate = dbl ? std::fmin(l->fwd_Bps, l->bwd_Bps) : l->fwd_Bps;
    if (l->hop_Bps) {
        rate = l->hop_Bps[0];
        for (int q = 1; q < p->n; ++q) rate = std::fmin(rate, l->hop_Bps[q]);
    }
    if (p->ring == COMPASS_RING_DOUBLE_SPLIT && l->fwd_Bps > 0 && l->bwd_Bps > 0) {
        step *= 2.0;                        // the whole chunk per step ...
        rate = l->fwd_Bps + l->bwd_Bps;     // ... over both rings at once
    }
    if (!(rate > 0)) {
        double e = (double)g_ctx.engines.size() / (dbl ? 2.0 : 1.0);
        if (p->pattern == COMPASS_GEMM_RS) e *= 2.0 / 3.0;
        rate = e * kEngineBps;
    }
    const double t_x = (p->n - 1) * step / rate;
    return t_x > 0 ? (flops / 1e15) / t_x : 1e9;
}

static int set_shape(GemmParams &g, int cfg, int M, int N, int K, const void *A, size_t a_rows, const void *W,
                     void *C, const float *P) {
    g.A = (const uint16_t *)A;
    g.W = (const uint16_t *)W;
    g.C = (uint16_t *)C;
    g.P = P;
    g.M = M; g.N = N; g.K = K;
    g.kslice = K;
    g.lda = K; g.ldw = K; g.ldc = N; g.ldp = N;
    g.a_bytes = (uint64_t)a_rows * (uint64_t)K * 2;
    g.w_bytes = (uint64_t)N * (uint64_t)K * 2;
    g.p_bytes = P ? (uint64_t)a_rows * (uint64_t)N * 4 : 0u;
    g.c_bytes = (uint64_t)a_rows * (uint64_t)N * 2;
    const int bm = tile_rows(cfg), bn = tile_cols(cfg);
    g.tiles_m = (M + bm - 1) / bm;
    g.tiles_n = (N + bn - 1) / bn;
    if (g.tiles_m > kMaxRowTiles) return set_error(COMPASS_ERR_UNSUPPORTED, "M too large for the tile table");
    const int total = g.tiles_m * g.tiles_n;
    const int cap = g_ctx.grid_override > 0 ? g_ctx.grid_override : g_ctx.num_cu * tile_wg_per_cu(cfg);
    g.grid = std::max(1, std::min(total, cap));
    g.nq = g.grid >= kMaxQueues ? kMaxQueues : 1;
    g.q_size = std::max(1, g.grid / g.nq);
    g.group_m = cfg == kTile256 ? 4 : 8;
    for (int t = 0; t < g.tiles_m; ++t) {
        g.rt_order[t] = (uint16_t)t;
        g.rt_lo[t] = 0;
        g.rt_hi[t] = 0;
    }
    return COMPASS_OK;
}

// Split K for a launch with too few tiles to occupy every workgroup slot:
// s slices per tile (at most kMaxSplit, each at least kMinSliceK deep, K
// slices multiples of 64), s * tiles <= slots, so that every slot gets a
// slice and the partials fit the workspace.
static void set_split(GemmParams &g, int cfg) {
    Ctx &c = g_ctx;
    const int tiles = g.tiles_m * g.tiles_n;
    const int slots = g_ctx.grid_override > 0 ? g_ctx.grid_override : c.num_cu * tile_wg_per_cu(cfg);
    if (!(c.sched & kSchedSplitK) || !c.split_ws || tiles > kMaxSplitTiles || 2 * tiles > slots) return;
    // at most 8 slices: the slice that completes a tile reads every partial,
    // and past 8 that costs more than the finer split gains (InterDecom at
    // d = 16 on the QKV shape: 850 us with up to 16 slices, 756 us with 8)
    int sp = std::min(std::min(slots / tiles, 8), std::max(1, g.K / kMinSliceK));
    if (sp < 2) return;
    const size_t tile_bytes = (size_t)tile_rows(cfg) * tile_cols(cfg) * sizeof(float);
    while (sp > 1 && (size_t)tiles * sp * tile_bytes > c.split_ws_bytes) --sp;
    if (sp < 2) return;
    const int kslice = ((g.K + sp - 1) / sp + 63) / 64 * 64;
    sp = (g.K + kslice - 1) / kslice;
    if (sp < 2) return;
    g.ksplit = sp;
    g.kslice = kslice;
    g.grid = std::min(tiles * sp, slots);
    g.nq = g.grid >= kMaxQueues ? kMaxQueues : 1;
    g.q_size = std::max(1, g.grid / g.nq);
}

// Tail split of a fused AllGather with 256 x 256 tiles: a tile runs K / 64
// pipeline stages (~300 us at K = 12288), so the tiles of the partitions
// that land last would keep a few dozen CUs busy long after the last arrival
// while the others idle (GPT-3 AllGather, 4 : 1 ring: 250 us of tail on at
// most 96 of 256 CUs). The row tiles of the ready order's last two groups
// (one partition each) split K into s slices, s = the workgroup slots over a
// group's tiles, at most 4, each at least kTailSliceK deep; the rest of the
// launch runs whole tiles. Only for K >= kTailMinK, where a whole tile's
// latency dwarfs the partial tiles' round trip through the workspace, and
// only when the transfer is not much shorter than the GEMM (estimated
// lambda below kTailMaxLambda): with the data there early the last tiles
// start with the rest, and the slices' round trips are pure cost (GPT-3
// AllGather, 4 : 1 ring: lambda ~ 0.7 split 1474 against 1616 us whole,
// lambda ~ 1 1117 against 1185 us; lambda ~ 2 split 1091 against 1038 us,
// links unpaced 1074 against 1024 us).
static void set_tail_split(GemmParams &g, int cfg, double lam_est) {
    Ctx &c = g_ctx;
    const int min_k = c.tail_min_k[cfg == kTile256 ? 0 : 1];
    if (!(c.sched & kSchedSplitK) || !c.split_ws || g.ksplit > 1 || min_k <= 0 || g.K < min_k) return;
    if (!(lam_est < kTailMaxLambda)) return;
    const int groups = (g.tiles_m + g.group_m - 1) / g.group_m;
    const int tail_groups = c.tail_groups;
    if (groups < 2 * tail_groups || g.tiles_m % g.group_m) return;
    const int tail_tiles = tail_groups * g.group_m * g.tiles_n;
    const int slots = g.grid;
    int sp = std::min(4, std::min(slots / (g.group_m * g.tiles_n), g.K / c.tail_slice_k));
    const size_t tile_bytes = (size_t)tile_rows(cfg) * tile_cols(cfg) * sizeof(float);
    while (sp > 1 && (size_t)tail_tiles * sp * tile_bytes > c.split_ws_bytes) --sp;
    if (sp < 2 || tail_tiles > kMaxSplitTiles) return;
    g.ksplit = sp;
    g.kslice = ((g.K + sp - 1) / sp + 63) / 64 * 64;
    g.split_from = (groups - tail_groups) * g.group_m * g.tiles_n;
}

// Head split of a fused AllGather (the tail split's gates: 256 x 256 tiles
// from K = kTailMinK, estimated lambda below kTailMaxLambda): until the
// first remote partition lands only the resident partitions' tiles can run,
// one per workgroup, and the other workgroups wait at their gates (GPT-3
// AllGather, 4 : 1 ring: 96 tiles on 256 CUs for 65-135 us). The leading
// row-tile groups of the ready order whose partitions are all resident
// split K into s = min(4, slots / their tiles) slices, each at least
// tail_slice_k deep, so that their work is spread over more workgroups and
// done sooner; the workspace holds both the head's and the tail's partials.
static void set_head_split(GemmParams &g, int cfg, double lam_est, uint64_t resident) {
    Ctx &c = g_ctx;
    const int min_k = c.tail_min_k[cfg == kTile256 ? 0 : 1];
    if (!c.head_split || !(c.sched & kSchedSplitK) || !c.split_ws || min_k <= 0 || g.K < min_k) return;
    if (!(lam_est < kTailMaxLambda) || !resident) return;
    int rt = 0;   // leading row tiles of the ready order with every partition resident
    while (rt < g.tiles_m) {
        const int t = g.rt_order[rt];
        const uint64_t lo = g.rt_lo[t], hi = g.rt_hi[t];
        const uint64_t touch = (hi >= 63 ? ~0ull : ((2ull << hi) - 1ull)) & ~((1ull << lo) - 1ull);
        if (touch & ~resident) break;
        ++rt;
    }
    rt -= rt % g.group_m;   // positions walk whole row-tile groups
    const int head = rt * g.tiles_n;
    if (head == 0 || 2 * head > g.grid) return;
    if (g.ksplit > 1 && g.split_from < head) return;
    int sh = std::min(4, std::min(g.grid / head, g.K / c.tail_slice_k));
    const size_t tile_bytes = (size_t)tile_rows(cfg) * tile_cols(cfg) * sizeof(float);
    const int tiles = g.tiles_m * g.tiles_n;
    const size_t tail_ws = g.ksplit > 1 ? (size_t)(tiles - g.split_from) * g.ksplit : 0;
    const int tail_cnt = g.ksplit > 1 ? tiles - g.split_from : 0;
    while (sh > 1 && ((size_t)head * sh + tail_ws) * tile_bytes > c.split_ws_bytes) --sh;
    if (sh < 2 || head + tail_cnt > kMaxSplitTiles) return;
    g.head_tiles = head;
    g.head_split = sh;
    g.head_kslice = ((g.K + sh - 1) / sh + 63) / 64 * 64;
}

static void touch_all(GemmParams &g, int nparts) {
    for (int t = 0; t < g.tiles_m; ++t) {
        g.rt_lo[t] = 0;
        g.rt_hi[t] = (uint8_t)(nparts - 1);
    }
}

// Row tiles ordered by when the last partition they touch is expected to
// land (ties: its schedule position); touched partitions from the identity
// row map. `arrive[q]` is that expectation for partition q (the schedule
// position itself when the links give no better one).
static void order_by_arrival(GemmParams &g, int cfg, const Geometry &geo, int M, bool main_gate,
                             const double *arrive) {
    const int bm = tile_rows(cfg);
    struct Key { double t; int pos, tile; };
    std::vector<Key> key;
    for (int t = 0; t < g.tiles_m; ++t) {
        const int r0 = t * bm, r1 = std::min(M, r0 + bm) - 1;
        const int p0 = part_of_row(geo, r0), p1 = part_of_row(geo, r1);
        Key k{0.0, 0, t};
        for (int q = p0; q <= p1; ++q) {
            k.t = std::max(k.t, arrive[q]);
            k.pos = std::max(k.pos, geo.pos[q]);
        }
        g.rt_lo[t] = (uint8_t)p0;
        g.rt_hi[t] = (uint8_t)p1;
        key.push_back(k);
    }
    std::stable_sort(key.begin(), key.end(),
                     [](const Key &a, const Key &b) { return a.t < b.t || (a.t == b.t && a.pos < b.pos); });
    for (int i = 0; i < g.tiles_m; ++i) g.rt_order[i] = (uint16_t)key[i].tile;
    // AllGather: the tiles of one arriving partition are consecutive in the
    // ready order and cannot start before it lands. Short super-blocks deal
    // them out over all XCD queues, and the second workgroup of each CU
    // waits for the first tickets to go one per CU. (ReduceScatter tiles
    // compute before they wait, so they keep the long super-blocks that let
    // each XCD's L2 reuse its rows of A and W.)
    if (!main_gate) return;
    if (g_ctx.sched & kSchedFineQueues) g.q_size = std::max(1, g.group_m);
    if ((g_ctx.sched & kSchedSpread) && g.nq == kMaxQueues && g.grid == g_ctx.num_cu * tile_wg_per_cu(cfg) &&
        tile_wg_per_cu(cfg) > 1)
        g.spread_wait = g_ctx.num_cu / kMaxQueues;
}

static inline uint64_t touched(const GemmParams &g, int t) {
    const int lo = g.rt_lo[t], hi = g.rt_hi[t];
    const uint64_t upto = hi >= 63 ? ~0ull : ((2ull << hi) - 1ull);
    return upto & ~((1ull << lo) - 1ull);
}

static hipError_t copy_if_needed(void *dst, const void *src, size_t bytes, hipStream_t s) {
    if (dst == src) return hipSuccess;
    return hipMemcpyAsync(dst, src, bytes, hipMemcpyDefault, s);
}

// Partition q's rows (identity map): base partition b = q / sub; chunk
// c = b (single ring) or b / 2 (double ring).
static inline int part_chunk(const Geometry &g, int q) { return g.dbl ? q / g.sub / 2 : q / g.sub; }
static inline int part_half(const Geometry &g, int q) { return g.dbl ? (q / g.sub) % 2 : 0; }
static inline bool part_fwd(const Geometry &g, int q) { return !g.dbl || (q / g.sub) % 2 == 1; }
// Rows [*off, *off + *cnt) of a block of r chunk rows that partition q carries.
static inline void part_rows(const Geometry &g, int r, int q, int *off, int *cnt) {
    int bo, bc;
    base_rows(g, r, part_half(g, q), &bo, &bc);
    const int t = q % g.sub;
    const int lo = piece_lo(bc, t, g.sub), hi = piece_lo(bc, t + 1, g.sub);
    *off = bo + lo;
    *cnt = hi - lo;
}

int op_partition_layout(int pattern, int ring, int n, int rank, int M, const compass_links *l, int32_t *order,
                        int32_t *row0, int32_t *rows, int cap) {
    if (!l || !order || !row0 || !rows) return set_error(COMPASS_ERR_INVALID, "partition_layout: NULL argument");
    Geometry g;
    const int rc = make_geometry(pattern, ring, n, rank, M, l, &g);
    if (rc != COMPASS_OK) return rc;
    if (cap < g.P) return set_error(COMPASS_ERR_INVALID, "partition_layout: cap below %d", g.P);
    for (int q = 0; q < g.P; ++q) {
        order[q] = g.sched[q];
        int off, cnt;
        part_rows(g, g.rows, q, &off, &cnt);
        row0[q] = part_chunk(g, q) * g.rows + off;
        rows[q] = cnt;
    }
    return g.P;
}

// A copy of `bytes` from src to dst; both ranges must lie inside the
// allocations that hold their first bytes (so that a buffer smaller than
// the problem says is refused before a copy engine writes past it).
static int make_item(Item *it, void *dst, const void *src, size_t bytes, int flag, int gate) {
    int rc;
    uintptr_t dst_end = 0, src_end = 0;
    if ((rc = agent_of(dst, &it->dst_agent, &dst_end)) != COMPASS_OK) return rc;
    if ((rc = agent_of(src, &it->src_agent, &src_end)) != COMPASS_OK) return rc;
    if ((uintptr_t)dst + bytes > dst_end || (uintptr_t)src + bytes > src_end)
        return set_error(COMPASS_ERR_INVALID, "a copy of %zu bytes from %p to %p runs past the end of its allocation",
                         bytes, src, dst);
    it->dst = dst;
    it->src = src;
    it->bytes = bytes;
    it->flag = flag;
    it->gate = gate;
    return COMPASS_OK;
}

static void fill_job(Job &j, const compass_links *l, bool fwd, uint32_t epoch, int role, const std::vector<int> &active,
                     const std::vector<double> &weight, bool paired) {
    j.rate = fwd ? l->fwd_Bps : l->bwd_Bps;
    j.slice = l->slice_bytes ? l->slice_bytes : kDefaultSlice;
    j.slice_default = l->slice_bytes == 0;
    j.epoch = epoch;
    j.engines = engines_for(role, active, weight, l->engines_per_ring, paired);
}

// Per-hop rates: the due times of the d * (n - 1) items this rank receives
// (sub-collective-major) for pieces of `piece_bytes`; empty without hop rates.
static int hop_arrivals(const compass_problem *p, const compass_links *l, int d, double piece_bytes,
                        std::vector<double> *out) {
    out->clear();
    if (!l->hop_Bps || p->n < 2) return COMPASS_OK;
    out->resize((size_t)d * (p->n - 1));
    const int k = ring_arrivals(p->n, p->rank, piece_bytes, l->hop_Bps, d, out->data(), (int)out->size());
    return k < 0 ? k : COMPASS_OK;
}

// Expected arrival of every partition of a fused operator (seconds after
// its start; resident partitions at 0), used only to order the tiles. Each
// ring direction delivers its partitions one after another in schedule
// order, a partition taking its bytes over the direction's rate; unpaced or
// half-paced links count as equal rates, so that the order falls back to
// the schedule's. Per-hop rates take the store-and-forward arrival times;
// the AlltoAll pattern keeps the schedule order.
static int expected_arrivals(const compass_problem *p, const Geometry &geo, const compass_links *l, uint64_t resident,
                             double *t) {
    for (int q = 0; q < geo.P; ++q) t[q] = (double)geo.pos[q];
    if (p->ring == COMPASS_RING_ALLTOALL) return COMPASS_OK;
    const double row_bytes = p->pattern == COMPASS_AG_GEMM ? 2.0 * p->K : 4.0 * p->N;
    if (l->hop_Bps) {
        std::vector<double> due;
        const int rc = hop_arrivals(p, l, 1, (double)geo.rows * row_bytes, &due);
        if (rc != COMPASS_OK) return rc;
        for (int s = 0; s < geo.P; ++s) {
            const int q = geo.sched[s];
            t[q] = (resident >> q) & 1ull ? 0.0 : due[(size_t)std::min(std::max(s, 1), geo.P - 1) - 1];
        }
        return COMPASS_OK;
    }
    const bool rated = l->fwd_Bps > 0 && (!geo.dbl || l->bwd_Bps > 0);
    double clock[2] = {0.0, 0.0};
    for (int s = 0; s < geo.P; ++s) {
        const int q = geo.sched[s];
        if ((resident >> q) & 1ull) {
            t[q] = 0.0;
            continue;
        }
        int off, cnt;
        part_rows(geo, geo.rows, q, &off, &cnt);
        const bool fwd = part_fwd(geo, q);
        const double rate = rated ? (fwd ? l->fwd_Bps : l->bwd_Bps) : 1.0;
        clock[fwd ? 0 : 1] += (double)cnt * row_bytes / rate;
        t[q] = clock[fwd ? 0 : 1];
    }
    return COMPASS_OK;
}

// ---------------------------------------------------------------- AllGather jobs
// Items: the remote partitions in schedule order (the local ones are already
// in place); forward-ring partitions go to role 0, backward-ring to role 1.
// `d` > 1: InterDecom sub-gathers, piece j of every remote partition, j-major,
// with flags j * P + partition.
static int ag_jobs(const compass_problem *p, const Geometry &geo, const compass_links *l, uint32_t epoch, int d,
                   bool wait_start, Job *fwd, Job *bwd) {
    const bool a2a = p->ring == COMPASS_RING_ALLTOALL;
    const int dom = std::max(1, p->n / 2);                          // AlltoAll: ranks per NUMA domain
    const std::vector<int> active = p->ring == COMPASS_RING_SINGLE ? std::vector<int>{0} : std::vector<int>{0, 1};
    // AlltoAll: role 0 carries the dom - 1 chunks of this rank's domain, role 1
    // the dom chunks of the other domain
    const std::vector<int> bytes = a2a ? std::vector<int>{std::max(1, dom - 1), dom} : std::vector<int>(active.size(), 1);
    std::vector<double> weight;
    const bool paired = !a2a && direction_weights(active, bytes, l, &weight);
    if (a2a) weight.assign(bytes.begin(), bytes.end());
    fill_job(*fwd, l, true, epoch, 0, active, weight, paired);
    fill_job(*bwd, l, false, epoch, 1, active, weight, paired);
    fwd->wait_start = bwd->wait_start = wait_start;
    if (a2a) {
        // every flow at once; the dom * dom flows into this domain share the
        // cross-domain link equally
        fwd->concurrent = bwd->concurrent = true;
        if (bwd->rate > 0) bwd->rate /= (double)dom * dom;
    }
    const size_t K = (size_t)p->K;
    const int pc = geo.rows / d;                                     // chunk rows per sub-operator
    std::vector<double> due;
    int rc0 = hop_arrivals(p, l, d, (double)pc * K * 2, &due);
    if (rc0 != COMPASS_OK) return rc0;
    if (!due.empty()) fwd->rate = l->hop_Bps[(p->rank + p->n - 1) % p->n];   // the hop into this rank
    for (int j = 0; j < d; ++j) {
        for (int s = 0; s < geo.P; ++s) {
            const int q = geo.sched[s];
            const int c = part_chunk(geo, q);
            if (c == p->rank) continue;
            if (q == g_ctx.drop_flag && d == 1) continue;
            int off, piece;                                          // rows of this item
            part_rows(geo, pc, q, &off, &piece);
            const size_t row_in_chunk = (size_t)j * pc + (size_t)off;
            const size_t row = (size_t)c * geo.rows + row_in_chunk;
            Item it;
            const int rc = make_item(&it, (char *)p->gathered + row * K * 2,
                                     (const char *)p->shard_src[c] + row_in_chunk * K * 2, (size_t)piece * K * 2,
                                     j * geo.P + q, -1);
            if (rc != COMPASS_OK) return rc;
            if (!due.empty()) it.due_at = due[(size_t)j * (p->n - 1) + (s - 1)];   // single ring: step s
            it.seq = j * geo.P + s;
            const bool on_fwd = a2a ? (c / dom == p->rank / dom) : part_fwd(geo, q);
            (on_fwd ? fwd : bwd)->items.push_back(it);
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
    // incoming fp32 partials carry twice the bytes of the outgoing bf16 sums
    std::vector<int> active{0}, bytes{2};
    const bool dbl = two_rings(p);
    if (dbl) { active.push_back(1); bytes.push_back(2); }
    if (p->send_dst) {
        active.push_back(2); bytes.push_back(1);
        if (dbl) { active.push_back(3); bytes.push_back(1); }
    }
    std::vector<double> weight;
    const bool paired = direction_weights(active, bytes, l, &weight);
    for (int r = 0; r < 4; ++r) {
        fill_job(jobs[r], l, r % 2 == 0, epoch, r, active, weight, paired);
        jobs[r].wait_start = wait_start;
    }
    const size_t N = (size_t)p->N;
    const int pc = geo.rows / d;
    std::vector<double> due;
    int rc0 = hop_arrivals(p, l, d, (double)pc * N * 4, &due);
    if (rc0 != COMPASS_OK) return rc0;
    if (!due.empty()) {
        jobs[0].rate = l->hop_Bps[(p->rank + p->n - 1) % p->n];   // the hop into this rank ...
        jobs[2].rate = l->hop_Bps[p->rank];                       // ... and out of it
    }
    for (int j = 0; j < d; ++j) {
        for (int s = 0; s < geo.P; ++s) {
            const int q = geo.sched[s];
            if (resident & (1ull << q)) continue;
            const int c = part_chunk(geo, q);
            int off, piece;
            part_rows(geo, pc, q, &off, &piece);
            const size_t row_in_chunk = (size_t)j * pc + (size_t)off;
            const size_t row = (size_t)c * geo.rows + row_in_chunk;
            Item it;
            const int rc = make_item(&it, (char *)p->partial_stage + row * N * 4,
                                     (const char *)p->partial_src[c] + row_in_chunk * N * 4, (size_t)piece * N * 4,
                                     j * geo.P + q, -1);
            if (rc != COMPASS_OK) return rc;
            if (!due.empty()) it.due_at = due[(size_t)j * (p->n - 1) + (s - 1)];   // single ring: step s >= 1
            it.seq = 2 * (j * geo.P + s) + 1;
            jobs[part_fwd(geo, q) ? 0 : 1].items.push_back(it);
        }
        if (!p->send_dst) continue;
        for (int s = 0; s < geo.P; ++s) {
            const int q = geo.sched[s];
            const int c = part_chunk(geo, q);
            if (c == p->rank) continue;
            int off, piece;
            part_rows(geo, pc, q, &off, &piece);
            const size_t row_in_chunk = (size_t)j * pc + (size_t)off;
            const size_t row = (size_t)c * geo.rows + row_in_chunk;
            Item it;
            const int rc = make_item(&it, (char *)p->send_dst[c] + row_in_chunk * N * 2,
                                     (const char *)p->C + row * N * 2, (size_t)piece * N * 2, -1,
                                     gate_out ? j * geo.P + q : -1);
            if (rc != COMPASS_OK) return rc;
            it.seq = 2 * (j * geo.P + s) + 2;   // right after its partition's incoming partial
            jobs[part_fwd(geo, q) ? 2 : 3].items.push_back(it);
        }
    }
    for (int r = 2; r < 4; ++r)
        if (!jobs[r].items.empty()) jobs[r].final_flag = kFinalFlag0 + r;
    return COMPASS_OK;
}

// The directions of an operator share every copy engine when all of its
// copies stay in device memory (COMPASS_OPT_POOL > 0): their items merge, in
// the operator's transfer order, into the first such job, which runs pooled
// on its role's thread (earliest due slice first); the other jobs are left
// empty. This covers paced links (with one direction too: its items then no
// longer wait for engine groups), per-hop due times and unpaced operators
// with more than one active direction. The AlltoAll pattern (flows sharing
// a link, each paced on its own) keeps a job per direction, and so do copies
// to or from host memory: across PCIe the link, not the engines, is the
// limit, a copy takes milliseconds, and a pooled engine's queue would hold
// an outgoing sum behind incoming partials that a direction of its own
// sends past (the fc2 ReduceScatter with pinned-host remote buffers: fused
// 3.03 ms pooled against the unfused 2.53 ms).
static void pool_jobs(Job *jobs, int count) {
    Ctx &c = g_ctx;
    if (c.pool_depth <= 0) return;
    int first = -1, active = 0;
    bool paced = false;
    for (int r = 0; r < count; ++r) {
        if (jobs[r].items.empty()) continue;
        if (jobs[r].concurrent) return;
        for (const Item &it : jobs[r].items)
            if (it.src_agent.handle != c.gpu.handle || it.dst_agent.handle != c.gpu.handle) return;
        paced |= jobs[r].rate > 0;
        for (const Item &it : jobs[r].items) paced |= it.due_at >= 0;
        if (first < 0) first = r;
        ++active;
    }
    if (active < 1 || (!paced && active < 2)) return;
    Job &m = jobs[first];
    for (int r = 0; r < count; ++r) {
        for (Item &it : jobs[r].items) {
            it.link = r;
            it.rate = jobs[r].rate;
            it.slice = !jobs[r].slice_default ? jobs[r].slice : paced ? kDefaultSlice : kPoolSlice;
        }
        if (r == first) continue;
        for (Item &it : jobs[r].items) m.items.push_back(it);
        jobs[r].items.clear();
        if (jobs[r].final_flag >= 0) {
            if (m.final_flag < 0) m.final_flag = jobs[r].final_flag;
            else m.more_finals.push_back(jobs[r].final_flag);
            jobs[r].final_flag = -1;
        }
    }
    std::stable_sort(m.items.begin(), m.items.end(), [](const Item &a, const Item &b) { return a.seq < b.seq; });
    m.engines = engines_for(first, std::vector<int>{first}, std::vector<double>{1.0}, 0);
    m.pool_depth = c.pool_depth;
}

// Partitions in place before the operator starts: the rank's own chunk
// (AllGather), or the first step's partials (ReduceScatter), all their pieces.
static uint64_t resident_mask(const compass_problem *p, const Geometry &geo) {
    uint64_t base = 0;
    if (p->pattern == COMPASS_AG_GEMM)
        base = geo.dbl ? 3ull << (2 * p->rank) : 1ull << p->rank;
    else
        base = geo.dbl ? (1ull << (geo.sched[0] / geo.sub)) | (1ull << (geo.sched[geo.sub] / geo.sub))
                       : 1ull << (geo.sched[0] / geo.sub);
    uint64_t m = 0;
    for (int q = 0; q < geo.P; ++q)
        if (base & (1ull << (q / geo.sub))) m |= 1ull << q;
    return m;
}

static uint64_t nonlocal_mask(const compass_problem *p, const Geometry &geo) {
    uint64_t m = 0;
    for (int q = 0; q < geo.P; ++q)
        if (part_chunk(geo, q) != p->rank) m |= 1ull << q;
    return m;
}

static int stage_local_shard(const compass_problem *p, const Geometry &geo, hipStream_t s) {
    const size_t K = (size_t)p->K;
    void *dst = (char *)p->gathered + (size_t)p->rank * geo.rows * K * 2;
    const hipError_t e = copy_if_needed(dst, p->shard_src[p->rank], (size_t)geo.rows * K * 2, s);
    return e == hipSuccess ? COMPASS_OK : hip_fail(e, "local shard copy");
}

// The first step's partials (the resident partitions) read by the kernel
// straight from the caller's buffers, with no staging copy: per chunk, the
// rows its resident partitions cover, contiguous in the chunk, become an
// aliased row range of the landing buffer (GemmParams::palt) whose partial
// the epilogue reads from partial_src[c]. Needs device memory 16-byte
// aligned, the identity row map, range ends on tile boundaries (no tile
// reads two buffers) and at most two ranges; *aliased false otherwise, and
// the caller stages them.
static int alias_resident_partials(GemmParams &g, const compass_problem *p, const Geometry &geo, uint64_t resident,
                                   int cfg, bool *aliased) {
    *aliased = false;
    if (g.piece != 0) return COMPASS_OK;
    const int bm = tile_rows(cfg);
    int lo[2], hi[2], chunk[2], k = 0;
    for (int c = 0; c < p->n; ++c) {
        int a = geo.rows, b = -1, rows = 0;
        for (int q = 0; q < geo.P; ++q) {
            if (!((resident >> q) & 1ull) || part_chunk(geo, q) != c) continue;
            int off, cnt;
            part_rows(geo, geo.rows, q, &off, &cnt);
            a = std::min(a, off);
            b = std::max(b, off + cnt);
            rows += cnt;
        }
        if (b < 0) continue;
        const int plo = c * geo.rows + a, phi = c * geo.rows + b;
        if (k == 2 || rows != b - a || plo % bm || (phi % bm && phi != p->M)) return COMPASS_OK;
        // (the epilogue reads the partial 16 bytes at a time)
        if ((uintptr_t)p->partial_src[c] % 16) return COMPASS_OK;
        hsa_agent_t owner;
        const int rc = agent_of(p->partial_src[c], &owner);
        if (rc != COMPASS_OK) return rc;
        if (owner.handle != g_ctx.gpu.handle) return COMPASS_OK;
        lo[k] = plo;
        hi[k] = phi;
        chunk[k] = c;
        ++k;
    }
    for (int i = 0; i < k; ++i) {
        g.palt[i] = (const float *)((const char *)p->partial_src[chunk[i]] + (size_t)(lo[i] - chunk[i] * geo.rows) *
                                                                               (size_t)p->N * 4);
        g.palt_lo[i] = lo[i];
        g.palt_hi[i] = hi[i];
    }
    *aliased = true;
    return COMPASS_OK;
}

// The partials of the resident partitions, for each of the d sub-operators
// the rows its piece of the partition covers (rs_jobs moves the others).
static int stage_resident_partials(const compass_problem *p, const Geometry &geo, uint64_t resident, int d,
                                   hipStream_t s) {
    const size_t N = (size_t)p->N;
    const int pc = geo.rows / d;
    for (int q = 0; q < geo.P; ++q) {
        if (!(resident & (1ull << q))) continue;
        const int c = part_chunk(geo, q);
        int off, cnt;
        part_rows(geo, pc, q, &off, &cnt);
        for (int j = 0; j < d; ++j) {
            const size_t row_in_chunk = (size_t)j * pc + (size_t)off;
            void *dst = (char *)p->partial_stage + ((size_t)c * geo.rows + row_in_chunk) * N * 4;
            const void *src = (const char *)p->partial_src[c] + row_in_chunk * N * 4;
            const hipError_t e = copy_if_needed(dst, src, (size_t)cnt * N * 4, s);
            if (e != hipSuccess) return hip_fail(e, "resident partial copy");
        }
    }
    return COMPASS_OK;
}

static int launch(const GemmParams &g0, int cfg, bool rs, hipStream_t s) {
    Ctx &c = g_ctx;
    GemmParams g = g0;
    if (++c.launch_seq == 0) c.launch_seq = 1;
    g.launch_seq = c.launch_seq;
    if (c.tile_trace) {
        g.tile_trace = c.tile_trace;
        g.trace_base = c.trace_used;
        g.trace_cap = c.trace_cap;
        const uint64_t work = (uint64_t)work_items(g0);
        c.trace_used = std::min<uint64_t>(c.trace_cap, (uint64_t)c.trace_used + work);
    }
    const bool timed = c.timing && c.timed_count < Ctx::kTimed;
    if (timed) (void)hipEventRecord(c.ev_begin[c.timed_count], s);
    const hipError_t e = launch_gemm(g, cfg, rs, s);
    if (e != hipSuccess) return hip_fail(e, "GEMM launch");
    if (timed) (void)hipEventRecord(c.ev_end[c.timed_count++], s);
    return COMPASS_OK;
}

int op_kernel_times(double *us, int cap) {
    Ctx &c = g_ctx;
    if (!c.ready || !c.timing) return set_error(COMPASS_ERR_INVALID, "kernel timing is not enabled");
    if (cap < 0 || (cap > 0 && !us)) return set_error(COMPASS_ERR_INVALID, "bad output buffer");
    const int n = std::min(cap, c.timed_count);
    for (int i = 0; i < n; ++i) {
        float ms = 0.f;
        hipError_t e = hipEventSynchronize(c.ev_end[i]);
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, c.ev_begin[i], c.ev_end[i]);
        if (e != hipSuccess) return hip_fail(e, "kernel event");
        us[i] = (double)ms * 1e3;
    }
    c.timed_count = 0;
    return n;
}

int op_tile_trace(uint32_t *out, int cap) {
    Ctx &c = g_ctx;
    if (!c.ready || !c.tile_trace) return set_error(COMPASS_ERR_INVALID, "tile trace is not enabled");
    if (cap < 0 || (cap > 0 && !out)) return set_error(COMPASS_ERR_INVALID, "bad output buffer");
    const int n = (int)std::min<uint32_t>((uint32_t)cap, c.trace_used);
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess && n > 0)
        e = hipMemcpy(out, c.tile_trace, (size_t)n * kTraceWords * sizeof(uint32_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "tile trace read");
    c.trace_used = 0;
    return n;
}

static int join(uint32_t epoch, const std::vector<int> &flags, bool write_start, hipStream_t s) {
    JoinParams j;
    std::memset(&j, 0, sizeof j);
    Ctx &c = g_ctx;
    j.flags = &c.hw[kHwFlags];
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
    // allocations seen by an earlier call may have been freed and their
    // addresses reused by others (of another size or owner) since
    g_ctx.ranges.clear();
    return take_async_error();
}

int op_probe_mfma(int iters, double *tflops, double *sclk_ghz) {
    if (iters < 1 || iters > (1 << 22)) return set_error(COMPASS_ERR_INVALID, "iters out of range [1, 2^22]");
    if (!tflops || !sclk_ghz) return set_error(COMPASS_ERR_INVALID, "null output pointer");
    int rc = begin();
    if (rc != COMPASS_OK) return rc;
    Ctx &c = g_ctx;
    const int grid = c.num_cu;
    const size_t waves = (size_t)grid * (kProbeThreads / 64);
    hipError_t e = hipSuccess;
    if (!c.probe_out) e = hipMalloc((void **)&c.probe_out, waves * 3 * sizeof(uint64_t));
    if (e != hipSuccess) return hip_fail(e, "probe buffer");
    hipEvent_t a = nullptr, b = nullptr;
    e = hipEventCreate(&a);
    if (e == hipSuccess) e = hipEventCreate(&b);
    if (e == hipSuccess) e = hipEventRecord(a, nullptr);
    if (e == hipSuccess) e = launch_mfma_probe(c.probe_out, grid, iters, nullptr);
    if (e == hipSuccess) e = hipEventRecord(b, nullptr);
    if (e == hipSuccess) e = hipEventSynchronize(b);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
    std::vector<uint64_t> h(waves * 3);
    if (e == hipSuccess) e = hipMemcpy(h.data(), c.probe_out, h.size() * sizeof(uint64_t), hipMemcpyDeviceToHost);
    if (a) (void)hipEventDestroy(a);
    if (b) (void)hipEventDestroy(b);
    if (e != hipSuccess) return hip_fail(e, "matrix-core probe");
    double cyc = 0.0, rt = 0.0;
    for (size_t w = 0; w < waves; ++w) {
        cyc += (double)h[3 * w];
        rt += (double)h[3 * w + 1];
    }
    if (!(rt > 0.0) || !(ms > 0.f)) return set_error(COMPASS_ERR_HIP, "matrix-core probe recorded no time");
    const double flops = 2.0 * 32 * 32 * 16 * 8.0 * (double)iters * (double)waves;
    *tflops = flops / ((double)ms * 1e-3) / 1e12;
    *sclk_ghz = cyc / rt * 0.1;   // real-time counter ticks at 100 MHz
    return COMPASS_OK;
}

// ---------------------------------------------------------------- operators
int op_ag_gemm(const compass_problem *p, const compass_links *l, void *stream) {
    Geometry geo;
    int rc = validate(p, l, COMPASS_AG_GEMM, &geo);
    if (rc != COMPASS_OK) return rc;
    if ((rc = begin()) != COMPASS_OK) return rc;
    hipStream_t s = (hipStream_t)stream;
    const uint32_t epoch = next_epoch();
    Job ag[2];
    if ((rc = ag_jobs(p, geo, l, epoch, 1, true, &ag[0], &ag[1])) != COMPASS_OK) return rc;
    pool_jobs(ag, 2);
    if ((rc = stage_local_shard(p, geo, s)) != COMPASS_OK) return rc;
    GemmParams g;
    init_params(g, epoch);
    // (rate-proportional parts: a 256-row tile may span both parts of a
    // chunk and waits for the later one, which an AllGather tolerates)
    const double lam = lambda_estimate(p, geo, l);
    const int cfg = pick_tile(p->M, p->N, true, geo.fb != 0.5 && geo.sub == 1 ? geo.rows : min_part_rows(geo), lam);
    if ((rc = set_shape(g, cfg, p->M, p->N, p->K, p->gathered, p->M, p->W, p->C, nullptr)) != COMPASS_OK) return rc;
    // 256-row tiles: one row-tile group per partition, so that the dealing
    // and the tail split follow partitions
    if (cfg == kTile256 && geo.sub == 1 && geo.fb == 0.5 && min_part_rows(geo) % 256 == 0)
        g.group_m = std::max(1, std::min(4, min_part_rows(geo) / 256));
    double arrive[2 * kMaxRanks];
    if ((rc = expected_arrivals(p, geo, l, resident_mask(p, geo), arrive)) != COMPASS_OK) return rc;
    order_by_arrival(g, cfg, geo, p->M, true, arrive);
    set_tail_split(g, cfg, lam);
    set_head_split(g, cfg, lam, resident_mask(p, geo));
    g.gate = kGateMain;
    g.nparts = geo.P;
    g.resident_mask = resident_mask(p, geo);
    g.start_word = &g_ctx.hw[kHwStart];
    submit(0, std::move(ag[0]));
    submit(1, std::move(ag[1]));
    return launch(g, cfg, false, s);
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
    GemmParams g;
    init_params(g, epoch);
    const int cfg = pick_tile(p->M, p->N, true, min_part_rows(geo), lambda_estimate(p, geo, l), true);
    if ((rc = set_shape(g, cfg, p->M, p->N, p->K, p->A, p->M, p->W, p->C, p->partial_stage)) != COMPASS_OK) return rc;
    bool aliased = false;
    if ((rc = alias_resident_partials(g, p, geo, res, cfg, &aliased)) != COMPASS_OK) return rc;
    if (!aliased && (rc = stage_resident_partials(p, geo, res, 1, s)) != COMPASS_OK) return rc;
    // ReduceScatter tiles compute before their partial is needed, so they
    // run in ring-step order (a step's partitions on both rings together),
    // not in arrival order: under a 4 : 1 ring the faster ring's partials
    // land early, and taking their tiles first left the slower ring's last
    // partitions computing long after their partials landed, their sends
    // then queued one after another on the slow link (GPT-3 ReduceScatter:
    // 220 us after the kernel)
    double arrive[2 * kMaxRanks];
    for (int q = 0; q < geo.P; ++q) arrive[q] = (double)geo.pos[q];
    order_by_arrival(g, cfg, geo, p->M, false, arrive);
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
                if (touched(g, t) & (1ull << q)) cnt += g.tiles_n;
            g.done_expect[q] = cnt;
        }
        for (int r = 2; r < 4; ++r)
            if (jobs[r].final_flag >= 0) finals.push_back(jobs[r].final_flag);
    }
    pool_jobs(jobs, 4);
    for (int r = 0; r < 4; ++r) submit(r, std::move(jobs[r]));
    if ((rc = launch(g, cfg, true, s)) != COMPASS_OK) return rc;
    if (!finals.empty()) return join(epoch, finals, false, s);
    return COMPASS_OK;
}

int op_decomp(const compass_problem *p, int d, const compass_links *l, void *stream) {
    Geometry geo;
    int rc = validate(p, l, -1, &geo);
    if (rc != COMPASS_OK) return rc;
    if (d < 1 || (d & (d - 1)) || geo.prow % d)
        return set_error(COMPASS_ERR_INVALID, "d must be a power of two dividing %d", geo.prow);
    if (d > 1 && p->ring == COMPASS_RING_ALLTOALL)
        return set_error(COMPASS_ERR_UNSUPPORTED, "InterDecom runs over the rings only");
    if (d > 1 && geo.sub > 1)
        return set_error(COMPASS_ERR_UNSUPPORTED, "InterDecom takes one flag per piece (sub_chunks <= 1)");
    if (d * geo.P > kFinalFlag0) return set_error(COMPASS_ERR_UNSUPPORTED, "d * partitions exceeds the flag slots");
    if (d > 1) {
        // a sub-GEMM's tile of 256 logical rows covers up to 255 / piece + 1
        // row pieces, each a chunk's rows apart in A and the partial
        const uint64_t piece = (uint64_t)(geo.rows / d);
        const uint64_t span = (255 / piece + 1) * (uint64_t)geo.rows;
        if (!spans_fit(p->K, p->N, p->pattern == COMPASS_GEMM_RS, span))
            return set_error(COMPASS_ERR_UNSUPPORTED, "d = %d: a sub-GEMM tile would span more than 1 GiB of A or the "
                                                      "partial", d);
    }
    if ((rc = begin()) != COMPASS_OK) return rc;
    hipStream_t s = (hipStream_t)stream;
    const uint32_t epoch = next_epoch();
    const uint64_t res = resident_mask(p, geo);
    const int piece = geo.rows / d;   // rows of a chunk per sub-operator
    std::vector<int> finals;
    Job agj[2], rs[4];
    if (p->pattern == COMPASS_AG_GEMM) {
        if ((rc = ag_jobs(p, geo, l, epoch, d, true, &agj[0], &agj[1])) != COMPASS_OK) return rc;
        if ((rc = stage_local_shard(p, geo, s)) != COMPASS_OK) return rc;
    } else {
        if ((rc = rs_jobs(p, geo, l, epoch, d, res, true, true, rs)) != COMPASS_OK) return rc;
        if ((rc = stage_resident_partials(p, geo, res, d, s)) != COMPASS_OK) return rc;
        if (p->send_dst)
            for (int r = 2; r < 4; ++r)
                if (rs[r].final_flag >= 0) finals.push_back(rs[r].final_flag);
    }
    std::vector<GemmParams> launches(d);
    const int cfg = pick_tile(p->M / d, p->N, false);
    for (int j = 0; j < d; ++j) {
        GemmParams &g = launches[j];
        init_params(g, epoch);
        const bool ag = p->pattern == COMPASS_AG_GEMM;
        if ((rc = set_shape(g, cfg, p->M / d, p->N, p->K, ag ? p->gathered : p->A, p->M, p->W, p->C,
                            ag ? nullptr : p->partial_stage)) != COMPASS_OK)
            return rc;
        if (d > 1) {
            g.piece = piece;
            g.pstride = geo.rows;
            g.poff = j * piece;
        }
        g.gate = ag ? kGateMain : kGateEpilogue;
        g.flag_base = j * geo.P;
        g.nparts = geo.P;
        g.resident_mask = res;
        touch_all(g, geo.P);   // a sub-operator needs its whole sub-collective
        if (j == 0) g.start_word = &g_ctx.hw[kHwStart];
        if (!ag && p->send_dst) {
            g.done_host = &g_ctx.hw[kHwDone];
            g.send_mask = nonlocal_mask(p, geo);
            for (int q = 0; q < geo.P; ++q)
                if (g.send_mask & (1ull << q)) g.done_expect[q] = (uint32_t)(g.tiles_m * g.tiles_n);
        }
        set_split(g, cfg);
    }
    if (p->pattern == COMPASS_AG_GEMM) {
        pool_jobs(agj, 2);
        submit(0, std::move(agj[0]));
        submit(1, std::move(agj[1]));
    } else {
        pool_jobs(rs, 4);
        for (int r = 0; r < 4; ++r) submit(r, std::move(rs[r]));
    }
    for (int j = 0; j < d; ++j)
        if ((rc = launch(launches[j], cfg, p->pattern == COMPASS_GEMM_RS, s)) != COMPASS_OK) return rc;
    if (!finals.empty()) return join(epoch, finals, false, s);
    return COMPASS_OK;
}

int op_gemm(int M, int N, int K, const void *A, const void *W, void *C, const float *P, void *stream) {
    if (M < 1 || N < 1 || K < 1 || K % 8 || N % 8) return set_error(COMPASS_ERR_INVALID, "need positive M, N, K with K, N multiples of 8");
    if (!A || !W || !C) return set_error(COMPASS_ERR_INVALID, "A, W and C are required");
    if ((M + 127) / 128 > kMaxRowTiles) return set_error(COMPASS_ERR_UNSUPPORTED, "M too large");
    if (!spans_fit(K, N, P != nullptr, 256))
        return set_error(COMPASS_ERR_UNSUPPORTED, "K = %d, N = %d: a 256-row tile would span more than 1 GiB of A, W "
                                                  "or the partial", K, N);
    int rc = begin();
    if (rc != COMPASS_OK) return rc;
    GemmParams g;
    init_params(g, g_ctx.epoch);
    const int cfg = pick_tile(M, N, false);
    if ((rc = set_shape(g, cfg, M, N, K, A, M, W, C, P)) != COMPASS_OK) return rc;
    g.gate = kGateNone;
    set_split(g, cfg);
    return launch(g, cfg, P != nullptr, (hipStream_t)stream);
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
        Job ag[2];
        if ((rc = ag_jobs(p, geo, l, epoch, 1, true, &ag[0], &ag[1])) != COMPASS_OK) return rc;
        for (int r = 0; r < 2; ++r)
            for (auto &it : ag[r].items) wait.push_back(it.flag);
        if ((rc = join(epoch, wait, true, s)) != COMPASS_OK) return rc;
        pool_jobs(ag, 2);
        submit(0, std::move(ag[0]));
        submit(1, std::move(ag[1]));
    } else {
        Job jobs[4];
        if ((rc = rs_jobs(p, geo, l, epoch, 1, resident_mask(p, geo), false, true, jobs)) != COMPASS_OK) return rc;
        for (int r = 0; r < 2; ++r)
            for (auto &it : jobs[r].items) wait.push_back(it.flag);
        for (int r = 2; r < 4; ++r)
            if (jobs[r].final_flag >= 0) wait.push_back(jobs[r].final_flag);
        if ((rc = join(epoch, wait, true, s)) != COMPASS_OK) return rc;
        pool_jobs(jobs, 4);
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
    GemmParams g;
    init_params(g, epoch);
    const int cfg = pick_tile(p->M, p->N, false);
    if ((rc = set_shape(g, cfg, p->M, p->N, p->K, p->A, p->M, p->W, p->C, p->partial_stage)) != COMPASS_OK) return rc;
    bool aliased = false;
    if ((rc = alias_resident_partials(g, p, geo, res, cfg, &aliased)) != COMPASS_OK) return rc;
    if (!aliased && (rc = stage_resident_partials(p, geo, res, 1, s)) != COMPASS_OK) return rc;
    g.gate = kGateNone;
    set_split(g, cfg);
    if ((rc = launch(g, cfg, true, s)) != COMPASS_OK) return rc;
    std::vector<int> wait;
    for (int r = 0; r < 2; ++r)
        for (auto &it : jobs[r].items) wait.push_back(it.flag);
    for (int r = 2; r < 4; ++r)
        if (jobs[r].final_flag >= 0) wait.push_back(jobs[r].final_flag);
    if ((rc = join(epoch, wait, true, s)) != COMPASS_OK) return rc;
    pool_jobs(jobs, 4);
    for (int r = 0; r < 4; ++r) submit(r, std::move(jobs[r]));
    return COMPASS_OK;
}

int op_sync() {
    int rc = ensure_init();
    if (rc != COMPASS_OK) return rc;
    // a job ends within its own stall bound (the host timeout), then lets a
    // failed job's copies land (the same bound again, at least 1 s); copy
    // jobs still running past both are treated as copies in flight
    const double t0 = now_s();
    while (!pacers_idle()) {
        if (now_s() - t0 > 2.0 * g_ctx.host_timeout + 2.0) {
            g_ctx.in_flight.store(true);
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
    case COMPASS_OPT_TILE:
        if (v < 0 || v > 2) return set_error(COMPASS_ERR_INVALID, "tile option must be 0, 1 or 2");
        c.tile_override = (int)v;
        return COMPASS_OK;
    case COMPASS_OPT_PACE_HEADROOM:
        if (v < 0 || v > 100) return set_error(COMPASS_ERR_INVALID, "pacing headroom must lie in [0, 100] percent");
        c.pace_headroom = (double)v / 100.0;
        return COMPASS_OK;
    case COMPASS_OPT_POOL:
        if (v < 0 || v > 8) return set_error(COMPASS_ERR_INVALID, "pool option must lie in [0, 8]");
        c.pool_depth = (int)v;
        return COMPASS_OK;
    case COMPASS_OPT_ENGINE_MASK:
        if (v < 0 || v > 0xFFFF) return set_error(COMPASS_ERR_INVALID, "engine mask out of range");
        c.engine_mask = (uint32_t)v;
        return COMPASS_OK;
    case COMPASS_OPT_KERNEL_TIMING: {
        if (v != 0 && v != 1) return set_error(COMPASS_ERR_INVALID, "kernel timing option must be 0 or 1");
        if (v == 1 && !c.timing) {
            const int rc = ensure_init();
            if (rc != COMPASS_OK) return rc;
            for (int i = 0; i < Ctx::kTimed; ++i) {
                if (!c.ev_begin[i] && hipEventCreate(&c.ev_begin[i]) != hipSuccess)
                    return set_error(COMPASS_ERR_HIP, "hipEventCreate failed");
                if (!c.ev_end[i] && hipEventCreate(&c.ev_end[i]) != hipSuccess)
                    return set_error(COMPASS_ERR_HIP, "hipEventCreate failed");
            }
        }
        c.timing = v == 1;
        c.timed_count = 0;
        return COMPASS_OK;
    }
    case COMPASS_OPT_TILE_TRACE: {
        if (v < 0 || v > (1 << 20)) return set_error(COMPASS_ERR_INVALID, "tile trace capacity out of range");
        const int rc = ensure_init();
        if (rc != COMPASS_OK) return rc;
        if (c.tile_trace) {
            hipError_t e = hipDeviceSynchronize();
            if (e == hipSuccess) e = hipFree(c.tile_trace);
            c.tile_trace = nullptr;
            c.trace_cap = c.trace_used = 0;
            if (e != hipSuccess) return hip_fail(e, "tile trace free");
        }
        if (v > 0) {
            const hipError_t e = hipMalloc((void **)&c.tile_trace, (size_t)v * kTraceWords * sizeof(uint32_t));
            if (e != hipSuccess) {
                c.tile_trace = nullptr;
                return hip_fail(e, "tile trace allocation");
            }
            c.trace_cap = (uint32_t)v;
        }
        return COMPASS_OK;
    }
    case COMPASS_OPT_SCHED:
        if (v < 0 || v > 7) return set_error(COMPASS_ERR_INVALID, "schedule option must be in [0, 7]");
        c.sched = (int)v;
        return COMPASS_OK;
    case COMPASS_OPT_TAIL_MIN_K:
    case COMPASS_OPT_TAIL_MIN_K_128:
        if (v < 0 || v > (1 << 21)) return set_error(COMPASS_ERR_INVALID, "tail split depth out of range");
        c.tail_min_k[key == COMPASS_OPT_TAIL_MIN_K ? 0 : 1] = (int)v;
        return COMPASS_OK;
    case COMPASS_OPT_TAIL_SLICE_K:
        if (v < 64 || v > (1 << 21) || v % 64) return set_error(COMPASS_ERR_INVALID, "tail slice depth must be a "
                                                                 "positive multiple of 64");
        c.tail_slice_k = (int)v;
        return COMPASS_OK;
    case COMPASS_OPT_HEAD_SPLIT:
        if (v != 0 && v != 1) return set_error(COMPASS_ERR_INVALID, "head split option must be 0 or 1");
        c.head_split = v == 1;
        return COMPASS_OK;
    case COMPASS_OPT_TAIL_GROUPS:
        if (v < 1 || v > 8) return set_error(COMPASS_ERR_INVALID, "tail groups must lie in [1, 8]");
        c.tail_groups = (int)v;
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
