// api.cpp -- the C ABI: argument checks, program cache, upload and launch.
//
// Mirrors the host side of the paper's compiled model (Section III-B-2 "Data Path"; Section V-B
// "Host-side Performance"): a collective call is validated, lowered into a complete program
// (or found in the cache of compiled work packets, which then costs only a re-enqueue),
// copied to device memory once, and enqueued as one executor launch on the caller's stream.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <thread>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <strings.h>
#include <list>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "compiler.h"
#include "hccl.h"
#include "program.h"

namespace hccl {
hipError_t launch_executor(const LaunchArgs& a, uint32_t blocks, int kind, hipStream_t stream);
hipError_t launch_executor_inline(const InlineArgs& a, uint32_t blocks, int kind, hipStream_t stream);
hipError_t launch_fill_u32(uint32_t* p, uint64_t n, uint32_t v, hipStream_t stream);
hipError_t launch_signal(uint64_t* word, uint64_t value, const ErrorRecord* err, hipStream_t stream);
hipError_t executor_occupancy(int kind, int* blocks_per_cu);
hipError_t launch_resident(const ResidentArgs& r, uint32_t blocks, hipStream_t stream);
hipError_t resident_occupancy(int* blocks_per_cu);
int executor_waves_per_block();
size_t workspace_bytes();
hipError_t workspace_address(void** ptr);
}  // namespace hccl

using namespace hccl;

namespace {

thread_local std::string g_last_error;

constexpr uint32_t kResidentDefaultBlocks = 32;       // 128 wavefronts, 4 workgroups per XCD
constexpr uint32_t kResidentDefaultIdleMs = 10000;
constexpr uint32_t kResidentMaxIdleMs = 600000;

hcclResult_t fail(hcclResult_t code, const std::string& msg) {
    g_last_error = msg;
    return code;
}

hcclResult_t hip_fail(hipError_t e, const char* what) {
    return fail(hcclHipError, std::string(what) + ": " + hipGetErrorString(e));
}

struct Call {
    CollectiveSpec spec;
    std::vector<const void*> send;
    std::vector<void*> recv;
    std::vector<void*> meta;   // device metadata arrays of a dynamic call (MetaSlot order)
    hipStream_t stream = nullptr;
};

struct DeviceProgram {
    std::vector<CollectiveSpec> specs;
    HostProgram prog;
    uint8_t* d_image = nullptr;
    uint32_t* d_state = nullptr;
    hipEvent_t done = nullptr;       // recorded after each launch
    hipStream_t last_stream = nullptr;
    bool launched = false;
    bool captured = false;           // a graph holds its image and state: never freed before the communicator
    double compile_us = 0;
};

}  // namespace

struct hcclComm {
    int nranks = 0;
    int device = HCCL_NO_DEVICE;
    hcclConfig_t cfg;
    int cus = 0;
    int blocks_per_cu[kNumKinds] = {0};
    uint64_t wall_clock_khz = 100000;
    ErrorRecord* d_error = nullptr;
    void* d_scratch = nullptr;
    uint64_t scratch_bytes = 0;
    hipEvent_t scratch_done = nullptr;  // recorded after each launch that uses the scratch
    hipStream_t scratch_stream = nullptr;
    bool scratch_launched = false;
    bool scratch_captured = false;      // a graph holds d_scratch: growth keeps the old allocation
    std::vector<void*> retired_scratch;
    hipStream_t setup_stream = nullptr;  // non-blocking: program uploads never wait for other streams
    std::list<std::unique_ptr<DeviceProgram>> cache;  // most recently used first
    std::vector<std::unique_ptr<DeviceProgram>> retired;  // evicted programs that a graph holds
    size_t cache_limit = 64;
    // tile dispatch (use_tickets): static, or by ticket for dependent programs while a waiting
    // executor holds CUs; HCCL_DISPATCH=static / dynamic forces one for every program
    int dispatch_mode = 0;           // 0 auto, 1 static, 2 tickets
    bool inline_single_step = true;  // one-step programs travel in the launch packet
    int group_depth = 0;             // > 0 between hccl_group_start and hccl_group_end
    std::vector<Call> pending;       // calls recorded inside a group
    bool has_trigger = false;        // hccl_set_trigger for the next work packet
    hcclTrigger_t trigger{};
    hcclProgramInfo_t last{};
    const HostProgram* last_prog = nullptr;  // the program `last` describes (NULL once evicted)
    // resident executor (hccl_resident_start .. hccl_resident_stop)
    bool resident = false;
    ResidentQueue* rq = nullptr;      // coherent pinned host memory, shared with the executor
    uint32_t* d_ctl = nullptr;
    hipStream_t resident_stream = nullptr;
    uint64_t resident_seq = 0;        // last packet published
    // environment overrides (read at creation): HCCL_ALGO, HCCL_CHUNK_BYTES, HCCL_DEBUG
    int env_algo = -1;                // hcclAlgo_t forced for every call, -1 = the configuration's
    uint64_t env_chunk = 0;           // chunk bytes forced for every call, 0 = the configuration's
    int log_level = 0;                // 0 off, 1 WARN, 2 INFO, 3 TRACE
    // per-tile trace of the last traced launch (cfg.trace)
    TileStamp* d_trace = nullptr;
    uint64_t trace_cap = 0;           // records the buffer holds
    uint32_t trace_tiles = 0;         // records the last traced launch wrote
    // allocation-free calls: this device's static workspace and host-only compiled programs
    void* workspace = nullptr;
    std::string workspace_error;
    std::list<std::pair<CollectiveSpec, std::unique_ptr<HostProgram>>> host_cache;
};

namespace {

// Log lines on stderr at HCCL_DEBUG=WARN (1), INFO (2) or TRACE (3).
void hlog(const hcclComm* c, int level, const char* fmt, ...) __attribute__((format(printf, 3, 4)));
void hlog(const hcclComm* c, int level, const char* fmt, ...) {
    if (!c || c->log_level < level) return;
    static const char* kNames[] = {"", "WARN", "INFO", "TRACE"};
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    std::fprintf(stderr, "[hccl %s] comm %p: %s\n", kNames[level], (const void*)c, buf);
}

const char* kCollNames[] = {"allreduce", "reduce_scatter", "allgather", "alltoallv", "alltoallv_dynamic"};
const char* kAlgoNames[] = {"auto", "direct", "ring", "two_level", "rhd"};

// The environment overrides of a new communicator. Unknown values are ignored with a warning.
void read_env(hcclComm* c) {
    if (const char* v = std::getenv("HCCL_DEBUG")) {
        if (!strcasecmp(v, "WARN")) c->log_level = 1;
        else if (!strcasecmp(v, "INFO")) c->log_level = 2;
        else if (!strcasecmp(v, "TRACE")) c->log_level = 3;
    }
    if (const char* v = std::getenv("HCCL_ALGO")) {
        for (int a = 0; a <= hcclAlgoRhd; ++a)
            if (!strcasecmp(v, kAlgoNames[a])) c->env_algo = a;
        if (c->env_algo < 0) hlog(c, 1, "HCCL_ALGO=%s is not a schedule (auto, direct, ring, two_level, rhd): ignored", v);
    }
    if (const char* v = std::getenv("HCCL_CHUNK_BYTES")) {
        char* end = nullptr;
        const unsigned long long n = std::strtoull(v, &end, 10);
        uint64_t mul = 1;
        if (end && (*end == 'K' || *end == 'k')) mul = 1024, ++end;
        else if (end && (*end == 'M' || *end == 'm')) mul = 1024 * 1024, ++end;
        if (end && *end == '\0' && n > 0 && n < (1ull << 40)) c->env_chunk = n * mul;
        else hlog(c, 1, "HCCL_CHUNK_BYTES=%s is not a byte count: ignored", v);
    }
}

// Triggered packets still waiting on a device (any communicator of the process). While one is,
// the library makes no call that could wait for every stream of that device (a free, a device
// synchronisation): the host thread that would release the trigger might be the one waiting.
struct PendingTrigger {
    int device;
    hipEvent_t done;  // recorded behind the packet (and its completion-word kernel)
};
std::mutex g_trigger_mu;
std::vector<PendingTrigger> g_triggers;

void note_trigger(int device, hipStream_t s) {
    hipEvent_t ev = nullptr;
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) return;
    if (hipEventRecord(ev, s) != hipSuccess) {
        (void)hipEventDestroy(ev);
        return;
    }
    std::lock_guard<std::mutex> lock(g_trigger_mu);
    g_triggers.push_back({device, ev});
}

// Resident executors running on each device (any communicator of the process).
std::mutex g_resident_mu;
std::vector<int> g_resident_devices;

void note_resident(int device, bool running) {
    std::lock_guard<std::mutex> lock(g_resident_mu);
    if (running) {
        g_resident_devices.push_back(device);
        return;
    }
    for (size_t i = 0; i < g_resident_devices.size(); ++i)
        if (g_resident_devices[i] == device) {
            g_resident_devices.erase(g_resident_devices.begin() + (long)i);
            return;
        }
}

bool resident_running(int device) {
    std::lock_guard<std::mutex> lock(g_resident_mu);
    for (int d : g_resident_devices)
        if (d == device) return true;
    return false;
}

bool trigger_pending(int device) {
    std::lock_guard<std::mutex> lock(g_trigger_mu);
    bool any = false;
    for (size_t i = 0; i < g_triggers.size();) {
        if (hipEventQuery(g_triggers[i].done) == hipSuccess) {
            (void)hipEventDestroy(g_triggers[i].done);
            g_triggers[i] = g_triggers.back();
            g_triggers.pop_back();
            continue;
        }
        any |= g_triggers[i].device == device;
        ++i;
    }
    return any;
}

bool env_flag(const char* name) {
    const char* v = std::getenv(name);
    return v && *v && std::strcmp(v, "0") != 0;
}

struct DeviceGuard {
    int prev = -1;
    bool changed = false;
    explicit DeviceGuard(int dev) {
        if (dev < 0) return;
        if (hipGetDevice(&prev) == hipSuccess && prev != dev) changed = hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard() {
        if (changed) (void)hipSetDevice(prev);
    }
};

void free_program(DeviceProgram* p) {
    if (p->done) (void)hipEventSynchronize(p->done);
    if (p->d_image) (void)hipFree(p->d_image);
    if (p->d_state) (void)hipFree(p->d_state);
    if (p->done) (void)hipEventDestroy(p->done);
    p->d_image = nullptr;
    p->d_state = nullptr;
    p->done = nullptr;
}

hcclResult_t check_dtype(hcclDataType_t dt) {
    if (dt != hcclBf16 && dt != hcclFp16 && dt != hcclFp32 && dt != hcclInt32)
        return fail(hcclInvalidArgument, "unknown data type");
    return hcclSuccess;
}

hcclResult_t check_op(hcclRedOp_t op) {
    if (op != hcclSum && op != hcclMax && op != hcclMin) return fail(hcclInvalidArgument, "unknown reduction operator");
    return hcclSuccess;
}

struct Range {
    uintptr_t lo, hi;
    int id;
};

// Buffers must be non-null (when non-empty), aligned to the element size, and must not
// overlap each other except where `allow` accepts the pair.
template <typename Allow>
hcclResult_t check_buffers(const std::vector<Range>& v, size_t es, Allow allow) {
    for (const Range& r : v) {
        if (r.hi == r.lo) continue;
        if (r.lo == 0) return fail(hcclInvalidArgument, "null buffer pointer");
        if (r.lo % es) return fail(hcclInvalidArgument, "buffer not aligned to its element size");
    }
    std::vector<Range> s;
    for (const Range& r : v)
        if (r.hi > r.lo) s.push_back(r);
    std::sort(s.begin(), s.end(), [](const Range& a, const Range& b) { return a.lo < b.lo; });
    for (size_t i = 0; i < s.size(); ++i)
        for (size_t j = i + 1; j < s.size() && s[j].lo < s[i].hi; ++j)
            if (!allow(s[i], s[j])) return fail(hcclInvalidArgument, "buffers overlap");
    return hcclSuccess;
}

// Compiles (or finds in the cache) the program of one work packet: one collective, or the
// collectives of a group, merged into one program whose steps use disjoint buffer ids.
// `may_compile` is false while the stream is being captured into a graph: compiling uploads
// the image with a synchronous copy, which a capture does not allow.
hcclResult_t compile_program(hcclComm* c, const std::vector<CollectiveSpec>& specs, DeviceProgram*& out, bool& hit,
                             bool may_compile) {
    for (auto it = c->cache.begin(); it != c->cache.end(); ++it) {
        if ((*it)->specs == specs) {
            if (it != c->cache.begin()) c->cache.splice(c->cache.begin(), c->cache, it);
            out = c->cache.front().get();
            hit = true;
            return hcclSuccess;
        }
    }
    hit = false;
    if (!may_compile)
        return fail(hcclUnsupported, "the stream is capturing a graph and this program is not compiled yet: "
                                     "make the same call once outside the capture first");
    auto t0 = std::chrono::steady_clock::now();
    auto dp = std::make_unique<DeviceProgram>();
    dp->specs = specs;
    std::string err;
    const bool check = c->cfg.validate || c->device == HCCL_NO_DEVICE || env_flag("HCCL_VALIDATE");
    std::vector<HostProgram> parts(specs.size());
    for (size_t k = 0; k < specs.size(); ++k) {
        if (!lower(specs[k], parts[k], err)) return fail(hcclUnsupported, err);
        if (specs[k].fuse) fuse(parts[k]);
        if (check) {
            HostProgram probe = parts[k];
            if (!finalize(probe, specs[k].tile_bytes, err)) return fail(hcclInternalError, err);
            if (!validate(probe, specs[k], err)) return fail(hcclInternalError, "program validation failed: " + err);
        }
    }
    if (parts.size() == 1) {
        dp->prog = std::move(parts[0]);
    } else if (!merge(parts, specs, dp->prog, err)) {
        return fail(hcclUnsupported, err);
    }
    if (!finalize(dp->prog, specs[0].tile_bytes, err)) return fail(hcclInternalError, err);
    dp->compile_us = std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count();
    hlog(c, 2, "compiled %s%s: schedule %s%s, %zu steps, %u tiles, %u dependencies, %u phases, %llu bytes read, "
               "%llu written, %llu scratch, kernel kind %d, %.1f us",
         specs.size() == 1 ? kCollNames[specs[0].coll] : "group of ", specs.size() == 1 ? "" : std::to_string(specs.size()).c_str(),
         kAlgoNames[dp->prog.algo], dp->prog.fused ? " (fused)" : "", dp->prog.descs.size(), dp->prog.ntiles,
         dp->prog.ndeps, dp->prog.nphase(), (unsigned long long)dp->prog.bytes_read, (unsigned long long)dp->prog.bytes_written,
         (unsigned long long)dp->prog.scratch_bytes, dp->prog.kind, dp->compile_us);

    if (c->device != HCCL_NO_DEVICE) {
        const auto& img = dp->prog.image;
        hipError_t e = hipMalloc(&dp->d_image, img.size());
        if (e != hipSuccess) return fail(hcclOutOfMemory, "program image allocation failed");
        e = hipMemcpyAsync(dp->d_image, img.data(), img.size(), hipMemcpyHostToDevice, c->setup_stream);
        if (e != hipSuccess) {
            free_program(dp.get());
            return hip_fail(e, "program upload");
        }
        e = hipMalloc(&dp->d_state, (size_t)dp->prog.nstate * sizeof(uint32_t));
        if (e != hipSuccess) {
            free_program(dp.get());
            return fail(hcclOutOfMemory, "program state allocation failed");
        }
        e = launch_fill_u32(dp->d_state, dp->prog.nstate, 0u, c->setup_stream);
        // only the upload and the fill are waited for, on a stream that waits for no other: a
        // resident executor, or a triggered one whose release is still to come, may be running
        if (e == hipSuccess) e = hipStreamSynchronize(c->setup_stream);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&dp->done, hipEventDisableTiming);
        if (e != hipSuccess) {
            free_program(dp.get());
            return hip_fail(e, "program state setup");
        }
    }
    c->cache.push_front(std::move(dp));
    while (c->cache.size() > c->cache_limit) {
        // (a free could wait for a running resident executor, which ends only when stopped, or
        // for a triggered one: those programs are kept until the communicator is destroyed)
        if (c->cache.back()->captured || c->resident || trigger_pending(c->device))
            c->retired.push_back(std::move(c->cache.back()));
        else {
            if (c->last_prog == &c->cache.back()->prog) c->last_prog = nullptr;
            free_program(c->cache.back().get());
        }
        c->cache.pop_back();
    }
    out = c->cache.front().get();
    return hcclSuccess;
}

hcclResult_t ensure_scratch(hcclComm* c, uint64_t bytes) {
    if (bytes <= c->scratch_bytes) return hcclSuccess;
    // The old scratch may still be in use. A graph may hold it, and while a triggered packet
    // waits a free could wait for it too: then it is kept until the communicator is destroyed.
    // Otherwise the last launch that used it is waited for, and it is freed.
    const bool keep = c->scratch_captured || trigger_pending(c->device);
    if (c->d_scratch && !keep && c->scratch_launched) {
        hipError_t e = hipEventSynchronize(c->scratch_done);
        if (e != hipSuccess) return hip_fail(e, "wait before scratch growth");
    }
    if (c->d_scratch && keep)
        c->retired_scratch.push_back(c->d_scratch);
    else if (c->d_scratch)
        (void)hipFree(c->d_scratch);
    hipError_t e;
    c->d_scratch = nullptr;
    c->scratch_captured = false;
    c->scratch_bytes = 0;
    e = hipMalloc(&c->d_scratch, bytes);
    if (e != hipSuccess) return fail(hcclOutOfMemory, "scratch allocation failed");
    c->scratch_bytes = bytes;
    c->scratch_launched = false;
    return hcclSuccess;
}

uint32_t stream_cu_count(hcclComm* c, hipStream_t s) {
    if (!s) return (uint32_t)c->cus;
    uint32_t mask[16] = {0};
    if (hipExtStreamGetCUMask(s, 16, mask) != hipSuccess) return (uint32_t)c->cus;
    uint32_t n = 0;
    for (uint32_t w : mask) n += (uint32_t)__builtin_popcount(w);
    if (n == 0 || n > (uint32_t)c->cus) return (uint32_t)c->cus;
    return n;
}

// ---- resident executor: host side of the doorbell
uint64_t resident_done(const hcclComm* c) { return __atomic_load_n(&c->rq->done_seq, __ATOMIC_ACQUIRE); }
bool resident_exited(const hcclComm* c) { return __atomic_load_n(&c->rq->exited, __ATOMIC_ACQUIRE) != 0u; }

// Why the resident executor ended, for messages.
std::string resident_exit_reason(const hcclComm* c) {
    const uint32_t why = __atomic_load_n(&c->rq->exited, __ATOMIC_ACQUIRE);
    return why == RESIDENT_EXIT_IDLE         ? "no packet arrived within the idle limit"
           : why == RESIDENT_EXIT_WORKGROUPS ? "its workgroups did not all finish a packet within the watchdog"
           : why == RESIDENT_EXIT_STOP       ? "a stop request"
                                             : "exit code " + std::to_string(why);
}

// Waits until packet `seq` has completed; fails if the executor stopped or `ms` passed first.
hcclResult_t resident_wait_for(hcclComm* c, uint64_t seq, uint64_t ms) {
    if (resident_done(c) >= seq) return hcclSuccess;
    const auto t0 = std::chrono::steady_clock::now();
    for (uint32_t spin = 0;; ++spin) {
        if (resident_done(c) >= seq) return hcclSuccess;
        if (resident_exited(c) && resident_done(c) < seq)
            return fail(hcclTimeout, "the resident executor stopped before packet " + std::to_string(seq) +
                                         " completed (" + resident_exit_reason(c) + "; packets completed: " +
                                         std::to_string(resident_done(c)) + ")");
        if ((spin & 1023u) == 1023u) {
            const double el = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
            if (el > (double)ms) return fail(hcclTimeout, "the resident executor did not complete the packet in time");
            std::this_thread::yield();
        }
    }
}

// Publishes one packet: its arguments into the next ring slot, then the slot's sequence number.
hcclResult_t resident_submit(hcclComm* c, const LaunchArgs& a, DeviceProgram* dp) {
    const uint64_t k = c->resident_seq + 1;
    const uint64_t ms = c->cfg.timeout_ms ? c->cfg.timeout_ms : 2000u;
    if (resident_exited(c))
        return fail(hcclTimeout, "the resident executor has stopped (" + resident_exit_reason(c) + "): restart it");
    // the slot last held packet k - kResidentSlots, whose arguments every workgroup has read
    // once it has completed
    if (k > kResidentSlots) {
        hcclResult_t r = resident_wait_for(c, k - kResidentSlots, ms);
        if (r != hcclSuccess) return r;
    }
    ResidentSlot& slot = c->rq->slots[(k - 1) % kResidentSlots];
    std::memcpy((void*)&slot.args, &a, sizeof a);
    std::atomic_thread_fence(std::memory_order_release);
    __atomic_store_n(&slot.seq, k, __ATOMIC_RELEASE);
    c->resident_seq = k;
    dp->captured = true;  // the executor may read the image after the call returns: never freed early
    return hcclSuccess;
}

// Largest grid of one wavefront per tile: a program has under 2^31 tiles, so the kernel's tile
// numbers (t + W, 32 bits) cannot wrap; larger phases loop as a resident grid does.
constexpr uint32_t kMaxGridWorkers = 1u << 24;

// Executor kernel and grid of a launch: the leanest kernel that covers the program (the aligned
// copy kernel only if every user buffer is 16-byte aligned), and its grid, capped by the
// configuration and by the tiles of the phase.
//  * A launch whose tiles never wait (no dependencies inside it, no trigger, no tickets, not
//    traced) gets one wavefront per tile. The hardware starts each workgroup as soon as a
//    resident one ends, in grid order, so the CUs work on a window of neighbouring tiles that
//    moves through the phase and no wavefront ends up with more tiles than the others. Measured
//    against a grid of the CUs' resident capacity: the grouped AllToAllv of 8 ranks x 2^18
//    embedding rows 192-193 -> 182-184 us, a 1 GiB copy 400-407 -> 340-343 us, the
//    reduce-scatter P=8 x 256 MiB bf16 423 -> 400-404 us.
//  * Otherwise the grid is the resident capacity of the CUs the stream may use: a dependent tile
//    waits for lower tiles, and static dispatch relies on the whole grid being resident; a
//    triggered launch holds its CUs while it waits; a traced launch records wavefront numbers.
// Sets a.nworkers and `blocks`; returns the kernel kind.
int launch_shape(hcclComm* c, const HostProgram& prog, uint32_t phase, LaunchArgs& a, uint32_t nuser, hipStream_t s,
                 uint32_t& blocks) {
    const uint32_t wpb = (uint32_t)executor_waves_per_block();
    uint32_t cus = stream_cu_count(c, s);
    int kind = prog.phase_kind.empty() ? prog.kind : prog.phase_kind[phase];
    a.tile_begin = prog.phase_tile.empty() ? 0u : prog.phase_tile[phase];
    a.tile_end = prog.phase_tile.empty() ? prog.ntiles : prog.phase_tile[phase + 1];
    a.xcd_order = prog.phase_xcd.empty() ? 0u : prog.phase_xcd[phase];
    if (a.trace) kind = kKindGeneric;  // the kernel that records the trace
    if (kind == kKindCopyAligned) {
        for (uint32_t i = 0; i < nuser; ++i)
            if ((uintptr_t)a.bufs[i] % 16) kind = kKindCopyOnly;
    }
    const uint32_t tiles = a.tile_end - a.tile_begin;
    uint32_t slots = cus * (uint32_t)std::max(1, c->blocks_per_cu[kind]) * wpb;
    const bool never_waits = (prog.flags & PF_HAS_DEPS) == 0 && a.wait_addr == nullptr && !a.dynamic && !a.trace;
    if (never_waits) slots = std::max(slots, std::min<uint32_t>(tiles, kMaxGridWorkers));
    if (c->cfg.max_workers > 0) slots = std::min<uint32_t>(slots, (uint32_t)c->cfg.max_workers);
    uint32_t workers = std::min<uint32_t>(slots, tiles);
    blocks = (workers + wpb - 1) / wpb;
    if (blocks == 0) blocks = 1;
    a.nworkers = blocks * wpb;
    return kind;
}

// How a launch hands out tiles. Static dispatch of a dependent program needs its whole grid
// resident at once; that fails when a kernel that waits for something still to come holds CUs:
// a triggered packet whose release is not enqueued yet, or a resident executor. While one of
// those (of any communicator of the process) is on the device, dependent programs take their
// tiles by ticket, which drains on whatever part of the grid is resident, at the price of one
// same-address atomic per tile (the unfused ring all-reduce P=4 x 2^20 fp32: 86 -> 131 us).
// HCCL_DISPATCH=static or =dynamic forces one way for every program.
bool use_tickets(const hcclComm* c, const HostProgram& prog, bool triggered) {
    if (c->dispatch_mode == 1) return false;
    if (c->dispatch_mode == 2) return true;
    if ((prog.flags & PF_HAS_DEPS) == 0) return false;
    return triggered || trigger_pending(c->device) || resident_running(c->device);
}

// A program of one plain step without dependencies travels in the launch packet itself.
bool inline_eligible(const hcclComm* c, const HostProgram& prog, bool triggered) {
    const bool plain_step = prog.descs.size() == 1 && (prog.descs[0].op == OP_COPY || prog.descs[0].op == OP_REDUCE);
    return c->inline_single_step && plain_step && (prog.flags & PF_HAS_DEPS) == 0 && c->dispatch_mode != 2 &&
           !triggered && !c->cfg.trace;
}

// Trace buffer for `tiles` records (grown on demand; traced launches are a diagnostic mode).
hcclResult_t ensure_trace(hcclComm* c, uint64_t tiles) {
    if (tiles <= c->trace_cap) return hcclSuccess;
    if (trigger_pending(c->device)) {
        if (c->d_trace) c->retired_scratch.push_back(c->d_trace);  // freed with the communicator
    } else {
        hipError_t e = hipDeviceSynchronize();  // the old buffer may still be written
        if (e != hipSuccess) return hip_fail(e, "synchronize before trace growth");
        if (c->d_trace) (void)hipFree(c->d_trace);
    }
    c->d_trace = nullptr;
    c->trace_cap = 0;
    c->trace_tiles = 0;
    hipError_t e = hipMalloc(&c->d_trace, tiles * sizeof(TileStamp));
    if (e != hipSuccess) return fail(hcclOutOfMemory, "trace buffer allocation failed");
    c->trace_cap = tiles;
    return hcclSuccess;
}

hipError_t launch_inline_step(const HostProgram& prog, const LaunchArgs& a, uint32_t blocks, int kind, hipStream_t s) {
    const HostDesc& d = prog.descs[0];
    InlineArgs ia;
    std::memset(&ia, 0, sizeof ia);
    ia.nelem = d.nelem;
    ia.tile_elems = prog.tile_elems;
    ia.ntiles = prog.ntiles;
    ia.nworkers = a.nworkers;
    ia.op = d.op;
    ia.redop = d.redop;
    ia.nsrc = (uint32_t)d.srcs.size();
    ia.ndst = (uint32_t)d.dsts.size();
    ia.group = d.group;
    ia.fold = d.fold;
    ia.requant = d.requant ? 1u : 0u;
    ia.es_first = dtype_size(d.srcs[0].dtype);
    ia.es_rest = dtype_size(d.srcs.size() > 1 ? d.srcs[1].dtype : d.srcs[0].dtype);
    ia.es_out = dtype_size(d.dsts[0].dtype);
    ia.sig = reduce_signature(d.srcs[0].dtype, d.srcs.size() > 1 ? d.srcs[1].dtype : d.srcs[0].dtype, d.dsts[0].dtype);
    for (size_t j = 0; j < d.srcs.size(); ++j) ia.src[j] = (uint64_t)(uintptr_t)a.bufs[d.srcs[j].buf] + d.srcs[j].offset;
    for (size_t j = 0; j < d.dsts.size(); ++j) ia.dst[j] = (uint64_t)(uintptr_t)a.bufs[d.dsts[j].buf] + d.dsts[j].offset;
    return launch_executor_inline(ia, blocks, kind, s);
}

// Program description for hccl_comm_last_program.
void describe(hcclProgramInfo_t& info, const std::vector<CollectiveSpec>& specs, const HostProgram& prog, bool hit,
              double compile_us) {
    std::memset(&info, 0, sizeof info);
    info.collective = specs.size() == 1 ? specs[0].coll : -1;
    info.algo = prog.algo;
    info.fused = prog.fused ? 1 : 0;
    info.cache_hit = hit ? 1 : 0;
    info.num_descs = (uint32_t)prog.descs.size();
    info.num_tiles = prog.ntiles;
    info.num_deps = prog.ndeps;
    info.num_operands = prog.noperands;
    info.max_srcs = prog.max_srcs;
    info.bytes_read = prog.bytes_read;
    info.bytes_written = prog.bytes_written;
    info.scratch_bytes = prog.scratch_bytes;
    info.program_bytes = prog.image.size();
    info.compile_us = compile_us;
    info.step_tile_min = prog.step_tile_min;
    info.step_tile_max = prog.step_tile_max;
    info.num_phases = prog.nphase();
}

// Compiles and enqueues one work packet (a list of collective calls on one stream).
hcclResult_t run_packet(hcclComm* c, const std::vector<Call>& calls) {
    DeviceProgram* dp = nullptr;
    bool hit = false;
    DeviceGuard guard(c->device);
    std::vector<CollectiveSpec> specs;
    for (const Call& k : calls) specs.push_back(k.spec);
    // the trigger belongs to this packet, whether it is enqueued or rejected
    const bool triggered = c->has_trigger;
    const hcclTrigger_t trig = c->trigger;
    c->has_trigger = false;
    // Under graph capture the packet may only enqueue: kernel launches on the capturing stream.
    // (The null stream is never captured, and querying it during another stream's capture is
    // itself an error, so it is not asked.)
    hipStream_t s = calls[0].stream;
    bool capturing = false;
    if (c->device != HCCL_NO_DEVICE && s) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        hipError_t e = hipStreamIsCapturing(s, &cs);
        if (e != hipSuccess) return hip_fail(e, "stream capture query");
        capturing = cs != hipStreamCaptureStatusNone;
    }
    hcclResult_t r = compile_program(c, specs, dp, hit, !capturing);
    if (r != hcclSuccess) {
        hlog(c, 1, "%s", g_last_error.c_str());
        return r;
    }
    if (hit) hlog(c, 3, "cached program: %zu steps, %u tiles", dp->prog.descs.size(), dp->prog.ntiles);

    hcclProgramInfo_t& info = c->last;
    describe(info, specs, dp->prog, hit, dp->compile_us);
    c->last_prog = &dp->prog;

    if (triggered) {
        if (dp->prog.ntiles == 0) return fail(hcclInvalidArgument, "a triggered work packet has no work to run");
        // the trigger words must not overlap a buffer of the packet
        for (const Call& k : calls) {
            BufferSizes sz = buffer_sizes(k.spec, 0);
            for (int i = 0; i < k.spec.P; ++i) {
                const std::pair<uintptr_t, uint64_t> spans[2] = {{(uintptr_t)k.send[i], sz.bytes[send_buf(i)]},
                                                                 {(uintptr_t)k.recv[i], sz.bytes[recv_buf(k.spec.P, i)]}};
                for (const auto& sp : spans)
                    for (const void* w : {(const void*)trig.wait_addr, (const void*)trig.done_addr})
                        if (w && (uintptr_t)w + 8 > sp.first && (uintptr_t)w < sp.first + sp.second)
                            return fail(hcclInvalidArgument, "a trigger word overlaps a buffer of the collective");
            }
        }
    }
    if (c->resident) {
        if (triggered) return fail(hcclUnsupported, "a triggered work packet cannot go to the resident executor");
        if (capturing)
            return fail(hcclUnsupported, "the resident executor takes packets from the host, not from a captured stream");
        if (dp->prog.scratch_bytes > c->scratch_bytes)
            return fail(hcclUnsupported, "the communicator's scratch must grow, which cannot happen while the resident "
                                         "executor runs: make the same call once before hccl_resident_start");
    }
    if (c->device == HCCL_NO_DEVICE || dp->prog.ntiles == 0) return hcclSuccess;

    if (capturing && dp->prog.scratch_bytes > c->scratch_bytes)
        return fail(hcclUnsupported, "the stream is capturing a graph and the communicator's scratch must grow: "
                                     "make the same call once outside the capture first");
    r = ensure_scratch(c, dp->prog.scratch_bytes);
    if (r != hcclSuccess) return r;
    const bool traced = c->cfg.trace != 0 && !capturing && !c->resident;
    if (traced && (r = ensure_trace(c, dp->prog.ntiles)) != hcclSuccess) return r;
    if (capturing) {  // the graph keeps this image, state and scratch address
        dp->captured = true;
        if (dp->prog.scratch_bytes > 0) c->scratch_captured = true;
    }

    LaunchArgs a;
    std::memset(&a, 0, sizeof a);
    a.prog = dp->d_image;
    a.state = dp->d_state;
    a.error = c->d_error;
    uint32_t base = 0;
    for (const Call& k : calls) {
        const int P = k.spec.P;
        for (int i = 0; i < P; ++i) {
            a.bufs[base + send_buf(i)] = (char*)k.send[i];
            a.bufs[base + recv_buf(P, i)] = (char*)k.recv[i];
        }
        base += 2 * (uint32_t)P;
    }
    a.bufs[base] = (char*)c->d_scratch;  // the scratch id follows every call's buffers
    const uint32_t nuser = base;
    uint32_t mb = base + 1;              // then the metadata arrays of the dynamic calls
    for (const Call& k : calls)
        for (void* m : k.meta) a.bufs[mb++] = (char*)m;
    const bool has_deps = (dp->prog.flags & PF_HAS_DEPS) != 0;
    a.dynamic = use_tickets(c, dp->prog, triggered) ? 1u : 0u;
    const uint64_t ms = c->cfg.timeout_ms ? c->cfg.timeout_ms : 2000u;
    a.timeout_ticks = ms * c->wall_clock_khz;
    if (triggered) {
        a.wait_addr = trig.wait_addr;
        a.wait_value = trig.wait_value;
        a.wait_cmp = (uint32_t)trig.wait_cmp;
    }
    const bool signals = triggered && trig.done_addr != nullptr;
    if (traced) a.trace = c->d_trace;

    const uint32_t nph = dp->prog.nphase();
    if (c->resident) {
        // one packet per phase: the executor finishes a packet everywhere before the next starts
        for (uint32_t q = 0; q < nph; ++q) {
            a.tile_begin = dp->prog.phase_tile[q];
            a.tile_end = dp->prog.phase_tile[q + 1];
            if ((r = resident_submit(c, a, dp)) != hcclSuccess) return r;
        }
        return hcclSuccess;
    }

    uint32_t blocks = 0;
    int kind = launch_shape(c, dp->prog, 0, a, nuser, s, blocks);
    info.workers = a.nworkers;
    info.tickets = a.dynamic;

    if (nph == 1 && inline_eligible(c, dp->prog, triggered)) {
        info.inline_launch = 1;
        hipError_t e = launch_inline_step(dp->prog, a, blocks, kind, s);
        if (e != hipSuccess) return hip_fail(e, "inline executor launch");
        return hcclSuccess;
    }

    // a program's counters serve one launch at a time, and the communicator's scratch one
    // program at a time: order such launches across streams. A captured launch is left out of
    // this bookkeeping: an event recorded outside a capture cannot be waited on inside it, and
    // one recorded inside stands for a graph node, not for a launch. Replays run in the order
    // of the stream they are launched on; the caller orders them against eager launches of the
    // same program, or of programs that use scratch, on other streams.
    if (traced) {  // every record of this launch starts cleared, then each tile writes its own
        c->trace_tiles = dp->prog.ntiles;
        hipError_t e = launch_fill_u32((uint32_t*)c->d_trace, (uint64_t)dp->prog.ntiles * sizeof(TileStamp) / 4, 0u, s);
        if (e != hipSuccess) return hip_fail(e, "trace clear");
    }
    const bool stateful = (has_deps || a.dynamic != 0) && !capturing;
    const bool scratch = dp->prog.scratch_bytes > 0 && !capturing;
    if (stateful && dp->launched && dp->last_stream != s) {
        hipError_t e = hipStreamWaitEvent(s, dp->done, 0);
        if (e != hipSuccess) return hip_fail(e, "cross-stream ordering");
    }
    if (scratch && c->scratch_launched && c->scratch_stream != s) {
        hipError_t e = hipStreamWaitEvent(s, c->scratch_done, 0);
        if (e != hipSuccess) return hip_fail(e, "cross-stream ordering");
    }
    hipError_t e = hipSuccess;
    for (uint32_t q = 0; q < nph; ++q) {
        if (q > 0) {
            // later phases follow the first on the stream: only the first waits for a trigger
            a.wait_addr = nullptr;
            kind = launch_shape(c, dp->prog, q, a, nuser, s, blocks);
            info.workers = std::max(info.workers, a.nworkers);
        }
        e = launch_executor(a, blocks, kind, s);
        if (e != hipSuccess) return hip_fail(e, "executor launch");
        hlog(c, 3, "launched phase %u of %u, kernel kind %d: %u workgroups, %u wavefronts, tiles %u..%u, %s dispatch%s",
             q + 1, nph, kind, blocks, a.nworkers, a.tile_begin, a.tile_end, a.dynamic ? "ticket" : "static",
             a.trace ? ", traced" : "");
    }
    if (signals) {
        e = launch_signal(trig.done_addr, trig.done_value, c->d_error, s);
        if (e != hipSuccess) return hip_fail(e, "completion word");
    }
    if (triggered) note_trigger(c->device, s);
    if (stateful) {
        e = hipEventRecord(dp->done, s);
        if (e != hipSuccess) return hip_fail(e, "completion event");
        dp->last_stream = s;
        dp->launched = true;
    }
    if (scratch) {
        e = hipEventRecord(c->scratch_done, s);
        if (e != hipSuccess) return hip_fail(e, "completion event");
        c->scratch_stream = s;
        c->scratch_launched = true;
    }
    return hcclSuccess;
}

hcclResult_t run(hcclComm* c, const CollectiveSpec& spec, const void* const* send, void* const* recv, void* stream,
                 std::vector<void*> meta = {}) {
    Call k;
    k.spec = spec;
    k.send.assign(send, send + spec.P);
    k.recv.assign(recv, recv + spec.P);
    k.meta = std::move(meta);
    k.stream = (hipStream_t)stream;
    if (c->group_depth > 0) {
        c->pending.push_back(std::move(k));
        return hcclSuccess;
    }
    std::vector<Call> one;
    one.push_back(std::move(k));
    return run_packet(c, one);
}

hcclResult_t fill_spec(hcclComm* c, CollectiveSpec& s, int coll, hcclDataType_t dt, hcclRedOp_t op) {
    s.coll = coll;
    s.P = c->nranks;
    s.dtype = (int)dt;
    s.redop = (int)op;
    s.algo = c->cfg.algo;
    s.group_size = c->cfg.group_size;
    s.chunk_bytes = c->cfg.chunk_bytes;
    s.fuse = c->cfg.fuse != 0;
    s.tile_bytes = c->cfg.tile_bytes;
    s.order = c->cfg.order;
    s.requant = c->cfg.requantize != 0;
    s.phases = c->cfg.phases;
    if (c->env_algo >= 0) s.algo = c->env_algo;
    if (c->env_chunk) s.chunk_bytes = c->env_chunk;
    if (s.algo < hcclAlgoAuto || s.algo > hcclAlgoRhd) return fail(hcclInvalidArgument, "unknown algorithm");
    if (s.order < hcclOrderAscending || s.order > hcclOrderHalving) return fail(hcclInvalidArgument, "unknown order");
    if (s.phases < hcclPhasesAuto || s.phases > hcclPhasesLevels) return fail(hcclInvalidArgument, "unknown phase mode");
    return hcclSuccess;
}

hcclResult_t check_comm(hcclComm_t comm) {
    if (!comm) return fail(hcclInvalidArgument, "null communicator");
    return hcclSuccess;
}

hcclResult_t check_ptr_arrays(const void* a, const void* b) {
    if (!a || !b) return fail(hcclInvalidArgument, "null buffer array");
    return hcclSuccess;
}

}  // namespace

extern "C" {

hcclResult_t hccl_config_init(hcclConfig_t* cfg) {
    if (!cfg) return fail(hcclInvalidArgument, "null config");
    std::memset(cfg, 0, sizeof *cfg);
    cfg->algo = hcclAlgoAuto;
    cfg->fuse = 1;
    return hcclSuccess;
}

hcclResult_t hccl_comm_create(int nranks, int device, const hcclConfig_t* cfg, hcclComm_t* out) {
    if (!out) return fail(hcclInvalidArgument, "null output pointer");
    *out = nullptr;
    if (nranks < 1 || nranks > HCCL_MAX_RANKS) return fail(hcclInvalidArgument, "nranks must be in [1, 64]");
    auto c = std::make_unique<hcclComm>();
    c->nranks = nranks;
    c->device = device < 0 ? HCCL_NO_DEVICE : device;
    if (cfg) c->cfg = *cfg;
    else hccl_config_init(&c->cfg);
    read_env(c.get());
    if (c->device != HCCL_NO_DEVICE) {
        int n = 0;
        hipError_t e = hipGetDeviceCount(&n);
        if (e != hipSuccess || device >= n) return fail(hcclInvalidArgument, "no such HIP device");
        DeviceGuard guard(c->device);
        e = hipDeviceGetAttribute(&c->cus, hipDeviceAttributeMultiprocessorCount, c->device);
        if (e != hipSuccess) return hip_fail(e, "device attributes");
        int khz = 0;
        if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, c->device) == hipSuccess && khz > 0)
            c->wall_clock_khz = (uint64_t)khz;
        c->inline_single_step = !(std::getenv("HCCL_INLINE") && std::strcmp(std::getenv("HCCL_INLINE"), "0") == 0);
        const char* disp = std::getenv("HCCL_DISPATCH");
        c->dispatch_mode = !disp ? 0 : std::strcmp(disp, "static") == 0 ? 1 : std::strcmp(disp, "dynamic") == 0 ? 2 : 0;
        const char* bpc = std::getenv("HCCL_BLOCKS_PER_CU");
        for (int k = 0; k < kNumKinds; ++k) {
            if (k > SIG_INT32 && k < kKindCopyOnly) continue;  // no kernel of its own
            e = executor_occupancy(k, &c->blocks_per_cu[k]);
            if (e != hipSuccess) return hip_fail(e, "executor occupancy");
            if (bpc && std::atoi(bpc) > 0) c->blocks_per_cu[k] = std::min(c->blocks_per_cu[k], std::atoi(bpc));
        }
        e = hipEventCreateWithFlags(&c->scratch_done, hipEventDisableTiming);
        if (e != hipSuccess) return hip_fail(e, "scratch event");
        e = hipStreamCreateWithFlags(&c->setup_stream, hipStreamNonBlocking);
        if (e != hipSuccess) return hip_fail(e, "setup stream");
        e = hipMalloc(&c->d_error, sizeof(ErrorRecord));
        if (e != hipSuccess) return fail(hcclOutOfMemory, "error record allocation failed");
        // cleared on the communicator's own stream and waited for: launches go to the caller's
        // streams, which need not be ordered after the null stream
        e = launch_fill_u32((uint32_t*)c->d_error, sizeof(ErrorRecord) / sizeof(uint32_t), 0u, c->setup_stream);
        if (e == hipSuccess) e = hipStreamSynchronize(c->setup_stream);
        if (e != hipSuccess) return hip_fail(e, "error record init");
        // the device address of the static workspace, looked up once per device (allocation-free calls)
        void* ws = nullptr;
        e = workspace_address(&ws);
        if (e == hipSuccess) c->workspace = ws;
        else c->workspace_error = hipGetErrorString(e);
    }
    hlog(c.get(), 2, "created: %d ranks on device %d (%d CUs)%s%s", c->nranks, c->device, c->cus,
         c->env_algo >= 0 ? ", schedule forced by HCCL_ALGO" : "", c->env_chunk ? ", chunk forced by HCCL_CHUNK_BYTES" : "");
    *out = c.release();
    return hcclSuccess;
}

hcclResult_t hccl_comm_destroy(hcclComm_t comm) {
    if (!comm) return hcclSuccess;
    {
        DeviceGuard guard(comm->device);
        (void)hccl_resident_stop(comm);
        if (comm->device != HCCL_NO_DEVICE) (void)hipDeviceSynchronize();
        for (auto& p : comm->cache) free_program(p.get());
        for (auto& p : comm->retired) free_program(p.get());
        comm->cache.clear();
        comm->retired.clear();
        if (comm->d_scratch) (void)hipFree(comm->d_scratch);
        for (void* p : comm->retired_scratch) (void)hipFree(p);
        if (comm->d_error) (void)hipFree(comm->d_error);
        if (comm->d_trace) (void)hipFree(comm->d_trace);
        if (comm->scratch_done) (void)hipEventDestroy(comm->scratch_done);
        if (comm->setup_stream) (void)hipStreamDestroy(comm->setup_stream);
    }
    delete comm;
    return hcclSuccess;
}

hcclResult_t hccl_comm_set_config(hcclComm_t comm, const hcclConfig_t* cfg) {
    if (check_comm(comm) != hcclSuccess) return hcclInvalidArgument;
    if (!cfg) return fail(hcclInvalidArgument, "null config");
    comm->cfg = *cfg;
    return hcclSuccess;
}

}  // extern "C"

namespace {

// Argument checks of an all-reduce and its collective spec.
hcclResult_t allreduce_spec(hcclComm_t comm, const void* const* sendbufs, void* const* recvbufs, size_t count,
                            hcclDataType_t dtype, hcclRedOp_t op, CollectiveSpec& s) {
    hcclResult_t r;
    if ((r = check_comm(comm)) || (r = check_ptr_arrays(sendbufs, recvbufs)) || (r = check_dtype(dtype)) ||
        (r = check_op(op)))
        return r;
    const int P = comm->nranks;
    const size_t es = dtype_size((uint32_t)dtype);
    bool in_place = true;
    std::vector<Range> v;
    for (int i = 0; i < P; ++i) {
        v.push_back({(uintptr_t)sendbufs[i], (uintptr_t)sendbufs[i] + count * es, i});
        v.push_back({(uintptr_t)recvbufs[i], (uintptr_t)recvbufs[i] + count * es, P + i});
        in_place &= (sendbufs[i] == recvbufs[i]);
    }
    if (count) {
        if (!in_place)
            for (int i = 0; i < P; ++i)
                if (sendbufs[i] == recvbufs[i])
                    return fail(hcclInvalidArgument, "allreduce in place must be in place on every rank");
        r = check_buffers(v, es, [&](const Range& a, const Range& b) {
            return in_place && (a.id % P == b.id % P) && a.lo == b.lo && a.hi == b.hi;
        });
        if (r) return r;
    }
    if ((r = fill_spec(comm, s, COLL_ALLREDUCE, dtype, op))) return r;
    s.count = count;
    s.in_place = in_place && count > 0;
    return hcclSuccess;
}

// Host-only program of an allocation-free call: lowered, fused, packed (and validated on
// request), kept in a small cache on the communicator. Only host memory is used.
hcclResult_t host_program(hcclComm* c, const CollectiveSpec& s, const HostProgram*& out, bool& hit,
                          double& compile_us) {
    for (auto it = c->host_cache.begin(); it != c->host_cache.end(); ++it) {
        if (it->first == s) {
            if (it != c->host_cache.begin()) c->host_cache.splice(c->host_cache.begin(), c->host_cache, it);
            out = c->host_cache.front().second.get();
            hit = true;
            compile_us = 0;
            return hcclSuccess;
        }
    }
    hit = false;
    const auto t0 = std::chrono::steady_clock::now();
    auto hp = std::make_unique<HostProgram>();
    std::string err;
    if (!lower(s, *hp, err)) return fail(hcclUnsupported, err);
    if (s.fuse) fuse(*hp);
    if (!finalize(*hp, s.tile_bytes, err)) return fail(hcclInternalError, err);
    if ((c->cfg.validate || env_flag("HCCL_VALIDATE")) && !validate(*hp, s, err))
        return fail(hcclInternalError, "program validation failed: " + err);
    compile_us = std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count();
    c->host_cache.emplace_front(s, std::move(hp));
    while (c->host_cache.size() > 16) {
        if (c->last_prog == c->host_cache.back().second.get()) c->last_prog = nullptr;
        c->host_cache.pop_back();
    }
    out = c->host_cache.front().second.get();
    return hcclSuccess;
}

uint64_t align256(uint64_t x) { return (x + 255) & ~uint64_t(255); }

}  // namespace

extern "C" {

hcclResult_t hccl_allreduce(hcclComm_t comm, const void* const* sendbufs, void* const* recvbufs, size_t count,
                            hcclDataType_t dtype, hcclRedOp_t op, void* stream) {
    CollectiveSpec s;
    hcclResult_t r = allreduce_spec(comm, sendbufs, recvbufs, count, dtype, op, s);
    if (r != hcclSuccess) return r;
    return run(comm, s, sendbufs, recvbufs, stream);
}

hcclResult_t hccl_allreduce_noalloc(hcclComm_t comm, const void* const* sendbufs, void* const* recvbufs,
                                    size_t count, hcclDataType_t dtype, hcclRedOp_t op, void* stream) {
    CollectiveSpec s;
    hcclResult_t r = allreduce_spec(comm, sendbufs, recvbufs, count, dtype, op, s);
    if (r != hcclSuccess) return r;
    if (comm->device == HCCL_NO_DEVICE)
        return fail(hcclInvalidArgument, "hccl_allreduce_noalloc needs a communicator with a device");
    if (comm->group_depth > 0) return fail(hcclUnsupported, "hccl_allreduce_noalloc cannot be recorded in a group");
    if (comm->resident)
        return fail(hcclUnsupported, "hccl_allreduce_noalloc is launched on its stream, not handed to the resident executor");
    if (comm->has_trigger)
        return fail(hcclUnsupported, "a trigger is set for the next work packet; hccl_allreduce_noalloc takes none");
    if (!comm->workspace)
        return fail(hcclHipError, "the static workspace is not available on this device: " + comm->workspace_error);
    DeviceGuard guard(comm->device);
    const HostProgram* hp = nullptr;
    bool hit = false;
    double compile_us = 0;
    if ((r = host_program(comm, s, hp, hit, compile_us)) != hcclSuccess) return r;
    describe(comm->last, {s}, *hp, hit, compile_us);
    comm->last_prog = hp;
    if (hp->ntiles == 0) return hcclSuccess;

    // workspace layout of this call: program image, counters, FP32 partials
    const uint64_t off_state = align256(hp->image.size());
    const uint64_t off_scratch = align256(off_state + (uint64_t)hp->nstate * sizeof(uint32_t));
    const uint64_t need = off_scratch + hp->scratch_bytes;
    if (need > workspace_bytes())
        return fail(hcclInvalidArgument, "hccl_allreduce_noalloc: this all-reduce needs " + std::to_string(need) +
                                             " bytes of workspace (program, counters and partials); the static "
                                             "workspace holds " + std::to_string(workspace_bytes()));
    char* ws = (char*)comm->workspace;
    hipStream_t st = (hipStream_t)stream;
    LaunchArgs a;
    std::memset(&a, 0, sizeof a);
    a.prog = (const uint8_t*)ws;
    a.state = (uint32_t*)(ws + off_state);
    a.error = comm->d_error;
    const int P = s.P;
    for (int i = 0; i < P; ++i) {
        a.bufs[send_buf(i)] = (char*)sendbufs[i];
        a.bufs[recv_buf(P, i)] = (char*)recvbufs[i];
    }
    a.bufs[scratch_buf(P)] = ws + off_scratch;
    a.dynamic = use_tickets(comm, *hp, false) ? 1u : 0u;
    const uint64_t ms = comm->cfg.timeout_ms ? comm->cfg.timeout_ms : 2000u;
    a.timeout_ticks = ms * comm->wall_clock_khz;
    uint32_t blocks = 0;
    int kind = launch_shape(comm, *hp, 0, a, 2u * (uint32_t)P, st, blocks);
    comm->last.workers = a.nworkers;
    comm->last.tickets = a.dynamic;
    hipError_t e;
    if (hp->nphase() == 1 && inline_eligible(comm, *hp, false)) {
        comm->last.inline_launch = 1;
        e = launch_inline_step(*hp, a, blocks, kind, st);
        if (e != hipSuccess) return hip_fail(e, "inline executor launch");
        return hcclSuccess;
    }
    // the image goes in with a copy on the stream, the counters start from zero (a fill kernel),
    // the partials need no clearing: every one is written before it is read
    e = hipMemcpyAsync(ws, hp->image.data(), hp->image.size(), hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return hip_fail(e, "program copy into the static workspace");
    e = launch_fill_u32(a.state, hp->nstate, 0u, st);
    if (e != hipSuccess) return hip_fail(e, "counter clear in the static workspace");
    for (uint32_t q = 0; q < hp->nphase(); ++q) {
        if (q > 0) {
            kind = launch_shape(comm, *hp, q, a, 2u * (uint32_t)P, st, blocks);
            comm->last.workers = std::max(comm->last.workers, a.nworkers);
        }
        e = launch_executor(a, blocks, kind, st);
        if (e != hipSuccess) return hip_fail(e, "executor launch");
    }
    return hcclSuccess;
}

hcclResult_t hccl_reduce_scatter(hcclComm_t comm, const void* const* sendbufs, void* const* recvbufs,
                                 size_t recvcount, hcclDataType_t dtype, hcclRedOp_t op, void* stream) {
    hcclResult_t r;
    if ((r = check_comm(comm)) || (r = check_ptr_arrays(sendbufs, recvbufs)) || (r = check_dtype(dtype)) ||
        (r = check_op(op)))
        return r;
    const int P = comm->nranks;
    const size_t es = dtype_size((uint32_t)dtype);
    std::vector<Range> v;
    for (int i = 0; i < P; ++i) {
        v.push_back({(uintptr_t)sendbufs[i], (uintptr_t)sendbufs[i] + (size_t)P * recvcount * es, i});
        v.push_back({(uintptr_t)recvbufs[i], (uintptr_t)recvbufs[i] + recvcount * es, P + i});
    }
    if (recvcount && (r = check_buffers(v, es, [](const Range&, const Range&) { return false; }))) return r;
    CollectiveSpec s;
    if ((r = fill_spec(comm, s, COLL_REDUCE_SCATTER, dtype, op))) return r;
    if (s.algo == hcclAlgoTwoLevel) return fail(hcclUnsupported, "the two-level schedule is for allreduce");
    s.count = recvcount;
    return run(comm, s, sendbufs, recvbufs, stream);
}

hcclResult_t hccl_allgather(hcclComm_t comm, const void* const* sendbufs, void* const* recvbufs, size_t sendcount,
                            hcclDataType_t dtype, void* stream) {
    hcclResult_t r;
    if ((r = check_comm(comm)) || (r = check_ptr_arrays(sendbufs, recvbufs)) || (r = check_dtype(dtype))) return r;
    const int P = comm->nranks;
    const size_t es = dtype_size((uint32_t)dtype);
    std::vector<Range> v;
    for (int i = 0; i < P; ++i) {
        v.push_back({(uintptr_t)sendbufs[i], (uintptr_t)sendbufs[i] + sendcount * es, i});
        v.push_back({(uintptr_t)recvbufs[i], (uintptr_t)recvbufs[i] + (size_t)P * sendcount * es, P + i});
    }
    if (sendcount && (r = check_buffers(v, es, [](const Range&, const Range&) { return false; }))) return r;
    CollectiveSpec s;
    if ((r = fill_spec(comm, s, COLL_ALLGATHER, dtype, hcclSum))) return r;
    if (s.algo == hcclAlgoTwoLevel) return fail(hcclUnsupported, "the two-level schedule is for allreduce");
    s.count = sendcount;
    return run(comm, s, sendbufs, recvbufs, stream);
}

hcclResult_t hccl_alltoallv(hcclComm_t comm, const void* const* sendbufs, const size_t* sendcounts,
                            const size_t* sdispls, void* const* recvbufs, const size_t* recvcounts,
                            const size_t* rdispls, hcclDataType_t dtype, void* stream) {
    hcclResult_t r;
    if ((r = check_comm(comm)) || (r = check_ptr_arrays(sendbufs, recvbufs)) || (r = check_dtype(dtype))) return r;
    if (!sendcounts || !sdispls || !recvcounts || !rdispls) return fail(hcclInvalidArgument, "null count array");
    const int P = comm->nranks;
    const size_t es = dtype_size((uint32_t)dtype);
    const size_t PP = (size_t)P * P;
    CollectiveSpec s;
    if ((r = fill_spec(comm, s, COLL_ALLTOALLV, dtype, hcclSum))) return r;
    s.sendcounts.assign(sendcounts, sendcounts + PP);
    s.sdispls.assign(sdispls, sdispls + PP);
    s.recvcounts.assign(recvcounts, recvcounts + PP);
    s.rdispls.assign(rdispls, rdispls + PP);
    const uint64_t kLimit = (1ull << 62) / 8;
    for (int src = 0; src < P; ++src) {
        for (int dst = 0; dst < P; ++dst) {
            uint64_t n = sendcounts[(size_t)src * P + dst];
            if (recvcounts[(size_t)dst * P + src] != n)
                return fail(hcclInvalidArgument, "recvcounts[dst*P+src] must equal sendcounts[src*P+dst]");
            if (n > kLimit || sdispls[(size_t)src * P + dst] > kLimit || rdispls[(size_t)dst * P + src] > kLimit)
                return fail(hcclInvalidArgument, "count or displacement out of range");
        }
    }
    // receive ranges of one destination must not overlap
    for (int dst = 0; dst < P; ++dst) {
        std::vector<std::pair<uint64_t, uint64_t>> rr;
        for (int src = 0; src < P; ++src) {
            uint64_t n = recvcounts[(size_t)dst * P + src];
            if (n) rr.push_back({rdispls[(size_t)dst * P + src], rdispls[(size_t)dst * P + src] + n});
        }
        std::sort(rr.begin(), rr.end());
        for (size_t i = 1; i < rr.size(); ++i)
            if (rr[i].first < rr[i - 1].second) return fail(hcclInvalidArgument, "receive ranges overlap");
    }
    // every send / receive buffer span must be disjoint from every other
    BufferSizes sizes = buffer_sizes(s, 0);
    std::vector<Range> v;
    for (int i = 0; i < P; ++i) {
        v.push_back({(uintptr_t)sendbufs[i], (uintptr_t)sendbufs[i] + sizes.bytes[send_buf(i)], i});
        v.push_back({(uintptr_t)recvbufs[i], (uintptr_t)recvbufs[i] + sizes.bytes[recv_buf(P, i)], P + i});
    }
    // send buffers may alias each other (read-only); nothing may alias a receive buffer
    if ((r = check_buffers(v, es, [&](const Range& a, const Range& b) { return a.id < P && b.id < P; })))
        return r;
    return run(comm, s, sendbufs, recvbufs, stream);
}

hcclResult_t hccl_alltoallv_dynamic(hcclComm_t comm, const void* const* sendbufs, const int64_t* sendcounts,
                                    const int64_t* sdispls, void* const* recvbufs, int64_t* recvcounts,
                                    const int64_t* rdispls, size_t row_elems, size_t send_capacity,
                                    size_t recv_capacity, hcclDataType_t dtype, void* stream) {
    hcclResult_t r;
    if ((r = check_comm(comm)) || (r = check_ptr_arrays(sendbufs, recvbufs)) || (r = check_dtype(dtype))) return r;
    if (!sendcounts) return fail(hcclInvalidArgument, "null count array");
    if (row_elems == 0) return fail(hcclInvalidArgument, "row_elems must be at least 1");
    const int P = comm->nranks;
    const uint64_t es = dtype_size((uint32_t)dtype);
    const uint64_t kLimit = (1ull << 62) / 8;
    if (row_elems > kLimit || send_capacity > kLimit / row_elems / es || recv_capacity > kLimit / row_elems / es)
        return fail(hcclInvalidArgument, "capacity out of range");
    const void* meta[kMetaPerDynamicCall] = {sendcounts, sdispls, rdispls, recvcounts};
    for (const void* m : meta)
        if ((uintptr_t)m % alignof(int64_t)) return fail(hcclInvalidArgument, "metadata arrays must be 8-byte aligned");
    CollectiveSpec s;
    if ((r = fill_spec(comm, s, COLL_ALLTOALLV_DYNAMIC, dtype, hcclSum))) return r;
    s.row_elems = row_elems;
    s.send_cap = send_capacity;
    s.recv_cap = recv_capacity;
    s.dyn_sdispls = sdispls != nullptr;
    s.dyn_rdispls = rdispls != nullptr;
    s.dyn_recvcounts = recvcounts != nullptr;
    // ids: sends [0, P), receives [P, 2P), metadata 2P + slot. Sends and the metadata inputs
    // are only read and may alias each other; receives and the count output alias nothing.
    const uint64_t sb = send_capacity * row_elems * es, rb = recv_capacity * row_elems * es;
    const uint64_t mbytes = (uint64_t)P * P * sizeof(int64_t);
    std::vector<Range> v;
    for (int i = 0; i < P; ++i) {
        v.push_back({(uintptr_t)sendbufs[i], (uintptr_t)sendbufs[i] + sb, i});
        v.push_back({(uintptr_t)recvbufs[i], (uintptr_t)recvbufs[i] + rb, P + i});
    }
    for (int m = 0; m < kMetaPerDynamicCall; ++m)
        if (meta[m]) v.push_back({(uintptr_t)meta[m], (uintptr_t)meta[m] + mbytes, 2 * P + m});
    auto read_only = [&](int id) { return id < P || (id >= 2 * P && id < 2 * P + META_RECVCOUNTS); };
    if ((r = check_buffers(v, es, [&](const Range& a, const Range& b) { return read_only(a.id) && read_only(b.id); })))
        return r;
    std::vector<void*> mv;
    for (const void* m : meta) mv.push_back(const_cast<void*>(m));
    return run(comm, s, sendbufs, recvbufs, stream, std::move(mv));
}

hcclResult_t hccl_set_trigger(hcclComm_t comm, const hcclTrigger_t* t) {
    if (check_comm(comm) != hcclSuccess) return hcclInvalidArgument;
    if (!t) {
        comm->has_trigger = false;
        return hcclSuccess;
    }
    if (t->wait_cmp < hcclCmpEq || t->wait_cmp > hcclCmpLt) return fail(hcclInvalidArgument, "unknown comparator");
    if ((uintptr_t)t->wait_addr % 8 || (uintptr_t)t->done_addr % 8)
        return fail(hcclInvalidArgument, "trigger words must be 8-byte aligned");
    if (t->wait_addr && (const void*)t->wait_addr == (const void*)t->done_addr)
        return fail(hcclInvalidArgument, "the wait and completion words must differ");
    comm->trigger = *t;
    comm->has_trigger = true;
    return hcclSuccess;
}

hcclResult_t hccl_group_start(hcclComm_t comm) {
    if (check_comm(comm) != hcclSuccess) return hcclInvalidArgument;
    comm->group_depth += 1;
    return hcclSuccess;
}

hcclResult_t hccl_group_end(hcclComm_t comm) {
    if (check_comm(comm) != hcclSuccess) return hcclInvalidArgument;
    if (comm->group_depth == 0) return fail(hcclInvalidArgument, "hccl_group_end without hccl_group_start");
    if (--comm->group_depth > 0) return hcclSuccess;
    std::vector<Call> calls;
    calls.swap(comm->pending);
    if (calls.empty()) return hcclSuccess;
    for (const Call& k : calls)
        if (k.stream != calls[0].stream) return fail(hcclInvalidArgument, "calls of one group must use one stream");
    uint32_t nbuf = 0, nmeta = 0;
    for (const Call& k : calls) {
        nbuf += 2 * (uint32_t)k.spec.P;
        nmeta += meta_buffers(k.spec);
    }
    if (nbuf > 2u * (uint32_t)kMaxRanks) return fail(hcclUnsupported, "a group may name at most 128 rank buffers");
    if (nmeta > (uint32_t)kMaxMetaBuffers) return fail(hcclUnsupported, "a group may hold at most two dynamic calls");
    // buffers of different calls must not overlap unless both are only read (each call was
    // checked on its own): ids are 2 * call + 1 for what a call writes, 2 * call for what it reads
    if (calls.size() > 1) {
        std::vector<Range> v;
        int id = 0;
        for (const Call& k : calls) {
            BufferSizes sz = buffer_sizes(k.spec, 0);
            for (int i = 0; i < k.spec.P; ++i) {
                v.push_back({(uintptr_t)k.send[i], (uintptr_t)k.send[i] + sz.bytes[send_buf(i)], 2 * id});
                v.push_back({(uintptr_t)k.recv[i], (uintptr_t)k.recv[i] + sz.bytes[recv_buf(k.spec.P, i)], 2 * id + 1});
            }
            const uint64_t mbytes = (uint64_t)k.spec.P * k.spec.P * sizeof(int64_t);
            for (size_t m = 0; m < k.meta.size(); ++m)
                if (k.meta[m])
                    v.push_back({(uintptr_t)k.meta[m], (uintptr_t)k.meta[m] + mbytes,
                                 2 * id + (m == META_RECVCOUNTS ? 1 : 0)});
            ++id;
        }
        hcclResult_t r = check_buffers(v, 1, [](const Range& a, const Range& b) {
            return a.id / 2 == b.id / 2 || (a.id % 2 == 0 && b.id % 2 == 0);
        });
        if (r != hcclSuccess) return fail(hcclInvalidArgument, "buffers of different calls in a group overlap");
    }
    return run_packet(comm, calls);
}

const char* hccl_get_last_error(void) { return g_last_error.c_str(); }

const char* hccl_result_string(hcclResult_t r) {
    switch (r) {
        case hcclSuccess: return "hcclSuccess";
        case hcclInvalidArgument: return "hcclInvalidArgument";
        case hcclUnsupported: return "hcclUnsupported";
        case hcclHipError: return "hcclHipError";
        case hcclOutOfMemory: return "hcclOutOfMemory";
        case hcclTimeout: return "hcclTimeout";
        case hcclInternalError: return "hcclInternalError";
    }
    return "unknown hcclResult_t";
}

namespace {

// The result code and message of a device error record.
hcclResult_t device_error(uint32_t code, uint32_t desc, uint32_t tile) {
    char buf[200];
    if (code == 2) {
        std::snprintf(buf, sizeof buf,
                      "the device-resident layout read by step %u was invalid (row or column %u): "
                      "a count or offset left its buffer, or receive ranges overlapped; nothing was moved",
                      desc, tile);
        return fail(hcclInvalidArgument, buf);
    }
    if (code == 3) {
        std::snprintf(buf, sizeof buf,
                      "the trigger word did not satisfy its comparison within the watchdog limit "
                      "(workgroup %u gave up); the collective's outputs are unspecified",
                      tile);
        return fail(hcclTimeout, buf);
    }
    std::snprintf(buf, sizeof buf, "a dependency wait of step %u (tile %u) exceeded the watchdog limit", desc, tile);
    return fail(hcclTimeout, buf);
}

}  // namespace

hcclResult_t hccl_get_async_error(hcclComm_t comm) {
    if (check_comm(comm) != hcclSuccess) return hcclInvalidArgument;
    if (comm->device == HCCL_NO_DEVICE) return hcclSuccess;
    if (comm->resident)
        return fail(hcclInvalidArgument, "the resident executor is running: hccl_resident_wait reports its errors");
    DeviceGuard guard(comm->device);
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "synchronize");
    ErrorRecord rec;
    e = hipMemcpy(&rec, comm->d_error, sizeof rec, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "read error record");
    if (rec.code == 0) return hcclSuccess;
    // cleared before anything else can be enqueued (the caller's streams need not follow the
    // null stream)
    e = launch_fill_u32((uint32_t*)comm->d_error, sizeof(ErrorRecord) / sizeof(uint32_t), 0u, comm->setup_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(comm->setup_stream);
    if (e != hipSuccess) return hip_fail(e, "clear error record");
    return device_error(rec.code, rec.desc, rec.tile);
}

hcclResult_t hccl_resident_start(hcclComm_t comm, uint32_t blocks, uint32_t idle_ms) {
    if (check_comm(comm) != hcclSuccess) return hcclInvalidArgument;
    if (comm->device == HCCL_NO_DEVICE) return fail(hcclInvalidArgument, "the resident executor needs a device");
    if (comm->resident) return fail(hcclInvalidArgument, "the resident executor is already running");
    if (comm->group_depth > 0) return fail(hcclInvalidArgument, "hccl_resident_start inside a group");
    DeviceGuard guard(comm->device);
    int per_cu = 0;
    hipError_t e = resident_occupancy(&per_cu);
    if (e != hipSuccess) return hip_fail(e, "resident executor occupancy");
    const uint32_t most = (uint32_t)comm->cus * (uint32_t)std::max(per_cu, 0);
    if (blocks == 0) blocks = std::min<uint32_t>(kResidentDefaultBlocks, most);
    if (blocks == 0 || blocks > most)
        return fail(hcclInvalidArgument, "blocks must fit on the device at once (at most " + std::to_string(most) + ")");
    if (idle_ms == 0) idle_ms = kResidentDefaultIdleMs;
    if (idle_ms > kResidentMaxIdleMs) return fail(hcclInvalidArgument, "idle_ms is above the limit of 10 minutes");

    void* q = nullptr;
    e = hipHostMalloc(&q, sizeof(ResidentQueue), hipHostMallocCoherent | hipHostMallocMapped);
    if (e != hipSuccess) return fail(hcclOutOfMemory, "pinned doorbell allocation failed");
    std::memset(q, 0, sizeof(ResidentQueue));
    void* qdev = nullptr;
    uint32_t* ctl = nullptr;
    hipStream_t st = nullptr;
    e = hipHostGetDevicePointer(&qdev, q, 0);
    // control words, then two device mirrors of packet arguments (one is filled ahead)
    const size_t ctl_bytes = 64 + 2 * sizeof(LaunchArgs);
    if (e == hipSuccess) e = hipMalloc(&ctl, ctl_bytes);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&st, hipStreamNonBlocking);
    // cleared on the executor's own stream: a non-blocking stream is not ordered after work on
    // the null stream, so a clear issued there could land after the executor has started
    if (e == hipSuccess) e = launch_fill_u32(ctl, ctl_bytes / sizeof(uint32_t), 0u, st);
    ResidentArgs r;
    std::memset(&r, 0, sizeof r);
    r.q = (ResidentQueue*)qdev;
    r.ctl = ctl;
    r.mirror = (uint64_t*)((char*)ctl + 64);
    r.error = comm->d_error;
    r.timeout_ticks = (comm->cfg.timeout_ms ? comm->cfg.timeout_ms : 2000u) * comm->wall_clock_khz;
    r.idle_ticks = (uint64_t)idle_ms * comm->wall_clock_khz;
    if (e == hipSuccess) e = launch_resident(r, blocks, st);
    if (e != hipSuccess) {
        if (st) (void)hipStreamDestroy(st);
        if (ctl) (void)hipFree(ctl);
        (void)hipHostFree(q);
        return hip_fail(e, "resident executor start");
    }
    comm->rq = (ResidentQueue*)q;
    comm->d_ctl = ctl;
    comm->resident_stream = st;
    comm->resident_seq = 0;
    comm->resident = true;
    note_resident(comm->device, true);
    return hcclSuccess;
}

hcclResult_t hccl_resident_stop(hcclComm_t comm) {
    if (check_comm(comm) != hcclSuccess) return hcclInvalidArgument;
    if (!comm->resident) return hcclSuccess;
    DeviceGuard guard(comm->device);
    hcclResult_t r = hcclSuccess;
    if (!resident_exited(comm)) {
        const uint64_t k = comm->resident_seq + 1;
        const uint64_t ms = comm->cfg.timeout_ms ? comm->cfg.timeout_ms : 2000u;
        if (k > kResidentSlots) r = resident_wait_for(comm, k - kResidentSlots, ms);
        if (r == hcclSuccess) {
            ResidentSlot& slot = comm->rq->slots[(k - 1) % kResidentSlots];
            __atomic_store_n(&slot.seq, k | kResidentStop, __ATOMIC_RELEASE);
        }
    }
    // every wait of the executor is bounded, so this returns
    hipError_t e = hipStreamSynchronize(comm->resident_stream);
    (void)hipStreamDestroy(comm->resident_stream);
    (void)hipFree(comm->d_ctl);
    (void)hipHostFree(comm->rq);
    comm->resident_stream = nullptr;
    comm->d_ctl = nullptr;
    comm->rq = nullptr;
    comm->resident = false;
    note_resident(comm->device, false);
    if (e != hipSuccess) return hip_fail(e, "resident executor stop");
    return r;
}

hcclResult_t hccl_resident_wait(hcclComm_t comm, uint64_t seq, uint32_t timeout_ms) {
    if (check_comm(comm) != hcclSuccess) return hcclInvalidArgument;
    if (!comm->resident) return fail(hcclInvalidArgument, "the resident executor is not running");
    if (seq == 0) seq = comm->resident_seq;
    if (seq > comm->resident_seq) return fail(hcclInvalidArgument, "no packet with that number was submitted");
    hcclResult_t r = resident_wait_for(comm, seq, timeout_ms ? timeout_ms : 2000u);
    if (r != hcclSuccess) return r;
    const uint32_t code = __atomic_load_n(&comm->rq->error, __ATOMIC_ACQUIRE);
    if (code == 0) return hcclSuccess;
    const uint32_t desc = comm->rq->err_desc, tile = comm->rq->err_tile;
    __atomic_store_n(&comm->rq->error, 0u, __ATOMIC_RELEASE);
    return device_error(code, desc, tile);
}

hcclResult_t hccl_resident_last_seq(hcclComm_t comm, uint64_t* seq) {
    if (check_comm(comm) != hcclSuccess) return hcclInvalidArgument;
    if (!seq) return fail(hcclInvalidArgument, "null output");
    *seq = comm->resident_seq;
    return hcclSuccess;
}

hcclResult_t hccl_comm_trace(hcclComm_t comm, hcclTileTrace_t* out, size_t capacity, size_t* count,
                             uint64_t* clock_khz) {
    if (check_comm(comm) != hcclSuccess) return hcclInvalidArgument;
    if (!count) return fail(hcclInvalidArgument, "null count");
    if (capacity && !out) return fail(hcclInvalidArgument, "null trace output");
    static_assert(sizeof(hcclTileTrace_t) == sizeof(TileStamp), "trace record layout");
    *count = 0;
    if (clock_khz) *clock_khz = comm->wall_clock_khz;
    if (comm->device == HCCL_NO_DEVICE || comm->trace_tiles == 0) return hcclSuccess;
    if (comm->resident)
        return fail(hcclInvalidArgument, "the resident executor is running: stop it before reading the trace");
    DeviceGuard guard(comm->device);
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "synchronize");
    const size_t n = std::min<size_t>(capacity, comm->trace_tiles);
    if (n) {
        e = hipMemcpy(out, comm->d_trace, n * sizeof(TileStamp), hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e, "read trace");
    }
    *count = comm->trace_tiles;
    return hcclSuccess;
}

hcclResult_t hccl_comm_program_image(hcclComm_t comm, void* out, size_t capacity, size_t* size) {
    if (check_comm(comm) != hcclSuccess) return hcclInvalidArgument;
    if (!size) return fail(hcclInvalidArgument, "null size");
    if (capacity && !out) return fail(hcclInvalidArgument, "null output");
    *size = 0;
    if (!comm->last_prog) return hcclSuccess;
    const std::vector<uint8_t>& img = comm->last_prog->image;
    *size = img.size();
    if (capacity) std::memcpy(out, img.data(), std::min(capacity, img.size()));
    return hcclSuccess;
}

hcclResult_t hccl_comm_last_program(hcclComm_t comm, hcclProgramInfo_t* info) {
    if (check_comm(comm) != hcclSuccess) return hcclInvalidArgument;
    if (!info) return fail(hcclInvalidArgument, "null info");
    *info = comm->last;
    return hcclSuccess;
}

}  // extern "C"
