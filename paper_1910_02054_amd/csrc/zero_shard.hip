// zero_shard.hip -- host side of libzeroshard: the C ABI declared in
// include/zero_shard.h (argument checks, partition layout, fp32 constants,
// per-(device, stream) workspace, launches, skip-flag readback, profiling).
//
// ZeRO (arXiv 1910.02054): Sec. 5.1 (P_os: N_d equal partitions, rank i
// updates partition i), Sec. 5.2 (P_g: the rank holds only its partition's
// reduced gradients), Sec. 3.1 (mixed-precision Adam state), Sec. 6.2
// (constant-size buffers: the workspace does not grow with the shard).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdlib>
#include <cstdio>
#include <cstring>
#include <algorithm>
#include <atomic>
#include <chrono>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <utility>
#include <vector>

#include "zero_shard.h"
#include "shard_kernels.hpp"
#include "probe_kernels.hpp"
#include "host_common.hpp"

namespace zsh {

thread_local std::string t_err;
thread_local zero_step_stats_t t_stats;
thread_local bool t_have_stats = false;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_err = buf;
    return code;
}

// ---------------------------------------------------------------------------
// Production launch policy of the streaming kernels (template knobs in
// shard_kernels.hpp), chosen by measurement on MI355X in the two-kernel step
// flow.  The HBM efficiency of these streams peaks well below full occupancy,
// so the statistics pass (persistent grid) and the update (one tile per
// workgroup) are launched with an LDS reservation that caps resident
// workgroups per CU.  The statistics pass uses cache-allocating loads, which
// leaves part of the gradient in the Infinity Cache for the update.
// ---------------------------------------------------------------------------
constexpr int kStatsBlock = 64, kStatsUnroll = 4, kStatsPerCU = 8;
constexpr bool kStatsNTL = false, kStatsXCD = false;
constexpr int kAdamBlock = 64, kAdamUnroll = 1, kAdamPerCU = 12;
constexpr bool kAdamNTL = true, kAdamNTS = true, kAdamXCD = false, kAdamREV = false;
constexpr int64_t kAdamMaxBlocks = 1 << 26;
constexpr int kCopyBlock = 64, kCopyUnroll = 1;
constexpr bool kCopyNTL = true, kCopyNTS = true, kCopyXCD = false;
// One-launch small-shard step (k_small_step): shards of at most kSmallMaxNumel
// elements whose arrays share one misalignment, on a grid of at most
// kSmallMaxGrid workgroups (each totals every workgroup's partial).
#ifndef ZS_SMALL_MAX_NUMEL
#define ZS_SMALL_MAX_NUMEL (1 << 22)
#endif
constexpr int64_t kSmallMaxNumel = ZS_SMALL_MAX_NUMEL;
constexpr int64_t kSmallMaxGrid = 512;
// A grid takes at most 1/share of the device's co-resident capacity, where
// share is the number of hardware queues the process may use (at least
// kSmallCapShare; HIP gives a process four unless GPU_MAX_HW_QUEUES says
// otherwise), so the barrier-waiting workgroups of small steps running at once
// on every queue always fit on the device together.
#ifndef ZS_SMALL_CAP_SHARE
#define ZS_SMALL_CAP_SHARE 4
#endif
constexpr int64_t kSmallCapShare = ZS_SMALL_CAP_SHARE;

int64_t small_cap_share() {
    int64_t share = kSmallCapShare;
    if (const char* e = std::getenv("GPU_MAX_HW_QUEUES")) {
        const long q = std::strtol(e, nullptr, 10);
        if (q > share)
            share = q;
    }
    return share;
}
constexpr int kSmallV[4] = {1, 2, 4, 8};
#ifndef ZS_SMALL_FIRST_V
#define ZS_SMALL_FIRST_V 0
#endif
constexpr int kSmallFirstV = ZS_SMALL_FIRST_V;  // index into kSmallV of the first variant tried

// ---------------------------------------------------------------------------
// Launch planning.  One function decides every launch shape from n and the
// arrays' alignments, so tests and benchmarks exercise the same configuration.
// ---------------------------------------------------------------------------
struct Plan {
    int64_t ghead, gvec;   // statistics: unaligned head elements, 8-element vectors
    int stats_blocks;
    bool vec;              // update: vector path (all arrays share misalignment)
    int64_t head, nvec;    // update: head elements, 4-element vectors
    int64_t adam_blocks;
    int small_v;           // one-launch small-shard step: vectors per thread (0: not taken)
    int64_t small_grid;
};

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

Plan plan_step(const uint16_t* g, const float* th, const float* m, const float* v, const uint16_t* p, int64_t n,
               int ncu) {
    Plan pl{};
    // statistics: 16-byte vectors of the gradient, at most kStatsPerCU workgroups per CU
    const uintptr_t ga = reinterpret_cast<uintptr_t>(g);
    int64_t gh = (int64_t)(((16 - (ga & 15)) & 15) / 2);
    pl.ghead = gh < n ? gh : n;
    pl.gvec = (n - pl.ghead) / 8;
    int64_t sb = ceil_div(pl.gvec, (int64_t)kStatsBlock * kStatsUnroll);
    const int64_t scap = std::min<int64_t>((int64_t)ncu * kStatsPerCU, zs::kMaxStatsBlocks);
    pl.stats_blocks = (int)(sb < 1 ? 1 : (sb > scap ? scap : sb));
    // update: 4-element vectors (16-byte fp32, 8-byte fp16) need one common misalignment
    const int64_t ef[3] = {(int64_t)((reinterpret_cast<uintptr_t>(th) & 15) / 4),
                           (int64_t)((reinterpret_cast<uintptr_t>(m) & 15) / 4),
                           (int64_t)((reinterpret_cast<uintptr_t>(v) & 15) / 4)};
    const int64_t eh[2] = {(int64_t)((reinterpret_cast<uintptr_t>(g) & 7) / 2),
                           (int64_t)((reinterpret_cast<uintptr_t>(p) & 7) / 2)};
    pl.vec = ef[0] == ef[1] && ef[0] == ef[2] && ef[0] == eh[0] && ef[0] == eh[1];
    if (pl.vec) {
        int64_t h = (4 - ef[0]) & 3;
        pl.head = h < n ? h : n;
        pl.nvec = (n - pl.head) / 4;
        int64_t ab = ceil_div(pl.nvec, (int64_t)kAdamBlock * kAdamUnroll);
        pl.adam_blocks = ab < 1 ? 1 : (ab > kAdamMaxBlocks ? kAdamMaxBlocks : ab);
    } else {
        pl.head = pl.nvec = 0;
        int64_t ab = ceil_div(n, zs::kScalarBlock);
        pl.adam_blocks = ab < 1 ? 1 : (ab > kAdamMaxBlocks ? kAdamMaxBlocks : ab);
    }
    return pl;
}

// The one-launch small-shard step when the shard qualifies: the fewest vectors
// per thread whose grid fits both kSmallMaxGrid and the device's co-resident
// capacity for that kernel.
void plan_small(Plan* pl, int64_t n, const DevInfo* info) {
    pl->small_v = 0;
    pl->small_grid = 0;
    if (!pl->vec || n > kSmallMaxNumel)
        return;
    for (int k = kSmallFirstV; k < 4; ++k) {
        int64_t grid = ceil_div(pl->nvec, (int64_t)zs::kSmallBlock * kSmallV[k]);
        if (grid < 1)
            grid = 1;
        if (grid <= kSmallMaxGrid && grid <= info->small_cap[k] / info->small_share) {
            pl->small_v = kSmallV[k];
            pl->small_grid = grid;
            return;
        }
    }
}

// Dynamic LDS that caps the resident workgroups of `kernel` (launched with
// `block` threads) at `per_cu` per CU: an equal share of the CU's LDS minus the
// kernel's own static LDS, lowered granule by granule until the runtime's
// occupancy calculator admits `per_cu` workgroups.  *resident receives what
// the calculator reports for the returned reservation.
size_t occupancy_lds(const void* kernel, int block, int per_cu, const hipDeviceProp_t& prop, int* resident) {
    const size_t granule = 512;
    *resident = 0;
    hipFuncAttributes attr;
    if (hipFuncGetAttributes(&attr, kernel) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    const size_t fixed = (attr.sharedSizeBytes + granule - 1) & ~(granule - 1);
    const size_t share = ((size_t)prop.maxSharedMemoryPerMultiProcessor / (size_t)per_cu) & ~(granule - 1);
    const size_t cap = (size_t)prop.sharedMemPerBlock > fixed + granule ? prop.sharedMemPerBlock - fixed - granule : 0;
    size_t r = share > fixed ? share - fixed : 0;
    if (r > cap)
        r = cap;
    for (;;) {
        int blocks = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel, block, r) != hipSuccess) {
            (void)hipGetLastError();
            return 0;
        }
        *resident = blocks;
        if (blocks >= per_cu || r < granule)
            return r;
        r -= granule;
    }
}

const void* small_kernel(int v) {
    switch (v) {
    case 1: return reinterpret_cast<const void*>(zs::k_small_step<1>);
    case 2: return reinterpret_cast<const void*>(zs::k_small_step<2>);
    case 4: return reinterpret_cast<const void*>(zs::k_small_step<4>);
    default: return reinterpret_cast<const void*>(zs::k_small_step<8>);
    }
}

// ---------------------------------------------------------------------------
// Per-device facts, computed once per device into a fixed table.
// ---------------------------------------------------------------------------
std::mutex g_dev_mu;
DevInfo g_dev[kMaxDevices];
std::atomic<bool> g_dev_ready[kMaxDevices];

int dev_info(int dev, const DevInfo** out) {
    if (dev < 0 || dev >= kMaxDevices)
        return fail(ZERO_EINVAL, "device %d is outside the library's table of %d devices", dev, kMaxDevices);
    if (!g_dev_ready[dev].load(std::memory_order_acquire)) {
        std::lock_guard<std::mutex> lk(g_dev_mu);
        if (!g_dev_ready[dev].load(std::memory_order_relaxed)) {
            hipDeviceProp_t prop;
            HIP_TRY(hipGetDeviceProperties(&prop, dev));
            DevInfo d;
            d.ncu = prop.multiProcessorCount;
            d.stats_lds = occupancy_lds(
                reinterpret_cast<const void*>(zs::k_stats<kStatsBlock, kStatsUnroll, kStatsNTL, kStatsXCD>),
                kStatsBlock, kStatsPerCU, prop, &d.stats_resident);
            d.adam_lds = occupancy_lds(
                reinterpret_cast<const void*>(
                    zs::k_adam_vec<kAdamBlock, kAdamUnroll, kAdamNTL, kAdamNTS, kAdamXCD, kAdamREV, false>),
                kAdamBlock, kAdamPerCU, prop, &d.adam_resident);
            d.probe_adam_lds = occupancy_lds(
                reinterpret_cast<const void*>(zs::k_probe_adam<kAdamBlock, kAdamUnroll, kAdamNTL, kAdamNTS, kAdamXCD>),
                kAdamBlock, kAdamPerCU, prop, &d.probe_adam_resident);
            for (int k = 0; k < 4; ++k) {
                int per_cu = 0;
                if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, small_kernel(kSmallV[k]), zs::kSmallBlock,
                                                                 0) != hipSuccess) {
                    (void)hipGetLastError();
                    per_cu = 0;
                }
                d.small_cap[k] = (int64_t)per_cu * d.ncu;
            }
            d.small_share = small_cap_share();
            g_dev[dev] = d;
            g_dev_ready[dev].store(true, std::memory_order_release);
        }
    }
    *out = &g_dev[dev];
    return ZERO_OK;
}

// ---------------------------------------------------------------------------
// Per-(device, stream) contexts (struct Ctx in host_common.hpp).
// ---------------------------------------------------------------------------

std::mutex g_ctx_mu;
std::map<std::pair<int, hipStream_t>, std::shared_ptr<Ctx>> g_ctx;

void free_ctx_buffers(Ctx* c) {
    if (c->part) (void)hipFree(c->part);
    if (c->res) (void)hipFree(c->res);
    if (c->sync) (void)hipFree(c->sync);
    if (c->host) (void)hipHostFree(c->host);
    c->part = nullptr;
    c->res = nullptr;
    c->sync = nullptr;
    c->host = c->host_dev = nullptr;
}

// Allocations made while `stream` may be capturing a graph switch this thread
// to the relaxed capture mode, in which allocating is permitted.
struct RelaxedCapture {
    bool on = false;
    hipStreamCaptureMode mode = hipStreamCaptureModeRelaxed;
    explicit RelaxedCapture(hipStream_t stream) {
        hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(stream, &st) != hipSuccess) {
            (void)hipGetLastError();
            return;
        }
        if (st != hipStreamCaptureStatusNone && hipThreadExchangeStreamCaptureMode(&mode) == hipSuccess)
            on = true;
    }
    ~RelaxedCapture() {
        if (on)
            (void)hipThreadExchangeStreamCaptureMode(&mode);
    }
};

int new_ctx(int dev, hipStream_t stream, const DevInfo* info, std::shared_ptr<Ctx>* out) {
    std::shared_ptr<Ctx> c = std::make_shared<Ctx>();
    c->dev = dev;
    c->stream = stream;
    c->info = info;
    RelaxedCapture relaxed(stream);
    // the barrier words are zeroed on the stream before the first small-shard launch
    bool ok = hipMalloc(reinterpret_cast<void**>(&c->part), sizeof(zs::Partial) * zs::kMaxStatsBlocks) == hipSuccess &&
              hipMalloc(reinterpret_cast<void**>(&c->res), sizeof(zs::Result)) == hipSuccess &&
              hipMalloc(reinterpret_cast<void**>(&c->sync), sizeof(uint64_t) * zs::kSyncWords) == hipSuccess &&
              hipHostMalloc(reinterpret_cast<void**>(&c->host), sizeof(zs::Result),
                            hipHostMallocMapped | hipHostMallocCoherent) == hipSuccess &&
              hipHostGetDevicePointer(reinterpret_cast<void**>(&c->host_dev), c->host, 0) == hipSuccess;
    if (!ok) {
        free_ctx_buffers(c.get());
        (void)hipGetLastError();
        return fail(ZERO_ENOMEM, "could not allocate the step workspace on device %d", dev);
    }
    std::memset(c->host, 0, sizeof(zs::Result));
    *out = std::move(c);
    return ZERO_OK;
}

// The device of the calling thread, and a check that `stream` belongs to it.
int current_device(hipStream_t stream, int* dev) {
    HIP_TRY(hipGetDevice(dev));
    if (stream) {
        hipDevice_t sdev = 0;
        HIP_TRY(hipStreamGetDevice(stream, &sdev));
        if ((int)sdev != *dev)
            return fail(ZERO_EINVAL, "stream belongs to device %d but the current device is %d", (int)sdev, *dev);
    }
    return ZERO_OK;
}

int lock_ctx(hipStream_t stream, CtxLock* out) {
    int dev = 0;
    int rc = current_device(stream, &dev);
    const DevInfo* info = nullptr;
    if (rc || (rc = dev_info(dev, &info)))
        return rc;
    const auto key = std::make_pair(dev, stream);
    for (;;) {
        std::shared_ptr<Ctx> c;
        {
            std::lock_guard<std::mutex> lk(g_ctx_mu);
            auto it = g_ctx.find(key);
            if (it != g_ctx.end()) {
                c = it->second;
            } else {
                if ((rc = new_ctx(dev, stream, info, &c)))
                    return rc;
                g_ctx.emplace(key, c);
            }
        }
        std::unique_lock<std::mutex> lk(c->mu);
        if (c->released)
            continue;  // released since the lookup: the registry holds a fresh one (or none)
        out->ref = std::move(c);
        out->lk = std::move(lk);
        return ZERO_OK;
    }
}

// ---------------------------------------------------------------------------
// Profiling: three events per sampled step (before the statistics, before the
// update, after it), each step with its own events.  Failures after a step's
// kernels are queued are deferred to the read call.
// ---------------------------------------------------------------------------
struct ProfRec {
    hipEvent_t start, mid, end;
    bool ok;
};

std::mutex g_prof_mu;
int32_t g_prof_every = 0;  // 0: off; k: profile one step in k on each stream
uint64_t g_prof_epoch = 1;
std::vector<ProfRec> g_prof_pending;
std::vector<hipEvent_t> g_prof_pool;
zero_profile_t g_prof_acc = {0, 0.0, 0.0};

std::mutex g_prof_err_mu;
std::string g_prof_err[2];
int g_prof_err_code[2] = {0, 0};

void prof_defer_error(int slot, const char* what, hipError_t e) {
    std::lock_guard<std::mutex> lk(g_prof_err_mu);
    if (g_prof_err_code[slot] == 0) {  // keep the first
        g_prof_err_code[slot] = ZERO_EHIP;
        g_prof_err[slot] = std::string("profiling: ") + what + ": " + hipGetErrorString(e);
    }
}

int prof_take_error(int slot) {
    std::lock_guard<std::mutex> lk(g_prof_err_mu);
    const int code = g_prof_err_code[slot];
    if (code) {
        t_err = g_prof_err[slot];
        g_prof_err_code[slot] = 0;
        g_prof_err[slot].clear();
    }
    return code;
}

hipEvent_t prof_event() {
    if (!g_prof_pool.empty()) {
        hipEvent_t e = g_prof_pool.back();
        g_prof_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    return e;
}

// Sums the pending records into the totals and returns their events to the
// pool; a failed query is deferred and the record dropped.
void prof_drain_locked() {
    for (ProfRec& r : g_prof_pending) {
        hipError_t e = hipEventSynchronize(r.end);
        float a = 0.f, b = 0.f;
        if (e == hipSuccess)
            e = hipEventElapsedTime(&a, r.start, r.mid);
        if (e == hipSuccess)
            e = hipEventElapsedTime(&b, r.mid, r.end);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            prof_defer_error(0, "reading step events", e);
            continue;
        }
        g_prof_acc.steps += 1;
        g_prof_acc.stats_ms += a;
        g_prof_acc.update_ms += b;
    }
    for (ProfRec& r : g_prof_pending) {
        g_prof_pool.push_back(r.start);
        g_prof_pool.push_back(r.mid);
        g_prof_pool.push_back(r.end);
    }
    g_prof_pending.clear();
}

// 1 when this step is sampled (rec holds three events), 0 when not, or an
// error (nothing queued yet) when the events cannot be had.
int prof_begin(uint64_t* tick, uint64_t* epoch, ProfRec* rec) {
    std::lock_guard<std::mutex> plk(g_prof_mu);
    if (g_prof_every <= 0)
        return 0;
    if (*epoch != g_prof_epoch) {
        *epoch = g_prof_epoch;
        *tick = 0;
    }
    if ((*tick)++ % (uint64_t)g_prof_every != 0)
        return 0;
    rec->start = prof_event();
    rec->mid = prof_event();
    rec->end = prof_event();
    rec->ok = rec->start && rec->mid && rec->end;
    if (!rec->ok) {
        for (hipEvent_t e : {rec->start, rec->mid, rec->end})
            if (e)
                g_prof_pool.push_back(e);
        return fail(ZERO_EHIP, "could not create a profiling event");
    }
    return 1;
}

void prof_record(hipEvent_t e, hipStream_t stream, ProfRec* rec) {
    if (!rec->ok)
        return;
    const hipError_t r = hipEventRecord(e, stream);
    if (r != hipSuccess) {
        (void)hipGetLastError();
        rec->ok = false;
        prof_defer_error(0, "hipEventRecord", r);
    }
}

void prof_end(const ProfRec& rec) {
    std::lock_guard<std::mutex> plk(g_prof_mu);
    if (!rec.ok) {
        for (hipEvent_t e : {rec.start, rec.mid, rec.end})
            g_prof_pool.push_back(e);
        return;
    }
    g_prof_pending.push_back(rec);
    if (g_prof_pending.size() >= 4096)
        prof_drain_locked();
}

bool is_fin(double x) { return std::isfinite(x); }

bool overlaps(uintptr_t a, size_t an, uintptr_t b, size_t bn) { return a < b + bn && b < a + an; }

// Call sequence numbers skip 0: the finalize kernel writes the host record with
// sequence number 0 before publishing the real one.
uint32_t next_seq(Ctx* ctx) {
    if (++ctx->seq == 0)
        ++ctx->seq;
    return ctx->seq;
}

// Argument checks shared by zero_shard_step and zero_shard_apply; nothing is
// launched unless every check passes.
constexpr size_t kElemSize[5] = {2, 4, 4, 4, 2};  // grad16, master32, m32, v32, param16_out

int check_arrays_basic(const char* fn, const uintptr_t a[5], int64_t n) {
    if (n < 0 || n > kMaxNumel)
        return fail(ZERO_EINVAL, "%s: n=%lld outside [0, 2^40]", fn, (long long)n);
    if (n > 0) {
        for (int i = 0; i < 5; ++i)
            if (!a[i])
                return fail(ZERO_EINVAL, "%s: NULL array with n > 0", fn);
        for (int i = 0; i < 5; ++i)
            if (a[i] % kElemSize[i])
                return fail(ZERO_EINVAL, "%s: array %d is not %zu-byte aligned", fn, i, kElemSize[i]);
    }
    return ZERO_OK;
}

int check_arrays_disjoint(const char* fn, const uintptr_t a[5], int64_t n) {
    for (int i = 0; i < 5; ++i)
        for (int j = i + 1; j < 5; ++j)
            if (overlaps(a[i], kElemSize[i] * (size_t)n, a[j], kElemSize[j] * (size_t)n))
                return fail(ZERO_EINVAL, "%s: arrays %d and %d overlap", fn, i, j);
    return ZERO_OK;
}

void array_addrs(const uint16_t* grad16, const float* master32, const float* m32, const float* v32,
                 const uint16_t* param16_out, uintptr_t a[5]) {
    a[0] = reinterpret_cast<uintptr_t>(grad16);
    a[1] = reinterpret_cast<uintptr_t>(master32);
    a[2] = reinterpret_cast<uintptr_t>(m32);
    a[3] = reinterpret_cast<uintptr_t>(v32);
    a[4] = reinterpret_cast<uintptr_t>(param16_out);
}

int check_arrays(const char* fn, const uint16_t* grad16, const float* master32, const float* m32, const float* v32,
                 const uint16_t* param16_out, int64_t n) {
    uintptr_t a[5];
    array_addrs(grad16, master32, m32, v32, param16_out, a);
    int rc = check_arrays_basic(fn, a, n);
    if (rc || n == 0)
        return rc;
    return check_arrays_disjoint(fn, a, n);
}

int check_hyper(const char* fn, double lr, double beta1, double beta2, double eps, double weight_decay, int64_t step,
                double loss_scale, double clip) {
    if (zs::hyper_ok(lr, beta1, beta2, eps, weight_decay, step, loss_scale, clip))
        return ZERO_OK;
    if (!is_fin(lr) || lr < 0.0 || !is_fin(eps) || eps < 0.0 || !is_fin(weight_decay))
        return fail(ZERO_EINVAL, "%s: need finite lr >= 0, eps >= 0, weight_decay", fn);
    if (!(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0))
        return fail(ZERO_EINVAL, "%s: beta1, beta2 must lie in [0, 1)", fn);
    if (step < 1)
        return fail(ZERO_EINVAL, "%s: step (t) must be >= 1, got %lld", fn, (long long)step);
    if (!is_fin(loss_scale) || !(loss_scale > 0.0))
        return fail(ZERO_EINVAL, "%s: loss_scale must be finite and > 0", fn);
    return fail(ZERO_EINVAL, "%s: clip is NaN", fn);
}

int check_update_args(const char* fn, const uint16_t* grad16, const float* master32, const float* m32,
                      const float* v32, const uint16_t* param16_out, int64_t n, double lr, double beta1,
                      double beta2, double eps, double weight_decay, int64_t step, double loss_scale, double clip) {
    const int rc = check_hyper(fn, lr, beta1, beta2, eps, weight_decay, step, loss_scale, clip);
    return rc ? rc : check_arrays(fn, grad16, master32, m32, v32, param16_out, n);
}

// Every array must lie inside one allocation the GPU can access: [p, p + bytes)
// within the range hipMemGetAddressRange reports for p.  This turns an n that
// overruns a buffer, or a pageable host pointer, into ZERO_EINVAL instead of a
// GPU memory fault.
int check_ranges(const char* fn, const void* const* ptrs, const size_t* bytes, int count) {
    for (int i = 0; i < count; ++i) {
        hipDeviceptr_t base = nullptr;
        size_t size = 0;
        if (hipMemGetAddressRange(&base, &size, const_cast<void*>(ptrs[i])) != hipSuccess || !base) {
            (void)hipGetLastError();
            return fail(ZERO_EINVAL, "%s: array %d is not in GPU-accessible memory", fn, i);
        }
        const uintptr_t b = reinterpret_cast<uintptr_t>(base), p = reinterpret_cast<uintptr_t>(ptrs[i]);
        if (p < b || p - b + bytes[i] > size)
            return fail(ZERO_EINVAL, "%s: array %d ([%p, +%zu B)) overruns its allocation ([%p, +%zu B))", fn, i,
                        ptrs[i], bytes[i], base, size);
    }
    return ZERO_OK;
}

int check_shard_ranges(const char* fn, const uint16_t* grad16, const float* master32, const float* m32,
                       const float* v32, const uint16_t* param16_out, int64_t n) {
    const void* ptrs[5] = {grad16, master32, m32, v32, param16_out};
    size_t bytes[5];
    for (int i = 0; i < 5; ++i)
        bytes[i] = kElemSize[i] * (size_t)n;
    return check_ranges(fn, ptrs, bytes, 5);
}

// fp32 constants, each computed in double and rounded once; the bias
// corrections come from the definition the resident step's kernel shares.
zs::AdamConst adam_const(double lr, double beta1, double beta2, double eps, double wd, int64_t step) {
    return zs::make_adam_const(lr, beta1, beta2, eps, wd, step);
}

// Statistics + finalize: the result record lands in res and host_dev.
int launch_stats_into(const DevInfo* info, zs::Partial* part, zs::Result* res, zs::Result* host_dev,
                      const uint16_t* grad16, int64_t n, const Plan& pl, double loss_scale, double clip, uint32_t seq,
                      hipStream_t stream) {
    zs::k_stats<kStatsBlock, kStatsUnroll, kStatsNTL, kStatsXCD>
        <<<pl.stats_blocks, kStatsBlock, info->stats_lds, stream>>>(grad16, n, pl.ghead, pl.gvec, part);
    HIP_TRY(hipGetLastError());
    zs::k_finalize<<<1, zs::kFinalBlock, 0, stream>>>(part, pl.stats_blocks, res, host_dev, loss_scale, clip, seq);
    HIP_TRY(hipGetLastError());
    return ZERO_OK;
}

int launch_stats_planned(Ctx* ctx, const uint16_t* grad16, int64_t n, double loss_scale, double clip, uint32_t seq,
                         hipStream_t stream) {
    const Plan pl = plan_step(grad16, nullptr, nullptr, nullptr, nullptr, n, ctx->info->ncu);
    return launch_stats_into(ctx->info, ctx->part, ctx->res, ctx->host_dev, grad16, n, pl, loss_scale, clip, seq,
                             stream);
}

int prof_every() {
    std::lock_guard<std::mutex> plk(g_prof_mu);
    return g_prof_every;
}

// The fused update reading its scalars from `res`; the fp32 constants are
// `c`, or the device copy at cdev when it is not NULL.
int launch_update_from(const DevInfo* info, const zs::Result* res, const uint16_t* grad16, float* master32,
                       float* m32, float* v32, uint16_t* param16_out, int64_t n, const Plan& pl,
                       const zs::AdamConst& c, hipStream_t stream, const zs::AdamConst* cdev = nullptr) {
    if (pl.vec && cdev)
        zs::k_adam_vec<kAdamBlock, kAdamUnroll, kAdamNTL, kAdamNTS, kAdamXCD, kAdamREV, true>
            <<<(unsigned)pl.adam_blocks, kAdamBlock, info->adam_lds, stream>>>(
                grad16, master32, m32, v32, param16_out, n, pl.head, pl.nvec, res, c, cdev);
    else if (pl.vec)
        zs::k_adam_vec<kAdamBlock, kAdamUnroll, kAdamNTL, kAdamNTS, kAdamXCD, kAdamREV, false>
            <<<(unsigned)pl.adam_blocks, kAdamBlock, info->adam_lds, stream>>>(
                grad16, master32, m32, v32, param16_out, n, pl.head, pl.nvec, res, c, nullptr);
    else if (cdev)
        zs::k_adam_scalar<true><<<(unsigned)pl.adam_blocks, zs::kScalarBlock, 0, stream>>>(
            grad16, master32, m32, v32, param16_out, n, res, c, cdev);
    else
        zs::k_adam_scalar<false><<<(unsigned)pl.adam_blocks, zs::kScalarBlock, 0, stream>>>(
            grad16, master32, m32, v32, param16_out, n, res, c, nullptr);
    HIP_TRY(hipGetLastError());
    return ZERO_OK;
}

int launch_update(Ctx* ctx, const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                  int64_t n, const Plan& pl, const zs::AdamConst& c, hipStream_t stream) {
    return launch_update_from(ctx->info, ctx->res, grad16, master32, m32, v32, param16_out, n, pl, c, stream);
}

// The one-launch small-shard step (pl.small_v > 0) with its partials in `part`
// and its barrier words at `sync` (zeroed on the stream first when
// *sync_ready is false).
int launch_small_into(uint64_t* part, uint64_t* sync, bool* sync_ready, zs::Result* res, zs::Result* host_dev,
                      const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                      int64_t n, const Plan& pl, double loss_scale, double clip, uint32_t seq, const zs::AdamConst& c,
                      hipStream_t stream) {
    if (!*sync_ready) {
        zs::k_zero_words<<<1, 256, 0, stream>>>(sync, zs::kSyncWords);
        HIP_TRY(hipGetLastError());
        *sync_ready = true;
    }
    const dim3 grid((unsigned)pl.small_grid), block(zs::kSmallBlock);
#define ZS_SMALL_LAUNCH(V)                                                                                      \
    zs::k_small_step<V><<<grid, block, 0, stream>>>(grad16, master32, m32, v32, param16_out, n, pl.head, pl.nvec, \
                                                    part, sync, res, host_dev, loss_scale, clip, seq, c)
    switch (pl.small_v) {
    case 1: ZS_SMALL_LAUNCH(1); break;
    case 2: ZS_SMALL_LAUNCH(2); break;
    case 4: ZS_SMALL_LAUNCH(4); break;
    default: ZS_SMALL_LAUNCH(8); break;
    }
#undef ZS_SMALL_LAUNCH
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return fail(ZERO_EHIP, "launch of the small-shard step (%lld workgroups): %s", (long long)pl.small_grid,
                    hipGetErrorString(e));
    return ZERO_OK;
}

// Wait until the finalize kernel has published call `seq` in the host-mapped
// record (it writes the record, then the sequence number with a system-scope
// release), then read it.  No event is recorded on the stream for this: event
// markers between kernels cost several microseconds of GPU idle time each.
int wait_result(Ctx* ctx, uint32_t seq, hipStream_t stream, zs::Result* out) {
    uint64_t polls = 0;
    while (__atomic_load_n(&ctx->host->seq, __ATOMIC_ACQUIRE) != seq) {
        // spin for the usual wait (the statistics of one shard: microseconds); once the stream
        // has been busy for a few milliseconds (other work queued ahead), sleep between checks
        // instead of holding a core
        if (polls < ((uint64_t)1 << 18))
            __builtin_ia32_pause();
        else
            std::this_thread::sleep_for(std::chrono::microseconds(50));
        if ((++polls & 0xFFF) == 0 || polls > ((uint64_t)1 << 18)) {
            const hipError_t e = hipStreamQuery(stream);
            if (e == hipSuccess) {  // everything queued has finished
                if (__atomic_load_n(&ctx->host->seq, __ATOMIC_ACQUIRE) == seq)
                    break;
                return fail(ZERO_EHIP, "result record %u not published although the stream is idle", seq);
            }
            if (e != hipErrorNotReady)
                return fail(ZERO_EHIP, "stream failed while waiting for the statistics: %s", hipGetErrorString(e));
        }
    }
    std::memcpy(out, (const void*)ctx->host, sizeof *out);
    return ZERO_OK;
}

void set_stats(const zs::Result& r, int64_t n, int32_t path) {
    t_stats.sumsq = r.sumsq;
    t_stats.norm = r.norm;
    t_stats.coef = r.coef;
    t_stats.mult = r.mult;
    t_stats.overflow = r.overflow;
    t_stats.skipped = r.skip;
    t_stats.path = path;
    t_stats.n = n;
    t_have_stats = true;
}

// ---------------------------------------------------------------------------
// Resident-step workspaces, one per (device, state record): every step taken
// with a record, eager or replayed from a captured graph, uses that record's
// workspace, so steps with different records never share one.
// ---------------------------------------------------------------------------
struct ResWs {
    zs::Partial* part = nullptr;
    zs::Result* res = nullptr;
    zs::AdamConst* dconst = nullptr;
    uint32_t seq = 0;          // call counter echoed in the result record
    uint64_t prof_tick = 0;    // sampled timing, as a stream context's
    uint64_t prof_epoch = 0;
};

std::mutex g_res_mu;
std::map<std::pair<int, const void*>, ResWs> g_res;  // node addresses stay valid until erased

void free_res_ws(ResWs* w) {
    if (w->part) (void)hipFree(w->part);
    if (w->res) (void)hipFree(w->res);
    if (w->dconst) (void)hipFree(w->dconst);
    *w = ResWs{};
}

// The workspace of `state` on device `dev`, allocated on first use (also while
// `stream` is capturing).  Steps with one record do not overlap, so the caller
// may use the entry without holding the lock.
int resident_ws(int dev, const void* state, hipStream_t stream, ResWs** out) {
    std::lock_guard<std::mutex> lk(g_res_mu);
    const auto key = std::make_pair(dev, state);
    auto it = g_res.find(key);
    if (it != g_res.end()) {
        *out = &it->second;
        return ZERO_OK;
    }
    RelaxedCapture relaxed(stream);
    ResWs w;
    const bool ok = hipMalloc(reinterpret_cast<void**>(&w.part), sizeof(zs::Partial) * zs::kMaxStatsBlocks) ==
                        hipSuccess &&
                    hipMalloc(reinterpret_cast<void**>(&w.res), sizeof(zs::Result)) == hipSuccess &&
                    hipMalloc(reinterpret_cast<void**>(&w.dconst), sizeof(zs::AdamConst)) == hipSuccess;
    if (!ok) {
        free_res_ws(&w);
        (void)hipGetLastError();
        return fail(ZERO_ENOMEM, "could not allocate the resident step's workspace on device %d", dev);
    }
    *out = &g_res.emplace(key, w).first->second;
    return ZERO_OK;
}

// ---------------------------------------------------------------------------
// The allocation-free step's workspace: one fixed device array per GPU (each
// device that loads the library holds its own copy until the process ends),
// laid out as the statistics partials, the one-launch step's barrier words,
// the result record and a second record that stands in for the host-mapped
// one (the host copies it out instead).  In host code `scratch` names a
// host-side stand-in; the device address comes from hipGetSymbolAddress.
// ---------------------------------------------------------------------------
constexpr size_t kScratchPart = 0;
constexpr size_t kScratchSync = kScratchPart + sizeof(zs::Partial) * zs::kMaxStatsBlocks;
constexpr size_t kScratchRes = kScratchSync + sizeof(uint64_t) * zs::kSyncWords;
constexpr size_t kScratchRes2 = kScratchRes + 256;
constexpr size_t kScratchBytes = kScratchRes2 + 256;
static_assert(kScratchRes % 256 == 0 && sizeof(zs::Result) <= 256, "scratch layout");

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

struct ScratchDev {
    std::mutex mu;           // serialises this device's allocation-free calls on the host side
    unsigned char* ptr = nullptr;  // the device's copy of `scratch`
    bool sync_ready = true;  // the barrier words are zero (as loaded) or were cleared
    uint32_t seq = 0;
};
ScratchDev g_scratch[kMaxDevices];

// The device address of `scratch` on `dev` (the current device), looked up
// once per device.  Caller holds g_scratch[dev].mu.
int scratch_ptr(int dev, unsigned char** out) {
    ScratchDev& sd = g_scratch[dev];
    if (!sd.ptr) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            (void)hipGetLastError();
            return fail(ZERO_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
        }
        sd.ptr = static_cast<unsigned char*>(p);
    }
    *out = sd.ptr;
    return ZERO_OK;
}

}  // namespace zsh

using namespace zsh;

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

const char* zero_last_error(void) { return t_err.c_str(); }

int zero_partition_layout(int64_t total_numel, int32_t nd, int32_t rank, zero_layout_t* out) {
    if (!out)
        return fail(ZERO_EINVAL, "zero_partition_layout: out is NULL");
    if (total_numel < 0 || total_numel > ((int64_t)1 << 62))
        return fail(ZERO_EINVAL, "zero_partition_layout: total_numel %lld outside [0, 2^62]", (long long)total_numel);
    if (nd < 1 || rank < 0 || rank >= nd)
        return fail(ZERO_EINVAL, "zero_partition_layout: need nd >= 1 and 0 <= rank < nd (nd=%d rank=%d)", nd, rank);
    const int64_t shard = total_numel / nd + (total_numel % nd ? 1 : 0);
    const int64_t first = shard * rank;
    int64_t valid = total_numel - first;
    valid = valid < 0 ? 0 : (valid > shard ? shard : valid);
    out->shard_numel = shard;
    out->offset = first;
    out->valid_numel = valid;
    out->padded_total = shard * nd;
    return ZERO_OK;
}

int zero_model_state_bytes(double psi, double nd, int32_t stage, double k, double* out) {
    if (!out || !(nd > 0.0) || !is_fin(nd) || !(psi >= 0.0) || !is_fin(psi) || !is_fin(k))
        return fail(ZERO_EINVAL, "zero_model_state_bytes: invalid psi/nd/k or NULL out");
    // fp16 parameters and gradients take 2 bytes each, the optimizer state K bytes per parameter.
    const double params = 2.0 * psi, grads = 2.0 * psi, opt = k * psi;
    switch (stage) {
    case ZERO_STAGE_DP: *out = params + grads + opt; break;
    case ZERO_STAGE_OS: *out = params + grads + opt / nd; break;
    case ZERO_STAGE_OS_G: *out = params + (grads + opt) / nd; break;
    case ZERO_STAGE_OS_G_P: *out = (params + grads + opt) / nd; break;
    default: return fail(ZERO_EINVAL, "zero_model_state_bytes: unknown stage %d", stage);
    }
    return ZERO_OK;
}

int zero_memory_bytes(double psi, int32_t nd, int32_t stage, int32_t k, double* bytes) {
    if (!bytes || nd < 1 || k < 0 || !(psi >= 0.0) || !is_fin(psi))
        return fail(ZERO_EINVAL, "zero_memory_bytes: need psi >= 0 finite, nd >= 1, k >= 0 and bytes != NULL");
    const int rc = zero_model_state_bytes(psi, (double)nd, stage, (double)k, bytes);
    if (rc)
        return fail(rc, "zero_memory_bytes: unknown stage %d", stage);
    return ZERO_OK;
}

int zero_scaler_init(zero_scaler_t* s, double scale, int64_t window, double min_scale) {
    if (!s || !is_fin(scale) || !(scale > 0.0) || !is_fin(min_scale) || !(min_scale > 0.0))
        return fail(ZERO_EINVAL, "zero_scaler_init: need finite scale > 0 and min_scale > 0");
    s->scale = scale;
    s->min_scale = min_scale;
    s->window = window;
    s->applied = 0;
    s->good = 0;
    return ZERO_OK;
}

int zero_scaler_update(zero_scaler_t* s, int32_t skipped) {
    if (!s)
        return fail(ZERO_EINVAL, "zero_scaler_update: NULL scaler");
    if (skipped) {
        const double halved = s->scale * 0.5;
        s->scale = halved > s->min_scale ? halved : s->min_scale;
        s->good = 0;
    } else {
        s->applied += 1;
        s->good += 1;
        if (s->window > 0 && s->good >= s->window) {
            s->scale *= 2.0;
            s->good = 0;
        }
    }
    return ZERO_OK;
}

int zero_shard_step_scaled(const zero_step_args_t* a, zero_scaler_t* s) {
    if (!a || !s)
        return fail(ZERO_EINVAL, "zero_shard_step_scaled: NULL args or scaler");
    if (s->applied < 0 || s->applied == INT64_MAX)
        return fail(ZERO_EINVAL, "zero_shard_step_scaled: scaler has %lld applied steps", (long long)s->applied);
    const int rc = zero_shard_step(a->grad16, a->master32, a->m32, a->v32, a->param16_out, a->n, a->lr, a->beta1,
                                   a->beta2, a->eps, a->weight_decay, s->applied + 1, s->scale, a->clip, a->stream);
    if (rc < 0)
        return rc;
    (void)zero_scaler_update(s, rc == ZERO_SKIPPED);
    return rc;
}

int zero_shard_last_step_stats(zero_step_stats_t* out) {
    if (!out)
        return fail(ZERO_EINVAL, "zero_shard_last_step_stats: NULL out");
    if (!t_have_stats)
        return fail(ZERO_EINVAL, "zero_shard_last_step_stats: no step on this thread yet");
    *out = t_stats;
    return ZERO_OK;
}

int zero_shard_last_stats(double* norm, float* mult, int* overflow) {
    if (!norm && !mult && !overflow)
        return fail(ZERO_EINVAL, "zero_shard_last_stats: every out pointer is NULL");
    if (!t_have_stats)
        return fail(ZERO_EINVAL, "zero_shard_last_stats: no step on this thread yet");
    if (norm)
        *norm = t_stats.norm;
    if (mult)
        *mult = t_stats.mult;
    if (overflow)
        *overflow = t_stats.overflow;
    return ZERO_OK;
}

int zero_bias_corrections(double beta1, double beta2, int64_t step, float* bc1, float* bc2) {
    if (!bc1 || !bc2 || step < 1 || !(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0))
        return fail(ZERO_EINVAL, "zero_bias_corrections: need beta1, beta2 in [0, 1), step >= 1, non-NULL outs");
    *bc1 = zs::bias_correction(beta1, step);
    *bc2 = zs::bias_correction(beta2, step);
    return ZERO_OK;
}

int zero_shard_step(const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                    int64_t n, double lr, double beta1, double beta2, double eps, double weight_decay,
                    int64_t step, double loss_scale, double clip, void* stream_) {
    // ---- argument checks: nothing is launched unless all pass ----
    int rc = check_update_args("zero_shard_step", grad16, master32, m32, v32, param16_out, n, lr, beta1, beta2, eps,
                               weight_decay, step, loss_scale, clip);
    if (rc)
        return rc;
    if (n == 0) {
        t_stats = zero_step_stats_t{0.0, 0.0, 1.0, (float)(1.0 / loss_scale), 0, 0, 0, 0};
        t_have_stats = true;
        return ZERO_OK;
    }
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    CtxLock ctx;
    if ((rc = lock_ctx(stream, &ctx)))
        return rc;
    if ((rc = check_shard_ranges("zero_shard_step", grad16, master32, m32, v32, param16_out, n)))
        return rc;
    const zs::AdamConst c = adam_const(lr, beta1, beta2, eps, weight_decay, step);
    Plan pl = plan_step(grad16, master32, m32, v32, param16_out, n, ctx->info->ncu);
    plan_small(&pl, n, ctx->info);
    const uint32_t seq = next_seq(ctx.get());

    ProfRec pr{};
    const int prof = prof_begin(&ctx->prof_tick, &ctx->prof_epoch, &pr);
    if (prof < 0)
        return prof;
    if (prof)
        prof_record(pr.start, stream, &pr);
    if (pl.small_v) {
        // one launch: its whole time counts as the update's
        if (prof)
            prof_record(pr.mid, stream, &pr);
        rc = launch_small_into(reinterpret_cast<uint64_t*>(ctx->part), ctx->sync, &ctx->sync_ready, ctx->res,
                               ctx->host_dev, grad16, master32, m32, v32, param16_out, n, pl, loss_scale, clip, seq,
                               c, stream);
    } else {
        rc = launch_stats_into(ctx->info, ctx->part, ctx->res, ctx->host_dev, grad16, n, pl, loss_scale, clip, seq,
                               stream);
        if (!rc && prof)
            prof_record(pr.mid, stream, &pr);
        if (!rc)
            rc = launch_update(ctx.get(), grad16, master32, m32, v32, param16_out, n, pl, c, stream);
    }
    if (rc) {
        if (prof) {
            pr.ok = false;
            prof_end(pr);
        }
        return rc;
    }
    if (prof) {
        prof_record(pr.end, stream, &pr);
        prof_end(pr);
    }
    // The update is already queued: wait only for the statistics.
    zs::Result r;
    if ((rc = wait_result(ctx.get(), seq, stream, &r))) {
        if (pl.small_v)
            ctx->sync_ready = false;  // an aborted launch's barrier words are cleared before the next
        return rc;
    }
    set_stats(r, n, pl.small_v ? 1 : 0);
    return r.skip ? ZERO_SKIPPED : ZERO_OK;
}

int zero_shard_stats(const uint16_t* grad16, int64_t n, double* local_sumsq, void* stream_) {
    if (!local_sumsq)
        return fail(ZERO_EINVAL, "zero_shard_stats: NULL local_sumsq");
    if (n < 0 || n > kMaxNumel)
        return fail(ZERO_EINVAL, "zero_shard_stats: n=%lld outside [0, 2^40]", (long long)n);
    if (n > 0 && (!grad16 || reinterpret_cast<uintptr_t>(grad16) % 2))
        return fail(ZERO_EINVAL, "zero_shard_stats: grad16 is NULL or not 2-byte aligned");
    if (n == 0) {
        *local_sumsq = 0.0;
        return ZERO_OK;
    }
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    CtxLock ctx;
    int rc = lock_ctx(stream, &ctx);
    if (rc)
        return rc;
    {
        const void* ptr = grad16;
        const size_t bytes = 2 * (size_t)n;
        if ((rc = check_ranges("zero_shard_stats", &ptr, &bytes, 1)))
            return rc;
    }
    const uint32_t seq = next_seq(ctx.get());
    if ((rc = launch_stats_planned(ctx.get(), grad16, n, 1.0, 0.0, seq, stream)))
        return rc;
    zs::Result r;
    if ((rc = wait_result(ctx.get(), seq, stream, &r)))
        return rc;
    *local_sumsq = r.sumsq;
    return ZERO_OK;
}

int zero_shard_apply(const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                     int64_t n, double global_sumsq, double lr, double beta1, double beta2, double eps,
                     double weight_decay, int64_t step, double loss_scale, double clip, void* stream_) {
    int rc = check_update_args("zero_shard_apply", grad16, master32, m32, v32, param16_out, n, lr, beta1, beta2, eps,
                               weight_decay, step, loss_scale, clip);
    if (rc)
        return rc;
    if (global_sumsq < 0.0)
        return fail(ZERO_EINVAL, "zero_shard_apply: global_sumsq is negative");
    const bool overflow = !is_fin(global_sumsq);
    if (n == 0 || overflow)
        return overflow ? ZERO_SKIPPED : ZERO_OK;
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    CtxLock ctx;
    if ((rc = lock_ctx(stream, &ctx)))
        return rc;
    if ((rc = check_shard_ranges("zero_shard_apply", grad16, master32, m32, v32, param16_out, n)))
        return rc;
    const zs::AdamConst c = adam_const(lr, beta1, beta2, eps, weight_decay, step);
    const Plan pl = plan_step(grad16, master32, m32, v32, param16_out, n, ctx->info->ncu);
    const uint32_t seq = next_seq(ctx.get());
    // sampled timing as in zero_shard_step: the "statistics" interval here is the
    // result-record kernel only (the statistics ran in zero_shard_stats)
    ProfRec pr{};
    const int prof = prof_begin(&ctx->prof_tick, &ctx->prof_epoch, &pr);
    if (prof < 0)
        return prof;
    if (prof)
        prof_record(pr.start, stream, &pr);
    zs::k_set_result<<<1, 64, 0, stream>>>(ctx->res, global_sumsq, loss_scale, clip, seq);
    rc = hipGetLastError() == hipSuccess ? ZERO_OK : fail(ZERO_EHIP, "zero_shard_apply: result-record launch failed");
    if (!rc && prof)
        prof_record(pr.mid, stream, &pr);
    if (!rc)
        rc = launch_update(ctx.get(), grad16, master32, m32, v32, param16_out, n, pl, c, stream);
    if (prof) {
        if (!rc)
            prof_record(pr.end, stream, &pr);
        else
            pr.ok = false;
        prof_end(pr);
    }
    return rc;
}

int zero_shard_stats_async(const uint16_t* grad16, int64_t n, double* local_sumsq, void* stream_) {
    const char* fn = "zero_shard_stats_async";
    if (n < 0 || n > kMaxNumel)
        return fail(ZERO_EINVAL, "%s: n=%lld outside [0, 2^40]", fn, (long long)n);
    if (n > 0 && (!grad16 || reinterpret_cast<uintptr_t>(grad16) % 2))
        return fail(ZERO_EINVAL, "%s: grad16 is NULL or not 2-byte aligned", fn);
    if (!local_sumsq || reinterpret_cast<uintptr_t>(local_sumsq) % 8)
        return fail(ZERO_EINVAL, "%s: local_sumsq must be an 8-byte aligned device pointer", fn);
    if (n > 0 && overlaps(reinterpret_cast<uintptr_t>(grad16), 2 * (size_t)n,
                          reinterpret_cast<uintptr_t>(local_sumsq), sizeof(double)))
        return fail(ZERO_EINVAL, "%s: local_sumsq overlaps grad16", fn);
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    CtxLock ctx;
    int rc = lock_ctx(stream, &ctx);
    if (rc)
        return rc;
    {
        const void* ptrs[2] = {local_sumsq, grad16};
        const size_t bytes[2] = {sizeof(double), 2 * (size_t)n};
        if ((rc = check_ranges(fn, ptrs, bytes, n > 0 ? 2 : 1)))
            return rc;
    }
    if (n == 0) {
        zs::k_set_value<<<1, 64, 0, stream>>>(local_sumsq, 0.0);
        HIP_TRY(hipGetLastError());
        return ZERO_OK;
    }
    const Plan pl = plan_step(grad16, nullptr, nullptr, nullptr, nullptr, n, ctx->info->ncu);
    zs::k_stats<kStatsBlock, kStatsUnroll, kStatsNTL, kStatsXCD>
        <<<pl.stats_blocks, kStatsBlock, ctx->info->stats_lds, stream>>>(grad16, n, pl.ghead, pl.gvec, ctx->part);
    HIP_TRY(hipGetLastError());
    zs::k_finalize_sum<<<1, zs::kFinalBlock, 0, stream>>>(ctx->part, pl.stats_blocks, local_sumsq);
    HIP_TRY(hipGetLastError());
    return ZERO_OK;
}

int zero_shard_apply_async(const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                           int64_t n, const double* global_sumsq, double lr, double beta1, double beta2, double eps,
                           double weight_decay, int64_t step, double loss_scale, double clip, int32_t* skipped,
                           void* stream_) {
    const char* fn = "zero_shard_apply_async";
    int rc = check_update_args(fn, grad16, master32, m32, v32, param16_out, n, lr, beta1, beta2, eps, weight_decay,
                               step, loss_scale, clip);
    if (rc)
        return rc;
    if (!global_sumsq || reinterpret_cast<uintptr_t>(global_sumsq) % 8)
        return fail(ZERO_EINVAL, "%s: global_sumsq must be an 8-byte aligned device pointer", fn);
    if (skipped && reinterpret_cast<uintptr_t>(skipped) % 4)
        return fail(ZERO_EINVAL, "%s: skipped must be 4-byte aligned", fn);
    {
        // the scalars must not alias the state the update writes
        uintptr_t a[5];
        array_addrs(grad16, master32, m32, v32, param16_out, a);
        for (int i = 0; i < 5 && n > 0; ++i) {
            if (overlaps(a[i], kElemSize[i] * (size_t)n, reinterpret_cast<uintptr_t>(global_sumsq), sizeof(double)) ||
                (skipped && overlaps(a[i], kElemSize[i] * (size_t)n, reinterpret_cast<uintptr_t>(skipped), 4)))
                return fail(ZERO_EINVAL, "%s: global_sumsq or skipped overlaps array %d", fn, i);
        }
    }
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    CtxLock ctx;
    if ((rc = lock_ctx(stream, &ctx)))
        return rc;
    {
        const void* ptrs[2] = {global_sumsq, skipped};
        const size_t bytes[2] = {sizeof(double), sizeof(int32_t)};
        if ((rc = check_ranges(fn, ptrs, bytes, skipped ? 2 : 1)))
            return rc;
    }
    if (n > 0 && (rc = check_shard_ranges(fn, grad16, master32, m32, v32, param16_out, n)))
        return rc;
    const uint32_t seq = next_seq(ctx.get());
    if (n == 0) {
        zs::k_set_result_dev<<<1, 64, 0, stream>>>(ctx->res, global_sumsq, loss_scale, clip, skipped, seq);
        HIP_TRY(hipGetLastError());
        return ZERO_OK;
    }
    const zs::AdamConst c = adam_const(lr, beta1, beta2, eps, weight_decay, step);
    const Plan pl = plan_step(grad16, master32, m32, v32, param16_out, n, ctx->info->ncu);
    ProfRec pr{};
    const int prof = prof_begin(&ctx->prof_tick, &ctx->prof_epoch, &pr);  // timed as zero_shard_apply
    if (prof < 0)
        return prof;
    if (prof)
        prof_record(pr.start, stream, &pr);
    zs::k_set_result_dev<<<1, 64, 0, stream>>>(ctx->res, global_sumsq, loss_scale, clip, skipped, seq);
    rc = hipGetLastError() == hipSuccess ? ZERO_OK : fail(ZERO_EHIP, "%s: result-record launch failed", fn);
    if (!rc && prof)
        prof_record(pr.mid, stream, &pr);
    if (!rc)
        rc = launch_update(ctx.get(), grad16, master32, m32, v32, param16_out, n, pl, c, stream);
    if (prof) {
        if (!rc)
            prof_record(pr.end, stream, &pr);
        else
            pr.ok = false;
        prof_end(pr);
    }
    return rc;
}

int zero_resident_state_init(zero_resident_state_t* out, double lr, double beta1, double beta2, double eps,
                             double weight_decay, double clip, double loss_scale, double min_scale, int64_t window,
                             int64_t t) {
    const char* fn = "zero_resident_state_init";
    if (!out)
        return fail(ZERO_EINVAL, "%s: NULL out", fn);
    int rc = check_hyper(fn, lr, beta1, beta2, eps, weight_decay, t, loss_scale, clip);
    if (rc)
        return rc;
    if (!is_fin(min_scale) || !(min_scale > 0.0))
        return fail(ZERO_EINVAL, "%s: min_scale must be finite and > 0", fn);
    zero_resident_state_t s;
    std::memset(&s, 0, sizeof s);
    s.lr = lr;
    s.beta1 = beta1;
    s.beta2 = beta2;
    s.eps = eps;
    s.weight_decay = weight_decay;
    s.clip = clip;
    s.loss_scale = loss_scale;
    s.min_scale = min_scale;
    s.window = window;
    s.t = t;
    *out = s;
    return ZERO_OK;
}

int zero_shard_step_resident(const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                             int64_t n, zero_resident_state_t* state, void* stream_) {
    const char* fn = "zero_shard_step_resident";
    int rc = check_arrays(fn, grad16, master32, m32, v32, param16_out, n);
    if (rc)
        return rc;
    if (!state || reinterpret_cast<uintptr_t>(state) % 8)
        return fail(ZERO_EINVAL, "%s: state must be an 8-byte aligned device pointer", fn);
    {
        uintptr_t a[5];
        array_addrs(grad16, master32, m32, v32, param16_out, a);
        for (int i = 0; i < 5 && n > 0; ++i)
            if (overlaps(a[i], kElemSize[i] * (size_t)n, reinterpret_cast<uintptr_t>(state), sizeof *state))
                return fail(ZERO_EINVAL, "%s: state overlaps array %d", fn, i);
    }
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    int dev = 0;
    const DevInfo* info = nullptr;
    if ((rc = current_device(stream, &dev)) || (rc = dev_info(dev, &info)))
        return rc;
    // While the stream is being captured into a graph only kernel launches are
    // recorded: the allocation lookups and the sampled timing run on eager calls.
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    HIP_TRY(hipStreamIsCapturing(stream, &cap));
    const bool capturing = cap != hipStreamCaptureStatusNone;
    if (!capturing) {
        const void* ptr = state;
        const size_t bytes = sizeof *state;
        if ((rc = check_ranges(fn, &ptr, &bytes, 1)))
            return rc;
        if (n > 0 && (rc = check_shard_ranges(fn, grad16, master32, m32, v32, param16_out, n)))
            return rc;
    }
    ResWs* ws = nullptr;
    if ((rc = resident_ws(dev, state, stream, &ws)))
        return rc;
    if (++ws->seq == 0)
        ++ws->seq;
    const uint32_t seq = ws->seq;
    const Plan pl = plan_step(grad16, master32, m32, v32, param16_out, n, info->ncu);
    ProfRec pr{};
    const int prof = !capturing && n > 0 ? prof_begin(&ws->prof_tick, &ws->prof_epoch, &pr) : 0;
    if (prof < 0)
        return prof;
    if (prof)
        prof_record(pr.start, stream, &pr);
    // statistics, then one workgroup that totals them, fills the result record and the
    // constants and advances the state record's loss-scale schedule (an empty shard has no
    // partials: its total is 0), then the update
    if (n > 0) {
        zs::k_stats<kStatsBlock, kStatsUnroll, kStatsNTL, kStatsXCD>
            <<<pl.stats_blocks, kStatsBlock, info->stats_lds, stream>>>(grad16, n, pl.ghead, pl.gvec, ws->part);
        rc = hipGetLastError() == hipSuccess ? ZERO_OK : fail(ZERO_EHIP, "%s: statistics launch failed", fn);
    }
    if (!rc) {
        zs::k_resident_begin<<<1, zs::kFinalBlock, 0, stream>>>(ws->part, n > 0 ? pl.stats_blocks : 0, state,
                                                                ws->res, ws->dconst, seq);
        rc = hipGetLastError() == hipSuccess ? ZERO_OK : fail(ZERO_EHIP, "%s: record kernel launch failed", fn);
    }
    if (!rc && prof)
        prof_record(pr.mid, stream, &pr);
    if (!rc && n > 0)
        rc = launch_update_from(info, ws->res, grad16, master32, m32, v32, param16_out, n, pl, zs::AdamConst{},
                                stream, ws->dconst);
    if (prof) {
        if (!rc)
            prof_record(pr.end, stream, &pr);
        else
            pr.ok = false;
        prof_end(pr);
    }
    return rc;
}

int zero_resident_release(const zero_resident_state_t* state) {
    if (!state)
        return fail(ZERO_EINVAL, "zero_resident_release: NULL state");
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    std::lock_guard<std::mutex> lk(g_res_mu);
    auto it = g_res.find(std::make_pair(dev, static_cast<const void*>(state)));
    if (it == g_res.end())
        return ZERO_OK;
    // replays of captured graphs may use the workspace on any stream of the device
    HIP_TRY(hipDeviceSynchronize());
    free_res_ws(&it->second);
    g_res.erase(it);
    return ZERO_OK;
}

int zero_stream_release(void* stream_) {
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    int dev = 0;
    int rc = current_device(stream, &dev);
    if (rc)
        return rc;
    std::shared_ptr<Ctx> c;
    {
        std::lock_guard<std::mutex> lk(g_ctx_mu);
        auto it = g_ctx.find(std::make_pair(dev, stream));
        if (it == g_ctx.end())
            return ZERO_OK;
        c = it->second;
    }
    std::lock_guard<std::mutex> lk(c->mu);
    if (c->released)
        return ZERO_OK;
    HIP_TRY(hipStreamSynchronize(stream));
    {
        std::lock_guard<std::mutex> glk(g_ctx_mu);
        auto it = g_ctx.find(std::make_pair(dev, stream));
        if (it != g_ctx.end() && it->second == c)
            g_ctx.erase(it);
    }
    c->released = true;
    free_ctx_buffers(c.get());
    return ZERO_OK;
}

int zero_workspace_count(int64_t* streams, int64_t* records) {
    if (!streams && !records)
        return fail(ZERO_EINVAL, "zero_workspace_count: every out pointer is NULL");
    if (streams) {
        std::lock_guard<std::mutex> lk(g_ctx_mu);
        *streams = (int64_t)g_ctx.size();
    }
    if (records) {
        std::lock_guard<std::mutex> lk(g_res_mu);
        *records = (int64_t)g_res.size();
    }
    return ZERO_OK;
}

int zero_shard_validate(const uint16_t* grad16, const float* master32, const float* m32, const float* v32,
                        const uint16_t* param16_out, int64_t n) {
    // The allocation check comes before the disjointness check here, so an n that
    // overruns the buffers is reported as such.
    uintptr_t a[5];
    array_addrs(grad16, master32, m32, v32, param16_out, a);
    int rc = check_arrays_basic("zero_shard_validate", a, n);
    if (rc || n == 0)
        return rc;
    if ((rc = check_shard_ranges("zero_shard_validate", grad16, master32, m32, v32, param16_out, n)))
        return rc;
    return check_arrays_disjoint("zero_shard_validate", a, n);
}

int zero_profile_enable(int32_t every) {
    if (every < 0)
        return fail(ZERO_EINVAL, "zero_profile_enable: every must be >= 0");
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof_every = every;
    g_prof_epoch += 1;  // every stream restarts its sampling count
    return ZERO_OK;
}

int zero_profile_read(zero_profile_t* out) {
    if (!out)
        return fail(ZERO_EINVAL, "zero_profile_read: NULL out");
    std::lock_guard<std::mutex> lk(g_prof_mu);
    prof_drain_locked();
    const int rc = prof_take_error(0);
    *out = g_prof_acc;
    g_prof_acc = zero_profile_t{0, 0.0, 0.0};
    return rc;
}

int zero_shard_step_noalloc(const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                            int64_t n, double lr, double beta1, double beta2, double eps, double weight_decay,
                            int64_t step, double loss_scale, double clip, void* stream_) {
    const char* fn = "zero_shard_step_noalloc";
    int rc = check_update_args(fn, grad16, master32, m32, v32, param16_out, n, lr, beta1, beta2, eps, weight_decay,
                               step, loss_scale, clip);
    if (rc)
        return rc;  // includes n above 2^40, the most the fixed workspace serves
    if (n == 0) {
        t_stats = zero_step_stats_t{0.0, 0.0, 1.0, (float)(1.0 / loss_scale), 0, 0, 0, 0};
        t_have_stats = true;
        return ZERO_OK;
    }
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    int dev = 0;
    const DevInfo* info = nullptr;
    if ((rc = current_device(stream, &dev)) || (rc = dev_info(dev, &info)))
        return rc;
    if ((rc = check_shard_ranges(fn, grad16, master32, m32, v32, param16_out, n)))
        return rc;
    ScratchDev& sd = g_scratch[dev];
    std::lock_guard<std::mutex> lk(sd.mu);
    unsigned char* base = nullptr;
    if ((rc = scratch_ptr(dev, &base)))
        return rc;
    zs::Partial* part = reinterpret_cast<zs::Partial*>(base + kScratchPart);
    uint64_t* sync = reinterpret_cast<uint64_t*>(base + kScratchSync);
    zs::Result* res = reinterpret_cast<zs::Result*>(base + kScratchRes);
    zs::Result* res2 = reinterpret_cast<zs::Result*>(base + kScratchRes2);
    const zs::AdamConst c = adam_const(lr, beta1, beta2, eps, weight_decay, step);
    Plan pl = plan_step(grad16, master32, m32, v32, param16_out, n, info->ncu);
    plan_small(&pl, n, info);
    if (pl.stats_blocks > zs::kMaxStatsBlocks || pl.small_grid > (int64_t)zs::kMaxStatsBlocks)
        return fail(ZERO_EINVAL, "%s: launch needs more partials than the fixed workspace holds", fn);
    if (++sd.seq == 0)
        ++sd.seq;
    const uint32_t seq = sd.seq;
    if (pl.small_v) {
        rc = launch_small_into(reinterpret_cast<uint64_t*>(part), sync, &sd.sync_ready, res, res2, grad16, master32,
                               m32, v32, param16_out, n, pl, loss_scale, clip, seq, c, stream);
    } else {
        rc = launch_stats_into(info, part, res, res2, grad16, n, pl, loss_scale, clip, seq, stream);
        if (!rc)
            rc = launch_update_from(info, res, grad16, master32, m32, v32, param16_out, n, pl, c, stream);
    }
    if (rc)
        return rc;
    // the record comes back with a copy after the update: the call returns once the whole
    // step has completed on the stream
    zs::Result r;
    std::memset(&r, 0, sizeof r);
    HIP_TRY(hipMemcpyAsync(&r, res2, sizeof r, hipMemcpyDeviceToHost, stream));
    HIP_TRY(hipStreamSynchronize(stream));
    if (r.seq != seq) {
        if (pl.small_v)
            sd.sync_ready = false;  // an aborted launch's barrier words are cleared before the next
        return fail(ZERO_EHIP, "%s: result record %u not published by the step's kernels", fn, seq);
    }
    set_stats(r, n, pl.small_v ? 1 : 0);
    return r.skip ? ZERO_SKIPPED : ZERO_OK;
}

int zero_probe_adam_mix(const uint16_t* grad16, float* master32, float* m32, float* v32, uint16_t* param16_out,
                        int64_t n, void* stream_) {
    const char* fn = "zero_probe_adam_mix";
    int rc = check_arrays(fn, grad16, master32, m32, v32, param16_out, n);
    if (rc || n == 0)
        return rc;
    const uintptr_t a16[3] = {reinterpret_cast<uintptr_t>(master32), reinterpret_cast<uintptr_t>(m32),
                              reinterpret_cast<uintptr_t>(v32)};
    for (int i = 0; i < 3; ++i)
        if (a16[i] % 16)
            return fail(ZERO_EINVAL, "%s: fp32 array %d must be 16-byte aligned", fn, i + 1);
    if (reinterpret_cast<uintptr_t>(grad16) % 8 || reinterpret_cast<uintptr_t>(param16_out) % 8)
        return fail(ZERO_EINVAL, "%s: grad16 and param16_out must be 8-byte aligned", fn);
    if ((rc = check_shard_ranges(fn, grad16, master32, m32, v32, param16_out, n)))
        return rc;
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    int dev = 0;
    const DevInfo* info = nullptr;
    if ((rc = current_device(stream, &dev)) || (rc = dev_info(dev, &info)))
        return rc;
    const int64_t nvec = n / 4;
    int64_t blocks = ceil_div(nvec, (int64_t)kAdamBlock * kAdamUnroll);
    blocks = blocks < 1 ? 1 : (blocks > kAdamMaxBlocks ? kAdamMaxBlocks : blocks);
    zs::k_probe_adam<kAdamBlock, kAdamUnroll, kAdamNTL, kAdamNTS, kAdamXCD>
        <<<(unsigned)blocks, kAdamBlock, info->probe_adam_lds, stream>>>(grad16, master32, m32, v32, param16_out,
                                                                          n, nvec);
    HIP_TRY(hipGetLastError());
    return ZERO_OK;
}

int zero_probe_copy(const void* src, void* dst, int64_t bytes, void* stream_) {
    const uintptr_t s = reinterpret_cast<uintptr_t>(src), d = reinterpret_cast<uintptr_t>(dst);
    if (bytes < 0 || bytes % 16 || (bytes > 0 && (!src || !dst || s % 16 || d % 16)))
        return fail(ZERO_EINVAL, "zero_probe_copy: need 16-byte aligned buffers and a multiple of 16 bytes");
    if (bytes > 0 && overlaps(s, (size_t)bytes, d, (size_t)bytes))
        return fail(ZERO_EINVAL, "zero_probe_copy: ranges overlap");
    if (bytes == 0)
        return ZERO_OK;
    {
        const void* ptrs[2] = {src, dst};
        const size_t sizes[2] = {(size_t)bytes, (size_t)bytes};
        int rc = check_ranges("zero_probe_copy", ptrs, sizes, 2);
        if (rc)
            return rc;
    }
    const int64_t nvec = bytes / 16;
    int64_t blocks = ceil_div(nvec, (int64_t)kCopyBlock * kCopyUnroll);
    blocks = blocks < 1 ? 1 : (blocks > kAdamMaxBlocks ? kAdamMaxBlocks : blocks);
    zs::k_probe_copy<kCopyBlock, kCopyUnroll, kCopyNTL, kCopyNTS, kCopyXCD>
        <<<(unsigned)blocks, kCopyBlock, 0, reinterpret_cast<hipStream_t>(stream_)>>>(
        reinterpret_cast<const zs::u32x4*>(src), reinterpret_cast<zs::u32x4*>(dst), nvec);
    HIP_TRY(hipGetLastError());
    return ZERO_OK;
}

}  // extern "C"
