// zero_lamb.hip -- host side of the LAMB shard step (declared in
// include/zero_shard.h): the layer-table plan and its work lists, argument
// checks, launches, split-phase entry points and sampled kernel timing.
//
// LAMB (You et al.) is listed in ZeRO's related work (Sec. 2.3) among the
// adaptive optimizers whose state ZeRO's partitioning (Sec. 5.1-5.2) makes
// affordable; the fp32 state per parameter is Adam's (Sec. 3.1, K = 12).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <memory>
#include <mutex>
#include <vector>

#include "zero_shard.h"
#include "shard_kernels.hpp"
#include "lamb_kernels.hpp"
#include "host_common.hpp"

// ---------------------------------------------------------------------------
// Launch policy of the two LAMB streaming passes (template knobs in
// lamb_kernels.hpp): one tile of BLOCK*U 4-element vectors per workgroup, at
// most kLambPerCU resident workgroups per CU (an LDS reservation).  Measured on
// MI355X over 250M-element shards: both passes run best with about 32 resident
// waves per CU (128 threads x 16 workgroups, one vector per thread), unlike
// the Adam update, whose optimum is 12 single-wave workgroups; each workgroup
// here also reads its tile's layer pieces and reduces a partial sum.
// ---------------------------------------------------------------------------
namespace {
constexpr int kLambBlock = 128, kLambUnroll = 1, kLambPerCU = 16;
constexpr bool kLambNTL = true, kLambNTS = true, kLambXCD = true;
constexpr int64_t kLambTile = 4 * (int64_t)kLambBlock * kLambUnroll;  // elements per tile
constexpr int64_t kLambMaxBlocks = 1 << 26;
constexpr int kPhases = 5;  // vector paths for element misalignment 0..3, then the scalar path
}  // namespace

using namespace zsh;

// The work lists of one array alignment, on the device: the items (tile pieces
// inside one layer, with the end sentinel), the first item of every tile, the
// level-1 chunks of the layer sums (item ranges inside one layer) and the first
// chunk of every layer (each list with its end sentinel).
struct LambWork {
    zs::LambItem* items = nullptr;
    int64_t* tile_first = nullptr;
    int64_t* chunk = nullptr;
    int64_t* chunk_first = nullptr;
    int64_t n_items = 0, ntiles = 0, n_chunks = 0;
    bool built = false;
};

struct LambProfRec {
    hipEvent_t e[5];
};

struct zero_lamb_plan {
    std::mutex mu;
    int dev = 0;
    int64_t n = 0;
    int32_t n_seg = 0;
    std::vector<int64_t> seg_off;
    LambWork work[kPhases];
    zs::LayerSums* part = nullptr;   // one partial per item (sized for the longest list)
    zs::LayerSums* cpart = nullptr;  // one partial per level-1 chunk
    zs::LayerSums* sums = nullptr;   // per-layer sums of zero_lamb_step
    int64_t max_items = 0, max_chunks = 0;
    hipEvent_t done = nullptr;       // recorded after each call's kernels (ordering across streams)
    hipStream_t last_stream = nullptr;
    bool used = false;
    uint64_t prof_tick = 0;
    size_t lds[2] = {0, 0};  // occupancy reservations of the moments and apply kernels (per phase kind)
    size_t lds_scalar[2] = {0, 0};
};

namespace {

std::mutex g_lprof_mu;
std::vector<LambProfRec> g_lprof_pending;
std::vector<hipEvent_t> g_lprof_pool;
zero_lamb_profile_t g_lprof_acc = {0, 0.0, 0.0, 0.0, 0.0};

template <bool VEC>
const void* moments_kernel() {
    return reinterpret_cast<const void*>(zs::k_lamb_moments<kLambBlock, kLambUnroll, kLambNTL, kLambNTS, VEC, kLambXCD>);
}
template <int PASS>
const void* probe_kernel() {
    return reinterpret_cast<const void*>(zs::k_probe_lamb<kLambBlock, kLambUnroll, kLambNTL, kLambNTS, kLambXCD, PASS>);
}
template <bool VEC>
const void* apply_kernel() {
    return reinterpret_cast<const void*>(zs::k_lamb_apply<kLambBlock, kLambUnroll, kLambNTL, kLambNTS, VEC, kLambXCD>);
}

// Upper bound on the items of any alignment: one per tile the shard touches
// (at most n/T + 2, counting the partial tile below the first aligned vector)
// plus one per interior layer boundary.
int64_t max_items_for(int64_t n, int32_t n_seg) { return n / kLambTile + 2 + (int64_t)n_seg; }

// Level-1 chunks: each layer's items cut into runs of at most kChunkItems.
int64_t max_chunks_for(int64_t max_items, int32_t n_seg) { return max_items / zs::kChunkItems + 1 + (int64_t)n_seg; }

// Tiles (as the kernels' tile_range defines them): [0, head) when head > 0,
// then runs of kLambTile elements from head on.
int64_t tile_of(int64_t pos, int64_t head) {
    const int64_t hs = head > 0 ? 1 : 0;
    return pos < head ? 0 : hs + (pos - head) / kLambTile;
}

int64_t tile_count(int64_t n, int64_t head) {
    if (n == 0)
        return 0;
    const int64_t hs = head > 0 ? 1 : 0;
    return n > head ? hs + (n - head + kLambTile - 1) / kLambTile : 1;
}

struct HostWork {
    std::vector<zs::LambItem> items;  // with the end sentinel
    std::vector<int64_t> tile_first;  // ntiles + 1
    std::vector<int64_t> chunk;       // n_chunks + 1 item indices
    std::vector<int64_t> chunk_first; // n_seg + 1 chunk indices
};

// Cut [0, n) at the tile boundaries and at the layer boundaries; index the
// pieces by tile, and each layer's pieces by level-1 chunk.
void build_work(const std::vector<int64_t>& off, int32_t n_seg, int64_t head, HostWork* w) {
    const int64_t n = n_seg ? off[n_seg] : 0;
    w->items.clear();
    std::vector<int64_t> first((size_t)n_seg + 1, 0);
    for (int32_t s = 0; s < n_seg; ++s) {
        first[s] = (int64_t)w->items.size();
        int64_t pos = off[s];
        const int64_t end = off[s + 1];
        while (pos < end) {
            const int64_t tile_end = pos < head ? head : head + ((pos - head) / kLambTile + 1) * kLambTile;
            w->items.push_back(zs::LambItem{pos, s, 0});
            pos = tile_end < end ? tile_end : end;
        }
    }
    first[n_seg] = (int64_t)w->items.size();
    const int64_t n_items = (int64_t)w->items.size();
    w->items.push_back(zs::LambItem{n, -1, 0});
    const int64_t ntiles = tile_count(n, head);
    w->tile_first.assign((size_t)ntiles + 1, n_items);
    int64_t next = 0;
    for (int64_t k = 0; k < n_items; ++k) {
        const int64_t t = tile_of(w->items[k].start, head);
        while (next <= t)
            w->tile_first[next++] = k;
    }
    w->chunk.clear();
    w->chunk_first.assign((size_t)n_seg + 1, 0);
    for (int32_t s = 0; s < n_seg; ++s) {
        w->chunk_first[s] = (int64_t)w->chunk.size();
        for (int64_t k = first[s]; k < first[s + 1]; k += zs::kChunkItems)
            w->chunk.push_back(k);
    }
    w->chunk_first[n_seg] = (int64_t)w->chunk.size();
    w->chunk.push_back(n_items);
}

template <typename T>
int upload(const std::vector<T>& h, T** d) {
    if (hipMalloc(reinterpret_cast<void**>(d), h.size() * sizeof(T)) != hipSuccess) {
        *d = nullptr;
        (void)hipGetLastError();
        return fail(ZERO_ENOMEM, "zero_lamb: could not allocate a work list of %zu entries", h.size());
    }
    HIP_TRY(hipMemcpy(*d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice));
    return ZERO_OK;
}

// The work list of `phase` (0..3: vector path with that head; 4: scalar path),
// built and uploaded on first use.  Caller holds plan->mu.
int get_work(zero_lamb_plan* plan, int phase, LambWork** out) {
    LambWork& w = plan->work[phase];
    if (!w.built) {
        HostWork h;
        const int64_t head = phase < 4 ? phase : 0;  // the kernels take the same head
        build_work(plan->seg_off, plan->n_seg, head, &h);
        const int64_t n_items = (int64_t)h.items.size() - 1, n_chunks = (int64_t)h.chunk.size() - 1;
        if (n_items > plan->max_items || n_chunks > plan->max_chunks)
            return fail(ZERO_EHIP, "zero_lamb: work lists (%lld items, %lld chunks) exceed their bounds",
                        (long long)n_items, (long long)n_chunks);
        int rc;
        if ((rc = upload(h.items, &w.items)) || (rc = upload(h.tile_first, &w.tile_first)) ||
            (rc = upload(h.chunk, &w.chunk)) || (rc = upload(h.chunk_first, &w.chunk_first)))
            return rc;
        w.n_items = n_items;
        w.ntiles = (int64_t)h.tile_first.size() - 1;
        w.n_chunks = n_chunks;
        w.built = true;
    }
    *out = &w;
    return ZERO_OK;
}

// Element misalignment shared by all arrays (0..3), or 4 when they differ (or
// when an fp16 array is only 2-byte aligned relative to its fp32 partners).
int phase_of(const uint16_t* g, const float* th, const float* m, const float* v, const uint16_t* p) {
    const uintptr_t ef[3] = {(reinterpret_cast<uintptr_t>(th) & 15) / 4, (reinterpret_cast<uintptr_t>(m) & 15) / 4,
                             (reinterpret_cast<uintptr_t>(v) & 15) / 4};
    bool same = ef[0] == ef[1] && ef[0] == ef[2];
    if (g)
        same = same && (reinterpret_cast<uintptr_t>(g) & 7) / 2 == ef[0];
    if (p)
        same = same && (reinterpret_cast<uintptr_t>(p) & 7) / 2 == ef[0];
    return same ? (int)((4 - ef[0]) & 3) : 4;
}

int check_plan(const char* fn, const zero_lamb_plan_t* plan) {
    if (!plan)
        return fail(ZERO_EINVAL, "%s: NULL plan", fn);
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    if (dev != plan->dev)
        return fail(ZERO_EINVAL, "%s: plan was created on device %d, current device is %d", fn, plan->dev, dev);
    return ZERO_OK;
}

int check_phi(const char* fn, double phi_lo, double phi_hi) {
    if (std::isnan(phi_lo) || std::isnan(phi_hi) || !(phi_lo >= 0.0) || !(phi_hi >= phi_lo) || std::isinf(phi_lo))
        return fail(ZERO_EINVAL, "%s: need 0 <= phi_lo <= phi_hi (phi_hi may be +inf)", fn);
    return ZERO_OK;
}

// Alignment, NULL, overlap and allocation checks of the arrays a call touches
// (NULL entries of ptrs are arrays the call does not take).
int check_lamb_arrays(const char* fn, const void* const ptrs[5], int64_t n) {
    static const size_t esz[5] = {2, 4, 4, 4, 2};
    size_t bytes[5];
    const void* live[5];
    size_t live_bytes[5];
    int k = 0;
    for (int i = 0; i < 5; ++i) {
        bytes[i] = esz[i] * (size_t)n;
        if (!ptrs[i])
            continue;
        if (reinterpret_cast<uintptr_t>(ptrs[i]) % esz[i])
            return fail(ZERO_EINVAL, "%s: array %d is not %zu-byte aligned", fn, i, esz[i]);
        live[k] = ptrs[i];
        live_bytes[k] = bytes[i];
        ++k;
    }
    if (n == 0)
        return ZERO_OK;
    for (int i = 0; i < 5; ++i)
        for (int j = i + 1; j < 5; ++j)
            if (ptrs[i] && ptrs[j] &&
                overlaps(reinterpret_cast<uintptr_t>(ptrs[i]), bytes[i], reinterpret_cast<uintptr_t>(ptrs[j]),
                         bytes[j]))
                return fail(ZERO_EINVAL, "%s: arrays %d and %d overlap", fn, i, j);
    return check_ranges(fn, live, live_bytes, k);
}

int check_layer_sums(const char* fn, const zero_lamb_plan_t* plan, const void* layer_sumsq,
                     const void* const arrays[5]) {
    if (!layer_sumsq || reinterpret_cast<uintptr_t>(layer_sumsq) % 16)
        return fail(ZERO_EINVAL, "%s: layer_sumsq must be a 16-byte aligned device array", fn);
    const size_t bytes = 16 * (size_t)plan->n_seg;
    for (int i = 0; i < 5; ++i)
        if (arrays[i] && overlaps(reinterpret_cast<uintptr_t>(arrays[i]), (i == 0 || i == 4 ? 2 : 4) * (size_t)plan->n,
                                  reinterpret_cast<uintptr_t>(layer_sumsq), bytes))
            return fail(ZERO_EINVAL, "%s: layer_sumsq overlaps array %d", fn, i);
    return check_ranges(fn, &layer_sumsq, &bytes, 1);
}

// Work queued on the plan's previous stream must finish before another
// stream reuses the plan's partials and sums: the new stream waits (on the
// device) for the event recorded after the plan's last call.  The event stays
// valid after that stream is destroyed, and no other stream or the host waits.
int switch_stream(zero_lamb_plan* plan, hipStream_t stream) {
    if (plan->used && plan->last_stream != stream)
        HIP_TRY(hipStreamWaitEvent(stream, plan->done, 0));
    plan->used = true;
    plan->last_stream = stream;
    return ZERO_OK;
}

// Marks the end of this call's kernels on `stream` (see switch_stream).
int mark_done(zero_lamb_plan* plan, hipStream_t stream) {
    HIP_TRY(hipEventRecord(plan->done, stream));
    return ZERO_OK;
}

unsigned grid_for(int64_t n_items) {
    int64_t b = n_items < 1 ? 1 : n_items;
    return (unsigned)(b > kLambMaxBlocks ? kLambMaxBlocks : b);
}

// Grid of the tile passes: a multiple of 8 (the XCD count) so that the XCD
// remapping of workgroups is a bijection; the extra workgroups find no tile.
unsigned tile_grid(int64_t ntiles) {
    int64_t b = ntiles < 1 ? 1 : ntiles;
    b = b > kLambMaxBlocks ? kLambMaxBlocks : b;
    return (unsigned)((b + 7) / 8 * 8);
}

int launch_moments(zero_lamb_plan* plan, const LambWork& w, int phase, const uint16_t* g, const float* th, float* m,
                   float* v, const zs::Result* res, const zs::AdamConst& c, hipStream_t stream) {
    const unsigned grid = tile_grid(w.ntiles);
    if (phase < 4)
        zs::k_lamb_moments<kLambBlock, kLambUnroll, kLambNTL, kLambNTS, true, kLambXCD>
            <<<grid, kLambBlock, plan->lds[0], stream>>>(g, th, m, v, w.items, w.tile_first, w.ntiles, plan->n,
                                                         phase, res, c, plan->part);
    else
        zs::k_lamb_moments<kLambBlock, kLambUnroll, kLambNTL, kLambNTS, false, kLambXCD>
            <<<grid, kLambBlock, plan->lds_scalar[0], stream>>>(g, th, m, v, w.items, w.tile_first, w.ntiles,
                                                                 plan->n, 0, res, c, plan->part);
    HIP_TRY(hipGetLastError());
    return ZERO_OK;
}

int launch_layer(zero_lamb_plan* plan, const LambWork& w, zs::LayerSums* sums, const zs::Result* res,
                 hipStream_t stream) {
    zs::k_lamb_chunks<<<grid_for(w.n_chunks), zs::kChunkBlock, 0, stream>>>(plan->part, w.chunk, w.n_chunks,
                                                                            plan->cpart, res);
    HIP_TRY(hipGetLastError());
    zs::k_lamb_layer<<<grid_for(plan->n_seg), zs::kLayerBlock, 0, stream>>>(plan->cpart, w.chunk_first,
                                                                            plan->n_seg, sums, res);
    HIP_TRY(hipGetLastError());
    return ZERO_OK;
}

int launch_apply(zero_lamb_plan* plan, const LambWork& w, int phase, float* th, const float* m, const float* v,
                 uint16_t* p, const zs::LayerSums* sums, const zs::Result* res, const zs::AdamConst& c, double lr,
                 double phi_lo, double phi_hi, hipStream_t stream) {
    const unsigned grid = tile_grid(w.ntiles);
    if (phase < 4)
        zs::k_lamb_apply<kLambBlock, kLambUnroll, kLambNTL, kLambNTS, true, kLambXCD>
            <<<grid, kLambBlock, plan->lds[1], stream>>>(th, m, v, p, w.items, w.tile_first, w.ntiles, plan->n,
                                                         phase, sums, res, c, lr, phi_lo, phi_hi);
    else
        zs::k_lamb_apply<kLambBlock, kLambUnroll, kLambNTL, kLambNTS, false, kLambXCD>
            <<<grid, kLambBlock, plan->lds_scalar[1], stream>>>(th, m, v, p, w.items, w.tile_first, w.ntiles,
                                                                 plan->n, 0, sums, res, c, lr, phi_lo, phi_hi);
    HIP_TRY(hipGetLastError());
    return ZERO_OK;
}

hipEvent_t lprof_event() {
    if (!g_lprof_pool.empty()) {
        hipEvent_t e = g_lprof_pool.back();
        g_lprof_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    return hipEventCreate(&e) == hipSuccess ? e : nullptr;
}

// Events of one sampled step, or false when this step is not sampled (or an
// event could not be created).  Caller holds plan->mu.
bool lprof_begin(zero_lamb_plan* plan, LambProfRec* rec) {
    const int every = prof_every();
    if (every <= 0 || plan->prof_tick++ % (uint64_t)every != 0)
        return false;
    std::lock_guard<std::mutex> lk(g_lprof_mu);
    bool ok = true;
    for (int i = 0; i < 5; ++i) {
        rec->e[i] = lprof_event();
        ok = ok && rec->e[i];
    }
    if (!ok) {
        for (int i = 0; i < 5; ++i)
            if (rec->e[i])
                g_lprof_pool.push_back(rec->e[i]);
        return false;
    }
    return true;
}

void lprof_drain_locked() {
    for (LambProfRec& r : g_lprof_pending) {
        hipError_t e = hipEventSynchronize(r.e[4]);
        float t[4] = {0.f, 0.f, 0.f, 0.f};
        for (int i = 0; i < 4 && e == hipSuccess; ++i)
            e = hipEventElapsedTime(&t[i], r.e[i], r.e[i + 1]);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            prof_defer_error(1, "reading LAMB step events", e);
            continue;
        }
        g_lprof_acc.steps += 1;
        g_lprof_acc.stats_ms += t[0];
        g_lprof_acc.moments_ms += t[1];
        g_lprof_acc.layer_ms += t[2];
        g_lprof_acc.apply_ms += t[3];
    }
    for (LambProfRec& r : g_lprof_pending)
        for (int i = 0; i < 5; ++i)
            g_lprof_pool.push_back(r.e[i]);
    g_lprof_pending.clear();
}

// Records event i of a sampled step; a failure drops the sample (deferred error).
void lprof_record(LambProfRec* rec, bool* ok, int i, hipStream_t stream) {
    if (!*ok)
        return;
    const hipError_t e = hipEventRecord(rec->e[i], stream);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        *ok = false;
        prof_defer_error(1, "hipEventRecord", e);
    }
}

// Queues a sampled step's record for the next read, or returns its events to
// the pool when a record failed.
void lprof_end(const LambProfRec& rec, bool ok) {
    std::lock_guard<std::mutex> lk(g_lprof_mu);
    if (!ok) {
        for (int i = 0; i < 5; ++i)
            g_lprof_pool.push_back(rec.e[i]);
        return;
    }
    g_lprof_pending.push_back(rec);
    if (g_lprof_pending.size() >= 4096)
        lprof_drain_locked();
}

void set_last_stats(const zs::Result& r, int64_t n) {
    t_stats.sumsq = r.sumsq;
    t_stats.norm = r.norm;
    t_stats.coef = r.coef;
    t_stats.mult = r.mult;
    t_stats.overflow = r.overflow;
    t_stats.skipped = r.skip;
    t_stats.path = 0;
    t_stats.n = n;
    t_have_stats = true;
}

void free_plan(zero_lamb_plan* p) {
    for (LambWork& w : p->work)
        for (void* d : {(void*)w.items, (void*)w.tile_first, (void*)w.chunk, (void*)w.chunk_first})
            if (d) (void)hipFree(d);
    if (p->part) (void)hipFree(p->part);
    if (p->cpart) (void)hipFree(p->cpart);
    if (p->sums) (void)hipFree(p->sums);
    if (p->done) (void)hipEventDestroy(p->done);
}

}  // namespace

extern "C" {

int zero_lamb_plan_create(const int64_t* seg_off, int32_t n_seg, int64_t n, zero_lamb_plan_t** out) {
    if (!out)
        return fail(ZERO_EINVAL, "zero_lamb_plan_create: NULL out");
    *out = nullptr;
    if (n < 0 || n > kMaxNumel)
        return fail(ZERO_EINVAL, "zero_lamb_plan_create: n=%lld outside [0, 2^40]", (long long)n);
    if (n_seg < 0 || (n == 0) != (n_seg == 0))
        return fail(ZERO_EINVAL, "zero_lamb_plan_create: need n_seg > 0 for n > 0 and n_seg = 0 for n = 0");
    if (n_seg > 0) {
        if (!seg_off)
            return fail(ZERO_EINVAL, "zero_lamb_plan_create: NULL seg_off");
        if (seg_off[0] != 0 || seg_off[n_seg] != n)
            return fail(ZERO_EINVAL, "zero_lamb_plan_create: seg_off must start at 0 and end at n");
        for (int32_t s = 0; s < n_seg; ++s)
            if (seg_off[s + 1] <= seg_off[s])
                return fail(ZERO_EINVAL, "zero_lamb_plan_create: seg_off must rise strictly (layer %d)", s);
    }
    std::unique_ptr<zero_lamb_plan> p(new zero_lamb_plan);
    HIP_TRY(hipGetDevice(&p->dev));
    p->n = n;
    p->n_seg = n_seg;
    if (n_seg > 0)
        p->seg_off.assign(seg_off, seg_off + n_seg + 1);
    else
        p->seg_off.assign(1, 0);
    p->max_items = max_items_for(n, n_seg);
    p->max_chunks = max_chunks_for(p->max_items, n_seg);
    if (hipEventCreateWithFlags(&p->done, hipEventDisableTiming) != hipSuccess) {
        p->done = nullptr;
        (void)hipGetLastError();
        return fail(ZERO_EHIP, "zero_lamb_plan_create: could not create the plan's event");
    }
    if (n > 0) {
        if (hipMalloc(reinterpret_cast<void**>(&p->part), (size_t)p->max_items * sizeof(zs::LayerSums)) !=
                hipSuccess ||
            hipMalloc(reinterpret_cast<void**>(&p->cpart), (size_t)p->max_chunks * sizeof(zs::LayerSums)) !=
                hipSuccess ||
            hipMalloc(reinterpret_cast<void**>(&p->sums), (size_t)n_seg * sizeof(zs::LayerSums)) != hipSuccess) {
            (void)hipGetLastError();
            free_plan(p.get());
            return fail(ZERO_ENOMEM, "zero_lamb_plan_create: could not allocate the plan workspace");
        }
        hipDeviceProp_t prop;
        if (hipGetDeviceProperties(&prop, p->dev) != hipSuccess) {
            (void)hipGetLastError();
            free_plan(p.get());
            return fail(ZERO_EHIP, "zero_lamb_plan_create: hipGetDeviceProperties failed");
        }
        int resident = 0;
        p->lds[0] = occupancy_lds(moments_kernel<true>(), kLambBlock, kLambPerCU, prop, &resident);
        p->lds[1] = occupancy_lds(apply_kernel<true>(), kLambBlock, kLambPerCU, prop, &resident);
        p->lds_scalar[0] = occupancy_lds(moments_kernel<false>(), kLambBlock, kLambPerCU, prop, &resident);
        p->lds_scalar[1] = occupancy_lds(apply_kernel<false>(), kLambBlock, kLambPerCU, prop, &resident);
    }
    *out = p.release();
    return ZERO_OK;
}

int zero_lamb_plan_destroy(zero_lamb_plan_t* plan) {
    if (!plan)
        return ZERO_OK;
    int rc = ZERO_OK;
    {
        std::lock_guard<std::mutex> lk(plan->mu);
        int cur = 0;
        if (hipGetDevice(&cur) == hipSuccess && cur != plan->dev)
            (void)hipSetDevice(plan->dev);
        // the plan's last call recorded `done` after its kernels, and every call waited
        // for the previous one's, so this waits for all of the plan's work
        if (plan->used && hipEventSynchronize(plan->done) != hipSuccess) {
            (void)hipGetLastError();
            rc = fail(ZERO_EHIP, "zero_lamb_plan_destroy: waiting for the plan's work failed");
        }
        free_plan(plan);
        if (cur != plan->dev)
            (void)hipSetDevice(cur);
    }
    delete plan;
    return rc;
}

int zero_lamb_step(const zero_lamb_plan_t* plan_, const uint16_t* grad16, float* master32, float* m32, float* v32,
                   uint16_t* param16_out, double lr, double beta1, double beta2, double eps, double weight_decay,
                   int64_t step, double loss_scale, double clip, double phi_lo, double phi_hi, void* stream_) {
    const char* fn = "zero_lamb_step";
    zero_lamb_plan* plan = const_cast<zero_lamb_plan*>(plan_);
    int rc = check_plan(fn, plan);
    if (rc || (rc = check_hyper(fn, lr, beta1, beta2, eps, weight_decay, step, loss_scale, clip)) ||
        (rc = check_phi(fn, phi_lo, phi_hi)))
        return rc;
    const int64_t n = plan->n;
    if (n > 0 && (!grad16 || !master32 || !m32 || !v32 || !param16_out))
        return fail(ZERO_EINVAL, "%s: NULL array with n > 0", fn);
    const void* arrays[5] = {grad16, master32, m32, v32, param16_out};
    if ((rc = check_lamb_arrays(fn, arrays, n)))
        return rc;
    if (n == 0) {
        t_stats = zero_step_stats_t{0.0, 0.0, 1.0, (float)(1.0 / loss_scale), 0, 0, 0, 0};
        t_have_stats = true;
        return ZERO_OK;
    }
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    std::lock_guard<std::mutex> plk(plan->mu);
    CtxLock ctx;
    if ((rc = lock_ctx(stream, &ctx)))
        return rc;
    const int phase = phase_of(grad16, master32, m32, v32, param16_out);
    LambWork* w = nullptr;
    if ((rc = get_work(plan, phase, &w)) || (rc = switch_stream(plan, stream)))
        return rc;
    const zs::AdamConst c = adam_const(lr, beta1, beta2, eps, weight_decay, step);
    const uint32_t seq = next_seq(ctx.get());
    LambProfRec pr;
    bool prof = lprof_begin(plan, &pr);
    const bool sampled = prof;
    lprof_record(&pr, &prof, 0, stream);
    rc = launch_stats_planned(ctx.get(), grad16, n, loss_scale, clip, seq, stream);
    lprof_record(&pr, &prof, 1, stream);
    if (!rc)
        rc = launch_moments(plan, *w, phase, grad16, master32, m32, v32, ctx->res, c, stream);
    lprof_record(&pr, &prof, 2, stream);
    if (!rc)
        rc = launch_layer(plan, *w, plan->sums, ctx->res, stream);
    lprof_record(&pr, &prof, 3, stream);
    if (!rc)
        rc = launch_apply(plan, *w, phase, master32, m32, v32, param16_out, plan->sums, ctx->res, c, lr, phi_lo,
                          phi_hi, stream);
    lprof_record(&pr, &prof, 4, stream);
    if (sampled)
        lprof_end(pr, prof && !rc);
    const int rc_done = mark_done(plan, stream);
    if (rc || (rc = rc_done))
        return rc;
    zs::Result r;
    if ((rc = wait_result(ctx.get(), seq, stream, &r)))
        return rc;
    set_last_stats(r, n);
    return r.skip ? ZERO_SKIPPED : ZERO_OK;
}

int zero_lamb_moments(const zero_lamb_plan_t* plan_, const uint16_t* grad16, const float* master32, float* m32,
                      float* v32, double global_sumsq, double beta1, double beta2, double eps, double weight_decay,
                      int64_t step, double loss_scale, double clip, double* layer_sumsq, void* stream_) {
    const char* fn = "zero_lamb_moments";
    zero_lamb_plan* plan = const_cast<zero_lamb_plan*>(plan_);
    int rc = check_plan(fn, plan);
    if (rc || (rc = check_hyper(fn, 0.0, beta1, beta2, eps, weight_decay, step, loss_scale, clip)))
        return rc;
    if (std::isnan(global_sumsq) || global_sumsq < 0.0)
        return fail(ZERO_EINVAL, "%s: global_sumsq must be >= 0 (+inf for an overflow)", fn);
    const int64_t n = plan->n;
    if (n > 0 && (!grad16 || !master32 || !m32 || !v32))
        return fail(ZERO_EINVAL, "%s: NULL array with n > 0", fn);
    const void* arrays[5] = {grad16, master32, m32, v32, nullptr};
    if ((rc = check_lamb_arrays(fn, arrays, n)))
        return rc;
    if (n > 0 && (rc = check_layer_sums(fn, plan, layer_sumsq, arrays)))
        return rc;
    if (!std::isfinite(global_sumsq))
        return ZERO_SKIPPED;
    if (n == 0)
        return ZERO_OK;
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    std::lock_guard<std::mutex> plk(plan->mu);
    CtxLock ctx;
    if ((rc = lock_ctx(stream, &ctx)))
        return rc;
    const int phase = phase_of(grad16, master32, m32, v32, nullptr);
    LambWork* w = nullptr;
    if ((rc = get_work(plan, phase, &w)) || (rc = switch_stream(plan, stream)))
        return rc;
    const zs::AdamConst c = adam_const(0.0, beta1, beta2, eps, weight_decay, step);
    const uint32_t seq = next_seq(ctx.get());
    zs::k_set_result<<<1, 64, 0, stream>>>(ctx->res, global_sumsq, loss_scale, clip, seq);
    rc = hipGetLastError() == hipSuccess ? ZERO_OK : fail(ZERO_EHIP, "%s: result-record launch failed", fn);
    if (!rc)
        rc = launch_moments(plan, *w, phase, grad16, master32, m32, v32, ctx->res, c, stream);
    if (!rc)
        rc = launch_layer(plan, *w, reinterpret_cast<zs::LayerSums*>(layer_sumsq), ctx->res, stream);
    const int rc_done = mark_done(plan, stream);
    return rc ? rc : rc_done;
}

int zero_lamb_apply(const zero_lamb_plan_t* plan_, float* master32, const float* m32, const float* v32,
                    uint16_t* param16_out, double global_sumsq, const double* layer_sumsq, double lr, double beta1,
                    double beta2, double eps, double weight_decay, int64_t step, double phi_lo, double phi_hi,
                    void* stream_) {
    const char* fn = "zero_lamb_apply";
    zero_lamb_plan* plan = const_cast<zero_lamb_plan*>(plan_);
    int rc = check_plan(fn, plan);
    if (rc || (rc = check_hyper(fn, lr, beta1, beta2, eps, weight_decay, step, 1.0, 0.0)) ||
        (rc = check_phi(fn, phi_lo, phi_hi)))
        return rc;
    if (std::isnan(global_sumsq) || global_sumsq < 0.0)
        return fail(ZERO_EINVAL, "%s: global_sumsq must be >= 0 (+inf for an overflow)", fn);
    const int64_t n = plan->n;
    if (n > 0 && (!master32 || !m32 || !v32 || !param16_out))
        return fail(ZERO_EINVAL, "%s: NULL array with n > 0", fn);
    const void* arrays[5] = {nullptr, master32, m32, v32, param16_out};
    if ((rc = check_lamb_arrays(fn, arrays, n)))
        return rc;
    if (n > 0 && (rc = check_layer_sums(fn, plan, layer_sumsq, arrays)))
        return rc;
    if (!std::isfinite(global_sumsq))
        return ZERO_SKIPPED;
    if (n == 0)
        return ZERO_OK;
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    std::lock_guard<std::mutex> plk(plan->mu);
    CtxLock ctx;
    if ((rc = lock_ctx(stream, &ctx)))
        return rc;
    const int phase = phase_of(nullptr, master32, m32, v32, param16_out);
    LambWork* w = nullptr;
    if ((rc = get_work(plan, phase, &w)) || (rc = switch_stream(plan, stream)))
        return rc;
    const zs::AdamConst c = adam_const(lr, beta1, beta2, eps, weight_decay, step);
    const uint32_t seq = next_seq(ctx.get());
    // the apply kernel reads only the skip flag of the record: not skipped here
    zs::k_set_result<<<1, 64, 0, stream>>>(ctx->res, 0.0, 1.0, 0.0, seq);
    rc = hipGetLastError() == hipSuccess ? ZERO_OK : fail(ZERO_EHIP, "%s: result-record launch failed", fn);
    if (!rc)
        rc = launch_apply(plan, *w, phase, master32, m32, v32, param16_out,
                          reinterpret_cast<const zs::LayerSums*>(layer_sumsq), ctx->res, c, lr, phi_lo, phi_hi,
                          stream);
    const int rc_done = mark_done(plan, stream);
    return rc ? rc : rc_done;
}

int zero_probe_lamb_pass(int32_t pass, const uint16_t* grad16, float* master32, float* m32, float* v32,
                         uint16_t* param16_out, int64_t n, void* stream_) {
    const char* fn = "zero_probe_lamb_pass";
    if (pass != 0 && pass != 1)
        return fail(ZERO_EINVAL, "%s: pass must be 0 (moments) or 1 (apply)", fn);
    if (n < 0 || n > kMaxNumel)
        return fail(ZERO_EINVAL, "%s: n=%lld outside [0, 2^40]", fn, (long long)n);
    if (n == 0)
        return ZERO_OK;
    const void* arrays[5] = {pass == 0 ? grad16 : nullptr, master32, m32, v32, pass == 1 ? param16_out : nullptr};
    static const size_t align[5] = {8, 16, 16, 16, 8};
    for (int i = 0; i < 5; ++i)
        if (arrays[i] == nullptr && ((pass == 0 && i != 4) || (pass == 1 && i != 0)))
            return fail(ZERO_EINVAL, "%s: NULL array %d", fn, i);
        else if (arrays[i] && reinterpret_cast<uintptr_t>(arrays[i]) % align[i])
            return fail(ZERO_EINVAL, "%s: array %d must be %zu-byte aligned", fn, i, align[i]);
    int rc = check_lamb_arrays(fn, arrays, n);
    if (rc)
        return rc;
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    hipDeviceProp_t prop;
    HIP_TRY(hipGetDeviceProperties(&prop, dev));
    const void* kern = pass == 0 ? probe_kernel<0>() : probe_kernel<1>();
    int resident = 0;
    const size_t lds = occupancy_lds(kern, kLambBlock, kLambPerCU, prop, &resident);
    const int64_t ntiles = (n + kLambTile - 1) / kLambTile;
    const unsigned grid = tile_grid(ntiles);
    hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
    if (pass == 0)
        zs::k_probe_lamb<kLambBlock, kLambUnroll, kLambNTL, kLambNTS, kLambXCD, 0>
            <<<grid, kLambBlock, lds, stream>>>(grad16, master32, m32, v32, param16_out, ntiles, n);
    else
        zs::k_probe_lamb<kLambBlock, kLambUnroll, kLambNTL, kLambNTS, kLambXCD, 1>
            <<<grid, kLambBlock, lds, stream>>>(grad16, master32, m32, v32, param16_out, ntiles, n);
    HIP_TRY(hipGetLastError());
    return ZERO_OK;
}

int zero_lamb_profile_read(zero_lamb_profile_t* out) {
    if (!out)
        return fail(ZERO_EINVAL, "zero_lamb_profile_read: NULL out");
    std::lock_guard<std::mutex> lk(g_lprof_mu);
    lprof_drain_locked();
    const int rc = prof_take_error(1);
    *out = g_lprof_acc;
    g_lprof_acc = zero_lamb_profile_t{0, 0.0, 0.0, 0.0, 0.0};
    return rc;
}

}  // extern "C"
