// host_common.hpp -- host-side internals of libzeroshard shared by its
// translation units (zero_shard.hip: Adam step, layout, accounting, scaler,
// profiling; zero_lamb.hip: the LAMB step).  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <memory>
#include <mutex>
#include <string>

#include "zero_shard.h"
#include "shard_kernels.hpp"

namespace zsh {

// Thread-local error text (zero_last_error) and statistics of the calling
// thread's last successful step (zero_shard_last_stats).
extern thread_local std::string t_err;
extern thread_local zero_step_stats_t t_stats;
extern thread_local bool t_have_stats;

// Records the message for zero_last_error and returns `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

#define HIP_TRY(expr)                                                                        \
    do {                                                                                     \
        hipError_t e_ = (expr);                                                              \
        if (e_ != hipSuccess)                                                                \
            return ::zsh::fail(ZERO_EHIP, "%s: %s", #expr, hipGetErrorString(e_));           \
    } while (0)

constexpr int64_t kMaxNumel = (int64_t)1 << 40;

// Per-device launch facts, computed once per device (no allocation): compute
// units and the dynamic-LDS reservations that cap resident workgroups of the
// streaming kernels (occupancy_lds), the update's byte-mix probe included.
struct DevInfo {
    int ncu = 0;
    size_t stats_lds = 0, adam_lds = 0, probe_adam_lds = 0;
    int stats_resident = 0, adam_resident = 0, probe_adam_resident = 0;
    int64_t small_cap[4] = {};  // co-resident workgroups of k_small_step<1, 2, 4, 8>
    int64_t small_share = 4;    // a one-launch grid takes at most small_cap / small_share
};

// The facts of device `dev` (0 <= dev < kMaxDevices), filled on first use.
int dev_info(int dev, const DevInfo** out);
constexpr int kMaxDevices = 64;

// Per-(device, stream) context: the constant-size workspace of the gradient
// statistics and the result record the update kernels read.  A context is
// shared (std::shared_ptr) between the registry and the calls using it, so a
// release (zero_stream_release) never frees memory under a running call: the
// releasing thread takes `mu`, waits for the stream, frees the device buffers
// and marks the context released; a call that locks it afterwards sees the
// mark and takes a fresh context.
struct Ctx {
    std::mutex mu;
    int dev = 0;
    hipStream_t stream = nullptr;
    zs::Partial* part = nullptr;    // kMaxStatsBlocks partial records (device)
    zs::Result* res = nullptr;      // result record (device), read by the update kernel
    zs::Result* host = nullptr;     // host-mapped, GPU-uncached copy of the result record
    zs::Result* host_dev = nullptr; // its device-side address
    uint64_t* sync = nullptr;       // grid-barrier words of the small-shard step (device)
    bool sync_ready = false;        // the words have been zeroed on the stream
    uint64_t prof_tick = 0;         // steps seen while profiling (for sampling)
    uint64_t prof_epoch = 0;        // profiling period the tick belongs to
    uint32_t seq = 0;               // call counter echoed in the result record
    bool released = false;
    const DevInfo* info = nullptr;
};

// A context of (current device, stream), locked for the duration of a call.
struct CtxLock {
    std::shared_ptr<Ctx> ref;
    std::unique_lock<std::mutex> lk;
    Ctx* operator->() const { return ref.get(); }
    Ctx* get() const { return ref.get(); }
};

// The locked context of (current device, stream), created on first use;
// rejects a stream of another device.
int lock_ctx(hipStream_t stream, CtxLock* out);

// Next call sequence number of a context (never 0).  Caller holds ctx->mu.
uint32_t next_seq(Ctx* ctx);

bool is_fin(double x);
bool overlaps(uintptr_t a, size_t an, uintptr_t b, size_t bn);

// Scalar arguments shared by every update: finite lr >= 0, eps >= 0, finite
// weight decay, beta1/beta2 in [0, 1), step >= 1, finite loss_scale > 0,
// clip not NaN.
int check_hyper(const char* fn, double lr, double beta1, double beta2, double eps, double weight_decay, int64_t step,
                double loss_scale, double clip);

// Each ptrs[i] .. ptrs[i] + bytes[i] inside one GPU-accessible allocation.
int check_ranges(const char* fn, const void* const* ptrs, const size_t* bytes, int count);

// Dynamic LDS that caps resident workgroups of `kernel` at `per_cu` per CU.
size_t occupancy_lds(const void* kernel, int block, int per_cu, const hipDeviceProp_t& prop, int* resident);

// The fp32 constants of the Adam moments and direction.
zs::AdamConst adam_const(double lr, double beta1, double beta2, double eps, double wd, int64_t step);

// Statistics + finalize of grad16[0, n) with the production launch shape; the
// result record lands in ctx->res and in the host-mapped ctx->host.
int launch_stats_planned(Ctx* ctx, const uint16_t* grad16, int64_t n, double loss_scale, double clip, uint32_t seq,
                         hipStream_t stream);

// Waits (host polling) until the finalize kernel has published call `seq`.
int wait_result(Ctx* ctx, uint32_t seq, hipStream_t stream, zs::Result* out);

// Sampling period of kernel profiling (0 = off), set by zero_profile_enable.
int prof_every();

// Records a profiling failure that happened after a step's kernels were
// queued (slot 0: Adam steps, read by zero_profile_read; slot 1: LAMB steps,
// read by zero_lamb_profile_read), so the step itself does not fail.
void prof_defer_error(int slot, const char* what, hipError_t e);

// The deferred profiling error of `slot` as a return code (0 if none), its
// message moved to zero_last_error; clears the slot.
int prof_take_error(int slot);

}  // namespace zsh
