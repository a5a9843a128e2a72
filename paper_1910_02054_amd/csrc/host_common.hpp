// host_common.hpp -- host-side internals of libzeroshard shared by its
// translation units (zero_shard.hip: Adam step, layout, accounting, scaler,
// profiling; zero_lamb.hip: the LAMB step).  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
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

// Per-(device, stream) context: the constant-size workspace of the gradient
// statistics and the result record the update kernels read.
struct Ctx {
    std::mutex mu;
    zs::Partial* part = nullptr;    // kMaxStatsBlocks partial records (device)
    zs::Result* res = nullptr;      // result record (device), read by the update kernel
    zs::Result* host = nullptr;     // host-mapped, GPU-uncached copy of the result record
    zs::Result* host_dev = nullptr; // its device-side address
    zs::AdamConst* dconst = nullptr; // fp32 constants of the resident step (device)
    hipEvent_t prof_last_end = nullptr;  // end event of the last profiled update on this stream
    uint64_t prof_tick = 0;              // steps seen while profiling (for sampling)
    uint32_t seq = 0;               // call counter echoed in the result record
    int ncu = 0;
    size_t stats_lds = 0, adam_lds = 0;   // occupancy reservations (dynamic LDS per workgroup)
    int stats_resident = 0, adam_resident = 0;
};

// The context of (current device, stream), created on first use; rejects a
// stream of another device.
int get_ctx(hipStream_t stream, Ctx** out);

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

}  // namespace zsh
