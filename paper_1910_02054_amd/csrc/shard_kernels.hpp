// shard_kernels.hpp -- gfx950 kernels of the ZeRO P_os+g shard step.
//
// ZeRO (arXiv 1910.02054) Sec. 5.1-5.2: after the reduce-scatter each
// data-parallel rank holds the fp16 gradients of its 1/N_d partition and
// updates only that partition's fp32 master parameters, momentum and variance
// (Sec. 3.1's mixed-precision Adam), then publishes the fp16 parameters.
//
// Three kernels run per step, all HBM-streaming (no dense contraction, so no
// MFMA):
//   k_stats     one read of the fp16 gradients; per-workgroup fp64 sum of the
//               exact fp32 squares (wave shuffle, then LDS across waves).  The
//               sum is non-finite iff some gradient is inf or NaN, which is the
//               overflow test (every finite square is below 2^32, so no finite
//               sum over fewer than 2^990 elements overflows fp64).
//   k_finalize  one workgroup: fixed-order reduction of the partials; the norm
//               of the unscaled gradient, the global-norm clipping coefficient,
//               the fp32 gradient multiplier and the skip flag, written to
//               device memory and to a host-mapped record.
//   k_adam_*    the fused update: unscale+clip, Adam with bias correction, fp16
//               cast; 14 bytes read and 14 bytes written per element.
// Small shards take one launch instead (k_small_step): every thread keeps
// its elements in registers, the workgroups meet at a grid barrier after the
// statistics, each totals the partials in the same fixed order, and the update
// follows from the registers (28 bytes per element, one launch).
// The other ways of running the same step swap only the one-thread kernels
// around these: the split phase takes the global sum from the host
// (k_set_result) or from device memory (k_finalize_sum writes a rank's local
// sum, k_set_result_dev reads the combined one); the resident step's
// k_resident_begin takes the finalize's place and also derives the fp32
// constants from a state record in device memory and runs the loss-scale
// schedule there.
//
// Numerics: every fp32 operation of the update is correctly rounded (IEEE
// division and square root, no contraction), in the order Adam's bias-corrected
// form is written, so an element's result depends only on its own inputs and
// the shared scalars.  The bias corrections 1 - beta^t come from one
// definition shared by the host and the device (bias_correction below).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "zero_shard.h"

namespace zs {

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kMaxStatsBlocks = 4096;  // partial-sum records in the workspace
constexpr int kScalarBlock = 256;

// Launch-policy knobs of the streaming kernels are template parameters:
//   BLOCK  threads per workgroup;  U  vectors per thread per tile;
//   NTL/NTS  non-temporal (streaming) loads/stores;
//   XCD    remap workgroups so that each of the 8 XCDs walks a contiguous run of
//          tiles (the dispatcher assigns workgroup b to XCD b mod 8);
//   REV    walk the tiles from the end of the shard to its start.
template <bool NT, typename T>
__device__ __forceinline__ T ld(const T* p) {
    if constexpr (NT)
        return __builtin_nontemporal_load(p);
    else
        return *p;
}

template <bool NT, typename T>
__device__ __forceinline__ void st(T v, T* p) {
    if constexpr (NT)
        __builtin_nontemporal_store(v, p);
    else
        *p = v;
}

template <bool XCD>
__device__ __forceinline__ int64_t logical_block() {
    const unsigned b = blockIdx.x, grid = gridDim.x;
    if constexpr (XCD) {
        if (grid % 8 == 0)
            return (int64_t)(b % 8) * (grid / 8) + b / 8;  // a bijection of [0, grid)
    }
    return b;
}

// Per-workgroup partial of the statistics pass.
struct alignas(16) Partial {
    double sumsq;
    double unused;
};

// The step's shared scalars, produced on the device by k_finalize and read by
// the update kernel (and by the host through a mapped copy for the skip
// decision).
struct alignas(16) Result {
    double sumsq;    // sum of grad16^2 (loss-scaled); non-finite iff overflow
    double norm;     // sqrt(sumsq) / loss_scale
    double coef;     // clipping coefficient
    float mult;      // (float)(coef / loss_scale)
    int32_t skip;    // 1 = overflow: the update kernel writes nothing
    int32_t overflow;
    uint32_t seq;    // call sequence number, echoed so the host can check freshness
    int32_t unused[2];
};

// fp32 constants of the update, each rounded once from a double (on the host,
// or on the device for the resident step).
struct AdamConst {
    float lr, b1, omb1, b2, omb2, bc1, bc2, eps, wd;
};

// beta^t for an integer t >= 0, as the double nearest the exact power.  Binary
// powering in double-double arithmetic: each product's rounding error is
// recovered exactly with a fused multiply-add, so the pair carries the power to
// about 2^-90 relative error before the one final rounding to double (the
// exact power of a double is never a midpoint between doubles for t >= 2).
// Every operation is a correctly rounded IEEE multiply, add or fused
// multiply-add, so the host and the device compute the same bits.
struct DDouble {
    double hi, lo;
};

__host__ __device__ inline DDouble dd_mul(DDouble a, DDouble b) {
    const double p = a.hi * b.hi;
    double e = __builtin_fma(a.hi, b.hi, -p);
    e = e + (a.hi * b.lo + a.lo * b.hi);
    const double s = p + e;
    return DDouble{s, e - (s - p)};
}

__host__ __device__ inline double pow_int(double b, int64_t t) {
    DDouble r{1.0, 0.0}, x{b, 0.0};
    while (t > 0) {
        if (t & 1)
            r = dd_mul(r, x);
        t >>= 1;
        if (t)
            x = dd_mul(x, x);
    }
    return r.hi;
}

// The fp32 bias correction 1 - beta^t of Adam's moment estimates: the power
// rounded to double, the difference in double, then one rounding to fp32.
__host__ __device__ inline float bias_correction(double beta, int64_t t) {
    return (float)(1.0 - pow_int(beta, t));
}

// The fp32 constants from the hyperparameters (each computed in double and
// rounded once).
__host__ __device__ inline AdamConst make_adam_const(double lr, double beta1, double beta2, double eps, double wd,
                                                     int64_t t) {
    AdamConst c;
    c.lr = (float)lr;
    c.b1 = (float)beta1;
    c.omb1 = (float)(1.0 - beta1);
    c.b2 = (float)beta2;
    c.omb2 = (float)(1.0 - beta2);
    c.bc1 = bias_correction(beta1, t);
    c.bc2 = bias_correction(beta2, t);
    c.eps = (float)eps;
    c.wd = (float)wd;
    return c;
}

// The hyperparameter ranges every step accepts (the synchronous entry points
// check the same on the host): lr, eps >= 0 and finite, weight decay finite,
// beta1, beta2 in [0, 1), t >= 1, loss scale finite and > 0, clip not NaN.
__host__ __device__ inline bool hyper_ok(double lr, double beta1, double beta2, double eps, double wd, int64_t t,
                                         double loss_scale, double clip) {
    return __builtin_isfinite(lr) && lr >= 0.0 && __builtin_isfinite(eps) && eps >= 0.0 && __builtin_isfinite(wd) &&
           beta1 >= 0.0 && beta1 < 1.0 && beta2 >= 0.0 && beta2 < 1.0 && t >= 1 && __builtin_isfinite(loss_scale) &&
           loss_scale > 0.0 && !__builtin_isnan(clip);
}

// A resident state record the step can run from: hyper_ok plus a finite
// min_scale > 0.
__host__ __device__ inline bool resident_record_ok(const zero_resident_state_t& s) {
    return hyper_ok(s.lr, s.beta1, s.beta2, s.eps, s.weight_decay, s.t, s.loss_scale, s.clip) &&
           __builtin_isfinite(s.min_scale) && s.min_scale > 0.0;
}

__device__ __forceinline__ float f16_to_f32(uint32_t bits16) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

__device__ __forceinline__ uint32_t f32_to_f16(float x) {
    // v_cvt_f16_f32 in the default round-to-nearest-even mode, fp16 denormals kept.
    return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)x);
}

// acc + g^2 for both halves of a 32-bit word; the square of a binary16 value
// is exact in fp32 (22 significant bits) and in fp64.
__device__ __forceinline__ double acc_sq2(uint32_t w, double acc) {
    double lo = (double)f16_to_f32(w & 0xFFFFu);
    double hi = (double)f16_to_f32(w >> 16);
    acc = __builtin_fma(lo, lo, acc);
    return __builtin_fma(hi, hi, acc);
}

__device__ __forceinline__ double sq1(uint32_t bits16) {
    double d = (double)f16_to_f32(bits16);
    return d * d;
}

__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        x += __shfl_xor(x, off, 64);
    return x;
}

// Fixed-order sum of one double per thread over a workgroup of BLOCK threads;
// the total is returned to thread 0.
template <int BLOCK>
__device__ __forceinline__ double block_sum(double x) {
    __shared__ double lds[BLOCK / 64];
    x = wave_sum(x);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if constexpr (BLOCK == 64) {
        return x;
    } else {
        if (lane == 0)
            lds[wave] = x;
        __syncthreads();
        double s = 0.0;
        if (threadIdx.x == 0) {
#pragma unroll
            for (int w = 0; w < BLOCK / 64; ++w)
                s += lds[w];
        }
        return s;
    }
}

// Norm, clipping coefficient, multiplier and skip flag from the global sum of
// squares (all in double; the multiplier rounded once to fp32).
__device__ __forceinline__ Result make_result(double tot, double loss_scale, double clip, uint32_t seq) {
    Result r;
    r.sumsq = tot;
    r.overflow = __builtin_isfinite(tot) ? 0 : 1;
    r.skip = r.overflow;
    if (r.overflow) {
        r.norm = __builtin_inf();
        r.coef = 1.0;
        r.mult = 0.0f;
    } else {
        r.norm = __builtin_sqrt(tot) / loss_scale;
        r.coef = (clip > 0.0 && r.norm > clip) ? clip / r.norm : 1.0;
        r.mult = (float)(r.coef / loss_scale);
    }
    r.seq = seq;
    r.unused[0] = r.unused[1] = 0;
    return r;
}

// ---------------------------------------------------------------------------
// K1: statistics.  `head` leading elements (0..7) are not 16-byte aligned and
// `nvec` 8-element vectors follow; elements [head + 8*nvec, n) are the tail.
// Grid: 1 .. kMaxStatsBlocks workgroups of BLOCK threads; workgroup b writes
// part[b].
// ---------------------------------------------------------------------------
template <int BLOCK, int U, bool NTL, bool XCD>
__global__ __launch_bounds__(BLOCK) void k_stats(const uint16_t* __restrict__ g, int64_t n, int64_t head,
                                                 int64_t nvec, Partial* __restrict__ part) {
    double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
    const u32x4* __restrict__ gv = reinterpret_cast<const u32x4*>(g + head);
    const int64_t tile = (int64_t)BLOCK * U;
    const int64_t stride = (int64_t)gridDim.x * tile;
    for (int64_t base = logical_block<XCD>() * tile + threadIdx.x; base < nvec; base += stride) {
        u32x4 q[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = base + (int64_t)u * BLOCK;
            q[u] = i < nvec ? ld<NTL>(gv + i) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            a0 = acc_sq2(q[u].x, a0);
            a1 = acc_sq2(q[u].y, a1);
            a2 = acc_sq2(q[u].z, a2);
            a3 = acc_sq2(q[u].w, a3);
        }
    }
    if (blockIdx.x == 0) {
        const int64_t t = threadIdx.x;
        const int64_t tail0 = head + 8 * nvec;
        if (t < head)
            a0 += sq1(g[t]);
        if (t < 8 && tail0 + t < n)
            a1 += sq1(g[tail0 + t]);
    }
    const double s = block_sum<BLOCK>((a0 + a1) + (a2 + a3));
    if (threadIdx.x == 0)
        part[blockIdx.x].sumsq = s;
}

// ---------------------------------------------------------------------------
// K2: finalize.  One workgroup of kFinalBlock threads; fixed-order reduction,
// so the result depends only on the partials (bitwise reproducible for a given
// launch shape).  `res_host` is host-mapped and GPU-uncached; its sequence
// number is stored last, with release semantics at system scope, so a host
// that sees the expected sequence number sees the whole record.
// ---------------------------------------------------------------------------
constexpr int kFinalBlock = 256;

// The total of part[0, nparts) in a fixed order (every thread of the
// kFinalBlock-thread workgroup returns it); 0 for nparts = 0.
__device__ __forceinline__ double partials_total(const Partial* __restrict__ part, int nparts) {
    double s0 = 0.0, s1 = 0.0;
    int i = threadIdx.x;
    for (; i + kFinalBlock < nparts; i += 2 * kFinalBlock) {
        s0 += part[i].sumsq;
        s1 += part[i + kFinalBlock].sumsq;
    }
    if (i < nparts)
        s0 += part[i].sumsq;
    return block_sum<kFinalBlock>(s0 + s1);
}

[[maybe_unused]] static __global__ __launch_bounds__(kFinalBlock) void k_finalize(
    const Partial* __restrict__ part, int nparts, Result* __restrict__ res, Result* __restrict__ res_host,
    double loss_scale, double clip, uint32_t seq) {
    const double tot = partials_total(part, nparts);
    if (threadIdx.x == 0) {
        const Result r = make_result(tot, loss_scale, clip, seq);
        *res = r;
        // publish to the host: the record first, then its sequence number with a
        // system-scope release (the host polls the sequence number)
        Result rh = r;
        rh.seq = 0;
        *res_host = rh;
        __hip_atomic_store(&res_host->seq, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

// One double into device memory (the empty shard's local sum, enqueued in order).
[[maybe_unused]] static __global__ __launch_bounds__(64) void k_set_value(double* __restrict__ out, double value) {
    if (threadIdx.x == 0)
        *out = value;
}

// Zeroes n 64-bit words (counters cleared in stream order).
[[maybe_unused]] static __global__ __launch_bounds__(256) void k_zero_words(uint64_t* __restrict__ out, int64_t n) {
    for (int64_t i = threadIdx.x; i < n; i += 256)
        out[i] = 0;
}

// Statistics total into caller device memory (the asynchronous split phase:
// no result record, no host copy).
[[maybe_unused]] static __global__ __launch_bounds__(kFinalBlock) void k_finalize_sum(
    const Partial* __restrict__ part, int nparts, double* __restrict__ out) {
    const double tot = partials_total(part, nparts);
    if (threadIdx.x == 0)
        *out = tot;
}

// Result record from a global sum of squares in device memory (the
// asynchronous split phase); the skip flag also goes to `skipped` when given
// (device or host-mapped memory).
[[maybe_unused]] static __global__ __launch_bounds__(64) void k_set_result_dev(Result* __restrict__ res,
                                                                                const double* __restrict__ global,
                                                                                double loss_scale, double clip,
                                                                                int32_t* __restrict__ skipped,
                                                                                uint32_t seq) {
    if (threadIdx.x == 0) {
        double g = *global;
        if (!(g >= 0.0))
            g = __builtin_inf();  // negative or NaN: not a sum of squares, skip like an overflow
        const Result r = make_result(g, loss_scale, clip, seq);
        *res = r;
        if (skipped)
            *skipped = r.skip;
    }
}

// Resident step, before the update, in one workgroup: the statistics total
// (as k_finalize forms it), the result record from it and the state record's
// loss scale and clip, the fp32 constants from the record's hyperparameters
// and t (make_adam_const, the host's definition), and then the loss-scale
// schedule on the record: after an overflow the scale halves (not below
// min_scale) and t stays; otherwise t and the good-step count advance and the
// scale doubles after `window` good steps.  The update kernel reads only the
// result record and the constants, so the schedule need not wait for it.  A
// record outside the accepted ranges (resident_record_ok) is left unchanged
// except for skipped = -1, and the step writes nothing.
// The resident step's decision from the statistics total and the record `s`
// read before the step: the result record, and the record's new scaler fields
// written to *st (skipped = -1 and nothing else for a record out of range).
__device__ __forceinline__ Result resident_advance(zero_resident_state_t* __restrict__ st,
                                                   const zero_resident_state_t& s, double tot, uint32_t seq) {
    if (!resident_record_ok(s)) {
        Result r = make_result(0.0, 1.0, 0.0, seq);
        r.skip = 1;
        st->skipped = -1;
        return r;
    }
    const Result r = make_result(tot, s.loss_scale, s.clip, seq);
    st->steps = s.steps + 1;
    st->skipped = r.skip;
    if (r.skip) {
        const double h = s.loss_scale * 0.5;
        st->loss_scale = h > s.min_scale ? h : s.min_scale;
        st->good = 0;
    } else {
        st->t = s.t + 1;
        int64_t good = s.good + 1;
        if (s.window > 0 && good >= s.window) {
            st->loss_scale = s.loss_scale * 2.0;
            good = 0;
        }
        st->good = good;
    }
    return r;
}

[[maybe_unused]] static __global__ __launch_bounds__(kFinalBlock) void k_resident_begin(
    const Partial* __restrict__ part, int nparts, zero_resident_state_t* __restrict__ st, Result* __restrict__ res,
    AdamConst* __restrict__ cout, uint32_t seq) {
    const double tot = partials_total(part, nparts);
    if (threadIdx.x == 0) {
        const zero_resident_state_t s = *st;
        *cout = make_adam_const(s.lr, s.beta1, s.beta2, s.eps, s.weight_decay, s.t);
        *res = resident_advance(st, s, tot, seq);
    }
}

// Result record from a global sum of squares supplied by the caller (the
// split-phase step: each rank's local sums combined outside the library).
[[maybe_unused]] static __global__ __launch_bounds__(64) void k_set_result(Result* __restrict__ res,
                                                                            double global_sumsq, double loss_scale,
                                                                            double clip, uint32_t seq) {
    if (threadIdx.x == 0)
        *res = make_result(global_sumsq, loss_scale, clip, seq);
}

// ---------------------------------------------------------------------------
// The per-element update: one definition for the vector body, the unaligned
// head/tail and the scalar path, so every element is computed identically.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t adam_elem(uint32_t g16, float mult, float& th, float& m, float& v,
                                              const AdamConst& c) {
#pragma clang fp contract(off)
    const float g = f16_to_f32(g16) * mult;
    const float mi = c.b1 * m + c.omb1 * g;
    const float vi = c.b2 * v + c.omb2 * (g * g);
    const float mhat = mi / c.bc1;
    const float vhat = vi / c.bc2;
    const float denom = __builtin_sqrtf(vhat) + c.eps;
    float u = mhat / denom;
    if (c.wd != 0.0f)
        u = u + c.wd * th;
    th = th - c.lr * u;
    m = mi;
    v = vi;
    return f32_to_f16(th);
}

__device__ __forceinline__ void adam_one(const uint16_t* g, float* th, float* m, float* v, uint16_t* p, int64_t i,
                                         float mult, const AdamConst& c) {
    float t = th[i], mm = m[i], vv = v[i];
    uint32_t h = adam_elem(g[i], mult, t, mm, vv, c);
    th[i] = t;
    m[i] = mm;
    v[i] = vv;
    p[i] = (uint16_t)h;
}

// Four consecutive elements of the vector path: the loaded gradient word pair
// and fp32 vectors in, the updated fp32 vectors and fp16 word pair out.
__device__ __forceinline__ void adam_vec4(u32x2 gq, f32x4 tq, f32x4 mq, f32x4 vq, float mult, const AdamConst& c,
                                          f32x4& to, f32x4& mo, f32x4& vo, u32x2& po) {
    float t[4] = {tq.x, tq.y, tq.z, tq.w};
    float mm[4] = {mq.x, mq.y, mq.z, mq.w};
    float vvv[4] = {vq.x, vq.y, vq.z, vq.w};
    const uint32_t gw[4] = {gq.x & 0xFFFFu, gq.x >> 16, gq.y & 0xFFFFu, gq.y >> 16};
    uint32_t h[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
        h[k] = adam_elem(gw[k], mult, t[k], mm[k], vvv[k], c);
    to = f32x4{t[0], t[1], t[2], t[3]};
    mo = f32x4{mm[0], mm[1], mm[2], mm[3]};
    vo = f32x4{vvv[0], vvv[1], vvv[2], vvv[3]};
    po = u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
}

// K2 (vector path).  All five arrays share the same element misalignment, so
// after `head` (0..3) scalar elements every array is aligned for 4-element
// vectors: 16-byte fp32 and 8-byte fp16 accesses, consecutive lanes on
// consecutive vectors.  A tile is BLOCK*U vectors; each thread loads its U
// vectors of all four inputs before computing (with U = 1, the production
// shape, the loads, the update and the stores sit under one bounds test,
// which measured about 4 us faster per 250M-element launch than a separate
// test for the loads and for the rest).  Elements [head + 4*nvec, n) are the
// tail (0..3).  Any grid size is valid (tiles are strided by it).  The fp32
// constants come by value, or with CDEV from device memory (the resident step
// computes them on the device).
template <int BLOCK, int U, bool NTL, bool NTS, bool XCD, bool REV, bool CDEV>
__global__ __launch_bounds__(BLOCK) void k_adam_vec(const uint16_t* __restrict__ g, float* __restrict__ th,
                                                    float* __restrict__ m, float* __restrict__ v,
                                                    uint16_t* __restrict__ p, int64_t n, int64_t head, int64_t nvec,
                                                    const Result* __restrict__ res, AdamConst c_arg,
                                                    const AdamConst* __restrict__ cdev) {
    if (res->skip)
        return;
    const float mult = res->mult;
    AdamConst c = c_arg;
    if constexpr (CDEV)
        c = *cdev;
    if (blockIdx.x == 0 && threadIdx.x < 8) {
        const int64_t t = threadIdx.x;
        const int64_t i = t < 4 ? t : head + 4 * nvec + (t - 4);
        if ((t < 4 && i < head) || (t >= 4 && i < n))
            adam_one(g, th, m, v, p, i, mult, c);
    }
    const u32x2* __restrict__ gv = reinterpret_cast<const u32x2*>(g + head);
    f32x4* __restrict__ tv = reinterpret_cast<f32x4*>(th + head);
    f32x4* __restrict__ mv = reinterpret_cast<f32x4*>(m + head);
    f32x4* __restrict__ vv = reinterpret_cast<f32x4*>(v + head);
    u32x2* __restrict__ pv = reinterpret_cast<u32x2*>(p + head);
    const int64_t tile = (int64_t)BLOCK * U;
    const int64_t ntiles = (nvec + tile - 1) / tile;
    for (int64_t tb = logical_block<XCD>(); tb < ntiles; tb += gridDim.x) {
        const int64_t base = (REV ? ntiles - 1 - tb : tb) * tile + threadIdx.x;
        if constexpr (U == 1) {
            if (base < nvec) {
                f32x4 to, mo, vo;
                u32x2 po;
                adam_vec4(ld<NTL>(gv + base), ld<NTL>(tv + base), ld<NTL>(mv + base), ld<NTL>(vv + base), mult, c,
                          to, mo, vo, po);
                st<NTS>(to, tv + base);
                st<NTS>(mo, mv + base);
                st<NTS>(vo, vv + base);
                st<NTS>(po, pv + base);
            }
        } else {
            u32x2 gq[U];
            f32x4 tq[U], mq[U], vq[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t i = base + (int64_t)u * BLOCK;
                if (i < nvec) {
                    gq[u] = ld<NTL>(gv + i);
                    tq[u] = ld<NTL>(tv + i);
                    mq[u] = ld<NTL>(mv + i);
                    vq[u] = ld<NTL>(vv + i);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t i = base + (int64_t)u * BLOCK;
                if (i < nvec) {
                    f32x4 to, mo, vo;
                    u32x2 po;
                    adam_vec4(gq[u], tq[u], mq[u], vq[u], mult, c, to, mo, vo, po);
                    st<NTS>(to, tv + i);
                    st<NTS>(mo, mv + i);
                    st<NTS>(vo, vv + i);
                    st<NTS>(po, pv + i);
                }
            }
        }
    }
}

// K2 (scalar path) for arrays whose element misalignments differ.
template <bool CDEV>
__global__ __launch_bounds__(kScalarBlock) void k_adam_scalar(
    const uint16_t* __restrict__ g, float* __restrict__ th, float* __restrict__ m, float* __restrict__ v,
    uint16_t* __restrict__ p, int64_t n, const Result* __restrict__ res, AdamConst c_arg,
    const AdamConst* __restrict__ cdev) {
    if (res->skip)
        return;
    const float mult = res->mult;
    AdamConst c = c_arg;
    if constexpr (CDEV)
        c = *cdev;
    const int64_t stride = (int64_t)gridDim.x * kScalarBlock;
    for (int64_t i = (int64_t)blockIdx.x * kScalarBlock + threadIdx.x; i < n; i += stride)
        adam_one(g, th, m, v, p, i, mult, c);
}

// ---------------------------------------------------------------------------
// One-launch small-shard step.  The grid is small enough to be resident on
// the device at once (the host keeps it to a fraction of the co-resident
// capacity, so a few such steps on concurrent streams also fit together), which
// the grid barrier below relies on.  The shard's vector layout is
// k_adam_vec's (`head` scalar elements, `nvec` 4-element vectors, a tail of
// 0..3); workgroup b owns vectors (b*V + u)*kSmallBlock + threadIdx.x for
// u < V, so consecutive lanes touch consecutive vectors.
//   1. Thread 0 reads its group's wake flag (its value before this launch),
//      then the workgroup loads its gradient vectors, sums their exact squares
//      in fp64 (workgroup 0 also takes the head and tail elements) and stores
//      the workgroup's partial part[b].
//   2. Arrival, in two levels so that no address takes more than a few dozen
//      atomic additions (one address serialises them at about 12 ns each):
//      workgroup b counts itself in group b mod kSyncGroups; the last of a
//      group counts the group at the top; the last group's last workgroup is
//      the last arrival.  Counters are reset by their last arrival.
//   3. The state loads of theta, m and v are issued (they overlap the wait).
//   4. The last arrival claims the launch, totals part[0, gridDim.x) in a
//      fixed order, publishes the result record (device and host-mapped),
//      then writes every group's wake flag: a launch count in the high bits,
//      the skip flag and the fp32 multiplier in the low 33, so a waiter reads
//      the step's scalars from the word it polls.  The others wait for their
//      group's flag to change.
//   5. Unless the step is skipped, the update from the registers.
// The wait is bounded.  A workgroup that gives up tries to claim the launch
// as aborted; the claim word makes completion and abort exclusive, so either
// every workgroup updates or none does (then nothing is written, the record
// is not published and the host's wait ends with an error once the stream
// is idle).  Partials, counters, flags and the claim word are accessed with
// agent-scope atomic operations, which the device keeps coherent across its
// XCDs without writing back or invalidating the L2 caches; a store completes
// (s_waitcnt) before the operation that announces it is issued.
// ---------------------------------------------------------------------------
constexpr int kSmallBlock = 256;
constexpr int kSyncGroups = 16;
constexpr int kSyncStride = 32;                        // words between sync words (256 bytes)
constexpr uint32_t kBarrierSpinLimit = 1u << 22;       // polls of about 0.1-1 us each
// Word offsets in the sync area (each word on its own 256-byte line).
constexpr int kSyncGroupCtr = 0;                       // kSyncGroups group counters
constexpr int kSyncTop = kSyncGroups;                  // the count of complete groups
constexpr int kSyncFlag = kSyncGroups + 1;             // kSyncGroups wake flags
constexpr int kSyncClaim = 2 * kSyncGroups + 1;        // 0 open, 1 completed, 2 aborted
constexpr int kSyncWords = (2 * kSyncGroups + 2) * kSyncStride;
constexpr uint64_t kFlagCount = (uint64_t)1 << 33;     // a wake flag's launch count unit

__device__ __forceinline__ uint64_t* sync_word(uint64_t* sync, int k) { return sync + (int64_t)k * kSyncStride; }

__device__ __forceinline__ uint64_t aload(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void astore(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t aadd(uint64_t* p, uint64_t v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ bool acas(uint64_t* p, uint64_t expect, uint64_t v) {
    return __hip_atomic_compare_exchange_strong(p, &expect, v, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
}

// Waiter (thread 0 of a workgroup that is not the last arrival): true when its
// group's flag has moved on from `flag0` (the launch completed; *word is the
// new flag), false when the launch was aborted.  The last arrival writes every
// flag before it reopens the claim word, so a flag that has not moved while the
// claim reads "aborted" means a real abort.
__device__ __forceinline__ bool small_wait(uint64_t* sync, int grp, uint64_t flag0, uint64_t* word) {
    uint64_t* flag = sync_word(sync, kSyncFlag + grp);
    uint64_t* claim = sync_word(sync, kSyncClaim);
    const uint64_t count0 = flag0 / kFlagCount;
    uint32_t polls = 0;
    for (;;) {
        if ((*word = aload(flag)) / kFlagCount != count0)
            return true;
        ++polls;
        if ((polls & 1023) == 0 && aload(claim) == 2)
            return (*word = aload(flag)) / kFlagCount != count0;
        if (polls >= kBarrierSpinLimit) {
            polls = 0;
            if (acas(claim, 0, 2)) {
                __builtin_amdgcn_s_waitcnt(0);
                if ((*word = aload(flag)) / kFlagCount != count0) {
                    astore(claim, 0);  // the launch had completed just before: undo the claim
                    return true;
                }
                return false;
            }
            // claimed as completed (the flag follows) or as aborted (the check above sees it)
        }
        __builtin_amdgcn_s_sleep(2);
    }
}

template <int V>
__global__ __launch_bounds__(kSmallBlock) void k_small_step(
    const uint16_t* __restrict__ g, float* __restrict__ th, float* __restrict__ m, float* __restrict__ v,
    uint16_t* __restrict__ p, int64_t n, int64_t head, int64_t nvec, uint64_t* __restrict__ part,
    uint64_t* __restrict__ sync, Result* __restrict__ res, Result* __restrict__ res_host, double loss_scale,
    double clip, uint32_t seq, AdamConst c) {
    __shared__ float s_mult;
    __shared__ int s_state;  // 1: this workgroup is the last arrival; then 0 proceed, 1 skip, 2 abort
    const u32x2* __restrict__ gv = reinterpret_cast<const u32x2*>(g + head);
    f32x4* __restrict__ tv = reinterpret_cast<f32x4*>(th + head);
    f32x4* __restrict__ mv = reinterpret_cast<f32x4*>(m + head);
    f32x4* __restrict__ vv = reinterpret_cast<f32x4*>(v + head);
    u32x2* __restrict__ pv = reinterpret_cast<u32x2*>(p + head);
    const int64_t b = blockIdx.x;
    const int G = (int)gridDim.x;
    const int grp = (int)(b % kSyncGroups);
    const int ngroups = G < kSyncGroups ? G : kSyncGroups;
    uint64_t flag0 = 0;
    if (threadIdx.x == 0)
        flag0 = aload(sync_word(sync, kSyncFlag + grp));  // before arriving: it cannot move until then

    // 1. statistics of this workgroup's gradient vectors
    u32x2 gq[V];
    double a0 = 0.0, a1 = 0.0;
#pragma unroll
    for (int u = 0; u < V; ++u) {
        const int64_t i = (b * V + u) * kSmallBlock + threadIdx.x;
        gq[u] = i < nvec ? ld<true>(gv + i) : u32x2{0u, 0u};
        a0 = acc_sq2(gq[u].x, a0);
        a1 = acc_sq2(gq[u].y, a1);
    }
    if (b == 0) {
        const int64_t t = threadIdx.x;
        const int64_t tail0 = head + 4 * nvec;
        if (t < head)
            a0 += sq1(g[t]);
        if (t < 4 && tail0 + t < n)
            a1 += sq1(g[tail0 + t]);
    }
    const double ps = block_sum<kSmallBlock>(a0 + a1);

    // 2. publish the partial and arrive (two levels)
    if (threadIdx.x == 0) {
        astore(part + b, __builtin_bit_cast(uint64_t, ps));
        __builtin_amdgcn_s_waitcnt(0);
        const uint64_t gsize = (uint64_t)((G - grp + kSyncGroups - 1) / kSyncGroups);
        uint64_t* gctr = sync_word(sync, kSyncGroupCtr + grp);
        int last = 0;
        if (aadd(gctr, 1) == gsize - 1) {
            astore(gctr, 0);  // every member has counted: ready for the next launch
            last = aadd(sync_word(sync, kSyncTop), 1) == (uint64_t)(ngroups - 1);
        }
        s_state = last;
    }
    // 3. the state loads, overlapping the wait
    f32x4 tq[V], mq[V], vq[V];
#pragma unroll
    for (int u = 0; u < V; ++u) {
        const int64_t i = (b * V + u) * kSmallBlock + threadIdx.x;
        if (i < nvec) {
            tq[u] = ld<true>(tv + i);
            mq[u] = ld<true>(mv + i);
            vq[u] = ld<true>(vv + i);
        }
    }
    __syncthreads();

    // 4. the last arrival totals and publishes; the others wait for their flag
    if (s_state == 1) {
        double s0 = 0.0;
        for (int64_t i = threadIdx.x; i < G; i += kSmallBlock)
            s0 += __builtin_bit_cast(double, aload(part + i));
        const double tot = block_sum<kSmallBlock>(s0);
        if (threadIdx.x == 0) {
            uint64_t* claim = sync_word(sync, kSyncClaim);
            if (!acas(claim, 0, 1)) {
                s_state = 2;  // a waiter gave up first: nobody writes
            } else {
                const Result r = make_result(tot, loss_scale, clip, seq);
                *res = r;
                Result rh = r;
                rh.seq = 0;
                *res_host = rh;
                __hip_atomic_store(&res_host->seq, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
                s_mult = r.mult;
                s_state = r.skip;
                astore(sync_word(sync, kSyncTop), 0);
                // every flag is written, whatever the grid, so all of them always hold the same
                // launch count (a waiter's group flag then always changes)
                const uint64_t word = (flag0 / kFlagCount + 1) * kFlagCount +
                                      ((uint64_t)__builtin_bit_cast(uint32_t, r.mult) | ((uint64_t)(uint32_t)r.skip << 32));
                for (int k = 0; k < kSyncGroups; ++k)
                    astore(sync_word(sync, kSyncFlag + k), word);
                __builtin_amdgcn_s_waitcnt(0);
                astore(claim, 0);  // after the flags: see small_wait
            }
        }
    } else if (threadIdx.x == 0) {
        uint64_t w = 0;
        if (!small_wait(sync, grp, flag0, &w)) {
            s_state = 2;
        } else {
            s_mult = __builtin_bit_cast(float, (uint32_t)w);
            s_state = (int)((w >> 32) & 1);
        }
    }
    __syncthreads();
    if (s_state)
        return;
    const float mult = s_mult;

    // 5. the update from the registers (workgroup 0 also takes head and tail)
    if (b == 0 && threadIdx.x < 8) {
        const int64_t t = threadIdx.x;
        const int64_t i = t < 4 ? t : head + 4 * nvec + (t - 4);
        if ((t < 4 && i < head) || (t >= 4 && i < n))
            adam_one(g, th, m, v, p, i, mult, c);
    }
#pragma unroll
    for (int u = 0; u < V; ++u) {
        const int64_t i = (b * V + u) * kSmallBlock + threadIdx.x;
        if (i < nvec) {
            f32x4 to, mo, vo;
            u32x2 po;
            adam_vec4(gq[u], tq[u], mq[u], vq[u], mult, c, to, mo, vo, po);
            st<true>(to, tv + i);
            st<true>(mo, mv + i);
            st<true>(vo, vv + i);
            st<true>(po, pv + i);
        }
    }
}

// Streaming copy of nvec 16-byte vectors: the achievable-bandwidth reference
// for the update kernel (same tiling knobs) and the calibration kernel for
// hardware byte counters.
template <int BLOCK, int U, bool NTL, bool NTS, bool XCD>
__global__ __launch_bounds__(BLOCK) void k_probe_copy(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                      int64_t nvec) {
    const int64_t tile = (int64_t)BLOCK * U;
    const int64_t stride = (int64_t)gridDim.x * tile;
    for (int64_t base = logical_block<XCD>() * tile + threadIdx.x; base < nvec; base += stride) {
        u32x4 q[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = base + (int64_t)u * BLOCK;
            if (i < nvec)
                q[u] = ld<NTL>(src + i);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = base + (int64_t)u * BLOCK;
            if (i < nvec)
                st<NTS>(q[u], dst + i);
        }
    }
}

}  // namespace zs
