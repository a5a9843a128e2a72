// lamb_kernels.hpp -- gfx950 kernels of the LAMB shard step.
//
// LAMB (You et al., layer-wise adaptive large-batch optimization; one of the
// adaptive optimizers ZeRO's related work lists as made affordable by
// partitioning optimizer state) keeps Adam's fp32 moments but scales each
// layer's update direction u by the trust ratio phi(||theta||)/||u||.  The
// layer norms couple every element of a layer, so the step takes two
// streaming passes after the gradient statistics:
//   k_lamb_moments  reads g16, theta, m, v; writes m, v; one fp64 partial
//                   (sum theta^2, sum u^2) per work item (22 bytes/element).
//   k_lamb_layer    fixed-order sum of each layer's partials.
//   k_lamb_apply    reads theta, m, v; recomputes u from the stored moments
//                   (the same fp32 operations, so the same bits); writes
//                   theta - step*u and its fp16 copy (18 bytes/element).
// A work item is a run of at most one tile of elements inside one layer: the
// host cuts the shard's tiles at the layer boundaries, so no workgroup needs a
// segmented reduction and every item's partial belongs to one layer.
#pragma once

#include "shard_kernels.hpp"

namespace zs {

// Elements [start, next item's start) of layer `layer`.  The list ends with a
// sentinel item whose start is n.
struct alignas(16) LambItem {
    int64_t start;
    int32_t layer;
    int32_t unused;
};

// Sum of theta^2 and sum of u^2 (fp64) of one work item or one layer.
struct alignas(16) LayerSums {
    double wsq;
    double usq;
};

// Adam's moments of one element (the same fp32 sequence as adam_elem); m and v
// are updated in place.
__device__ __forceinline__ void lamb_moments_elem(uint32_t g16, float mult, float& m, float& v, const AdamConst& c) {
#pragma clang fp contract(off)
    const float g = f16_to_f32(g16) * mult;
    m = c.b1 * m + c.omb1 * g;
    v = c.b2 * v + c.omb2 * (g * g);
}

// The update direction from the new moments and the old parameter: bias
// correction, eps outside the square root, decoupled weight decay.
__device__ __forceinline__ float lamb_dir(float m, float v, float th, const AdamConst& c) {
#pragma clang fp contract(off)
    const float mhat = m / c.bc1;
    const float vhat = v / c.bc2;
    const float denom = __builtin_sqrtf(vhat) + c.eps;
    float u = mhat / denom;
    if (c.wd != 0.0f)
        u = u + c.wd * th;
    return u;
}

// The layer's fp32 step size lr * phi(||theta||) / ||u|| (1 for the ratio when
// either norm is zero), computed in double and rounded once.
__device__ __forceinline__ float lamb_step_size(LayerSums s, double lr, double phi_lo, double phi_hi) {
    double trust = 1.0;
    if (s.wsq > 0.0 && s.usq > 0.0) {
        double wn = __builtin_sqrt(s.wsq);
        if (wn < phi_lo)
            wn = phi_lo;
        if (wn > phi_hi)
            wn = phi_hi;
        trust = wn / __builtin_sqrt(s.usq);
    }
    return (float)(lr * trust);
}

// Fixed-order workgroup sum of two doubles per thread; thread 0 receives the
// totals.  Ends with a barrier so that a following call may reuse the LDS.
template <int BLOCK>
__device__ __forceinline__ void block_sum2(double& a, double& b) {
    a = wave_sum(a);
    b = wave_sum(b);
    if constexpr (BLOCK > 64) {
        __shared__ double lds[2][BLOCK / 64];
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        if (lane == 0) {
            lds[0][wave] = a;
            lds[1][wave] = b;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            double sa = 0.0, sb = 0.0;
#pragma unroll
            for (int w = 0; w < BLOCK / 64; ++w) {
                sa += lds[0][w];
                sb += lds[1][w];
            }
            a = sa;
            b = sb;
        }
        __syncthreads();
    }
}

// First element of the 4-element vector that holds element `start`, where
// vectors begin at indices congruent to `head` mod 4 (head in 0..3; a start
// below head lies in the partial vector that ends at head).
__device__ __forceinline__ int64_t vec_floor(int64_t start, int64_t head) {
    const int64_t d = start - head;
    return head + 4 * (d >= 0 ? d / 4 : -1);
}

// ---------------------------------------------------------------------------
// Moments pass.  Workgroup k handles item k (grid-strided): thread t covers the
// U vectors base + 4*(t + u*BLOCK) .. +3, where base is the vector holding the
// item's first element.  VEC: all arrays share the element misalignment
// `head`, so a vector wholly inside the item is one 16-byte fp32 access per
// array and one 8-byte fp16 access; elements of partial vectors (layer
// boundaries, the array's ends) and every element when !VEC (head = 0) take
// the scalar path.  Only elements of the item are read or written.
// ---------------------------------------------------------------------------
template <int BLOCK, int U, bool NTL, bool NTS, bool VEC>
__global__ __launch_bounds__(BLOCK) void k_lamb_moments(const uint16_t* __restrict__ g, const float* __restrict__ th,
                                                        float* __restrict__ m, float* __restrict__ v,
                                                        const LambItem* __restrict__ items, int64_t n_items,
                                                        int64_t head, const Result* __restrict__ res, AdamConst c,
                                                        LayerSums* __restrict__ part) {
    if (res->skip)
        return;
    const float mult = res->mult;
    for (int64_t k = blockIdx.x; k < n_items; k += gridDim.x) {
        const int64_t start = items[k].start, end = items[k + 1].start;
        const int64_t base = vec_floor(start, head);
        double aw = 0.0, au = 0.0;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t e0 = base + 4 * ((int64_t)threadIdx.x + (int64_t)u * BLOCK);
            if (VEC && e0 >= start && e0 + 4 <= end) {
                const u32x2 gq = ld<NTL>(reinterpret_cast<const u32x2*>(g + e0));
                const f32x4 tq = ld<NTL>(reinterpret_cast<const f32x4*>(th + e0));
                f32x4 mq = ld<NTL>(reinterpret_cast<const f32x4*>(m + e0));
                f32x4 vq = ld<NTL>(reinterpret_cast<const f32x4*>(v + e0));
                const uint32_t gw[4] = {gq.x & 0xFFFFu, gq.x >> 16, gq.y & 0xFFFFu, gq.y >> 16};
                float t4[4] = {tq.x, tq.y, tq.z, tq.w};
                float m4[4] = {mq.x, mq.y, mq.z, mq.w};
                float v4[4] = {vq.x, vq.y, vq.z, vq.w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    lamb_moments_elem(gw[j], mult, m4[j], v4[j], c);
                    const double ud = (double)lamb_dir(m4[j], v4[j], t4[j], c);
                    const double td = (double)t4[j];
                    aw = __builtin_fma(td, td, aw);
                    au = __builtin_fma(ud, ud, au);
                }
                st<NTS>(f32x4{m4[0], m4[1], m4[2], m4[3]}, reinterpret_cast<f32x4*>(m + e0));
                st<NTS>(f32x4{v4[0], v4[1], v4[2], v4[3]}, reinterpret_cast<f32x4*>(v + e0));
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int64_t i = e0 + j;
                    if (i >= start && i < end) {
                        float mm = m[i], vv = v[i];
                        const float t = th[i];
                        lamb_moments_elem(g[i], mult, mm, vv, c);
                        const double ud = (double)lamb_dir(mm, vv, t, c);
                        const double td = (double)t;
                        aw = __builtin_fma(td, td, aw);
                        au = __builtin_fma(ud, ud, au);
                        m[i] = mm;
                        v[i] = vv;
                    }
                }
            }
        }
        block_sum2<BLOCK>(aw, au);
        if (threadIdx.x == 0)
            part[k] = LayerSums{aw, au};
    }
}

// ---------------------------------------------------------------------------
// Layer sums: workgroup s adds the partials of layer s's items
// [first[s], first[s+1]) in a fixed order (strided per thread, then the
// workgroup tree), so the result is reproducible for a given item list.
// ---------------------------------------------------------------------------
constexpr int kLayerBlock = 256;

__global__ __launch_bounds__(kLayerBlock) void k_lamb_layer(const LayerSums* __restrict__ part,
                                                            const int64_t* __restrict__ first, int64_t n_layers,
                                                            LayerSums* __restrict__ sums,
                                                            const Result* __restrict__ res) {
    if (res->skip)
        return;
    for (int64_t s = blockIdx.x; s < n_layers; s += gridDim.x) {
        const int64_t a = first[s], b = first[s + 1];
        double w = 0.0, u = 0.0;
        for (int64_t i = a + threadIdx.x; i < b; i += kLayerBlock) {
            const LayerSums p = part[i];
            w += p.wsq;
            u += p.usq;
        }
        block_sum2<kLayerBlock>(w, u);
        if (threadIdx.x == 0)
            sums[s] = LayerSums{w, u};
    }
}

// ---------------------------------------------------------------------------
// Apply pass: same item walk as the moments pass; theta <- theta - step*u with
// the item's layer step size, and the fp16 copy.
// ---------------------------------------------------------------------------
template <int BLOCK, int U, bool NTL, bool NTS, bool VEC>
__global__ __launch_bounds__(BLOCK) void k_lamb_apply(float* __restrict__ th, const float* __restrict__ m,
                                                      const float* __restrict__ v, uint16_t* __restrict__ p,
                                                      const LambItem* __restrict__ items, int64_t n_items,
                                                      int64_t head, const LayerSums* __restrict__ sums,
                                                      const Result* __restrict__ res, AdamConst c, double lr,
                                                      double phi_lo, double phi_hi) {
#pragma clang fp contract(off)
    if (res->skip)
        return;
    for (int64_t k = blockIdx.x; k < n_items; k += gridDim.x) {
        const LambItem it = items[k];
        const int64_t start = it.start, end = items[k + 1].start;
        const float step = lamb_step_size(sums[it.layer], lr, phi_lo, phi_hi);
        const int64_t base = vec_floor(start, head);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t e0 = base + 4 * ((int64_t)threadIdx.x + (int64_t)u * BLOCK);
            if (VEC && e0 >= start && e0 + 4 <= end) {
                const f32x4 tq = ld<NTL>(reinterpret_cast<const f32x4*>(th + e0));
                const f32x4 mq = ld<NTL>(reinterpret_cast<const f32x4*>(m + e0));
                const f32x4 vq = ld<NTL>(reinterpret_cast<const f32x4*>(v + e0));
                const float t4[4] = {tq.x, tq.y, tq.z, tq.w};
                const float m4[4] = {mq.x, mq.y, mq.z, mq.w};
                const float v4[4] = {vq.x, vq.y, vq.z, vq.w};
                float o[4];
                uint32_t h[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    o[j] = t4[j] - step * lamb_dir(m4[j], v4[j], t4[j], c);
                    h[j] = f32_to_f16(o[j]);
                }
                st<NTS>(f32x4{o[0], o[1], o[2], o[3]}, reinterpret_cast<f32x4*>(th + e0));
                st<NTS>(u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)}, reinterpret_cast<u32x2*>(p + e0));
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int64_t i = e0 + j;
                    if (i >= start && i < end) {
                        const float t = th[i];
                        const float o = t - step * lamb_dir(m[i], v[i], t, c);
                        th[i] = o;
                        p[i] = (uint16_t)f32_to_f16(o);
                    }
                }
            }
        }
    }
}

}  // namespace zs
