// probe_kernels.hpp -- measurement probe of the update kernel's streams (not
// part of the step).  Kept apart from the step's kernels, whose source the
// committed counter summaries are keyed to.
#pragma once

#include "shard_kernels.hpp"

namespace zs {

// The probe's work on four consecutive elements: three adds and a conversion.
template <bool NTS>
__device__ __forceinline__ void probe_vec4(u32x2 gq, f32x4 tq, f32x4 mq, f32x4 vq, f32x4* __restrict__ tv,
                                           f32x4* __restrict__ mv, f32x4* __restrict__ vv, u32x2* __restrict__ pv,
                                           int64_t i) {
    const f32x4 gf = {f16_to_f32(gq.x & 0xFFFFu), f16_to_f32(gq.x >> 16), f16_to_f32(gq.y & 0xFFFFu),
                      f16_to_f32(gq.y >> 16)};
    const f32x4 to = tq + gf;
    st<NTS>(to, tv + i);
    st<NTS>(mq + tq, mv + i);
    st<NTS>(vq + mq, vv + i);
    st<NTS>(u32x2{f32_to_f16(to.x) | (f32_to_f16(to.y) << 16), f32_to_f16(to.z) | (f32_to_f16(to.w) << 16)}, pv + i);
}

// Byte-mix probe of the update: k_adam_vec's four reads and four writes per
// element (fp16 gradient, fp32 master, momentum and variance in; fp32 master,
// momentum, variance and fp16 parameters out), its tiles, vector widths,
// cache policy and launch shape, with three adds and a conversion per element
// in place of Adam.  Its time is the achievable time of the update's streams
// at the update's launch shape.  Arrays start 16-byte aligned (fp16 8-byte):
// nvec 4-element vectors, then the last 0..3 elements one by one.
template <int BLOCK, int U, bool NTL, bool NTS, bool XCD>
__global__ __launch_bounds__(BLOCK) void k_probe_adam(const uint16_t* __restrict__ g, float* __restrict__ th,
                                                      float* __restrict__ m, float* __restrict__ v,
                                                      uint16_t* __restrict__ p, int64_t n, int64_t nvec) {
    if (blockIdx.x == 0 && threadIdx.x < 4) {
        const int64_t i = 4 * nvec + threadIdx.x;
        if (i < n) {
            const float t = th[i], mm = m[i];
            th[i] = t + f16_to_f32(g[i]);
            m[i] = mm + t;
            v[i] = v[i] + mm;
            p[i] = (uint16_t)f32_to_f16(th[i]);
        }
    }
    const u32x2* __restrict__ gv = reinterpret_cast<const u32x2*>(g);
    f32x4* __restrict__ tv = reinterpret_cast<f32x4*>(th);
    f32x4* __restrict__ mv = reinterpret_cast<f32x4*>(m);
    f32x4* __restrict__ vv = reinterpret_cast<f32x4*>(v);
    u32x2* __restrict__ pv = reinterpret_cast<u32x2*>(p);
    const int64_t tile = (int64_t)BLOCK * U;
    const int64_t ntiles = (nvec + tile - 1) / tile;
    for (int64_t tb = logical_block<XCD>(); tb < ntiles; tb += gridDim.x) {
        const int64_t base = tb * tile + threadIdx.x;
        // as the update: with one vector per thread, one bounds test around loads, work and stores
        if constexpr (U == 1) {
            if (base < nvec)
                probe_vec4<NTS>(ld<NTL>(gv + base), ld<NTL>(tv + base), ld<NTL>(mv + base), ld<NTL>(vv + base), tv,
                                mv, vv, pv, base);
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
                if (i < nvec)
                    probe_vec4<NTS>(gq[u], tq[u], mq[u], vq[u], tv, mv, vv, pv, i);
            }
        }
    }
}

}  // namespace zs
