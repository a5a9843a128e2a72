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
//   k_lamb_chunks,  fixed-order two-level sum of each layer's partials.
//   k_lamb_layer
//   k_lamb_apply    reads theta, m, v; recomputes u from the stored moments
//                   (the same fp32 operations, so the same bits); writes
//                   theta - step*u and its fp16 copy (18 bytes/element).
// A work item is a tile's piece inside one layer: the host cuts the shard's
// tiles at the layer boundaries.  Each workgroup owns one tile and computes its
// addresses from its index alone; it reads the tile's items (almost always
// one) only to attribute its partial sums and step sizes to layers.
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

// Tiles of the shard: with head h (0..3) the 4-element vectors begin at
// indices congruent to h mod 4; tile 0 is [0, h) when h > 0, and the other
// tiles are T = 4*BLOCK*U elements long, aligned to the vectors.  Returns the
// first vector's element index (h - 4 for the partial tile [0, h)) and the
// tile's element range [ts, te).
template <int BLOCK, int U>
__device__ __forceinline__ int64_t tile_range(int64_t b, int64_t head, int64_t n, int64_t* ts, int64_t* te) {
    constexpr int64_t T = 4 * (int64_t)BLOCK * U;
    const int64_t hs = head > 0 ? 1 : 0;
    if (b < hs) {
        *ts = 0;
        *te = head < n ? head : n;
        return head - 4;
    }
    const int64_t base = head + (b - hs) * T;
    *ts = base;
    *te = base + T < n ? base + T : n;
    return base;
}

// ---------------------------------------------------------------------------
// Moments pass.  Workgroup b (grid-strided over the tiles; with XCD, remapped so
// that each XCD walks a contiguous run of tiles and the tiles' descriptors,
// which neighbouring tiles share cache lines of, stay in one L2) owns tile b: thread
// t covers the U vectors base + 4*(t + u*BLOCK) .. +3.  The data addresses
// depend on b only, so the loads are issued before the tile's work items
// (its layer pieces, [tile_first[b], tile_first[b+1]) of the item list) are
// read; the items are needed only to attribute each element's theta^2 and u^2
// to its layer piece.  VEC: all arrays share the element misalignment `head`,
// so a vector inside the tile is one 16-byte fp32 access per array and one
// 8-byte fp16 access; the partial vectors at the array's ends and every
// element when !VEC (head = 0) take the scalar path.
// ---------------------------------------------------------------------------
template <int BLOCK, int U, bool NTL, bool NTS, bool VEC, bool XCD>
__global__ __launch_bounds__(BLOCK) void k_lamb_moments(const uint16_t* __restrict__ g, const float* __restrict__ th,
                                                        float* __restrict__ m, float* __restrict__ v,
                                                        const LambItem* __restrict__ items,
                                                        const int64_t* __restrict__ tile_first, int64_t ntiles,
                                                        int64_t n, int64_t head, const Result* __restrict__ res,
                                                        AdamConst c, LayerSums* __restrict__ part) {
    if (res->skip)
        return;
    const float mult = res->mult;
    for (int64_t b = logical_block<XCD>(); b < ntiles; b += gridDim.x) {
        int64_t ts, te;
        const int64_t base = tile_range<BLOCK, U>(b, head, n, &ts, &te);
        double w2[U][4], u2[U][4];
        int64_t e0s[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t e0 = base + 4 * ((int64_t)threadIdx.x + (int64_t)u * BLOCK);
            e0s[u] = e0;
            if (VEC && e0 >= ts && e0 + 4 <= te) {
                const u32x2 gq = ld<NTL>(reinterpret_cast<const u32x2*>(g + e0));
                const f32x4 tq = ld<NTL>(reinterpret_cast<const f32x4*>(th + e0));
                f32x4 mq = ld<NTL>(reinterpret_cast<const f32x4*>(m + e0));
                f32x4 vq = ld<NTL>(reinterpret_cast<const f32x4*>(v + e0));
                const uint32_t gw[4] = {gq.x & 0xFFFFu, gq.x >> 16, gq.y & 0xFFFFu, gq.y >> 16};
                const float t4[4] = {tq.x, tq.y, tq.z, tq.w};
                float m4[4] = {mq.x, mq.y, mq.z, mq.w};
                float v4[4] = {vq.x, vq.y, vq.z, vq.w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    lamb_moments_elem(gw[j], mult, m4[j], v4[j], c);
                    const double ud = (double)lamb_dir(m4[j], v4[j], t4[j], c);
                    const double td = (double)t4[j];
                    w2[u][j] = td * td;
                    u2[u][j] = ud * ud;
                }
                st<NTS>(f32x4{m4[0], m4[1], m4[2], m4[3]}, reinterpret_cast<f32x4*>(m + e0));
                st<NTS>(f32x4{v4[0], v4[1], v4[2], v4[3]}, reinterpret_cast<f32x4*>(v + e0));
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int64_t i = e0 + j;
                    w2[u][j] = 0.0;
                    u2[u][j] = 0.0;
                    if (i >= ts && i < te) {
                        float mm = m[i], vv = v[i];
                        const float t = th[i];
                        lamb_moments_elem(g[i], mult, mm, vv, c);
                        const double ud = (double)lamb_dir(mm, vv, t, c);
                        const double td = (double)t;
                        w2[u][j] = td * td;
                        u2[u][j] = ud * ud;
                        m[i] = mm;
                        v[i] = vv;
                    }
                }
            }
        }
        // one partial per layer piece of the tile (almost always one piece)
        const int64_t f = tile_first[b], l = tile_first[b + 1];
        for (int64_t k = f; k < l; ++k) {
            const int64_t s0 = items[k].start, s1 = items[k + 1].start;
            double aw = 0.0, au = 0.0;
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int64_t i = e0s[u] + j;
                    if (i >= s0 && i < s1) {
                        aw += w2[u][j];
                        au += u2[u][j];
                    }
                }
            block_sum2<BLOCK>(aw, au);
            if (threadIdx.x == 0)
                part[k] = LayerSums{aw, au};
        }
    }
}

// ---------------------------------------------------------------------------
// Layer sums, two levels in a fixed order.  Level 1: workgroup c adds the
// partials of item chunk c, items [chunk[c], chunk[c+1]) (a chunk never
// spans two layers).  Level 2: workgroup s adds the chunk sums of layer s,
// chunks [chunk_first[s], chunk_first[s+1]).
// ---------------------------------------------------------------------------
constexpr int kChunkBlock = 256;
constexpr int kChunkItems = 1024;   // items per level-1 chunk (4 per thread)
constexpr int kLayerBlock = 64;

__global__ __launch_bounds__(kChunkBlock) void k_lamb_chunks(const LayerSums* __restrict__ part,
                                                             const int64_t* __restrict__ chunk, int64_t n_chunks,
                                                             LayerSums* __restrict__ cpart,
                                                             const Result* __restrict__ res) {
    if (res->skip)
        return;
    for (int64_t cb = blockIdx.x; cb < n_chunks; cb += gridDim.x) {
        const int64_t a = chunk[cb], e = chunk[cb + 1];
        double w = 0.0, u = 0.0;
        for (int64_t i = a + threadIdx.x; i < e; i += kChunkBlock) {
            const LayerSums p = part[i];
            w += p.wsq;
            u += p.usq;
        }
        block_sum2<kChunkBlock>(w, u);
        if (threadIdx.x == 0)
            cpart[cb] = LayerSums{w, u};
    }
}

__global__ __launch_bounds__(kLayerBlock) void k_lamb_layer(const LayerSums* __restrict__ cpart,
                                                            const int64_t* __restrict__ chunk_first,
                                                            int64_t n_layers, LayerSums* __restrict__ sums,
                                                            const Result* __restrict__ res) {
    if (res->skip)
        return;
    for (int64_t s = blockIdx.x; s < n_layers; s += gridDim.x) {
        const int64_t a = chunk_first[s], e = chunk_first[s + 1];
        double w = 0.0, u = 0.0;
        for (int64_t i = a + threadIdx.x; i < e; i += kLayerBlock) {
            const LayerSums p = cpart[i];
            w += p.wsq;
            u += p.usq;
        }
        block_sum2<kLayerBlock>(w, u);
        if (threadIdx.x == 0)
            sums[s] = LayerSums{w, u};
    }
}

// ---------------------------------------------------------------------------
// Apply pass: same tile walk as the moments pass; each element moves by its
// layer piece's step size (theta <- theta - step*u) and gets its fp16 copy.
// ---------------------------------------------------------------------------
template <int BLOCK, int U, bool NTL, bool NTS, bool VEC, bool XCD>
__global__ __launch_bounds__(BLOCK) void k_lamb_apply(float* __restrict__ th, const float* __restrict__ m,
                                                      const float* __restrict__ v, uint16_t* __restrict__ p,
                                                      const LambItem* __restrict__ items,
                                                      const int64_t* __restrict__ tile_first, int64_t ntiles,
                                                      int64_t n, int64_t head, const LayerSums* __restrict__ sums,
                                                      const Result* __restrict__ res, AdamConst c, double lr,
                                                      double phi_lo, double phi_hi) {
#pragma clang fp contract(off)
    if (res->skip)
        return;
    for (int64_t b = logical_block<XCD>(); b < ntiles; b += gridDim.x) {
        int64_t ts, te;
        const int64_t base = tile_range<BLOCK, U>(b, head, n, &ts, &te);
        float t4[U][4], u4[U][4];
        bool full[U];
        int64_t e0s[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t e0 = base + 4 * ((int64_t)threadIdx.x + (int64_t)u * BLOCK);
            e0s[u] = e0;
            full[u] = VEC && e0 >= ts && e0 + 4 <= te;
            if (full[u]) {
                const f32x4 tq = ld<NTL>(reinterpret_cast<const f32x4*>(th + e0));
                const f32x4 mq = ld<NTL>(reinterpret_cast<const f32x4*>(m + e0));
                const f32x4 vq = ld<NTL>(reinterpret_cast<const f32x4*>(v + e0));
                const float tt[4] = {tq.x, tq.y, tq.z, tq.w};
                const float mm[4] = {mq.x, mq.y, mq.z, mq.w};
                const float vv[4] = {vq.x, vq.y, vq.z, vq.w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    t4[u][j] = tt[j];
                    u4[u][j] = lamb_dir(mm[j], vv[j], tt[j], c);
                }
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int64_t i = e0 + j;
                    t4[u][j] = 0.0f;
                    u4[u][j] = 0.0f;
                    if (i >= ts && i < te) {
                        t4[u][j] = th[i];
                        u4[u][j] = lamb_dir(m[i], v[i], t4[u][j], c);
                    }
                }
            }
        }
        // the step size of every element's layer piece (almost always one piece per tile)
        float step[U][4];
        const int64_t f = tile_first[b], l = tile_first[b + 1];
        {
            const LambItem it = items[f];
            const float s = lamb_step_size(sums[it.layer], lr, phi_lo, phi_hi);
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    step[u][j] = s;
        }
        for (int64_t k = f + 1; k < l; ++k) {
            const LambItem it = items[k];
            const float s = lamb_step_size(sums[it.layer], lr, phi_lo, phi_hi);
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (e0s[u] + j >= it.start)
                        step[u][j] = s;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t e0 = e0s[u];
            float o[4];
            uint32_t h[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                o[j] = t4[u][j] - step[u][j] * u4[u][j];
                h[j] = f32_to_f16(o[j]);
            }
            if (full[u]) {
                st<NTS>(f32x4{o[0], o[1], o[2], o[3]}, reinterpret_cast<f32x4*>(th + e0));
                st<NTS>(u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)}, reinterpret_cast<u32x2*>(p + e0));
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int64_t i = e0 + j;
                    if (i >= ts && i < te) {
                        th[i] = o[j];
                        p[i] = (uint16_t)h[j];
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Byte-mix probes of the two passes: the same arrays, tile walk (XCD-contiguous
// tiles of 4*BLOCK*U elements, one tile per workgroup), vector width and cache
// policy as k_lamb_moments (PASS 0: reads g16, theta, m, v; writes m, v) and
// k_lamb_apply (PASS 1: reads theta, m, v; writes theta, p16), with one or two
// adds per element in place of the pass's arithmetic and no work lists.  Their
// time is the achievable time of each pass's streams at its launch shape.
// Arrays 16-byte aligned (fp16 8-byte); the last partial vector is scalar.
// ---------------------------------------------------------------------------
template <int BLOCK, int U, bool NTL, bool NTS, bool XCD, int PASS>
__global__ __launch_bounds__(BLOCK) void k_probe_lamb(const uint16_t* __restrict__ g, float* __restrict__ th,
                                                      float* __restrict__ m, float* __restrict__ v,
                                                      uint16_t* __restrict__ p, int64_t ntiles, int64_t n) {
    constexpr int64_t T = 4 * (int64_t)BLOCK * U;
    for (int64_t b = logical_block<XCD>(); b < ntiles; b += gridDim.x) {
        const int64_t te = (b + 1) * T < n ? (b + 1) * T : n;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t e0 = b * T + 4 * ((int64_t)threadIdx.x + (int64_t)u * BLOCK);
            if (e0 + 4 <= te) {
                if constexpr (PASS == 0) {
                    const u32x2 gq = ld<NTL>(reinterpret_cast<const u32x2*>(g + e0));
                    const f32x4 tq = ld<NTL>(reinterpret_cast<const f32x4*>(th + e0));
                    const f32x4 mq = ld<NTL>(reinterpret_cast<const f32x4*>(m + e0));
                    const f32x4 vq = ld<NTL>(reinterpret_cast<const f32x4*>(v + e0));
                    const f32x4 gf = {f16_to_f32(gq.x & 0xFFFFu), f16_to_f32(gq.x >> 16), f16_to_f32(gq.y & 0xFFFFu),
                                      f16_to_f32(gq.y >> 16)};
                    st<NTS>(mq + gf, reinterpret_cast<f32x4*>(m + e0));
                    st<NTS>(vq + tq, reinterpret_cast<f32x4*>(v + e0));
                } else {
                    const f32x4 tq = ld<NTL>(reinterpret_cast<const f32x4*>(th + e0));
                    const f32x4 mq = ld<NTL>(reinterpret_cast<const f32x4*>(m + e0));
                    const f32x4 vq = ld<NTL>(reinterpret_cast<const f32x4*>(v + e0));
                    const f32x4 o = tq + mq + vq;
                    st<NTS>(o, reinterpret_cast<f32x4*>(th + e0));
                    st<NTS>(u32x2{f32_to_f16(o.x) | (f32_to_f16(o.y) << 16), f32_to_f16(o.z) | (f32_to_f16(o.w) << 16)},
                            reinterpret_cast<u32x2*>(p + e0));
                }
            } else {
                for (int64_t i = e0; i < te && i < e0 + 4; ++i) {
                    if constexpr (PASS == 0) {
                        m[i] = m[i] + f16_to_f32(g[i]);
                        v[i] = v[i] + th[i];
                    } else {
                        const float o = th[i] + m[i] + v[i];
                        th[i] = o;
                        p[i] = (uint16_t)f32_to_f16(o);
                    }
                }
            }
        }
    }
}

}  // namespace zs
