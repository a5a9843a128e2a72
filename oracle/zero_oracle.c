/*
 * zero_oracle.c -- CPU oracle for the ZeRO P_os+g shard optimizer step.
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg load this library.  It shares no source,
 * header, table or helper with the GPU library and does not include or call it.
 *
 * What it computes, and where each piece comes from (ZeRO, Rajbhandari et al.,
 * arXiv 1910.02054, plus the methods that paper cites):
 *
 *   zo_layout         Sec. 5.1: the optimizer state is cut into N_d equal
 *                     partitions and rank i owns partition i.  The paper does
 *                     not say what happens when N_d does not divide Psi; this
 *                     oracle pads the flat index space at its tail
 *                     (S = ceil(Psi/N_d), shard r = [r*S, r*S+S)).
 *   zo_f16_to_f32     IEEE 754 binary16 decoding (the fp16 gradients and
 *   zo_f32_to_f16     parameters of Sec. 3.1's mixed-precision training),
 *   zo_f32_to_f16_array
 *                     written from the format definition; encoding rounds to
 *                     nearest, ties to even.
 *   zo_local_stats    Sec. 3.2 names the gradient-norm computation over the
 *                     flattened gradients.  The sum of squares is taken
 *                     EXACTLY: a finite binary16 value is k * 2^-24 for an
 *                     integer |k| < 2^40, so sum(k^2) is an integer that fits
 *                     128 bits for any n < 2^48.  The overflow test (an inf or
 *                     NaN gradient, as in mixed-precision training with loss
 *                     scaling) is an exponent-field test.
 *   zo_scalars        Global-norm clipping (Pascanu et al.) of the unscaled
 *                     gradient: norm = sqrt(sum g16^2) / loss_scale,
 *                     coef = clip/norm if clip > 0 and norm > clip, else 1;
 *                     the fp32 gradient multiplier is (float)(coef/loss_scale).
 *   zo_hyper          The fp32 constants of the update, each computed in
 *                     double and rounded once to fp32.
 *   zo_adam           Adam with bias correction (Kingma & Ba, Algorithm 1),
 *                     cited by Sec. 3.1 as the optimizer whose fp32 master
 *                     parameters, momentum and variance make K = 12; optional
 *                     decoupled weight decay; every operation in fp32
 *                     round-to-nearest-even, in the order written, with no
 *                     contraction.  The fp16 parameter copy is written last.
 *   zo_shard_step     stats -> scalars -> skip or Adam, for one shard whose
 *                     own norm is the global norm.
 *   zo_model_state_bytes
 *                     Sec. 3.1 and Sec. 5.1-5.3: bytes of model state per
 *                     device for standard DP and the three ZeRO-DP stages.
 *   zo_scaler_update  Dynamic loss scaling (mixed-precision training): halve
 *                     on overflow, double after a window of good steps.
 *   zo_sumsq_f32      The sum of squares of fp32 values taken EXACTLY in a
 *                     640-bit fixed-point accumulator (every fp32 square is an
 *                     integer multiple of 2^-298) and rounded once to double.
 *   zo_lamb           LAMB (You et al.), a layer-wise adaptive optimizer that
 *   zo_lamb_step      ZeRO's related work lists among the optimizers whose
 *                     state partitioning makes affordable: Adam's moments,
 *                     then each layer's update scaled by the trust ratio
 *                     phi(||theta||)/||u|| with exact norms.
 *
 * Build: cc -std=gnu11 -O2 -ffp-contract=off -fno-fast-math -fPIC -shared
 * (x86-64: SSE arithmetic, so every float operation rounds once to fp32).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 zo_u128;

/* ------------------------------------------------------------------------ */
/* Partition layout (Sec. 5.1, equal partitions; tail padding)              */
/* ------------------------------------------------------------------------ */

/* out[0] = S (shard length), out[1] = r*S (shard offset in the padded flat
 * index space), out[2] = valid elements of the shard, out[3] = N_d*S.
 * Returns 0, or -1 on invalid arguments. */
int zo_layout(int64_t psi, int32_t nd, int32_t rank, int64_t out[4])
{
    if (!out || psi < 0 || psi > ((int64_t)1 << 62) || nd <= 0 || rank < 0 || rank >= nd)
        return -1;
    int64_t S = psi / nd;
    if (psi % nd != 0)
        S += 1;
    int64_t off = (int64_t)rank * S;
    int64_t valid = psi - off;
    if (valid < 0)
        valid = 0;
    if (valid > S)
        valid = S;
    out[0] = S;
    out[1] = off;
    out[2] = valid;
    out[3] = (int64_t)nd * S;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* binary16 <-> binary32, from the IEEE 754 format definition               */
/* ------------------------------------------------------------------------ */

/* 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.  Exponent field 0
 * holds zero and subnormals f * 2^-24; field 31 holds inf (f = 0) and NaN. */
float zo_f16_to_f32(uint16_t h)
{
    int sign = h >> 15;
    int e = (h >> 10) & 31;
    int f = h & 1023;
    double mag;
    if (e == 31)
        return f ? (float)NAN : (sign ? -(float)INFINITY : (float)INFINITY);
    if (e == 0)
        mag = ldexp((double)f, -24);
    else
        mag = ldexp((double)(1024 + f), e - 25);
    return (float)(sign ? -mag : mag); /* exact: at most 11 significant bits */
}

/* Round |x| to a multiple of the binary16 quantum of its binade, ties to even. */
uint16_t zo_f32_to_f16(float x)
{
    uint32_t bits;
    memcpy(&bits, &x, sizeof bits);
    uint16_t sign = (uint16_t)((bits >> 16) & 0x8000u);
    if (isnan(x))
        return (uint16_t)(sign | 0x7E00u);
    if (isinf(x))
        return (uint16_t)(sign | 0x7C00u);
    double a = fabs((double)x);
    if (a == 0.0)
        return sign;
    int ex;
    (void)frexp(a, &ex);       /* a = fr * 2^ex, fr in [0.5, 1): binade 2^(ex-1) */
    int E = ex - 1;
    if (E > 15)
        return (uint16_t)(sign | 0x7C00u);
    /* quantum: 2^(E-10) for normal binades, 2^-24 below the smallest normal */
    int qexp = (E < -14) ? -24 : E - 10;
    double r = ldexp(a, -qexp); /* exact: a power-of-two scaling */
    double k = floor(r);
    double frac = r - k;
    if (frac > 0.5 || (frac == 0.5 && fmod(k, 2.0) != 0.0))
        k += 1.0;
    /* k*2^qexp is the rounded magnitude.  Subnormal range: the bit pattern is
     * k itself (k == 1024 is exactly the smallest normal, 0x0400). */
    if (qexp == -24)
        return (uint16_t)(sign | (uint16_t)k);
    if (k >= 2048.0) { /* rounded up into the next binade */
        k = 1024.0;
        E += 1;
    }
    if (E > 15)
        return (uint16_t)(sign | 0x7C00u);
    return (uint16_t)(sign | (uint16_t)((E + 15) << 10) | (uint16_t)(k - 1024.0));
}

/* Element-wise zo_f32_to_f16 over an array (for exhaustive checks). */
void zo_f32_to_f16_array(const float* x, uint16_t* out, int64_t n)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = zo_f32_to_f16(x[i]);
}

/* ------------------------------------------------------------------------ */
/* Gradient statistics: exact sum of squares and the overflow test           */
/* ------------------------------------------------------------------------ */

/* A finite binary16 h equals k * 2^-24 with integer k (sign dropped):
 * subnormal: k = f; normal: k = (1024 + f) * 2^(e-1). */
static uint64_t f16_units(uint16_t h)
{
    int e = (h >> 10) & 31;
    uint64_t f = h & 1023u;
    if (e == 0)
        return f;
    return (1024u + f) << (e - 1);
}

/* sumsq_units = sum over finite g16[i] of k_i^2, i.e. sum g^2 in units of
 * 2^-48, returned as {low 64 bits, high 64 bits}.  *overflow = 1 if any
 * element is inf or NaN (exponent field all ones), else 0. */
void zo_local_stats(const uint16_t* g16, int64_t n, uint64_t sumsq_units[2], int32_t* overflow)
{
    zo_u128 acc = 0;
    int32_t ovf = 0;
    for (int64_t i = 0; i < n; ++i) {
        uint16_t h = g16[i];
        if ((h & 0x7C00u) == 0x7C00u) {
            ovf = 1;
            continue;
        }
        zo_u128 k = f16_units(h);
        acc += k * k;
    }
    sumsq_units[0] = (uint64_t)acc;
    sumsq_units[1] = (uint64_t)(acc >> 64);
    *overflow = ovf;
}

/* The 128-bit integer rounded once to the nearest double (ties to even). */
double zo_u128_to_double(const uint64_t v[2])
{
    zo_u128 x = ((zo_u128)v[1] << 64) | v[0];
    return (double)x;
}

/* ------------------------------------------------------------------------ */
/* Step scalars: norm, clip coefficient, gradient multiplier, skip           */
/* ------------------------------------------------------------------------ */

typedef struct {
    double sumsq;     /* sum of g16^2, still loss-scaled                   */
    double norm;      /* sqrt(sumsq) / loss_scale: norm of the true gradient */
    double coef;      /* clipping coefficient in (0, 1]                    */
    float mult;       /* (float)(coef / loss_scale): applied to each g16   */
    int32_t skip;     /* 1 when the gradients overflowed                   */
} zo_scalars_t;

void zo_scalars(const uint64_t sumsq_units[2], int32_t overflow, double loss_scale, double clip,
                zo_scalars_t* out)
{
    out->skip = overflow ? 1 : 0;
    if (overflow) {
        out->sumsq = INFINITY;
        out->norm = INFINITY;
        out->coef = 1.0;
        out->mult = 0.0f;
        return;
    }
    out->sumsq = ldexp(zo_u128_to_double(sumsq_units), -48);
    out->norm = sqrt(out->sumsq) / loss_scale;
    out->coef = (clip > 0.0 && out->norm > clip) ? clip / out->norm : 1.0;
    out->mult = (float)(out->coef / loss_scale);
}

/* ------------------------------------------------------------------------ */
/* Adam with bias correction, fp32                                           */
/* ------------------------------------------------------------------------ */

typedef struct {
    float lr, b1, omb1, b2, omb2, bc1, bc2, eps, wd;
} zo_hyper_t;

/* t is the 1-based count of applied updates including this one. */
void zo_hyper(double lr, double beta1, double beta2, double eps, double wd, int64_t t, zo_hyper_t* h)
{
    h->lr = (float)lr;
    h->b1 = (float)beta1;
    h->omb1 = (float)(1.0 - beta1);
    h->b2 = (float)beta2;
    h->omb2 = (float)(1.0 - beta2);
    h->bc1 = (float)(1.0 - pow(beta1, (double)t));
    h->bc2 = (float)(1.0 - pow(beta2, (double)t));
    h->eps = (float)eps;
    h->wd = (float)wd;
}

/* One Adam update of n elements.  g = g16 * mult is the unscaled, clipped
 * fp32 gradient.  With first moment m, second moment v and parameter theta:
 *   m     <- b1*m + (1-b1)*g
 *   v     <- b2*v + (1-b2)*g^2
 *   mhat  =  m / (1 - b1^t)
 *   vhat  =  v / (1 - b2^t)
 *   u     =  mhat / (sqrt(vhat) + eps)   [+ wd*theta, decoupled decay]
 *   theta <- theta - lr*u
 *   p16   =  binary16(theta) */
/* The moments of one element and its update direction u (before any step
 * size); shared by Adam and LAMB, which differ only in how u is scaled. */
static float adam_direction(float g, float* m, float* v, float theta, const zo_hyper_t* h)
{
    float mi = h->b1 * *m + h->omb1 * g;
    float vi = h->b2 * *v + h->omb2 * (g * g);
    float mhat = mi / h->bc1;
    float vhat = vi / h->bc2;
    float denom = sqrtf(vhat) + h->eps;
    float u = mhat / denom;
    if (h->wd != 0.0f)
        u = u + h->wd * theta;
    *m = mi;
    *v = vi;
    return u;
}

void zo_adam(const uint16_t* g16, float* theta, float* m, float* v, uint16_t* p16, int64_t n,
             float mult, const zo_hyper_t* h)
{
    for (int64_t i = 0; i < n; ++i) {
        float g = zo_f16_to_f32(g16[i]) * mult;
        float u = adam_direction(g, &m[i], &v[i], theta[i], h);
        float th = theta[i] - h->lr * u;
        theta[i] = th;
        p16[i] = zo_f32_to_f16(th);
    }
}

/* The whole step on one shard whose own statistics are the global ones.
 * Returns 1 (skipped: nothing written) or 0 (applied).  *out receives the
 * scalars when out is not NULL. */
int zo_shard_step(const uint16_t* g16, float* theta, float* m, float* v, uint16_t* p16, int64_t n,
                  double lr, double beta1, double beta2, double eps, double wd, int64_t t,
                  double loss_scale, double clip, zo_scalars_t* out)
{
    uint64_t s[2];
    int32_t ovf;
    zo_scalars_t sc;
    zo_local_stats(g16, n, s, &ovf);
    zo_scalars(s, ovf, loss_scale, clip, &sc);
    if (out)
        *out = sc;
    if (sc.skip)
        return 1;
    zo_hyper_t h;
    zo_hyper(lr, beta1, beta2, eps, wd, t, &h);
    zo_adam(g16, theta, m, v, p16, n, sc.mult, &h);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Model-state memory per device (Sec. 3.1, Sec. 5.1-5.3)                    */
/* ------------------------------------------------------------------------ */

/* stage 0: standard DP,  (2 + 2 + K) * Psi
 * stage 1: P_os,         2*Psi + 2*Psi + K*Psi/N_d
 * stage 2: P_os+g,       2*Psi + (2 + K)*Psi/N_d
 * stage 3: P_os+g+p,     (2 + 2 + K)*Psi/N_d
 * Returns bytes, or -1 for an unknown stage or N_d <= 0. */
double zo_model_state_bytes(double psi, double nd, int32_t stage, double k)
{
    if (nd <= 0.0)
        return -1.0;
    switch (stage) {
    case 0: return (2.0 + 2.0 + k) * psi;
    case 1: return 2.0 * psi + 2.0 * psi + k * psi / nd;
    case 2: return 2.0 * psi + (2.0 + k) * psi / nd;
    case 3: return (2.0 + 2.0 + k) * psi / nd;
    default: return -1.0;
    }
}

/* ------------------------------------------------------------------------ */
/* Dynamic loss scaling                                                      */
/* ------------------------------------------------------------------------ */

/* state[0] = loss scale, applied = updates applied so far, good = applied
 * steps since the last overflow or growth.  After an overflow the scale
 * halves (not below min_scale) and nothing else advances; after an applied
 * step applied and good advance and, once good reaches window, the scale
 * doubles and good restarts. */
void zo_scaler_update(double* scale, int64_t* applied, int64_t* good, int32_t skipped,
                      int64_t window, double min_scale)
{
    if (skipped) {
        double s = *scale / 2.0;
        *scale = s < min_scale ? min_scale : s;
        *good = 0;
        return;
    }
    *applied += 1;
    *good += 1;
    if (window > 0 && *good >= window) {
        *scale *= 2.0;
        *good = 0;
    }
}

/* ------------------------------------------------------------------------ */
/* Exact sum of squares of fp32 values                                       */
/* ------------------------------------------------------------------------ */

/* A finite binary32 x equals M * 2^E with integer 0 <= M < 2^24 and
 * -149 <= E <= 104, so x^2 = M^2 * 2^(2E) is M^2 (below 2^48) shifted to bit
 * 2E + 298 >= 0 of a fixed-point number whose unit is 2^-298.  The largest
 * square reaches bit 554; 640 bits leave room for 2^85 terms.  Limbs are
 * little-endian 64-bit words. */
#define ZO_ACC_LIMBS 10

typedef struct {
    uint64_t limb[ZO_ACC_LIMBS];
    int32_t has_inf, has_nan;
} zo_acc_t;

static void acc_add_at(zo_acc_t* a, uint64_t value, int bit)
{
    int q = bit / 64, r = bit % 64;
    zo_u128 wide = (zo_u128)value << r;
    uint64_t parts[2] = {(uint64_t)wide, (uint64_t)(wide >> 64)};
    uint64_t carry = 0;
    for (int i = q; i < ZO_ACC_LIMBS; ++i) {
        zo_u128 s = (zo_u128)a->limb[i] + carry + (i - q < 2 ? parts[i - q] : 0);
        a->limb[i] = (uint64_t)s;
        carry = (uint64_t)(s >> 64);
        if (i - q >= 1 && carry == 0)
            break;
    }
}

static void acc_add_square(zo_acc_t* a, float x)
{
    uint32_t b;
    memcpy(&b, &x, 4);
    uint32_t e = (b >> 23) & 255u, f = b & 0x7FFFFFu;
    if (e == 255u) {
        if (f)
            a->has_nan = 1;
        else
            a->has_inf = 1;
        return;
    }
    uint64_t M = e ? (f | 0x800000u) : f;
    int E = e ? (int)e - 150 : -149;
    if (M)
        acc_add_at(a, M * M, 2 * E + 298);
}

/* The fixed-point value rounded once to the nearest double, ties to even. */
static double acc_to_double(const zo_acc_t* a)
{
    if (a->has_nan)
        return NAN;
    if (a->has_inf)
        return INFINITY;
    int top = -1;
    for (int i = ZO_ACC_LIMBS - 1; i >= 0 && top < 0; --i)
        if (a->limb[i])
            top = 64 * i + 63 - __builtin_clzll(a->limb[i]);
    if (top < 0)
        return 0.0;
    if (top < 64)
        return ldexp((double)a->limb[0], -298);  /* one 64-bit word: C rounds to nearest even */
    /* the 64 bits [top-63, top] and whether anything below them is nonzero */
    int lo = top - 63, q = lo / 64, r = lo % 64;
    uint64_t head = a->limb[q] >> r;
    if (r)
        head |= a->limb[q + 1] << (64 - r);
    int sticky = r ? (a->limb[q] & ((1ull << r) - 1)) != 0 : 0;
    for (int i = 0; i < q && !sticky; ++i)
        sticky = a->limb[i] != 0;
    uint64_t mant = head >> 11, rem = head & 0x7FFu;
    if (rem > 0x400u || (rem == 0x400u && (sticky || (mant & 1u))))
        mant += 1;  /* may reach 2^53, still exact as a double */
    return ldexp((double)mant, lo + 11 - 298);
}

/* sum of x[i]^2 over i < n, exact, then rounded once to double; +inf if an
 * element is infinite, NaN if one is NaN. */
double zo_sumsq_f32(const float* x, int64_t n)
{
    zo_acc_t a;
    memset(&a, 0, sizeof a);
    for (int64_t i = 0; i < n; ++i)
        acc_add_square(&a, x[i]);
    return acc_to_double(&a);
}

/* ------------------------------------------------------------------------ */
/* LAMB: Adam's moments with a per-layer trust ratio                         */
/* ------------------------------------------------------------------------ */

/* Layer-wise adaptive large-batch optimization (You et al., LAMB, one of the
 * adaptive optimizers ZeRO's related-work section lists as made affordable by
 * partitioning the optimizer state).  The flat vector is cut into layers
 * [seg_off[s], seg_off[s+1]).  Per element, in fp32, exactly as zo_adam up to
 * the update direction:
 *   m <- b1*m + (1-b1)*g;  v <- b2*v + (1-b2)*g^2
 *   u  = (m/(1-b1^t)) / (sqrt(v/(1-b2^t)) + eps)   [+ wd*theta]
 * then per layer, with the norms of the layer's old theta and of u taken
 * exactly and rounded once to double:
 *   trust = phi(||theta||) / ||u||   (1 when either norm is zero),
 *   phi(z) = min(max(z, phi_lo), phi_hi),
 *   step   = (float)(lr * trust)      (computed in double, rounded once)
 *   theta <- theta - step*u;  p16 = binary16(theta).
 * seg_out (3 doubles per layer, may be NULL) receives sum theta^2, sum u^2
 * and the trust ratio.  Returns 0, or -1 on a malformed layer table
 * (seg_off must rise strictly from 0 to n) or an allocation failure. */
int zo_lamb(const uint16_t* g16, float* theta, float* m, float* v, uint16_t* p16, int64_t n,
            const int64_t* seg_off, int32_t n_seg, float mult, const zo_hyper_t* h, double lr,
            double phi_lo, double phi_hi, double* seg_out)
{
    if (n_seg < 0 || (n_seg == 0 && n != 0) || (n_seg > 0 && (seg_off[0] != 0 || seg_off[n_seg] != n)))
        return -1;
    int64_t longest = 0;
    for (int32_t s = 0; s < n_seg; ++s) {
        if (seg_off[s + 1] <= seg_off[s])
            return -1;
        if (seg_off[s + 1] - seg_off[s] > longest)
            longest = seg_off[s + 1] - seg_off[s];
    }
    float* u = (float*)malloc((size_t)(longest ? longest : 1) * sizeof(float));
    if (!u)
        return -1;
    for (int32_t s = 0; s < n_seg; ++s) {
        const int64_t a = seg_off[s], len = seg_off[s + 1] - a;
        for (int64_t j = 0; j < len; ++j) {
            const int64_t i = a + j;
            float g = zo_f16_to_f32(g16[i]) * mult;
            u[j] = adam_direction(g, &m[i], &v[i], theta[i], h);
        }
        const double st = zo_sumsq_f32(theta + a, len);
        const double su = zo_sumsq_f32(u, len);
        double trust = 1.0;
        if (st > 0.0 && su > 0.0) {
            double wn = sqrt(st);
            if (wn < phi_lo)
                wn = phi_lo;
            if (wn > phi_hi)
                wn = phi_hi;
            trust = wn / sqrt(su);
        }
        const float step = (float)(lr * trust);
        for (int64_t j = 0; j < len; ++j) {
            const int64_t i = a + j;
            float th = theta[i] - step * u[j];
            theta[i] = th;
            p16[i] = zo_f32_to_f16(th);
        }
        if (seg_out) {
            seg_out[3 * s] = st;
            seg_out[3 * s + 1] = su;
            seg_out[3 * s + 2] = trust;
        }
    }
    free(u);
    return 0;
}

/* The whole LAMB step: gradient statistics and scalars as for Adam, then
 * skip (returns 1, nothing written) or the update (returns 0); -1 on a
 * malformed layer table. */
int zo_lamb_step(const uint16_t* g16, float* theta, float* m, float* v, uint16_t* p16, int64_t n,
                 const int64_t* seg_off, int32_t n_seg, double lr, double beta1, double beta2, double eps,
                 double wd, int64_t t, double loss_scale, double clip, double phi_lo, double phi_hi,
                 zo_scalars_t* out, double* seg_out)
{
    uint64_t s[2];
    int32_t ovf;
    zo_scalars_t sc;
    zo_local_stats(g16, n, s, &ovf);
    zo_scalars(s, ovf, loss_scale, clip, &sc);
    if (out)
        *out = sc;
    if (sc.skip != 0)
        return 1;
    zo_hyper_t h;
    zo_hyper(lr, beta1, beta2, eps, wd, t, &h);
    return zo_lamb(g16, theta, m, v, p16, n, seg_off, n_seg, sc.mult, &h, lr, phi_lo, phi_hi, seg_out);
}
