/*
 * c_abi_driver.c -- a plain C99 program that drives libzeroshard through its C
 * ABI alone: HIP's C runtime API for device memory and streams, the library
 * for the shard step (ZeRO Sec. 5.1-5.2 P_os+g rank step with Sec. 3.1's
 * mixed-precision Adam state), and the CPU oracle for the expected bytes.  No
 * Python and no PyTorch are involved.
 *
 * Test infrastructure: it links the oracle.  Exit status 0 = every check
 * passed, 1 = a mismatch or an error (described on stdout), 77 = no GPU.
 *
 * Cases: shards of several lengths, with all arrays 16-byte aligned, all
 * shifted by the same element count (vector path with a scalar head) and
 * shifted by different counts (scalar path); per case three fused steps, the
 * second with an inf gradient (skipped, nothing written), then one split-phase
 * step (zero_shard_stats, then zero_shard_apply with that sum as the global
 * one), each compared byte for byte with the oracle; then LAMB steps through a
 * layer-table plan (tiny layers, layers across tile boundaries) at the same
 * three alignments.
 */
#include <hip/hip_runtime_api.h>

#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "zero_shard.h"

/* The oracle's shard steps (oracle/zero_oracle.c); the scalar and per-layer outputs may be NULL. */
int zo_shard_step(const uint16_t* g16, float* theta, float* m, float* v, uint16_t* p16, int64_t n, double lr,
                  double beta1, double beta2, double eps, double wd, int64_t t, double loss_scale, double clip,
                  void* scalars_out);
int zo_lamb_step(const uint16_t* g16, float* theta, float* m, float* v, uint16_t* p16, int64_t n,
                 const int64_t* seg_off, int32_t n_seg, double lr, double beta1, double beta2, double eps,
                 double wd, int64_t t, double loss_scale, double clip, double phi_lo, double phi_hi,
                 void* scalars_out, double* seg_out);
/* The oracle's model-state accounting and fp32 update constants. */
double zo_model_state_bytes(double psi, double nd, int32_t stage, double k);
typedef struct {
    float lr, b1, omb1, b2, omb2, bc1, bc2, eps, wd;
} zo_hyper_t;
void zo_hyper(double lr, double beta1, double beta2, double eps, double wd, int64_t t, zo_hyper_t* h);
/* The oracle's loss-scale schedule. */
void zo_scaler_update(double* scale, int64_t* applied, int64_t* good, int32_t skipped, int64_t window,
                      double min_scale);

#define LR 1e-4
#define B1 0.9
#define B2 0.999
#define EPS 1e-8
#define WD 0.01
#define SCALE 65536.0
#define CLIP 1.0
#define PAD 8        /* spare elements per buffer, for the shifted cases */
#define SENTINEL 0xA5A5u

#define HIPCHECK(x)                                                                                  \
    do {                                                                                             \
        hipError_t e_ = (x);                                                                         \
        if (e_ != hipSuccess) {                                                                      \
            printf("FAIL: %s: %s (line %d)\n", #x, hipGetErrorString(e_), __LINE__);                 \
            exit(1);                                                                                 \
        }                                                                                            \
    } while (0)

/* SplitMix64: a counter-based generator for the test inputs (bit patterns only). */
static uint64_t g_rng;
static uint64_t rnd(void) {
    uint64_t z = (g_rng += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* A float with a random sign (unless positive), a biased exponent in [elo, ehi] and random mantissa. */
static float rnd_f32(unsigned elo, unsigned ehi, int positive) {
    const uint64_t r = rnd();
    const uint32_t e = elo + (uint32_t)(r % (ehi - elo + 1));
    const uint32_t bits = (positive ? 0u : ((uint32_t)(r >> 63) << 31)) | (e << 23) | (uint32_t)((r >> 8) & 0x7FFFFF);
    float f;
    memcpy(&f, &bits, sizeof f);
    return f;
}

/* A finite fp16 pattern: random sign, biased exponent in [1, 22], random mantissa. */
static uint16_t rnd_f16(void) {
    const uint64_t r = rnd();
    const uint32_t e = 1 + (uint32_t)(r % 22);
    return (uint16_t)(((r >> 63) << 15) | (e << 10) | ((r >> 20) & 0x3FF));
}

typedef struct {
    void* d[5];          /* device allocations: grad16, master32, m32, v32, param16_out */
    char* view[5];       /* shifted views into them */
    uint16_t *g, *p;     /* host copies */
    float *th, *m, *v;
} shard_t;

static const size_t kSize[5] = {2, 4, 4, 4, 2};

static void upload(shard_t* s, int i, const void* src, int64_t n) {
    HIPCHECK(hipMemcpy(s->view[i], src, kSize[i] * (size_t)n, hipMemcpyHostToDevice));
}

static int same(const shard_t* s, int i, const void* ref, int64_t n, const char* what) {
    void* got = malloc(kSize[i] * (size_t)(n ? n : 1));
    HIPCHECK(hipMemcpy(got, s->view[i], kSize[i] * (size_t)n, hipMemcpyDeviceToHost));
    const int ok = memcmp(got, ref, kSize[i] * (size_t)n) == 0;
    if (!ok) {
        int64_t k = 0;
        while (memcmp((char*)got + k * kSize[i], (const char*)ref + k * kSize[i], kSize[i]) == 0)
            ++k;
        printf("FAIL: %s: array %d differs from the oracle first at element %lld\n", what, i, (long long)k);
    }
    free(got);
    return ok;
}

static int check_all(const shard_t* s, int64_t n, const char* what) {
    return same(s, 1, s->th, n, what) && same(s, 2, s->m, n, what) && same(s, 3, s->v, n, what) &&
           same(s, 4, s->p, n, what);
}

static int run_case(int64_t n, const int shift[5], hipStream_t stream) {
    shard_t s;
    char what[128];
    for (int i = 0; i < 5; ++i) {
        HIPCHECK(hipMalloc(&s.d[i], kSize[i] * (size_t)(n + PAD)));
        s.view[i] = (char*)s.d[i] + kSize[i] * (size_t)shift[i];
    }
    s.g = malloc(2 * (size_t)n + 2);
    s.p = malloc(2 * (size_t)n + 2);
    s.th = malloc(4 * (size_t)n + 4);
    s.m = malloc(4 * (size_t)n + 4);
    s.v = malloc(4 * (size_t)n + 4);
    for (int64_t k = 0; k < n; ++k) {
        s.th[k] = rnd_f32(110, 126, 0);
        s.m[k] = rnd_f32(100, 115, 0);
        s.v[k] = rnd_f32(90, 110, 1);
        s.p[k] = SENTINEL;
    }
    upload(&s, 1, s.th, n);
    upload(&s, 2, s.m, n);
    upload(&s, 3, s.v, n);
    upload(&s, 4, s.p, n);

    int ok = 1;
    int64_t t = 1;
    for (int k = 1; k <= 3 && ok; ++k) {
        for (int64_t j = 0; j < n; ++j)
            s.g[j] = rnd_f16();
        if (k == 2 && n > 0)
            s.g[n / 2] = 0x7C00; /* +inf: the step must be skipped */
        upload(&s, 0, s.g, n);
        const int rc = zero_shard_step((const uint16_t*)s.view[0], (float*)s.view[1], (float*)s.view[2],
                                       (float*)s.view[3], (uint16_t*)s.view[4], n, LR, B1, B2, EPS, WD, t, SCALE,
                                       CLIP, stream);
        HIPCHECK(hipStreamSynchronize(stream));
        const int want = zo_shard_step(s.g, s.th, s.m, s.v, s.p, n, LR, B1, B2, EPS, WD, t, SCALE, CLIP, NULL);
        snprintf(what, sizeof what, "n=%lld shifts=%d%d%d%d%d step %d", (long long)n, shift[0], shift[1], shift[2],
                 shift[3], shift[4], k);
        if (rc != want) {
            printf("FAIL: %s: zero_shard_step returned %d (%s), the oracle %d\n", what, rc, zero_last_error(), want);
            ok = 0;
            break;
        }
        zero_step_stats_t st;
        if (n > 0 && (zero_shard_last_step_stats(&st) != ZERO_OK || st.skipped != want || st.n != n)) {
            printf("FAIL: %s: last stats disagree (skipped %d, n %lld)\n", what, st.skipped, (long long)st.n);
            ok = 0;
            break;
        }
        double norm = -1.0;
        float mult = -1.0f;
        int ovf = -1;
        if (n > 0 && (zero_shard_last_stats(&norm, &mult, &ovf) != ZERO_OK || ovf != want ||
                      memcmp(&norm, &st.norm, sizeof norm) != 0 || memcmp(&mult, &st.mult, sizeof mult) != 0)) {
            printf("FAIL: %s: three-pointer last stats disagree with the record\n", what);
            ok = 0;
            break;
        }
        ok = check_all(&s, n, what);
        if (!want)
            ++t;
    }
    if (ok && n > 0) {
        /* one split-phase step: this shard's sum is the global sum of a one-rank job */
        for (int64_t j = 0; j < n; ++j)
            s.g[j] = rnd_f16();
        upload(&s, 0, s.g, n);
        double local = -1.0;
        int rc = zero_shard_stats((const uint16_t*)s.view[0], n, &local, stream);
        if (rc == ZERO_OK)
            rc = zero_shard_apply((const uint16_t*)s.view[0], (float*)s.view[1], (float*)s.view[2],
                                  (float*)s.view[3], (uint16_t*)s.view[4], n, local, LR, B1, B2, EPS, WD, t, SCALE,
                                  CLIP, stream);
        HIPCHECK(hipStreamSynchronize(stream));
        const int want = zo_shard_step(s.g, s.th, s.m, s.v, s.p, n, LR, B1, B2, EPS, WD, t, SCALE, CLIP, NULL);
        snprintf(what, sizeof what, "n=%lld split phase", (long long)n);
        if (rc != want) {
            printf("FAIL: %s: returned %d (%s), the oracle %d\n", what, rc, zero_last_error(), want);
            ok = 0;
        } else {
            ok = check_all(&s, n, what);
        }
    }
    if (ok && n > 0) {
        /* two scaler-driven steps, the second skipped (window 1: the scale doubles after every
           applied step); the library's scaler against the oracle's schedule */
        zero_scaler_t sc;
        if (zero_scaler_init(&sc, SCALE, 1, 1.0) != ZERO_OK) {
            printf("FAIL: zero_scaler_init\n");
            ok = 0;
        }
        sc.applied = t - 1;
        double o_scale = SCALE;
        int64_t o_applied = t - 1, o_good = 0;
        const zero_step_args_t args = {(const uint16_t*)s.view[0], (float*)s.view[1], (float*)s.view[2],
                                       (float*)s.view[3], (uint16_t*)s.view[4], n, LR, B1, B2, EPS, WD, CLIP,
                                       stream};
        for (int k = 0; k < 2 && ok; ++k) {
            for (int64_t j = 0; j < n; ++j)
                s.g[j] = rnd_f16();
            if (k == 1)
                s.g[0] = 0x7E00; /* NaN: skipped */
            upload(&s, 0, s.g, n);
            const int rc = zero_shard_step_scaled(&args, &sc);
            HIPCHECK(hipStreamSynchronize(stream));
            const int want = zo_shard_step(s.g, s.th, s.m, s.v, s.p, n, LR, B1, B2, EPS, WD, o_applied + 1, o_scale,
                                           CLIP, NULL);
            zo_scaler_update(&o_scale, &o_applied, &o_good, want, 1, 1.0);
            snprintf(what, sizeof what, "n=%lld scaled step %d", (long long)n, k);
            if (rc != want || sc.scale != o_scale || sc.applied != o_applied || sc.good != o_good) {
                printf("FAIL: %s: returned %d (%s), the oracle %d; scaler (%g, %lld, %lld), oracle (%g, %lld, %lld)\n",
                       what, rc, zero_last_error(), want, sc.scale, (long long)sc.applied, (long long)sc.good,
                       o_scale, (long long)o_applied, (long long)o_good);
                ok = 0;
            } else {
                ok = check_all(&s, n, what);
            }
        }
    }
    for (int i = 0; i < 5; ++i)
        HIPCHECK(hipFree(s.d[i]));
    free(s.g);
    free(s.p);
    free(s.th);
    free(s.m);
    free(s.v);
    if (ok)
        printf("ok: n=%lld shifts=%d%d%d%d%d\n", (long long)n, shift[0], shift[1], shift[2], shift[3], shift[4]);
    fflush(stdout);
    return ok;
}

/* LAMB (ZeRO Sec. 2.3 lists it among the optimizers whose state partitioning
 * makes affordable): one step over a layer table with a few tiny layers and
 * layers that do not line up with the kernels' tiles, through a plan. */
static int run_lamb_case(int64_t n, const int shift[5], hipStream_t stream) {
    shard_t s;
    char what[128];
    int64_t off[16];
    int32_t n_seg = 0;
    const int64_t cuts[] = {1, 2, 5, 517, 4096, 4099, 70001};
    off[n_seg] = 0;
    for (size_t k = 0; k < sizeof cuts / sizeof cuts[0]; ++k)
        if (cuts[k] > off[n_seg] && cuts[k] < n)
            off[++n_seg] = cuts[k];
    off[++n_seg] = n;
    for (int i = 0; i < 5; ++i) {
        HIPCHECK(hipMalloc(&s.d[i], kSize[i] * (size_t)(n + PAD)));
        s.view[i] = (char*)s.d[i] + kSize[i] * (size_t)shift[i];
    }
    s.g = malloc(2 * (size_t)n);
    s.p = malloc(2 * (size_t)n);
    s.th = malloc(4 * (size_t)n);
    s.m = malloc(4 * (size_t)n);
    s.v = malloc(4 * (size_t)n);
    for (int64_t k = 0; k < n; ++k) {
        s.g[k] = rnd_f16();
        s.th[k] = rnd_f32(110, 126, 0);
        s.m[k] = rnd_f32(100, 115, 0);
        s.v[k] = rnd_f32(90, 110, 1);
        s.p[k] = SENTINEL;
    }
    for (int i = 0; i < 5; ++i)
        upload(&s, i, i == 0 ? (const void*)s.g : i == 1 ? (const void*)s.th : i == 2 ? (const void*)s.m
                                                  : i == 3 ? (const void*)s.v : (const void*)s.p, n);
    zero_lamb_plan_t* plan = NULL;
    int ok = 1;
    int rc = zero_lamb_plan_create(off, n_seg, n, &plan);
    snprintf(what, sizeof what, "lamb n=%lld layers=%d shifts=%d%d%d%d%d", (long long)n, n_seg, shift[0], shift[1],
             shift[2], shift[3], shift[4]);
    if (rc != ZERO_OK) {
        printf("FAIL: %s: plan: %s\n", what, zero_last_error());
        ok = 0;
    } else {
        rc = zero_lamb_step(plan, (const uint16_t*)s.view[0], (float*)s.view[1], (float*)s.view[2],
                            (float*)s.view[3], (uint16_t*)s.view[4], LR, B1, B2, 1e-6, WD, 3, SCALE, CLIP, 0.0,
                            10.0, stream);
        HIPCHECK(hipStreamSynchronize(stream));
        const int want = zo_lamb_step(s.g, s.th, s.m, s.v, s.p, n, off, n_seg, LR, B1, B2, 1e-6, WD, 3, SCALE,
                                      CLIP, 0.0, 10.0, NULL, NULL);
        if (rc != want) {
            printf("FAIL: %s: zero_lamb_step returned %d (%s), the oracle %d\n", what, rc, zero_last_error(), want);
            ok = 0;
        } else {
            ok = check_all(&s, n, what);
        }
        if (zero_lamb_plan_destroy(plan) != ZERO_OK) {
            printf("FAIL: %s: plan destroy: %s\n", what, zero_last_error());
            ok = 0;
        }
    }
    for (int i = 0; i < 5; ++i)
        HIPCHECK(hipFree(s.d[i]));
    free(s.g);
    free(s.p);
    free(s.th);
    free(s.m);
    free(s.v);
    if (ok)
        printf("ok: %s\n", what);
    fflush(stdout);
    return ok;
}

/* Host-only entry points against the oracle (no GPU needed): the accounting of
 * every Table 1 cell's parameters and the bias corrections of the first 2000
 * steps of two Adam settings. */
static int host_checks(void) {
    const double psis[3] = {7.5e9, 128e9, 1e12};
    const int32_t nds[6] = {1, 4, 16, 64, 256, 1024};
    for (int a = 0; a < 3; ++a)
        for (int b = 0; b < 6; ++b)
            for (int32_t st = ZERO_STAGE_DP; st <= ZERO_STAGE_OS_G_P; ++st) {
                double got = -1.0;
                const double want = zo_model_state_bytes(psis[a], (double)nds[b], st, 12.0);
                if (zero_memory_bytes(psis[a], nds[b], st, 12, &got) != ZERO_OK || got != want) {
                    printf("FAIL: zero_memory_bytes(%g, %d, %d, 12) = %.17g, oracle %.17g\n", psis[a], nds[b], st,
                           got, want);
                    return 0;
                }
            }
    if (zero_memory_bytes(1e9, 0, ZERO_STAGE_OS, 12, NULL) != ZERO_EINVAL) {
        printf("FAIL: zero_memory_bytes accepted nd = 0 and a NULL out\n");
        return 0;
    }
    const double betas[2][2] = {{0.9, 0.999}, {0.95, 0.98}};
    for (int k = 0; k < 2; ++k)
        for (int64_t t = 1; t <= 2000; ++t) {
            float bc1 = 0.f, bc2 = 0.f;
            zo_hyper_t h;
            zo_hyper(LR, betas[k][0], betas[k][1], 1e-8, 0.0, t, &h);
            if (zero_bias_corrections(betas[k][0], betas[k][1], t, &bc1, &bc2) != ZERO_OK ||
                memcmp(&bc1, &h.bc1, sizeof bc1) != 0 || memcmp(&bc2, &h.bc2, sizeof bc2) != 0) {
                printf("FAIL: bias corrections at betas (%g, %g), t = %lld differ from the oracle\n", betas[k][0],
                       betas[k][1], (long long)t);
                return 0;
            }
        }
    printf("host checks ok\n");
    return 1;
}

int main(void) {
    if (!host_checks())
        return 1;
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) {
        printf("no GPU\n");
        return 77;
    }
    HIPCHECK(hipSetDevice(0));
    hipStream_t stream;
    HIPCHECK(hipStreamCreate(&stream));
    g_rng = 20191002u;
    const int aligned[5] = {0, 0, 0, 0, 0};
    const int equal[5] = {3, 3, 3, 3, 3};
    const int mixed[5] = {1, 2, 0, 3, 5};
    const int64_t sizes[] = {0, 1, 5, 1023, 65537, 1000003};
    int ok = 1;
    for (size_t k = 0; k < sizeof sizes / sizeof sizes[0] && ok; ++k) {
        ok = run_case(sizes[k], aligned, stream) && run_case(sizes[k], equal, stream) &&
             run_case(sizes[k], mixed, stream);
    }
    /* the null stream too */
    ok = ok && run_case(262147, equal, NULL);
    /* LAMB through its plan */
    const int64_t lamb_sizes[] = {3, 600, 100003};
    for (size_t k = 0; k < sizeof lamb_sizes / sizeof lamb_sizes[0] && ok; ++k)
        ok = run_lamb_case(lamb_sizes[k], aligned, stream) && run_lamb_case(lamb_sizes[k], equal, stream) &&
             run_lamb_case(lamb_sizes[k], mixed, stream);
    if (zero_stream_release(stream) != ZERO_OK) {
        printf("FAIL: zero_stream_release: %s\n", zero_last_error());
        ok = 0;
    }
    HIPCHECK(hipStreamDestroy(stream));
    printf(ok ? "c-abi driver: all cases match the oracle\n" : "c-abi driver: FAILED\n");
    return ok ? 0 : 1;
}
