/* Pure-C use of the DQGAN library (include/dqgan.h, libdqgan.so) with the
 * HIP runtime's C API for device memory: one fused iteration of Algorithm 2
 * for M workers with the s = 15 quantizer, checked against the C oracle
 * (oracle/libdqgan_oracle.so), teacher-forced with the GPU's segment scales:
 * every output bit for bit, the scales within 1e-5 of the oracle's own.
 * Test infrastructure: exits 0 and prints "c abi demo ok" on success. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "dqgan.h"

/* The oracle's iteration (oracle/dqgan_oracle.c). */
typedef struct {
    int64_t d, ld;
    int32_t M, n_seg;
    const int64_t *seg_offsets;
    int32_t kind, norm;
    int32_t levels;
    int64_t k;
    uint64_t seed;
} oracle_desc;
int oracle_step(const oracle_desc *D, float eta, uint32_t t, const float *G, float *E, float *W, float *WX,
                uint32_t *sign_words, uint32_t *level_words, float *scales, float *val, uint32_t *idx, float *qhat,
                const float *scales_in);

#define HIP_OK(x)                                                            \
    do {                                                                     \
        hipError_t e_ = (x);                                                 \
        if (e_ != hipSuccess) {                                              \
            fprintf(stderr, "%s:%d: %s\n", __FILE__, __LINE__, hipGetErrorString(e_)); \
            return 2;                                                        \
        }                                                                    \
    } while (0)

static uint64_t lcg = 0x9E3779B97F4A7C15ull;
static float uniform_pm1(void) { /* in (-1, 1), 24-bit grid */
    lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
    return ((float)(lcg >> 40) - 8388608.0f) / 8388608.0f;
}

static int same_bits(const char *name, const void *a, const void *b, size_t n) {
    if (memcmp(a, b, n) == 0) return 1;
    fprintf(stderr, "%s differs from the oracle\n", name);
    return 0;
}

int main(void) {
    const int64_t d = 10007, ld = 10240;
    const int32_t M = 5, S = 3;
    const int64_t offs[4] = {0, 1000, 6001, 10007};
    const float eta = 0.01f;
    const uint32_t t = 3;
    dqgan_desc desc;
    memset(&desc, 0, sizeof desc);
    desc.d = d;
    desc.ld = ld;
    desc.M = M;
    desc.n_seg = S;
    desc.seg_offsets = offs;
    desc.kind = DQGAN_QSGD;
    desc.norm = DQGAN_L2;
    desc.levels = 15;
    desc.seed = 0x5EEDull;
    dqgan_plan plan;
    dqgan_status st = dqgan_plan_create(&desc, &plan);
    if (st != DQGAN_OK) {
        fprintf(stderr, "plan: %s\n", dqgan_status_string(st));
        return 2;
    }
    size_t sb, lb, cb, vb, ib;
    dqgan_wire_bytes(plan, &sb, &lb, &cb, &vb, &ib);

    const size_t mat = (size_t)M * ld, vec = (size_t)ld;
    float *hG = calloc(mat, 4), *hE = calloc(mat, 4), *hW = calloc(vec, 4);
    for (int32_t m = 0; m < M; ++m)
        for (int64_t i = 0; i < d; ++i) {
            hG[m * ld + i] = uniform_pm1();
            hE[m * ld + i] = 1e-3f * uniform_pm1();
        }
    for (int64_t i = 0; i < d; ++i) hW[i] = 0.02f * uniform_pm1();

    float *G, *E, *W, *WX, *Q;
    dqgan_wire wire;
    memset(&wire, 0, sizeof wire);
    HIP_OK(hipMalloc((void **)&G, mat * 4));
    HIP_OK(hipMalloc((void **)&E, mat * 4));
    HIP_OK(hipMalloc((void **)&WX, mat * 4));
    HIP_OK(hipMalloc((void **)&W, vec * 4));
    HIP_OK(hipMalloc((void **)&Q, vec * 4));
    HIP_OK(hipMalloc((void **)&wire.sign, sb));
    HIP_OK(hipMalloc((void **)&wire.level, lb));
    HIP_OK(hipMalloc((void **)&wire.scale, cb));
    HIP_OK(hipMemcpy(G, hG, mat * 4, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(E, hE, mat * 4, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(W, hW, vec * 4, hipMemcpyHostToDevice));

    st = dqgan_step_fused(plan, eta, t, G, E, W, WX, &wire, Q, NULL);
    if (st != DQGAN_OK) {
        fprintf(stderr, "step: %s\n", dqgan_status_string(st));
        return 2;
    }
    HIP_OK(hipDeviceSynchronize());

    float *gE = malloc(mat * 4), *gW = malloc(vec * 4), *gWX = malloc(mat * 4), *gQ = malloc(vec * 4);
    float *gS = malloc(cb);
    uint32_t *gSign = malloc(sb), *gLevel = malloc(lb);
    HIP_OK(hipMemcpy(gE, E, mat * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gW, W, vec * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gWX, WX, mat * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gQ, Q, vec * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gS, wire.scale, cb, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gSign, wire.sign, sb, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gLevel, wire.level, lb, hipMemcpyDeviceToHost));

    /* the oracle from the same inputs, with the GPU's scales */
    oracle_desc od = {d, ld, M, S, offs, 1, 2, 15, 0, desc.seed};
    float *oE = malloc(mat * 4), *oW = malloc(vec * 4), *oWX = calloc(mat, 4), *oQ = calloc(vec, 4);
    float *oS = malloc(cb);
    uint32_t *oSign = calloc(sb / 4, 4), *oLevel = calloc(lb / 4, 4);
    memcpy(oE, hE, mat * 4);
    memcpy(oW, hW, vec * 4);
    if (oracle_step(&od, eta, t, hG, oE, oW, oWX, oSign, oLevel, oS, NULL, NULL, oQ, gS) != 0) return 2;

    int ok = same_bits("sign plane", gSign, oSign, sb) && same_bits("level plane", gLevel, oLevel, lb);
    for (int32_t m = 0; ok && m < M; ++m) {
        ok = same_bits("e_t", gE + m * ld, oE + m * ld, (size_t)d * 4) &&
             same_bits("WX", gWX + m * ld, oWX + m * ld, (size_t)d * 4);
    }
    ok = ok && same_bits("w_t", gW, oW, (size_t)d * 4) && same_bits("q-hat", gQ, oQ, (size_t)d * 4);

    /* the oracle's own scales */
    memcpy(oE, hE, mat * 4);
    memcpy(oW, hW, vec * 4);
    if (oracle_step(&od, eta, t, hG, oE, oW, oWX, oSign, oLevel, oS, NULL, NULL, oQ, NULL) != 0) return 2;
    for (int32_t j = 0; ok && j < M * S; ++j) {
        if (!(fabs((double)gS[j] - (double)oS[j]) <= 1e-5 * fabs((double)oS[j]))) {
            fprintf(stderr, "scale %d: %.9g vs %.9g\n", j, gS[j], oS[j]);
            ok = 0;
        }
    }
    dqgan_plan_destroy(plan);
    if (!ok) return 1;
    printf("c abi demo ok: %d workers, d = %lld, s = 15, every output identical to the oracle\n", M, (long long)d);
    return 0;
}
