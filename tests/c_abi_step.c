/*
 * A C program (no Python, no torch) that uses libssmq.so through include/ssmq.h:
 * device buffers from the HIP runtime, one fused bf16 Weyl step and one E4M3 SR
 * step on a small Mamba-2 layer, results checked against the CPU oracle
 * (test infrastructure, linked only here), and a rejected call's error path.
 * Prints "c_abi_step: ok" and exits 0 on success.
 */
#define __HIP_PLATFORM_AMD__
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "ssmq.h"

/* The oracle's entry points used here (oracle/ssmq_oracle.c). */
int orc_requantize(int f, int rule, uint32_t seed, uint32_t layer, uint32_t step,
                   uint64_t entry_base, uint64_t block, int64_t n, int64_t group, const float *h,
                   void *codes, float *scale);
int orc_state_update(int f, int rule, uint32_t seed, uint32_t layer, uint32_t step,
                     uint64_t entry_base, uint64_t block, int64_t group, int64_t batch,
                     int64_t nheads, int64_t headdim, int64_t dstate, int64_t ngroups,
                     int a_per_state, void *state, float *scale, const float *x, const float *dt,
                     const float *A, const float *B, const float *C, const float *D, double *y,
                     float *hnew);
int orc_code_rank(int f, uint32_t code);

#define CHECK_HIP(e)                                                          \
    do {                                                                      \
        hipError_t err_ = (e);                                                \
        if (err_ != hipSuccess) {                                             \
            fprintf(stderr, "HIP error %d at line %d\n", (int)err_, __LINE__); \
            return 1;                                                         \
        }                                                                     \
    } while (0)

enum { BATCH = 2, NHEADS = 4, HEADDIM = 64, DSTATE = 128, NGROUPS = 2 };
#define NENT (BATCH * NHEADS * HEADDIM * DSTATE)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static double uniform01(void) { /* xorshift64*, top 53 bits */
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (double)((rng_state * 0x2545F4914F6CDD1Dull) >> 11) * 0x1p-53;
}
static float normal(void) { /* Box-Muller */
    double u = uniform01(), v = uniform01();
    return (float)(sqrt(-2.0 * log(u + 1e-300)) * cos(6.283185307179586 * v));
}

static int run_case(int format, int rule, int code_bytes) {
    static float h0[NENT], x[BATCH * NHEADS * HEADDIM], dt[BATCH * NHEADS], A[NHEADS], D[NHEADS];
    static float B[BATCH * NGROUPS * DSTATE], C[BATCH * NGROUPS * DSTATE], y[BATCH * NHEADS * HEADDIM];
    static double y_ref[BATCH * NHEADS * HEADDIM];
    static float h_new[NENT];
    static uint8_t codes[NENT * 2], codes_ref[NENT * 2], codes_gpu[NENT * 2];
    float scale[BATCH * NHEADS], scale_ref[BATCH * NHEADS], scale_gpu[BATCH * NHEADS];
    const int scaled = (format == SSMQ_FP8_E4M3);
    for (int i = 0; i < NENT; ++i) h0[i] = 0.1f * normal();
    for (int i = 0; i < BATCH * NHEADS * HEADDIM; ++i) x[i] = normal();
    for (int i = 0; i < BATCH * NHEADS; ++i) dt[i] = log1pf(expf(normal() - 4.0f));
    for (int i = 0; i < NHEADS; ++i) { A[i] = -expf(2.5f * (float)uniform01()); D[i] = normal(); }
    for (int i = 0; i < BATCH * NGROUPS * DSTATE; ++i) { B[i] = normal(); C[i] = normal(); }
    /* initial codes: the oracle's round-to-nearest write of h0 (one scale per head) */
    if (orc_requantize(format, SSMQ_RTN, 0, 0, 0, 0, 128, NENT, HEADDIM * DSTATE, h0, codes,
                       scaled ? scale : NULL) != 0)
        return 1;
    memcpy(codes_ref, codes, (size_t)NENT * code_bytes);
    memcpy(scale_ref, scale, sizeof scale);

    void *d_state, *d_scale, *d_x, *d_dt, *d_A, *d_B, *d_C, *d_D, *d_y;
    CHECK_HIP(hipMalloc(&d_state, (size_t)NENT * code_bytes));
    CHECK_HIP(hipMalloc(&d_scale, sizeof scale));
    CHECK_HIP(hipMalloc(&d_x, sizeof x));
    CHECK_HIP(hipMalloc(&d_dt, sizeof dt));
    CHECK_HIP(hipMalloc(&d_A, sizeof A));
    CHECK_HIP(hipMalloc(&d_B, sizeof B));
    CHECK_HIP(hipMalloc(&d_C, sizeof C));
    CHECK_HIP(hipMalloc(&d_D, sizeof D));
    CHECK_HIP(hipMalloc(&d_y, sizeof y));
    CHECK_HIP(hipMemcpy(d_state, codes, (size_t)NENT * code_bytes, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_scale, scale, sizeof scale, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_x, x, sizeof x, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_dt, dt, sizeof dt, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_A, A, sizeof A, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_B, B, sizeof B, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_C, C, sizeof C, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_D, D, sizeof D, hipMemcpyHostToDevice));

    ssmq_dims dims = {BATCH, NHEADS, HEADDIM, DSTATE, NGROUPS, 0};
    ssmq_qparams q;
    memset(&q, 0, sizeof q);
    q.rule = rule;
    q.format = format;
    q.dither_block = 128;
    q.scale_group = 0;
    q.seed = 1;
    q.layer = 3;
    q.step = 42;
    ssmq_status st = ssmq_state_update(&dims, &q, d_state, scaled ? (float *)d_scale : NULL,
                                       (const float *)d_x, (const float *)d_dt, (const float *)d_A,
                                       (const float *)d_B, (const float *)d_C, (const float *)d_D,
                                       (float *)d_y, NULL);
    if (st != SSMQ_OK) {
        fprintf(stderr, "ssmq_state_update: %s (%s)\n", ssmq_status_string(st), ssmq_last_error());
        return 1;
    }
    CHECK_HIP(hipDeviceSynchronize());
    CHECK_HIP(hipMemcpy(codes_gpu, d_state, (size_t)NENT * code_bytes, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(scale_gpu, d_scale, sizeof scale, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(y, d_y, sizeof y, hipMemcpyDeviceToHost));
    if (orc_state_update(format, rule, 1, 3, 42, 0, 128, 0, BATCH, NHEADS, HEADDIM, DSTATE, NGROUPS,
                         0, codes_ref, scaled ? scale_ref : NULL, x, dt, A, B, C, D, y_ref,
                         h_new) != 0)
        return 1;

    int differ = 0, far = 0;
    for (int i = 0; i < NENT; ++i) {
        uint32_t g = code_bytes == 2 ? ((uint16_t *)codes_gpu)[i] : codes_gpu[i];
        uint32_t r = code_bytes == 2 ? ((uint16_t *)codes_ref)[i] : codes_ref[i];
        if (g != r) {
            ++differ;
            if (abs(orc_code_rank(format, g) - orc_code_rank(format, r)) > 1) ++far;
        }
    }
    /* y per element within 1e-5 of |y| + sum_n |C_n h_n| + |D x| (h_n before rounding) */
    int y_bad = 0;
    for (int i = 0; i < BATCH * NHEADS * HEADDIM; ++i) {
        const int b = i / (NHEADS * HEADDIM), hd = (i / HEADDIM) % NHEADS;
        const float *Cg = C + (b * NGROUPS + hd / (NHEADS / NGROUPS)) * DSTATE;
        double mag = fabs((double)D[hd] * x[i]) + fabs(y_ref[i]);
        for (int n = 0; n < DSTATE; ++n) mag += fabs((double)Cg[n] * h_new[i * DSTATE + n]);
        if (fabs((double)y[i] - y_ref[i]) > 1e-5 * mag) ++y_bad;
    }
    /* the group scales are fp32 outputs of the step: within 1e-5 relative */
    int scale_bad = 0, scale_differ = 0;
    for (int i = 0; scaled && i < BATCH * NHEADS; ++i) {
        if (scale_gpu[i] != scale_ref[i]) ++scale_differ;
        if (fabs((double)scale_gpu[i] - scale_ref[i]) > 1e-5 * fabs((double)scale_ref[i])) ++scale_bad;
    }
    printf("c_abi_step: format %d rule %d: %d of %d codes differ (%d by more than one step), "
           "%d y outside tolerance, %d scales differ (%d outside 1e-5)\n", format, rule, differ,
           NENT, far, y_bad, scale_differ, scale_bad);
    hipFree(d_state); hipFree(d_scale); hipFree(d_x); hipFree(d_dt); hipFree(d_A);
    hipFree(d_B); hipFree(d_C); hipFree(d_D); hipFree(d_y);
    return (differ * 10000 > NENT || far || y_bad || scale_bad) ? 1 : 0;
}

int main(void) {
    if (run_case(SSMQ_BF16, SSMQ_WEYL, 2) != 0) return 1;
    if (run_case(SSMQ_FP8_E4M3, SSMQ_SR, 1) != 0) return 1;
    /* a rejected call: validated on the host, nothing launched, a message left */
    ssmq_qparams q;
    memset(&q, 0, sizeof q);
    q.rule = SSMQ_WEYL;
    q.format = SSMQ_BF16;
    q.dither_block = 24; /* not a power of two */
    ssmq_dims dims = {1, 4, 64, 128, 2, 0};
    ssmq_status st = ssmq_state_update(&dims, &q, (void *)0x10000, NULL, (const float *)0x10000,
                                       (const float *)0x10000, (const float *)0x10000,
                                       (const float *)0x10000, (const float *)0x10000, NULL,
                                       (float *)0x10000, NULL);
    if (st != SSMQ_EINVAL || ssmq_last_error()[0] == '\0') {
        fprintf(stderr, "expected SSMQ_EINVAL with a message, got %d\n", (int)st);
        return 1;
    }
    printf("c_abi_step: ok\n");
    return 0;
}
