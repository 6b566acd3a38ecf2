/*
 * Address/undefined-behaviour sanitizer run of the C oracle (test
 * infrastructure).  Built with -fsanitize=address,undefined together with
 * oracle/pdec_oracle.c by tests/test_sanitizers.py; every entry point runs on
 * small inputs covering its branches (ended streams, full caches, both
 * element types, the plan mask, ragged batches, whole branches with and
 * without cross-stream visibility, the rotary append), and a few results are
 * checked against facts that hold at any size.  Exit status 0: no error.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_REAL double
#define ORACLE_SUFFIX f64
#include "../../oracle/pdec_oracle.c"

static uint32_t rng_state = 12345u;
static float frand(void)
{
    rng_state = rng_state * 1664525u + 1013904223u;
    return (float)((rng_state >> 8) & 0xffff) / 65536.0f - 0.5f;
}
static void fill_f32(float* x, size_t n) { for (size_t i = 0; i < n; ++i) x[i] = frand(); }
static void fill_bf16(uint16_t* x, size_t n)
{
    for (size_t i = 0; i < n; ++i) {
        float f = frand();
        uint32_t u;
        memcpy(&u, &f, 4);
        x[i] = (uint16_t)(u >> 16);
    }
}

#define CHECK(c)                                                   \
    do {                                                           \
        if (!(c)) {                                                \
            fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            return 1;                                              \
        }                                                          \
    } while (0)

static int step_case(int dtype, int plan_mask, int plan_T)
{
    enum { L = 9, E = 3, HQ = 4, HKV = 2, D = 8, CAP = 5 };
    const size_t es = dtype == 0 ? 4 : 2;
    void* q = malloc((size_t)E * HQ * D * es);
    void* kp = malloc((size_t)L * HKV * D * es);
    void* vp = malloc((size_t)L * HKV * D * es);
    void* ke = malloc((size_t)E * CAP * HKV * D * es);
    void* ve = malloc((size_t)E * CAP * HKV * D * es);
    if (dtype == 0) {
        fill_f32(q, (size_t)E * HQ * D); fill_f32(kp, (size_t)L * HKV * D); fill_f32(vp, (size_t)L * HKV * D);
        fill_f32(ke, (size_t)E * CAP * HKV * D); fill_f32(ve, (size_t)E * CAP * HKV * D);
    } else {
        fill_bf16(q, (size_t)E * HQ * D); fill_bf16(kp, (size_t)L * HKV * D); fill_bf16(vp, (size_t)L * HKV * D);
        fill_bf16(ke, (size_t)E * CAP * HKV * D); fill_bf16(ve, (size_t)E * CAP * HKV * D);
    }
    const int32_t n[E] = {2, 0, CAP};
    const int32_t cu_p[2] = {0, L}, cu_e[2] = {0, E};
    const long U = L + (long)E * CAP;
    double* out = malloc(sizeof(double) * E * HQ * D);
    double* lse = malloc(sizeof(double) * E * HQ);
    double* probs = malloc(sizeof(double) * E * HQ * U);
    uint8_t sel[E * HQ];
    for (int i = 0; i < E * HQ; ++i) sel[i] = 1;
    int rc = oracle_attn_step_f64(1, cu_p, cu_e, HQ, HKV, D, CAP, 0.0, dtype, plan_mask, plan_T, q, kp, vp, ke, ve,
                                  n, sel, out, lse, probs, 2);
    CHECK(rc == 0);
    for (int h = 0; h < HQ; ++h) {
        CHECK(isinf(lse[1 * HQ + h]) && lse[1 * HQ + h] < 0);  /* ended stream */
        double s = 0;
        for (long j = 0; j < U; ++j) s += probs[(0 * HQ + h) * U + j];
        CHECK(fabs(s - 1.0) < 1e-12);                           /* weights of a live row sum to 1 */
        for (int f = 0; f < E; ++f)                             /* other streams' rows stay hidden */
            if (f != 0)
                for (int t = 0; t < CAP; ++t) CHECK(probs[(0 * HQ + h) * U + L + f * CAP + t] == 0.0);
    }
    free(q); free(kp); free(vp); free(ke); free(ve); free(out); free(lse); free(probs);
    return 0;
}

static int ragged_case(void)
{
    enum { V = 2, HQ = 2, HKV = 1, D = 4, CAP = 3 };
    const int32_t cu_p[V + 1] = {0, 4, 4}, cu_e[V + 1] = {0, 2, 5};  /* second video: empty prefix */
    const int32_t n[5] = {1, 3, 0, 2, 1};
    float q[5 * HQ * D], kp[4 * HKV * D], vp[4 * HKV * D], ke[5 * CAP * HKV * D], ve[5 * CAP * HKV * D];
    fill_f32(q, sizeof(q) / 4); fill_f32(kp, sizeof(kp) / 4); fill_f32(vp, sizeof(vp) / 4);
    fill_f32(ke, sizeof(ke) / 4); fill_f32(ve, sizeof(ve) / 4);
    double out[5 * HQ * D], lse[5 * HQ];
    CHECK(oracle_attn_step_f64(V, cu_p, cu_e, HQ, HKV, D, CAP, 0.5, 0, 0, 0, q, kp, vp, ke, ve, n, NULL, out, lse,
                               NULL, 1) == 0);
    CHECK(isinf(lse[2 * HQ]) && lse[2 * HQ] < 0);
    /* inconsistent arguments are refused, not read out of bounds */
    const int32_t bad_n[5] = {1, 4, 0, 2, 1};
    CHECK(oracle_attn_step_f64(V, cu_p, cu_e, HQ, HKV, D, CAP, 0.5, 0, 0, 0, q, kp, vp, ke, ve, bad_n, NULL, out,
                               lse, NULL, 1) == -1);
    return 0;
}

static int mask_case(void)
{
    enum { L = 6, E = 3, CAP = 4 };
    const int32_t n[E] = {2, 0, 4};
    uint8_t m[E * (L + E * CAP)];
    CHECK(oracle_build_mask_f64(L, E, CAP, n, 0, 0, m) == 0);
    CHECK(oracle_build_mask_f64(L, E, CAP, n, 1, 2, m) == 0);
    CHECK(oracle_build_mask_f64(L, E, CAP, n, 1, 5, m) == -1); /* plan segment longer than the prefix */
    return 0;
}

static int loop_case(void)
{
    enum { S = 7, E = 3, HQ = 2, HKV = 1, D = 4, CAP = 6, L = 5 };
    float kp[L * HKV * D], vp[L * HKV * D], q[S * E * HQ * D], kn[S * E * HKV * D], vn[S * E * HKV * D];
    fill_f32(kp, sizeof(kp) / 4); fill_f32(vp, sizeof(vp) / 4); fill_f32(q, sizeof(q) / 4);
    fill_f32(kn, sizeof(kn) / 4); fill_f32(vn, sizeof(vn) / 4);
    const int32_t eos[E] = {2, 6, 0};
    double out[S * E * HQ * D], lse[S * E * HQ];
    CHECK(oracle_decode_loop_f64(S - 1, E, HQ, HKV, D, CAP, L, 0.0, 0, kp, vp, q, kn, vn, eos, out, lse, 1) == 0);
    CHECK(isinf(lse[(3 * E + 0) * HQ]));  /* stream 0 past its EOS step */
    const int32_t long_eos[E] = {7, 1, 1};  /* more live steps than the cache holds: refused */
    CHECK(oracle_decode_loop_f64(S, E, HQ, HKV, D, CAP, L, 0.0, 0, kp, vp, q, kn, vn, long_eos, out, lse, 1) == -1);
    return 0;
}

static int prefill_case(int cross)
{
    enum { HQ = 2, HKV = 1, D = 4, CAP = 4, N = 3 };
    const int32_t cu_p[2] = {0, 5}, cu_e[2] = {0, 2};
    const int32_t n[2] = {3, 2};
    uint16_t q[2 * N * HQ * D], kp[5 * HKV * D], vp[5 * HKV * D], ke[2 * CAP * HKV * D], ve[2 * CAP * HKV * D];
    fill_bf16(q, sizeof(q) / 2); fill_bf16(kp, sizeof(kp) / 2); fill_bf16(vp, sizeof(vp) / 2);
    fill_bf16(ke, sizeof(ke) / 2); fill_bf16(ve, sizeof(ve) / 2);
    double out[2 * N * HQ * D], lse[2 * N * HQ];
    CHECK(oracle_attn_prefill_f64(1, cu_p, cu_e, N, cross, HQ, HKV, D, CAP, 0.0, 1, q, kp, vp, ke, ve, n, out, lse,
                                  1) == 0);
    return 0;
}

static int rope_case(void)
{
    enum { V = 1, HQ = 2, HKV = 1, D = 8, CAP = 3, E = 3 };
    const int32_t cu_e[2] = {0, E}, pos[1] = {100};
    const int32_t lens[E] = {0, CAP, 1}, live[E] = {1, 1, 0};
    float q[E * HQ * D], kn[E * HKV * D];
    fill_f32(q, sizeof(q) / 4); fill_f32(kn, sizeof(kn) / 4);
    double qr[E * HQ * D], kr[E * HKV * D];
    int32_t nl[E];
    CHECK(oracle_rope_append_f64(V, cu_e, pos, HQ, HKV, D, CAP, 10000.0, 0, q, kn, lens, live, qr, kr, nl) == 0);
    CHECK(nl[0] == 1 && nl[1] == CAP && nl[2] == 0);
    /* a rotation keeps each (i, i + D/2) pair's length */
    for (int i = 0; i < D / 2; ++i) {
        const double a = (double)q[i] * q[i] + (double)q[i + D / 2] * q[i + D / 2];
        const double b = qr[i] * qr[i] + qr[i + D / 2] * qr[i + D / 2];
        CHECK(fabs(a - b) < 1e-9);
    }
    return 0;
}

int main(void)
{
    for (int dtype = 0; dtype < 2; ++dtype) {
        if (step_case(dtype, 0, 0)) return 1;
        if (step_case(dtype, 1, 2)) return 1;
    }
    if (ragged_case() || mask_case() || loop_case() || prefill_case(0) || prefill_case(1) || rope_case()) return 1;
    printf("oracle sanitizer driver: ok\n");
    return 0;
}
