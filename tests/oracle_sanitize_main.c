/*
 * Driver that runs every oracle function on small random and edge-case
 * inputs; built with the address and undefined-behaviour sanitizers by
 * tests/test_oracle_sanitize.py (so any out-of-bounds access, leak or
 * undefined operation in the oracle aborts the run).  Exit 0 when all calls
 * return as expected.  Argument: the oracle's thread count (default 1).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"

static uint64_t st = 0x9E3779B97F4A7C15ull;
static uint64_t rnd(void)
{
    st ^= st << 13;
    st ^= st >> 7;
    st ^= st << 17;
    return st;
}
static float rval(void) { return (float)((int64_t)(rnd() % 2001) - 1000) / 37.0f; }

/* a sorted random subset of [0, N) of size about k */
static uint64_t subset(uint32_t* out, uint64_t N, uint64_t k)
{
    uint64_t n = 0;
    for (uint64_t i = 0; i < N && n < k; ++i)
        if (rnd() % (N - i) < k - n) out[n++] = (uint32_t)i;
    return n;
}

#define CHECK(x)                                                        \
    do {                                                                \
        if (!(x)) {                                                     \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #x); \
            return 1;                                                   \
        }                                                               \
    } while (0)

int main(int argc, char** argv)
{
    /* optional argument: the oracle's thread count for every call */
    if (argc > 1) orc_set_threads(atoi(argv[1]));
    for (int it = 0; it < 200; ++it) {
        const int P = 1 + (int)(rnd() % 19);
        const uint64_t N = 1 + rnd() % 300;
        uint32_t* idx[19];
        float* val[19];
        uint64_t nnz[19], tot = 0;
        for (int r = 0; r < P; ++r) {
            idx[r] = malloc(sizeof(uint32_t) * N);
            val[r] = malloc(sizeof(float) * N);
            nnz[r] = subset(idx[r], N, rnd() % (N + 1));
            for (uint64_t i = 0; i < nnz[r]; ++i) val[r][i] = rval();
            tot += nnz[r];
        }
        const double deltas[4] = {1e-9, 0.05, 0.5, 4.0};
        const double delta = deltas[rnd() % 4];
        uint64_t cap = tot < N ? tot : N;
        uint32_t* oi = malloc(sizeof(uint32_t) * (cap ? cap : 1));
        float* ov = malloc(sizeof(float) * N);
        uint64_t onnz = 0, nn[32];
        int dense = 0;
        uint8_t nd[32];
        CHECK(orc_sparse_reduce(P, (const uint32_t* const*)idx, (const float* const*)val, nnz, N, delta, oi, cap,
                                ov, &onnz, &dense, P > 1 ? nn : NULL, P > 1 ? nd : NULL) == 0);
        CHECK(dense ? onnz == N : onnz <= cap);

        /* quantization, per stream and in buckets, and its inverse */
        const int bits = 2 << (rnd() % 3);
        uint8_t* q[19];
        float* dq[19];
        float scales[19 * 300];
        for (int r = 0; r < P; ++r) {
            q[r] = malloc(nnz[r] + 1);
            dq[r] = malloc(sizeof(float) * (nnz[r] + 1));
        }
        CHECK(orc_quantize(P, (const float* const*)val, nnz, bits, rnd(), q, scales, dq) == 0);
        CHECK(orc_dequantize(q[0], scales[0], bits, nnz[0], dq[0]) == 0);
        const uint64_t bucket = 1 + rnd() % 9;
        CHECK(orc_quantize_bucketed(P, (const float* const*)val, nnz, bits, bucket, rnd(), q, scales, dq) == 0);
        CHECK(orc_dequantize_bucketed(q[0], scales, bits, bucket, nnz[0], dq[0]) == 0);
        CHECK(orc_densify(idx[0], val[0], nnz[0], N, ov) == 0);

        /* top-k on the densified rows, plain and bucketed */
        float* x = malloc(sizeof(float) * P * N);
        for (uint64_t i = 0; i < (uint64_t)P * N; ++i) x[i] = (rnd() & 3) ? rval() : 0.0f;
        const uint64_t k = rnd() % (N + 1);
        uint32_t* ti = malloc(sizeof(uint32_t) * P * (k ? k : 1));
        float* tv = malloc(sizeof(float) * P * (k ? k : 1));
        float* res = malloc(sizeof(float) * P * N);
        CHECK(orc_topk(P, x, N, k, ti, tv, res) == 0);
        CHECK(orc_topk(P, x, N, k, ti, tv, x) == 0); /* residual aliasing the input */
        const uint64_t B = 64, kb = 1 + rnd() % 8;
        const uint64_t nb = (N + B - 1) / B;
        const uint64_t last = N - (nb - 1) * B;
        const uint64_t K = (nb - 1) * kb + (kb < last ? kb : last);
        uint32_t* bi = malloc(sizeof(uint32_t) * P * K);
        float* bv = malloc(sizeof(float) * P * K);
        CHECK(orc_topk_bucketed(P, res, x, N, 0.5f, B, kb, bi, bv) == 0);
        CHECK(orc_topk_bucketed(P, NULL, x, N, 0.5f, B, kb, bi, bv) == 0);

        free(bi);
        free(bv);
        free(res);
        free(ti);
        free(tv);
        free(x);
        for (int r = 0; r < P; ++r) {
            free(q[r]);
            free(dq[r]);
            free(idx[r]);
            free(val[r]);
        }
        free(oi);
        free(ov);
    }
    /* invalid input is refused without touching memory it should not */
    uint32_t bad[3] = {5, 3, 9};
    float bv3[3] = {1, 2, 3};
    const uint32_t* bi1[1] = {bad};
    const float* bv1[1] = {bv3};
    uint64_t n3 = 3, onnz;
    uint32_t oi3[3];
    float ov3[10];
    int dense;
    CHECK(orc_sparse_reduce(1, bi1, bv1, &n3, 10, 0.5, oi3, 3, ov3, &onnz, &dense, NULL, NULL) != 0);
    uint32_t ctr[4] = {1, 2, 3, 4}, key[2] = {5, 6}, out[4];
    orc_philox4x32_10(ctr, key, out);
    printf("oracle sanitizer run: ok\n");
    return 0;
}
