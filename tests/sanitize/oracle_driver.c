/*
 * Drives every entry point of the CPU oracle (oracle/sq_oracle.c) on small
 * seeded inputs, for a build with AddressSanitizer and UndefinedBehaviorSanitizer
 * (tests/test_oracle_sanitize.py).  Exits 0 and prints "ok" when nothing was
 * reported; a sanitizer finding aborts the run.  Shapes include a k range that
 * ends in a partial chunk of 256, band widths of zero, an all-zero row, every
 * fp16 bit pattern, and TAC block sizes 1 ... 128.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

float sqo_h2f(uint16_t h);
uint16_t sqo_f2h(float f);
void sqo_h2f_array(const uint16_t* h, float* f, int64_t n);
void sqo_f2h_array(const float* f, uint16_t* h, int64_t n);
void sqo_tac(const uint16_t* Z, const uint16_t* Mb, const uint16_t* d, int64_t M, int C, int g, uint16_t* out);
void sqo_transform(const uint16_t* X, const uint8_t* state, const float* P, int64_t M, int K, int dm, int du,
                   float* xp);
void sqo_quant_rows(const float* x, int64_t M, int K, uint8_t* packed, float* scale, int8_t* codes);
void sqo_quant_rows_q8(const float* x, int64_t M, int K, int8_t* codes, float* scale);
void sqo_unpack(const uint8_t* packed, int64_t M, int K, int8_t* codes);
void sqo_quant_act(const uint16_t* X, const uint8_t* state, const float* P, int64_t M, int K, int dm, int du,
                   const uint16_t* tacM, const uint16_t* tacd, int g, uint8_t* Aq, float* s_a);
void sqo_prepare_weights(const uint16_t* W, const float* P, int64_t N, int K, uint8_t* Wq, float* s_w);
void sqo_quant_act_q8(const uint16_t* X, const uint8_t* state, const float* P, int64_t M, int K, int dm, int du,
                      const uint16_t* tacM, const uint16_t* tacd, int g, int8_t* Aq, float* s_a);
void sqo_prepare_weights_q8(const uint16_t* W, const float* P, int64_t N, int K, int8_t* Wq, float* s_w);
int sqo_gemm_q8(const int8_t* Aq, const float* s_a, const int8_t* Wq, const float* s_w, int64_t M, int64_t N, int K,
                uint16_t* Y, int32_t* acc_out);
int sqo_gemm(const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w, int64_t M, int64_t N, int K,
             uint16_t* Y, int32_t* acc_out);

static uint64_t rng = 0x9e3779b97f4a7c15ull;
static double unif(void) {   /* xorshift64*, uniform in [0, 1) */
    rng ^= rng >> 12;
    rng ^= rng << 25;
    rng ^= rng >> 27;
    return (double)((rng * 2685821657736338717ull) >> 11) * (1.0 / 9007199254740992.0);
}
static double gauss(void) { return sqrt(-2.0 * log(1.0 - unif())) * cos(6.283185307179586 * unif()); }

static void* xmalloc(size_t n) {
    void* p = malloc(n ? n : 1);
    if (!p) { fprintf(stderr, "out of memory\n"); exit(2); }
    return p;
}

static void run_case(int64_t M, int K, int64_t N, int dm, int du, int g) {
    uint16_t* X = xmalloc(sizeof(uint16_t) * M * K);
    uint16_t* W = xmalloc(sizeof(uint16_t) * N * K);
    float* P = xmalloc(sizeof(float) * K * K);
    uint8_t* st = xmalloc((size_t)M);
    uint16_t* tM = xmalloc(sizeof(uint16_t) * (size_t)K * g);
    uint16_t* td = xmalloc(sizeof(uint16_t) * (size_t)K);
    for (int64_t i = 0; i < M * K; ++i) X[i] = sqo_f2h((float)(gauss() * (i % 17 == 0 ? 16.0 : 1.0)));
    for (int64_t i = 0; i < K; ++i) X[i] = 0;   /* an all-zero row */
    for (int64_t i = 0; i < N * K; ++i) W[i] = sqo_f2h((float)(0.02 * gauss()));
    for (int64_t i = 0; i < (int64_t)K * K; ++i) P[i] = (float)(gauss() / sqrt((double)K));
    for (int64_t i = 0; i < M; ++i) st[i] = unif() < 0.5;
    for (int64_t i = 0; i < (int64_t)K * g; ++i) tM[i] = sqo_f2h((float)((i % (g + 1) == 0 ? 1.0 : 0.0) + 0.01 * gauss()));
    for (int i = 0; i < K; ++i) td[i] = sqo_f2h((float)(0.01 * gauss()));

    float* xp = xmalloc(sizeof(float) * M * K);
    uint16_t* z = xmalloc(sizeof(uint16_t) * M * K);
    sqo_tac(X, tM, td, M, K, g, z);
    sqo_transform(z, st, P, M, K, dm, du, xp);
    sqo_transform(X, NULL, NULL, M, K, 0, 0, xp);

    uint8_t* packed = xmalloc((size_t)(M * K / 2));
    int8_t* codes = xmalloc((size_t)(M * K));
    float* sc = xmalloc(sizeof(float) * M);
    sqo_quant_rows(xp, M, K, packed, sc, codes);
    sqo_unpack(packed, M, K, codes);
    sqo_quant_rows_q8(xp, M, K, codes, sc);

    uint8_t* Aq = xmalloc((size_t)(M * K / 2));
    float* s_a = xmalloc(sizeof(float) * M);
    uint8_t* Wq = xmalloc((size_t)(N * K / 2));
    float* s_w = xmalloc(sizeof(float) * N);
    uint16_t* Y = xmalloc(sizeof(uint16_t) * M * N);
    int32_t* acc = xmalloc(sizeof(int32_t) * M * N);
    sqo_quant_act(X, st, P, M, K, dm, du, tM, td, g, Aq, s_a);
    sqo_quant_act(X, NULL, NULL, M, K, 0, 0, NULL, NULL, 0, Aq, s_a);
    sqo_prepare_weights(W, P, N, K, Wq, s_w);
    sqo_prepare_weights(W, NULL, N, K, Wq, s_w);
    if (sqo_gemm(Aq, s_a, Wq, s_w, M, N, K, Y, acc) != 0) { fprintf(stderr, "gemm range\n"); exit(3); }

    int8_t* Aq8 = xmalloc((size_t)(M * K));
    int8_t* Wq8 = xmalloc((size_t)(N * K));
    sqo_quant_act_q8(X, st, P, M, K, dm, du, tM, td, g, Aq8, s_a);
    sqo_prepare_weights_q8(W, P, N, K, Wq8, s_w);
    if (sqo_gemm_q8(Aq8, s_a, Wq8, s_w, M, N, K, Y, acc) != 0) { fprintf(stderr, "gemm_q8 range\n"); exit(3); }

    free(X); free(W); free(P); free(st); free(tM); free(td); free(xp); free(z); free(packed); free(codes); free(sc);
    free(Aq); free(s_a); free(Wq); free(s_w); free(Y); free(acc); free(Aq8); free(Wq8);
}

int main(void) {
    /* every fp16 bit pattern through both conversions */
    uint16_t* h = xmalloc(sizeof(uint16_t) * 65536);
    float* f = xmalloc(sizeof(float) * 65536);
    for (int i = 0; i < 65536; ++i) h[i] = (uint16_t)i;
    sqo_h2f_array(h, f, 65536);
    sqo_f2h_array(f, h, 65536);
    free(h);
    free(f);
    run_case(37, 320, 24, 10, 10, 16);     /* K ends in a partial chunk of 256 */
    run_case(5, 64, 8, 0, 0, 1);           /* no gating, g = 1 */
    run_case(9, 512, 16, 16, 16, 128);     /* the widest TAC block */
    run_case(3, 256, 8, 0, 32, 4);         /* one band empty */
    printf("ok\n");
    return 0;
}
