/*
 * STaR-Quant W4A4 hot path: CPU ORACLE.  Test infrastructure only.
 *
 * This file is the plain, slow reference that the HIP library is checked
 * against.  Only the test suite, the smoke check and the benchmark's CPU
 * baseline may load it; the product path never does.  It shares no code,
 * header, table or constant with the HIP library.
 *
 * Built with gcc -O2 -fno-fast-math -ffp-contract=off (IEEE binary32, no
 * contraction other than the explicit fmaf calls, no flush-to-zero).
 *
 * What it computes (paper sections cited per function):
 *   - symmetric uniform quantiser (Sec. 3.1, Eq. 2-3 with z = 0) at 4 bits,
 *     per token for activations and per output channel for weights (Eq. 5);
 *   - the SGAT state-conditioned transform x P G_s (Sec. 3.2, Eq. 8-11) and
 *     the shared static weight transform W~ = Q_w(P^T W^T) (Eq. 12);
 *   - the state-guided projection Q_a(Phi_s(X)) W~ (Eq. 13);
 *   - TAC, Z_b M_b^T + 1 d_b^T per block of g channels (Eq. 17, App. C).
 *
 * Readings of points the paper leaves open (each one is a stated choice):
 *   Q1 symmetric quantiser, s = absmax / 7 (fp32, correctly rounded divide),
 *      codes clamp(rint(fl(x / s)), -8, 7), ties to even on the fp32 quotient;
 *   Q4 a row whose scale is 0 gets all-zero codes;
 *   T3 the transform is fp32: split k into chunks of 256, accumulate each
 *      chunk with fmaf in ascending k from +0, add the chunk sums in ascending
 *      order to a +0 total;
 *   T4 columns of P are ordered [shared | masked band | unmasked band] with
 *      band widths d_m, d_u; gated columns are exactly +0;
 *   R2 TAC: fp32 fmaf over c ascending from +0, bias added last, result
 *      rounded to fp16 (round to nearest even);
 *   G1 GEMM: int32 sum of code products, y = fp16((float(acc) * s_a) * s_w);
 *   packing: byte t = (q[2t] & 15) | (q[2t+1] & 15) << 4.
 *   W8A8 (App. D): the same method with 8-bit codes, s = absmax / 127, codes
 *      clamp(rint(x / s), -128, 127), one signed byte per code.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define SQO_CHUNK 256

/* ------------------------------------------------------------------ fp16 */
/* IEEE 754 binary16 -> binary32: exact. */
float sqo_h2f(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 31;
    int m = h & 1023;
    float v;
    if (e == 0)
        v = ldexpf((float)m, -24);                 /* zero or subnormal */
    else if (e == 31)
        v = m ? NAN : INFINITY;
    else
        v = ldexpf((float)(1024 + m), e - 25);     /* (1 + m/1024) * 2^(e-15) */
    return sign ? -v : v;
}

/* IEEE 754 binary32 -> binary16, round to nearest, ties to even. */
uint16_t sqo_f2h(float f)
{
    uint16_t sign = signbit(f) ? 0x8000 : 0;
    float a = fabsf(f);
    if (isnan(f))
        return 0x7E00;
    if (a >= 65520.0f)                             /* halfway to 2^16 rounds up */
        return sign | 0x7C00;
    if (a < 0x1p-14f) {                            /* subnormal range, step 2^-24 */
        float n = rintf(a * 0x1p24f);              /* exact scaling, then RNE */
        return sign | (uint16_t)n;                 /* n == 1024 is the min normal */
    }
    int e;
    frexpf(a, &e);                                 /* a = fr * 2^e, fr in [0.5, 1) */
    e -= 1;                                        /* a in [2^e, 2^(e+1)) */
    float n = rintf(ldexpf(a, 10 - e));            /* in [1024, 2048] */
    if (n == 2048.0f) {
        n = 1024.0f;
        e += 1;
    }
    if (e > 15)
        return sign | 0x7C00;
    return sign | (uint16_t)(((e + 15) << 10) | ((int)n - 1024));
}

void sqo_h2f_array(const uint16_t* h, float* f, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) f[i] = sqo_h2f(h[i]);
}

void sqo_f2h_array(const float* f, uint16_t* h, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) h[i] = sqo_f2h(f[i]);
}

/* ------------------------------------------------------------------ TAC */
/* Eq. 17 in the row-major form of App. C: for token i, block b, row r,
 *   z'[i][b*g + r] = fp16( sum_c M_b[r][c] * z[i][b*g + c] + d[b*g + r] ). */
void sqo_tac(const uint16_t* Z, const uint16_t* Mb, const uint16_t* d,
             int64_t M, int C, int g, uint16_t* out)
{
    for (int64_t i = 0; i < M; ++i) {
        const uint16_t* z = Z + i * C;
        for (int b = 0; b < C / g; ++b) {
            for (int r = 0; r < g; ++r) {
                const uint16_t* mrow = Mb + ((int64_t)b * g + r) * g;
                float t = 0.0f;
                for (int c = 0; c < g; ++c)
                    t = fmaf(sqo_h2f(mrow[c]), sqo_h2f(z[b * g + c]), t);
                out[i * C + b * g + r] = sqo_f2h(t + sqo_h2f(d[b * g + r]));
            }
        }
    }
}

/* --------------------------------------------------------------- SGAT */
/* Gate G_s (Eq. 9): column j of the transformed row is kept for state s iff
 * it lies in the shared block or in s's own band. */
static int sqo_kept(int j, int K, int dm, int du, int masked)
{
    int m_lo = K - dm - du, u_lo = K - du;
    if (j < m_lo) return 1;                 /* shared */
    if (j < u_lo) return masked;            /* masked-specific band */
    return !masked;                         /* unmasked-specific band */
}

/* x'[i] = x_i P G_{s_i} (Eq. 11) for rows [0, M).  P == NULL means the input
 * already lies in the P basis (x' = x before gating).  state == NULL means
 * no gate (used for the weight side, Eq. 12).  Output fp32 [M][K]. */
void sqo_transform(const uint16_t* X, const uint8_t* state, const float* P,
                   int64_t M, int K, int dm, int du, float* xp)
{
    float* xin = (float*)malloc(sizeof(float) * K);
    float* acc = (float*)malloc(sizeof(float) * K);
    float* tot = (float*)malloc(sizeof(float) * K);
    for (int64_t i = 0; i < M; ++i) {
        for (int k = 0; k < K; ++k) xin[k] = sqo_h2f(X[i * K + k]);
        if (P) {
            /* Each output j follows its own fixed sequence; the loops are only
             * interleaved across different j. */
            for (int j = 0; j < K; ++j) tot[j] = 0.0f;
            for (int c0 = 0; c0 < K; c0 += SQO_CHUNK) {
                int c1 = c0 + SQO_CHUNK < K ? c0 + SQO_CHUNK : K;
                for (int j = 0; j < K; ++j) acc[j] = 0.0f;
                for (int k = c0; k < c1; ++k) {
                    const float* prow = P + (int64_t)k * K;
                    for (int j = 0; j < K; ++j) acc[j] = fmaf(xin[k], prow[j], acc[j]);
                }
                for (int j = 0; j < K; ++j) tot[j] = tot[j] + acc[j];
            }
        } else {
            memcpy(tot, xin, sizeof(float) * K);
        }
        for (int j = 0; j < K; ++j) {
            int keep = state ? sqo_kept(j, K, dm, du, state[i] != 0) : 1;
            xp[i * K + j] = keep ? tot[j] : 0.0f;
        }
    }
    free(xin);
    free(acc);
    free(tot);
}

/* --------------------------------------------------------- quantiser */
/* Symmetric 4-bit quantisation of each row of x [M][K] (Eq. 2 with z = 0):
 * s = absmax/7; q = clamp(rint(x/s), -8, 7); two codes per byte. */
void sqo_quant_rows(const float* x, int64_t M, int K, uint8_t* packed, float* scale, int8_t* codes)
{
    for (int64_t i = 0; i < M; ++i) {
        const float* row = x + i * K;
        float a = 0.0f;
        for (int j = 0; j < K; ++j)
            if (fabsf(row[j]) > a) a = fabsf(row[j]);
        float s = a / 7.0f;
        scale[i] = s;
        for (int j = 0; j < K; j += 2) {
            int q[2];
            for (int h = 0; h < 2; ++h) {
                int v = 0;
                if (s != 0.0f) {
                    float r = rintf(row[j + h] / s);
                    v = r < -8.0f ? -8 : (r > 7.0f ? 7 : (int)r);
                }
                q[h] = v;
                if (codes) codes[i * K + j + h] = (int8_t)v;
            }
            packed[i * (K / 2) + j / 2] = (uint8_t)((q[0] & 15) | ((q[1] & 15) << 4));
        }
    }
}

/* Symmetric 8-bit quantisation of each row (W8A8, App. D): s = absmax/127;
 * q = clamp(rint(x/s), -128, 127), one signed byte per code. */
void sqo_quant_rows_q8(const float* x, int64_t M, int K, int8_t* codes, float* scale)
{
    for (int64_t i = 0; i < M; ++i) {
        const float* row = x + i * K;
        float a = 0.0f;
        for (int j = 0; j < K; ++j)
            if (fabsf(row[j]) > a) a = fabsf(row[j]);
        float s = a / 127.0f;
        scale[i] = s;
        for (int j = 0; j < K; ++j) {
            int v = 0;
            if (s != 0.0f) {
                float r = rintf(row[j] / s);
                v = r < -128.0f ? -128 : (r > 127.0f ? 127 : (int)r);
            }
            codes[i * K + j] = (int8_t)v;
        }
    }
}

/* Two's-complement nibble -> code. */
static int sqo_nib(uint8_t byte, int hi)
{
    int v = hi ? (byte >> 4) : (byte & 15);
    return v >= 8 ? v - 16 : v;
}

void sqo_unpack(const uint8_t* packed, int64_t M, int K, int8_t* codes)
{
    for (int64_t i = 0; i < M; ++i)
        for (int j = 0; j < K; ++j)
            codes[i * K + j] = (int8_t)sqo_nib(packed[i * (K / 2) + j / 2], j & 1);
}

/* ------------------------------------------------------ composition */
/* Activation side of one SGAT linear (Eq. 11 then Q_a), with optional TAC on
 * the raw input first (TAC sits ahead of the O-projection, App. C).
 * Codes [M][K/2] and per-token scales [M]. */
void sqo_quant_act(const uint16_t* X, const uint8_t* state, const float* P,
                   int64_t M, int K, int dm, int du,
                   const uint16_t* tacM, const uint16_t* tacd, int g,
                   uint8_t* Aq, float* s_a)
{
    const uint16_t* src = X;
    uint16_t* z = NULL;
    if (tacM) {
        z = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)(M * K));
        sqo_tac(X, tacM, tacd, M, K, g, z);
        src = z;
    }
    float* xp = (float*)malloc(sizeof(float) * (size_t)(M * K));
    sqo_transform(src, state, P, M, K, dm, du, xp);
    sqo_quant_rows(xp, M, K, Aq, s_a, NULL);
    free(xp);
    free(z);
}

/* Weight side (Eq. 12): W' = rows of W times P, no gate; then per-output-
 * channel quantisation. */
void sqo_prepare_weights(const uint16_t* W, const float* P, int64_t N, int K,
                         uint8_t* Wq, float* s_w)
{
    float* wp = (float*)malloc(sizeof(float) * (size_t)(N * K));
    sqo_transform(W, NULL, P, N, K, 0, 0, wp);
    sqo_quant_rows(wp, N, K, Wq, s_w, NULL);
    free(wp);
}

/* W8A8 activation side: [TAC] -> x P G_s -> 8-bit per-token codes. */
void sqo_quant_act_q8(const uint16_t* X, const uint8_t* state, const float* P,
                      int64_t M, int K, int dm, int du,
                      const uint16_t* tacM, const uint16_t* tacd, int g,
                      int8_t* Aq, float* s_a)
{
    const uint16_t* src = X;
    uint16_t* z = NULL;
    if (tacM) {
        z = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)(M * K));
        sqo_tac(X, tacM, tacd, M, K, g, z);
        src = z;
    }
    float* xp = (float*)malloc(sizeof(float) * (size_t)(M * K));
    sqo_transform(src, state, P, M, K, dm, du, xp);
    sqo_quant_rows_q8(xp, M, K, Aq, s_a);
    free(xp);
    free(z);
}

/* W8A8 weight side: rows of W P, per-output-channel 8-bit codes. */
void sqo_prepare_weights_q8(const uint16_t* W, const float* P, int64_t N, int K, int8_t* Wq, float* s_w)
{
    float* wp = (float*)malloc(sizeof(float) * (size_t)(N * K));
    sqo_transform(W, NULL, P, N, K, 0, 0, wp);
    sqo_quant_rows_q8(wp, N, K, Wq, s_w);
    free(wp);
}

/* W8A8 projection: acc = sum_j qa[i][j] qw[n][j] (int32), y as in sqo_gemm.
 * Returns 1 if an accumulator left the int32 range. */
int sqo_gemm_q8(const int8_t* Aq, const float* s_a, const int8_t* Wq, const float* s_w,
                int64_t M, int64_t N, int K, uint16_t* Y, int32_t* acc_out)
{
    int bad = 0;
    for (int64_t i = 0; i < M; ++i) {
        const int8_t* a = Aq + i * K;
        for (int64_t n = 0; n < N; ++n) {
            const int8_t* w = Wq + n * K;
            int64_t acc = 0;
            for (int j = 0; j < K; ++j) acc += (int64_t)a[j] * w[j];
            if (acc > INT32_MAX || acc < INT32_MIN) bad = 1;
            if (acc_out) acc_out[i * N + n] = (int32_t)acc;
            if (Y) Y[i * N + n] = sqo_f2h(((float)acc * s_a[i]) * s_w[n]);
        }
    }
    return bad;
}

/* Quantised projection (Eq. 5 / Eq. 13): acc = sum_j qa[i][j] qw[n][j];
 * y = fp16((float(acc) * s_a[i]) * s_w[n]).  Returns 0, or 1 if an
 * accumulator left the int32 range. */
int sqo_gemm(const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w,
             int64_t M, int64_t N, int K, uint16_t* Y, int32_t* acc_out)
{
    int8_t* qa = (int8_t*)malloc((size_t)K);
    int8_t* qw = (int8_t*)malloc((size_t)(N * K));
    int bad = 0;
    sqo_unpack(Wq, N, K, qw);
    for (int64_t i = 0; i < M; ++i) {
        sqo_unpack(Aq + i * (K / 2), 1, K, qa);
        for (int64_t n = 0; n < N; ++n) {
            const int8_t* w = qw + n * K;
            int64_t acc = 0;
            for (int j = 0; j < K; ++j) acc += (int64_t)qa[j] * w[j];
            if (acc > INT32_MAX || acc < INT32_MIN) bad = 1;
            if (acc_out) acc_out[i * N + n] = (int32_t)acc;
            if (Y) Y[i * N + n] = sqo_f2h(((float)acc * s_a[i]) * s_w[n]);
        }
    }
    free(qa);
    free(qw);
    return bad;
}
