/*
 * starquant.h -- C ABI of the STaR-Quant W4A4 hot path for AMD MI355X (gfx950).
 *
 * STaR-Quant (arXiv 2606.04945) quantises the linear layers of a diffusion LLM
 * to 4-bit weights and 4-bit activations.  At every denoising step a quantised
 * linear layer runs:
 *   (1) the State-Guided Activation Transformation (SGAT): each token's row x is
 *       mapped to x P G_s, where P = [U_sh, U_m, U_u] is an orthogonal basis and
 *       the binary gate G_s keeps the shared columns plus the band of the token's
 *       own mask state s in {masked, unmasked} (Sec. 3.2, Eq. 8-11);
 *   (2) per-token symmetric int4 quantisation of the transformed row (Sec. 3.1,
 *       Eq. 2 and 5);
 *   (3) an int4 x int4 product with the shared, offline-quantised weight
 *       W~ = Q_w(P^T W^T) (Eq. 12-13), dequantised to fp16;
 *   (4) ahead of the attention output projection only, Temporal Attention
 *       Compensation (TAC): a block-diagonal affine map z_b -> M_b z_b + d_b on
 *       the attention output (Sec. 3.3, Eq. 17; App. C).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every tensor pointer is a DEVICE pointer owned by the caller; the library
 *    never allocates, frees or retains device memory, and keeps no state between
 *    calls other than the thread-local error message (one exception:
 *    w4a4_gemm_frag_noalloc, for callers that cannot allocate, uses a
 *    fixed-size scratch array the library holds on each GPU).
 *  - Row-major, dense.  fp16 tensors are passed as uint16_t* holding IEEE
 *    binary16 bits.  Packed int4 tensors are uint8_t* with two codes per byte:
 *    byte t of a row holds code 2t in bits 0-3 and code 2t+1 in bits 4-7, each a
 *    two's-complement nibble.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Work is enqueued on it
 *    and the call returns without synchronising.  Calls are reentrant.
 *  - Every argument is checked before anything is enqueued; on a non-zero
 *    return nothing was enqueued and no output was touched.  M == 0 (or N == 0)
 *    is a successful no-op.  sq_last_error() describes the last failure on the
 *    calling thread.
 *  - Shape rules: K % 64 == 0 and 64 <= K <= 131072; N % 8 == 0; all pointers
 *    16-byte aligned.  TAC block size g is a power of two, 1 <= g <= 128, g | C.
 *    w4a4_gemm, w8a8_gemm, tac_apply and sgat_quant_act with TAC take at most
 *    4194240 (65535 x 64) rows per call.
 *  - Debugging: with the environment variable SQ_DEBUG_SYNC set (to anything
 *    but "" or "0") when the library first checks it, every kernel launch is
 *    followed by hipDeviceSynchronize and an error check, so an asynchronous
 *    fault is returned as SQ_ERR_HIP by the call that launched the faulting
 *    kernel, named in sq_last_error().  This serialises the device and must
 *    not be used under stream capture.
 *  - Arithmetic is fixed so that results are a unique function of the inputs:
 *    fp32 IEEE throughout (correctly rounded divide, round-to-nearest-even, no
 *    flush of subnormals); the transform accumulates k in chunks of 256 with a
 *    fused multiply-add in ascending k from +0 and adds the chunk sums in
 *    ascending order; the quantiser is s = absmax / 7, q = clamp(rint(x / s),
 *    -8, 7), a zero scale giving zero codes.
 */
#ifndef STARQUANT_H
#define STARQUANT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define SQ_OK 0
#define SQ_ERR_NULL 1        /* a required pointer is NULL                     */
#define SQ_ERR_SHAPE 2       /* a size or band/block parameter breaks a rule   */
#define SQ_ERR_ALIGN 3       /* a pointer is not 16-byte aligned               */
#define SQ_ERR_WORKSPACE 4   /* workspace missing or smaller than required     */
#define SQ_ERR_HIP 5         /* the HIP runtime reported an error at launch    */

/* Message for the last non-zero return on the calling thread ("" if none). */
const char* sq_last_error(void);

/* Library version string. */
const char* sq_version(void);

/* TAC default block size (App. C): 16, or the largest g <= 16 dividing C;
 * 0 if C <= 0. */
int32_t sq_tac_default_block(int32_t C);

/* Device workspace, in bytes, that sgat_quant_act needs for these arguments
 * (has_P, has_tac: 0 or 1).  0 means ws may be NULL. */
size_t sq_quant_act_workspace_bytes(int32_t M, int32_t K, int32_t has_P, int32_t has_tac);

/* Device workspace, in bytes, that sgat_prepare_weights needs. */
size_t sq_prepare_weights_workspace_bytes(int32_t N, int32_t K, int32_t has_P);

/* Device workspace, in bytes, that w4a4_gemm needs for this shape (split-K
 * partial sums when few output tiles meet a long K); 0 means ws may be NULL. */
size_t sq_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K);

/* The same for w8a8_gemm. */
size_t sq_gemm_w8_workspace_bytes(int32_t M, int32_t N, int32_t K);

/*
 * sgat_prepare_weights -- offline weight side of SGAT (Eq. 12; App. A, App. B).
 * W~ = Q_w(P^T W^T) is stored transposed, as the rows of W P: for output channel
 * n, w'_n = W[n, :] P (no gate), then per-output-channel symmetric int4:
 * s_w[n] = max_j |w'_nj| / 7, codes clamp(rint(w'_nj / s_w[n]), -8, 7).
 *   W    [N][K] fp16, row n = output channel n's input weights.
 *   P    [K][K] fp32, P[k][j]; NULL = identity (W is already in the P basis).
 *   Wq   out [N][K/2] packed int4.     s_w  out [N] fp32.
 *   ws   device workspace of at least sq_prepare_weights_workspace_bytes().
 */
int sgat_prepare_weights(const uint16_t* W, const float* P, int32_t N, int32_t K,
                         uint8_t* Wq, float* s_w, void* ws, size_t ws_bytes, void* stream);

/*
 * sgat_transform -- the SGAT activation transform alone (Eq. 11): x'_i = x_i P G_{s_i}.
 * Columns of P are ordered [shared | masked band (d_m) | unmasked band (d_u)]
 * (Eq. 8); a masked token's unmasked band and an unmasked token's masked band
 * are exactly +0 (Eq. 9-10).
 *   X      [M][K] fp16 tokens.        state [M] uint8, 0 = unmasked, else masked;
 *                                     NULL = no gate (every column kept).
 *   P      [K][K] fp32, or NULL (X already in the P basis: x' = x, then gated).
 *   d_m, d_u  band widths, d_m, d_u >= 0, d_m + d_u < K (default K/32 each).
 *   Xp     out [M][K] fp32.
 */
int sgat_transform(const uint16_t* X, const uint8_t* state, const float* P,
                   int32_t M, int32_t K, int32_t d_m, int32_t d_u, float* Xp, void* stream);

/*
 * sgat_quantize -- per-row symmetric int4 quantisation of fp32 rows (Sec. 3.1,
 * Eq. 2 with zero point 0; per token for activations, Eq. 5):
 * s[i] = max_j |X[i][j]| / 7 and codes clamp(rint(X[i][j] / s[i]), -8, 7), all
 * codes 0 when s[i] == 0.  Used on the output of sgat_transform.
 *   Xp  [M][K] fp32.   Aq out [M][K/2] packed int4.   s out [M] fp32.
 */
int sgat_quantize(const float* Xp, int32_t M, int32_t K, uint8_t* Aq, float* s, void* stream);

/*
 * sgat_quant_act -- activation side of one SGAT linear, per denoising step:
 * [TAC] -> x P G_s (Eq. 11) -> per-token symmetric int4 (Eq. 2, 5).
 *   X      [M][K] fp16 tokens (for the O-projection: the attention output Z).
 *   state  [M] uint8, 0 = unmasked, else masked; NULL = no gate.
 *   P      [K][K] fp32 or NULL (X already in the P basis).
 *   d_m, d_u  band widths as in sgat_transform.
 *   tac_M  [K/g][g][g] fp16, tac_M[b][r][c] = M_b[r][c]; NULL = no TAC.
 *   tac_d  [K] fp16 bias d, required iff tac_M != NULL.  g: TAC block size.
 *          TAC output z'_{b g + r} = fp16(sum_c M_b[r][c] z_{b g + c} + d_{b g + r}),
 *          fp32 fused multiply-adds in ascending c from +0, bias added last.
 *   Aq     out [M][K/2] packed int4.   s_a out [M] fp32 per-token scales.
 *   ws     device workspace of at least sq_quant_act_workspace_bytes().
 */
int sgat_quant_act(const uint16_t* X, const uint8_t* state, const float* P,
                   int32_t M, int32_t K, int32_t d_m, int32_t d_u,
                   const uint16_t* tac_M, const uint16_t* tac_d, int32_t g,
                   uint8_t* Aq, float* s_a, void* ws, size_t ws_bytes, void* stream);

/*
 * w4a4_gemm -- the state-guided quantised projection (Eq. 13; Eq. 5):
 * acc[i][n] = sum_j qa[i][j] qw[n][j] (exact int32), and
 * Y[i][n] = fp16((float(acc[i][n]) * s_a[i]) * s_w[n]).
 *   Aq [M][K/2], s_a [M]: from sgat_quant_act.  Wq [N][K/2], s_w [N]: from
 *   sgat_prepare_weights.  Both operands are K-contiguous (Y = A B^T).
 *   Y    out [M][N] fp16 (may be NULL if acc is given).
 *   acc  out [M][N] int32, or NULL.
 *   ws   device workspace of at least sq_gemm_workspace_bytes(M, N, K).
 *   Each packed operand must be smaller than 2 GiB (M K / 2 and N K / 2 bytes).
 */
int w4a4_gemm(const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w,
              int32_t M, int32_t N, int32_t K, uint16_t* Y, int32_t* acc,
              void* ws, size_t ws_bytes, void* stream);

/*
 * tac_apply -- Temporal Attention Compensation on its own (Eq. 17, App. C):
 * for token i and block b of g channels, Z_out[i, b g + r] =
 * fp16(sum_c M_b[r][c] Z[i, b g + c] + d[b g + r]) with the arithmetic stated
 * at sgat_quant_act.  Not state-dependent; parameters fixed across steps.
 *   Z [M][C] fp16; tac_M [C/g][g][g] fp16; tac_d [C] fp16.
 *   Z_out out [M][C] fp16; must not overlap Z.
 */
int tac_apply(const uint16_t* Z, const uint16_t* tac_M, const uint16_t* tac_d,
              int32_t M, int32_t C, int32_t g, uint16_t* Z_out, void* stream);

/*
 * W8A8 variant (App. D: the same method at 8 bits).  Identical arguments and
 * arithmetic to the 4-bit calls above except for the quantiser, s = absmax / 127
 * and codes clamp(rint(x / s), -128, 127), and the code layout: one signed byte
 * per code, rows of K bytes.
 *   sgat_prepare_weights_w8 -- Wq out [N][K] int8 (as sgat_prepare_weights).
 *   sgat_quantize_w8        -- Aq out [M][K] int8 (as sgat_quantize).
 *   sgat_quant_act_w8       -- Aq out [M][K] int8 (as sgat_quant_act).
 *   w8a8_gemm               -- acc = sum_j qa qw (int32), Y = fp16((acc * s_a) * s_w);
 *                              K <= 65536 so |acc| < 2^31; operands under 2 GiB;
 *                              ws of at least sq_gemm_w8_workspace_bytes(M, N, K).
 */
int sgat_prepare_weights_w8(const uint16_t* W, const float* P, int32_t N, int32_t K,
                            int8_t* Wq, float* s_w, void* ws, size_t ws_bytes, void* stream);
int sgat_quantize_w8(const float* Xp, int32_t M, int32_t K, int8_t* Aq, float* s, void* stream);
int sgat_quant_act_w8(const uint16_t* X, const uint8_t* state, const float* P,
                      int32_t M, int32_t K, int32_t d_m, int32_t d_u,
                      const uint16_t* tac_M, const uint16_t* tac_d, int32_t g,
                      int8_t* Aq, float* s_a, void* ws, size_t ws_bytes, void* stream);
int w8a8_gemm(const int8_t* Aq, const float* s_a, const int8_t* Wq, const float* s_w,
              int32_t M, int32_t N, int32_t K, uint16_t* Y, int32_t* acc,
              void* ws, size_t ws_bytes, void* stream);

/*
 * Fast activation transform on the fp16 matrix cores (the matrix-core form of
 * Eq. 11).  The basis is split once: v = 2^14 P, hi = fp16(v), lo = fp16(v - hi),
 * stored as Ps [K][2K] fp16 with Ps[j][k] = hi(P[k][j]) and Ps[j][K + k] =
 * lo(P[k][j]) (4 K^2 bytes, the size of P itself).  sgat_transform_fast then
 * computes x' = 2^-14 ([x, x] . Ps^T) with fp32 accumulation and the gate of
 * sgat_transform; the result differs from the exact x P by at most
 * 2^-14 (sum_k |x_k||v_kj - hi_kj - lo_kj| + gamma_2K sum_k |x_k|(|hi_kj| + |lo_kj|)),
 * gamma_n = n u / (1 - n u), u = 2^-23.  It is not bit-identical to
 * sgat_transform, whose fixed order defines the codes; codes quantised from it
 * can differ where a value lies within that bound of a rounding boundary.
 *   sgat_split_basis:    P [K][K] fp32 in, Ps [K][2K] fp16 out; K^2 4 bytes < 2 GiB.
 *   sgat_transform_fast: X [M][K] fp16, state [M] or NULL (no gate), Ps from
 *                        sgat_split_basis, Xp out [M][K] fp32; X under 2 GiB.
 */
int sgat_split_basis(const float* P, int32_t K, uint16_t* Ps, void* stream);
int sgat_transform_fast(const uint16_t* X, const uint8_t* state, const uint16_t* Ps, int32_t M, int32_t K,
                        int32_t d_m, int32_t d_u, float* Xp, void* stream);

/*
 * int4 codes on the FP6 matrix cores: the same GEMM (Eq. 5 / Eq. 13) with both
 * operands re-encoded as 6-bit floats.  In e3m2 (sign, 3 exponent bits with
 * bias 3, 2 mantissa bits; OCP Microscaling Formats v1.0 FP6 E3M2) every code
 * -8..7 is exact, products are integers of magnitude <= 64 and sums of up to
 * 131072 of them are integers below 2^24, so the matrix cores' fp32
 * accumulation is exact: acc and Y equal w4a4_gemm's bit for bit.
 * Operand layout (A and W alike): per row, the K codes padded with zero codes to
 * whole blocks of 128; block b takes 96 bytes at 96 b; chunk c of it (codes
 * 128 b + 32 c .. + 31) is the 192-bit little-endian string with code j in bits
 * 6 j .. 6 j + 5, its bytes 0..15 stored at 96 b + 16 c and bytes 16..23 at
 * 96 b + 64 + 8 c.  Rows are sq_fp6_row_bytes(K) = 96 ceil(K / 128) bytes.
 *   sq_fp6_row_bytes: bytes per operand row, 0 for an invalid K.
 *   sq_codes_to_fp6:  codes [R][K/2] packed int4 (the sgat_* layout) in, out
 *                     [R][sq_fp6_row_bytes(K)] (must not overlap codes); under 2 GiB.
 *   w4a4_gemm_fp6:    A6 [M][row bytes], W6 [N][row bytes], s_a [M], s_w [N];
 *                     Y [M][N] fp16 and / or acc [M][N] int32 out; N % 8 == 0;
 *                     operands under 2 GiB; no workspace.
 */
size_t sq_fp6_row_bytes(int32_t K);
int sq_codes_to_fp6(const uint8_t* codes, int32_t R, int32_t K, uint8_t* out, void* stream);
int w4a4_gemm_fp6(const uint8_t* A6, const float* s_a, const uint8_t* W6, const float* s_w,
                  int32_t M, int32_t N, int32_t K, uint16_t* Y, int32_t* acc, void* stream);

/*
 * Fragment-ordered weights: the same GEMM (Eq. 13; Eq. 5) with the packed int4
 * weights stored in the order the GEMM kernels read them.  The weights are
 * fixed after sgat_prepare_weights (Eq. 12), so they can be reordered once,
 * offline; a load of 16 weight rows then reads one contiguous 1 KB block, which
 * the memory system serves faster than 16 runs of 64 bytes (decode-sized M,
 * where the GEMM streams the weights from HBM).
 * Layout: rows in groups of 16 (the last group padded with zero rows), k in
 * steps of 128 codes (64 bytes of a row; the last step padded with zero codes);
 * with G = ceil(N / 16), block (g, t) is 1024 bytes at (t G + g) 1024, and
 * within it the 16 bytes at 16 (16 j + r) are bytes 64 t + 16 j .. 64 t + 16 j
 * + 15 of row 16 g + r (j = 0..3, r = 0..15).  Every byte of Wq appears exactly
 * once.
 *   sq_frag_weight_bytes: G ceil(K / 128) 1024, 0 for an invalid K.
 *   sq_weights_to_frag:   Wq [N][K/2] (the sgat_prepare_weights layout) in, Wf
 *                         [sq_frag_weight_bytes(N, K)] out (must not overlap
 *                         Wq); under 2 GiB.  Any N >= 0.
 *   w4a4_gemm_frag:       as w4a4_gemm with Wf in place of Wq: same arguments,
 *                         rules and workspace (sq_gemm_workspace_bytes); acc and
 *                         Y equal w4a4_gemm's bit for bit.
 */
size_t sq_frag_weight_bytes(int32_t N, int32_t K);
int sq_weights_to_frag(const uint8_t* Wq, int32_t N, int32_t K, uint8_t* Wf, void* stream);
int w4a4_gemm_frag(const uint8_t* Aq, const float* s_a, const uint8_t* Wf, const float* s_w,
                   int32_t M, int32_t N, int32_t K, uint16_t* Y, int32_t* acc,
                   void* ws, size_t ws_bytes, void* stream);

/*
 * The same for the W8A8 variant (App. D): the int8 weights [N][K] of
 * sgat_prepare_weights_w8 in fragment order.  A row of K int8 codes is K bytes,
 * the bytes of 2 K int4 codes, and is reordered exactly as such a row (k steps
 * of 64 codes here).
 *   sq_frag_weight_w8_bytes: sq_frag_weight_bytes(N, 2 K) = G ceil(K / 64) 1024;
 *                            0 for an invalid K (64 <= K <= 65536, K % 64 == 0).
 *   sq_weights_to_frag_w8:   Wq [N][K] int8 in, Wf [sq_frag_weight_w8_bytes(N, K)]
 *                            out; sq_weights_to_frag(Wq, N, 2 K, Wf) with the
 *                            same rules.
 *   w8a8_gemm_frag:          as w8a8_gemm with Wf in place of Wq: same arguments,
 *                            rules and workspace (sq_gemm_w8_workspace_bytes);
 *                            acc and Y equal w8a8_gemm's bit for bit.
 */
size_t sq_frag_weight_w8_bytes(int32_t N, int32_t K);
int sq_weights_to_frag_w8(const int8_t* Wq, int32_t N, int32_t K, uint8_t* Wf, void* stream);
int w8a8_gemm_frag(const int8_t* Aq, const float* s_a, const uint8_t* Wf, const float* s_w,
                   int32_t M, int32_t N, int32_t K, uint16_t* Y, int32_t* acc,
                   void* ws, size_t ws_bytes, void* stream);

/*
 * w4a4_gemm_frag_noalloc -- for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): w4a4_gemm_frag without the workspace argument.  Same arguments
 * otherwise, same rules, same results bit for bit.  The K-split partial sums
 * that w4a4_gemm_frag keeps in the caller's workspace go to scratch memory the
 * library holds instead: a device array of SQ_NOALLOC_SCRATCH_BYTES per GPU,
 * held from the first call on that GPU until the process ends.  The call
 * allocates nothing (no hipMalloc, no library allocator); the first call on a
 * device looks up the array's address once.
 *   - A shape whose partial sums would exceed SQ_NOALLOC_SCRATCH_BYTES is
 *     rejected with SQ_ERR_WORKSPACE (sq_gemm_workspace_bytes(M, N, K) gives
 *     the need; no shape this GEMM splits needs more than 16 MiB).
 *   - `stream` must belong to the current device (SQ_ERR_SHAPE otherwise).
 *   - Every call on one GPU shares that GPU's array: calls that overlap in
 *     time on one GPU (on different streams, or from different threads
 *     without ordering) race on it and may return wrong results.  Calls
 *     ordered on one stream are safe.  Nothing in the array needs to start at
 *     zero; it keeps the last call's partial sums.
 */
#define SQ_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
int w4a4_gemm_frag_noalloc(const uint8_t* Aq, const float* s_a, const uint8_t* Wf, const float* s_w,
                           int32_t M, int32_t N, int32_t K, uint16_t* Y, int32_t* acc, void* stream);

/*
 * tac_calibrate -- the closed-form estimate of the TAC parameters (Sec. 3.3,
 * closed-form estimation; App. C), from paired attention outputs collected at
 * the TAC insertion point with the quantisers off (Z_fp) and on (Z_q).  Per
 * block b of g channels, in fp64:
 *   mu_b = (1/N) sum_i z_i, Sigma_b = (1/N) sum_i z_i z_i^T - mu_b mu_b^T (both inputs);
 *   lambda_b = rho max(Tr(Sigma_q) / g, eps);
 *   M_b = Sigma_fp^(1/2) (Sigma_q + lambda_b I)^(-1/2), each power through a
 *         symmetric eigendecomposition with eigenvalues clamped below at 1e-12;
 *   M_b = U diag(s) V^T -> U diag((1 - eta) s + eta mean(s)) V^T   (smoothing);
 *   M_b -> (1 - alpha) M_b + alpha I                                 (shrinkage);
 *   d_b = mu_fp - M_b mu_q.
 * The appendix's defaults are rho = 3e-4, eps = 1e-8, eta = 0.15, alpha = 0.55.
 *   Z_fp, Z_q [N][C] fp16, N >= 1 tokens; C as K (C % 64 == 0); g as for TAC.
 *   tac_M out [C/g][g][g] fp16 (M_b[r][c]), tac_d out [C] fp16: each one
 *         round-to-nearest-even from the fp64 value; the layout tac_apply and
 *         sgat_quant_act read.
 *   M64 out [C/g][g][g] fp64 and d64 out [C] fp64: the unrounded values, or NULL.
 *   ws    device workspace of at least sq_tac_calibrate_workspace_bytes(N, C, g)
 *         (required).
 * Sums run in a fixed order, so results depend only on the inputs; they agree
 * with any other fp64 evaluation to rounding, not bit for bit.  Offline: run
 * once per layer after the activation transform is fixed.
 */
size_t sq_tac_calibrate_workspace_bytes(int32_t N, int32_t C, int32_t g);
int tac_calibrate(const uint16_t* Z_fp, const uint16_t* Z_q, int32_t N, int32_t C, int32_t g,
                  double rho, double eps, double eta, double alpha,
                  uint16_t* tac_M, uint16_t* tac_d, double* M64, double* d64,
                  void* ws, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* STARQUANT_H */
