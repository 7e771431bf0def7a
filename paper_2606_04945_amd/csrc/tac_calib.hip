// TAC closed-form calibration (Sec. 3.3 closed-form estimation; App. C).
//
// From paired attention outputs Z_fp (quantisers off) and Z_q (quantisers on),
// fp16 [N][C], per block of g channels:
//   mu_b    = (1/N) sum_i z_i,   Sigma_b = (1/N) sum_i z_i z_i^T - mu_b mu_b^T   (both passes)
//   lambda  = rho max(Tr(Sigma_q) / g, eps)
//   M       = Sigma_fp^(1/2) (Sigma_q + lambda I)^(-1/2),  A^p = Q diag(max(l_i, 1e-12)^p) Q^T
//   M_sv    = U diag((1 - eta) sigma + eta mean(sigma)) V^T,  M = U diag(sigma) V^T
//   M_final = (1 - alpha) M_sv + alpha I,   d = mu_fp - M_final mu_q
// stored as fp16 (one round-to-nearest-even from fp64) in the layout the TAC
// kernels read, tac_M [C/g][g][g] (row r, column c) and tac_d [C].
//
// Two kernels, all arithmetic in fp64:
//  * tac_stats_kernel: the data-parallel part.  A workgroup takes a span of
//    channels (whole blocks, at least 64 channels so rows are read in 128-byte
//    runs) and a chunk of tokens, stages 32 tokens at a time in LDS as fp64,
//    and accumulates every (r, c) product of its blocks and every channel sum
//    in registers, in token order.  Partial sums per chunk go to the
//    workspace.
//  * tac_finalize_kernel: one workgroup per block.  Adds the chunk partials in
//    chunk order, forms the statistics, and runs the closed form: symmetric
//    eigendecompositions by cyclic Jacobi with the round-robin (parallel)
//    ordering, and the singular value decomposition of M by one-sided
//    (Hestenes) Jacobi, whose singular values keep full relative accuracy.
//    Matrices live in the workspace (g x g fp64, up to 128 KB each); the two
//    a Jacobi iteration updates every round are staged in LDS for g <= 64, and
//    for g = 128 the rotated matrix sits in LDS and the vectors in registers.
// Results depend only on the inputs (every sum has a fixed order); they agree
// with an fp64 LAPACK evaluation to rounding, not bit for bit.
#include "sq_internal.hpp"

namespace sq {
namespace {

constexpr int kCalThreads = 256;
constexpr int kTileTok = 32;            // tokens staged per LDS tile
constexpr int kMaxChunks = 64;
constexpr int kChunkTok = 128;          // tokens per chunk before the caps
constexpr double kEigFloor = 1e-12;
constexpr int kLdsBlock = 64;          // largest g whose Jacobi matrices stay in LDS

// ----------------------------------------------------------------- statistics

// part layout: [pass][chunk][block][g*g second moments, then g sums]
template <int G>
__global__ __launch_bounds__(kCalThreads) void tac_stats_kernel(const uint16_t* __restrict__ Zf,
                                                               const uint16_t* __restrict__ Zq, int N, int C,
                                                               int tok_per_chunk, int chunks,
                                                               double* __restrict__ part) {
    constexpr int S = G > 64 ? G : 64;                   // channels per workgroup
    constexpr int NB = S / G;                            // blocks per workgroup
    constexpr int P = S * G;                             // (block, r, c) products
    constexpr int PPT = (P + kCalThreads - 1) / kCalThreads;
    constexpr int VPT = kTileTok * S / 8 / kCalThreads;  // 16-byte loads per thread per tile
    static_assert(VPT >= 1 && VPT * 8 * kCalThreads == kTileTok * S, "tile split");
    __shared__ double tile[kTileTok][S + 1];

    const int tid = threadIdx.x;
    const int c0 = blockIdx.x * S;
    const int chunk = blockIdx.y;
    const int pass = blockIdx.z;
    const uint16_t* Z = pass == 0 ? Zf : Zq;
    const int t0 = chunk * tok_per_chunk;
    const int t1 = min(N, t0 + tok_per_chunk);

    double acc[PPT];
    int pr[PPT], pc[PPT];
#pragma unroll
    for (int k = 0; k < PPT; ++k) {
        acc[k] = 0.0;
        const int p = tid + k * kCalThreads;
        const int bs = p / (G * G), rc = p % (G * G);
        pr[k] = p < P ? bs * G + rc / G : 0;              // span-local channel of row r
        pc[k] = p < P ? bs * G + rc % G : 0;              // and of column c
    }
    double sum = 0.0;                                     // channel tid's sum (tid < S)

    for (int tb = t0; tb < t1; tb += kTileTok) {
#pragma unroll
        for (int v = 0; v < VPT; ++v) {
            const int e = (tid + v * kCalThreads) * 8;    // element index in the tile
            const int tt = e / S, ch = e % S;
            const int t = tb + tt;
            uint4 raw = make_uint4(0, 0, 0, 0);           // tokens past t1 contribute zeros
            if (t < t1) raw = *reinterpret_cast<const uint4*>(Z + (size_t)t * C + c0 + ch);
            const uint16_t* h = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
            for (int q = 0; q < 8; ++q) tile[tt][ch + q] = (double)h2f(h[q]);
        }
        __syncthreads();
        const int nt = min(kTileTok, t1 - tb);
        for (int tt = 0; tt < nt; ++tt) {
#pragma unroll
            for (int k = 0; k < PPT; ++k) acc[k] = fma(tile[tt][pr[k]], tile[tt][pc[k]], acc[k]);
            if (tid < S) sum += tile[tt][tid];
        }
        __syncthreads();
    }
    const int B = C / G;
    const size_t stride = (size_t)G * G + G;
    double* base = part + ((size_t)pass * chunks + chunk) * B * stride;
#pragma unroll
    for (int k = 0; k < PPT; ++k) {
        const int p = tid + k * kCalThreads;
        if (p < P) {
            const int bs = p / (G * G), rc = p % (G * G);
            base[(size_t)(blockIdx.x * NB + bs) * stride + rc] = acc[k];
        }
    }
    if (tid < S) base[(size_t)(blockIdx.x * NB + tid / G) * stride + G * G + tid % G] = sum;
}

// ----------------------------------------------------------------- closed form

// One RNE rounding of an fp64 value to fp16 bits (overflow to infinity).
__device__ uint16_t f64_to_f16(double x) {
    const uint64_t b = (uint64_t)__double_as_longlong(x);
    const uint16_t sign = (uint16_t)((b >> 48) & 0x8000u);
    const int e = (int)((b >> 52) & 0x7FF);
    const uint64_t frac = b & 0xFFFFFFFFFFFFFull;
    if (e == 0x7FF) return sign | 0x7C00u | (frac ? 0x200u : 0u);
    if (e == 0) return sign;                              // zero or an fp64 subnormal
    const uint64_t mant = frac | (1ull << 52);            // value = mant * 2^(E - 52)
    int E = e - 1023;
    int shift;                                            // bits dropped from mant
    if (E >= -14) {
        shift = 42;                                       // keep 11 bits (implicit one + 10)
    } else {
        shift = 28 - E;                                   // subnormal: units of 2^-24
        if (shift > 60) return sign;                      // below half the smallest subnormal
    }
    uint64_t q = mant >> shift;
    const uint64_t rem = mant & ((1ull << shift) - 1);
    const uint64_t half = 1ull << (shift - 1);
    if (rem > half || (rem == half && (q & 1))) ++q;
    if (E >= -14) {
        if (q == (1ull << 11)) {                          // mantissa carried into the exponent
            q >>= 1;
            ++E;
        }
        if (E > 15) return sign | 0x7C00u;
        return sign | (uint16_t)((E + 15) << 10) | (uint16_t)(q & 0x3FFu);
    }
    return sign | (uint16_t)q;                            // q == 1024 is the smallest normal
}

__device__ int rr_player(int i, int r, int n) { return i == 0 ? 0 : 1 + (i - 1 + r) % (n - 1); }

// Round-robin pair t of round r over n = g players (g even), p < q.
__device__ void rr_pair(int t, int r, int n, int& p, int& q) {
    const int a = rr_player(t, r, n), b = rr_player(n - 1 - t, r, n);
    p = a < b ? a : b;
    q = a < b ? b : a;
}

// Sum over the workgroup (fixed tree order).
__device__ double wg_sum(double v, double* red) {
    const int tid = threadIdx.x;
    red[tid] = v;
    __syncthreads();
    for (int s = kCalThreads / 2; s > 0; s >>= 1) {
        if (tid < s) red[tid] += red[tid + s];
        __syncthreads();
    }
    const double r = red[0];
    __syncthreads();
    return r;
}

// Symmetric eigendecomposition of A (overwritten; eigenvalues end on its
// diagonal), eigenvectors into the columns of V: cyclic Jacobi, round-robin.
__device__ void jacobi_eigh(double* A, double* V, int g, double* cs, double* red) {
    const int tid = threadIdx.x;
    for (int e = tid; e < g * g; e += kCalThreads) V[e] = (e / g == e % g) ? 1.0 : 0.0;
    __syncthreads();
    if (g == 1) return;
    const int h = g / 2;
    for (int sweep = 0; sweep < 60; ++sweep) {
        double off = 0.0, tot = 0.0;
        for (int e = tid; e < g * g; e += kCalThreads) {
            const double a2 = A[e] * A[e];
            tot += a2;
            if (e / g != e % g) off += a2;
        }
        off = wg_sum(off, red);
        tot = wg_sum(tot, red);
        if (!(off > 1e-30 * tot)) break;                  // also stops on a zero matrix
        for (int r = 0; r < g - 1; ++r) {
            if (tid < h) {
                int p, q;
                rr_pair(tid, r, g, p, q);
                const double apq = A[p * g + q];
                double c = 1.0, s = 0.0;
                if (apq != 0.0) {
                    const double tau = (A[q * g + q] - A[p * g + p]) / (2.0 * apq);
                    // for |tau| beyond 1e150, tau^2 would overflow; t = 1 / (2 tau) there
                    const double t = fabs(tau) > 1e150 ? 0.5 / tau
                                                       : (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
                    c = 1.0 / sqrt(1.0 + t * t);
                    s = t * c;
                }
                cs[2 * tid] = c;
                cs[2 * tid + 1] = s;
            }
            __syncthreads();
            for (int e = tid; e < g * h; e += kCalThreads) {      // columns: A J and V J
                const int i = e / h, t = e % h;
                int p, q;
                rr_pair(t, r, g, p, q);
                const double c = cs[2 * t], s = cs[2 * t + 1];
                const double ap = A[i * g + p], aq = A[i * g + q];
                A[i * g + p] = c * ap - s * aq;
                A[i * g + q] = s * ap + c * aq;
                const double vp = V[i * g + p], vq = V[i * g + q];
                V[i * g + p] = c * vp - s * vq;
                V[i * g + q] = s * vp + c * vq;
            }
            __syncthreads();
            for (int e = tid; e < g * h; e += kCalThreads) {      // rows: J^T (A J)
                const int j = e / h, t = e % h;
                int p, q;
                rr_pair(t, r, g, p, q);
                const double c = cs[2 * t], s = cs[2 * t + 1];
                const double ap = A[p * g + j], aq = A[q * g + j];
                A[p * g + j] = c * ap - s * aq;
                A[q * g + j] = s * ap + c * aq;
            }
            __syncthreads();
        }
    }
}

// R = V diag(max(l_i, 1e-12)^p) V^T for p = +1/2 or -1/2; l_i on the diagonal of D.
__device__ void eig_power(const double* D, const double* V, double* R, int g, bool inverse, double* w) {
    const int tid = threadIdx.x;
    for (int k = tid; k < g; k += kCalThreads) {
        const double l = fmax(D[k * g + k], kEigFloor);
        w[k] = inverse ? 1.0 / sqrt(l) : sqrt(l);
    }
    __syncthreads();
    for (int e = tid; e < g * g; e += kCalThreads) {
        const int r = e / g, c = e % g;
        double s = 0.0;
        for (int k = 0; k < g; ++k) s = fma(V[r * g + k] * w[k], V[c * g + k], s);
        R[e] = s;
    }
    __syncthreads();
}

// Singular value decomposition of G (g x g) by one-sided Jacobi: on return the
// columns of G are u_j sigma_j and V holds the right singular vectors.
__device__ void jacobi_svd(double* G, double* V, int g, double* cs, int* flag) {
    const int tid = threadIdx.x;
    for (int e = tid; e < g * g; e += kCalThreads) V[e] = (e / g == e % g) ? 1.0 : 0.0;
    __syncthreads();
    if (g == 1) return;
    const int h = g / 2;
    for (int sweep = 0; sweep < 60; ++sweep) {
        if (tid == 0) *flag = 0;
        __syncthreads();
        for (int r = 0; r < g - 1; ++r) {
            if (tid < h) {
                int p, q;
                rr_pair(tid, r, g, p, q);
                double al = 0.0, be = 0.0, ga = 0.0;
                for (int i = 0; i < g; ++i) {
                    const double x = G[i * g + p], y = G[i * g + q];
                    al = fma(x, x, al);
                    be = fma(y, y, be);
                    ga = fma(x, y, ga);
                }
                double c = 1.0, s = 0.0;
                if (ga != 0.0 && fabs(ga) > 1e-15 * sqrt(al * be)) {
                    const double zeta = (be - al) / (2.0 * ga);
                    const double t = fabs(zeta) > 1e150
                                         ? 0.5 / zeta
                                         : (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
                    c = 1.0 / sqrt(1.0 + t * t);
                    s = t * c;
                    *flag = 1;
                }
                cs[2 * tid] = c;
                cs[2 * tid + 1] = s;
            }
            __syncthreads();
            for (int e = tid; e < g * h; e += kCalThreads) {
                const int i = e / h, t = e % h;
                int p, q;
                rr_pair(t, r, g, p, q);
                const double c = cs[2 * t], s = cs[2 * t + 1];
                const double gp = G[i * g + p], gq = G[i * g + q];
                G[i * g + p] = c * gp - s * gq;
                G[i * g + q] = s * gp + c * gq;
                const double vp = V[i * g + p], vq = V[i * g + q];
                V[i * g + p] = c * vp - s * vq;
                V[i * g + q] = s * vp + c * vq;
            }
            __syncthreads();
        }
        if (*flag == 0) break;
        __syncthreads();
    }
}

// g = 128: two g x g fp64 matrices (256 KB) do not fit in LDS together, and
// updating them in global memory made every round a chain of dependent memory
// round trips.  The matrix the rotations act on two-sidedly (A) or whose
// columns they combine (G) stays in LDS; the vector matrix V lives in registers,
// each row split over a lane pair: lane 2 i + h holds half h of row i.  V's
// columns are kept in round-robin *position* order (position k holds column
// rr_player(k, r)), half 0 holding positions 0 .. g/2 - 1 at index k and half 1
// positions g - 1 .. g/2 at index k (position g - 1 - k), so that every round's
// pair t (positions t and g - 1 - t) sits at index t in both lanes and all
// register indices are static.  Between rounds positions 1 .. g - 1 shift
// cyclically by one.  After a whole sweep (g - 1 rounds) position order is
// column order again, and the sweep loops only stop at sweep boundaries.
// Rotations and sums are those of jacobi_eigh and jacobi_svd; only where the
// data lives differs (and, for the SVD, the column sums are split four ways and
// added in a fixed order).
constexpr int kRegBlock = 128;

// The value held by the other lane of this lane's pair (lanes 2 i, 2 i + 1).
__device__ __forceinline__ double pair_swap(double x) {
    const unsigned long long u = (unsigned long long)__double_as_longlong(x);
    const int lo = __builtin_amdgcn_mov_dpp((int)(unsigned)u, 0xB1, 0xF, 0xF, false);   // quad_perm [1, 0, 3, 2]
    const int hi = __builtin_amdgcn_mov_dpp((int)(unsigned)(u >> 32), 0xB1, 0xF, 0xF, false);
    return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

// Half h of row i of the identity, in position order at the start of a sweep.
template <int G>
__device__ __forceinline__ void half_identity(double (&v)[G / 2], int i, bool h1) {
#pragma unroll
    for (int k = 0; k < G / 2; ++k) v[k] = (h1 ? G - 1 - k : k) == i ? 1.0 : 0.0;
}

template <int G>
__device__ __forceinline__ void store_half(const double (&v)[G / 2], double* Vout, int i, bool h1) {
#pragma unroll
    for (int k = 0; k < G / 2; ++k) Vout[i * G + (h1 ? G - 1 - k : k)] = v[k];
}

// One round on the lane pair's row: pair t holds columns (a, b) = (rr_player(t),
// rr_player(g - 1 - t)); with p = min(a, b) the rotation is (v_p, v_q) <- (c v_p
// - s v_q, s v_p + c v_q), the same map on (v_a, v_b) with s negated when a > b;
// sg[t] holds that signed s.  Then the shift to the next round's positions.
template <int G>
__device__ __forceinline__ void rotate_pairs(double (&v)[G / 2], bool h1, const double* cs, const double* sg) {
    constexpr int H = G / 2, CH = 8;
    static_assert(H % CH == 0, "chunks of pairs");
    // chunks of pairs, so that the rotation parameters are read as they are used
    // and do not all sit in registers at once
#pragma unroll
    for (int t0 = 0; t0 < H; t0 += CH) {
#pragma unroll
        for (int t = t0; t < t0 + CH; ++t) {
            const double c = cs[2 * t], sp = sg[t];
            const double mine = v[t], other = pair_swap(mine);
            v[t] = h1 ? sp * other + c * mine : c * mine - sp * other;
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    // half 0 moves down one index and takes position g/2 from its partner's
    // last index; half 1 moves up one index and takes position 1 from its
    // partner's index 1; position 0 stays.  In place, in ascending index order,
    // carrying the old value of the previous index for half 1.
    const double from_hi = pair_swap(v[H - 1]), from_lo = pair_swap(v[1]);
    double prev = v[0];
    v[0] = h1 ? from_lo : v[0];
#pragma unroll
    for (int k = 1; k < H - 1; ++k) {
        const double cur = v[k];
        v[k] = h1 ? prev : v[k + 1];
        prev = cur;
    }
    v[H - 1] = h1 ? prev : from_hi;
}

// Symmetric eigendecomposition, A in LDS (eigenvalues end on its diagonal),
// eigenvectors into the columns of Vout (global), V by lane-pair rows as above.  One two-sided update per
// round over 2 x 2 blocks: block (t1, t2) takes rows (p1, q1) and columns (p2,
// q2), rotated first by columns (A J) then by rows (J^T), the order and
// arithmetic of jacobi_eigh's two passes.
template <int G>
__device__ __forceinline__ void jacobi_eigh_reg(double* A, double* Vout, double* cs, double* sg, int* pq, double* red) {
    constexpr int H = G / 2;
    static_assert(2 * G <= kCalThreads, "a lane pair per row");
    const int tid = threadIdx.x;
    const int row = tid / 2;
    const bool h1 = tid & 1;
    double v[H];
    half_identity<G>(v, row, h1);
    for (int sweep = 0; sweep < 60; ++sweep) {
        double off = 0.0, tot = 0.0;
        for (int e = tid; e < G * G; e += kCalThreads) {
            const double a2 = A[e] * A[e];
            tot += a2;
            if (e / G != e % G) off += a2;
        }
        off = wg_sum(off, red);
        tot = wg_sum(tot, red);
        if (!(off > 1e-30 * tot)) break;                  // also stops on a zero matrix
        for (int r = 0; r < G - 1; ++r) {
            if (tid < H) {
                int p, q;
                rr_pair(tid, r, G, p, q);
                const double apq = A[p * G + q];
                double c = 1.0, s = 0.0;
                if (apq != 0.0) {
                    const double tau = (A[q * G + q] - A[p * G + p]) / (2.0 * apq);
                    const double t = fabs(tau) > 1e150 ? 0.5 / tau
                                                       : (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
                    c = 1.0 / sqrt(1.0 + t * t);
                    s = t * c;
                }
                cs[2 * tid] = c;
                cs[2 * tid + 1] = s;
                sg[tid] = rr_player(tid, r, G) == p ? s : -s;
                pq[2 * tid] = p;
                pq[2 * tid + 1] = q;
            }
            __syncthreads();
#pragma unroll 2
            for (int blk = tid; blk < H * H; blk += kCalThreads) {
                const int t1 = blk / H, t2 = blk % H;
                const int p1 = pq[2 * t1], q1 = pq[2 * t1 + 1], p2 = pq[2 * t2], q2 = pq[2 * t2 + 1];
                const double c1 = cs[2 * t1], s1 = cs[2 * t1 + 1], c2 = cs[2 * t2], s2 = cs[2 * t2 + 1];
                const double a00 = A[p1 * G + p2], a01 = A[p1 * G + q2], a10 = A[q1 * G + p2], a11 = A[q1 * G + q2];
                const double b00 = c2 * a00 - s2 * a01, b01 = s2 * a00 + c2 * a01;   // columns: A J
                const double b10 = c2 * a10 - s2 * a11, b11 = s2 * a10 + c2 * a11;
                A[p1 * G + p2] = c1 * b00 - s1 * b10;                                  // rows: J^T (A J)
                A[q1 * G + p2] = s1 * b00 + c1 * b10;
                A[p1 * G + q2] = c1 * b01 - s1 * b11;
                A[q1 * G + q2] = s1 * b01 + c1 * b11;
            }
            rotate_pairs<G>(v, h1, cs, sg);
            __syncthreads();
        }
    }
    store_half<G>(v, Vout, row, h1);
    __syncthreads();
}

// One-sided Jacobi SVD of Gm (g x g, in LDS): on return its columns are
// u_j sigma_j and Vout (global) holds the right singular vectors.  Each pair's
// three column sums are split over four threads (rows i = 4 k + j ... ) and
// added in the fixed order (s0 + s1) + (s2 + s3).
template <int G>
__device__ __forceinline__ void jacobi_svd_reg(double* Gm, double* Vout, double* cs, double* sg, int* flag) {
    constexpr int H = G / 2;
    static_assert(4 * H <= kCalThreads && 2 * G <= kCalThreads, "four threads per pair, a lane pair per row");
    const int tid = threadIdx.x;
    const int row = tid / 2;
    const bool h1 = tid & 1;
    double v[H];
    half_identity<G>(v, row, h1);
    for (int sweep = 0; sweep < 60; ++sweep) {
        if (tid == 0) *flag = 0;
        __syncthreads();
        for (int r = 0; r < G - 1; ++r) {
            const int t = tid / 4, j = tid % 4;
            int p = 0, q = 1;
            double al = 0.0, be = 0.0, ga = 0.0;
            if (t < H) {
                rr_pair(t, r, G, p, q);
#pragma unroll 4
                for (int i = j; i < G; i += 4) {
                    const double x = Gm[i * G + p], y = Gm[i * G + q];
                    al = fma(x, x, al);
                    be = fma(y, y, be);
                    ga = fma(x, y, ga);
                }
            }
            // lanes 4 t .. 4 t + 3 are consecutive in one wave: (s0 + s1) + (s2 + s3)
            al += __shfl_xor(al, 1);
            be += __shfl_xor(be, 1);
            ga += __shfl_xor(ga, 1);
            al += __shfl_xor(al, 2);
            be += __shfl_xor(be, 2);
            ga += __shfl_xor(ga, 2);
            if (t < H && j == 0) {
                double c = 1.0, s = 0.0;
                if (ga != 0.0 && fabs(ga) > 1e-15 * sqrt(al * be)) {
                    const double zeta = (be - al) / (2.0 * ga);
                    const double tt = fabs(zeta) > 1e150
                                          ? 0.5 / zeta
                                          : (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
                    c = 1.0 / sqrt(1.0 + tt * tt);
                    s = tt * c;
                    *flag = 1;
                }
                cs[2 * t] = c;
                cs[2 * t + 1] = s;
                sg[t] = rr_player(t, r, G) == p ? s : -s;
            }
            __syncthreads();
#pragma unroll 2
            for (int e = tid; e < G * H; e += kCalThreads) {
                const int i = e / H, tt = e % H;
                int pp, qq;
                rr_pair(tt, r, G, pp, qq);
                const double c = cs[2 * tt], s = cs[2 * tt + 1];
                const double gp = Gm[i * G + pp], gq = Gm[i * G + qq];
                Gm[i * G + pp] = c * gp - s * gq;
                Gm[i * G + qq] = s * gp + c * gq;
            }
            rotate_pairs<G>(v, h1, cs, sg);
            __syncthreads();
        }
        if (*flag == 0) break;
        __syncthreads();
    }
    store_half<G>(v, Vout, row, h1);
    __syncthreads();
}

// REG: g = 128, the Jacobi matrix in LDS and V in registers (see jacobi_eigh_reg);
// otherwise both Jacobi matrices in LDS for g <= 64, in the workspace above.
template <bool REG>
__global__ __launch_bounds__(kCalThreads) void tac_finalize_kernel(const double* __restrict__ part, int chunks,
                                                                  int N, int C, int g, double rho, double eps,
                                                                  double eta, double alpha, double* __restrict__ wk,
                                                                  uint16_t* __restrict__ tac_M,
                                                                  uint16_t* __restrict__ tac_d,
                                                                  double* __restrict__ M64, double* __restrict__ d64) {
    __shared__ double red[kCalThreads];
    __shared__ double cs[128];
    __shared__ double w[128];
    __shared__ double sg[64];
    __shared__ int pq[128];
    __shared__ int flag;
    extern __shared__ double lds_mats[];               // 2 g^2 doubles when g <= 64, g^2 for REG
    const int tid = threadIdx.x;
    const int b = blockIdx.x;
    const int B = C / g;
    const size_t gg = (size_t)g * g;
    // the Jacobi iterations touch their two matrices every round: in LDS when
    // they fit, else in the workspace
    const bool local = !REG && g <= kLdsBlock;
    auto stage_in = [&](const double* src) {
        for (int e = tid; e < (int)gg; e += kCalThreads) lds_mats[e] = src[e];
        __syncthreads();
    };
    auto stage_out = [&](double* a, double* v) {
        for (int e = tid; e < (int)gg; e += kCalThreads) {
            a[e] = lds_mats[e];
            v[e] = lds_mats[gg + e];
        }
        __syncthreads();
    };
    auto stage_out_a = [&](double* a) {               // REG: V was written by the solver
        for (int e = tid; e < (int)gg; e += kCalThreads) a[e] = lds_mats[e];
        __syncthreads();
    };
    double* base = wk + (size_t)b * (6 * gg + 3 * g);
    double* Sf = base;                 // Sigma_fp, then its eigenvalues
    double* Sq = base + gg;            // Sigma_q + lambda I, then its eigenvalues
    double* V = base + 2 * gg;         // eigenvectors / right singular vectors
    double* R1 = base + 3 * gg;        // Sigma_fp^(1/2), later M_sv
    double* R2 = base + 4 * gg;        // (Sigma_q + lambda I)^(-1/2)
    double* G = base + 5 * gg;         // M, then U diag(sigma)
    double* mu_f = base + 6 * gg;
    double* mu_q = mu_f + g;
    double* sig = mu_q + g;
    const size_t stride = gg + g;

    // statistics: chunk partials added in chunk order
    for (int e = tid; e < (int)stride; e += kCalThreads) {
        double sf = 0.0, sq = 0.0;
        for (int k = 0; k < chunks; ++k) {
            sf += part[((size_t)k * B + b) * stride + e];
            sq += part[((size_t)(chunks + k) * B + b) * stride + e];
        }
        if (e < (int)gg) {
            Sf[e] = sf / (double)N;
            Sq[e] = sq / (double)N;
        } else {
            mu_f[e - gg] = sf / (double)N;
            mu_q[e - gg] = sq / (double)N;
        }
    }
    __syncthreads();
    for (int e = tid; e < (int)gg; e += kCalThreads) {
        const int r = e / g, c = e % g;
        Sf[e] = Sf[e] - mu_f[r] * mu_f[c];
        Sq[e] = Sq[e] - mu_q[r] * mu_q[c];
    }
    __syncthreads();
    // damping
    double tr = 0.0;
    for (int k = tid; k < g; k += kCalThreads) tr += Sq[k * g + k];
    tr = wg_sum(tr, red);
    const double lam = rho * fmax(tr / g, eps);
    for (int k = tid; k < g; k += kCalThreads) Sq[k * g + k] += lam;
    __syncthreads();
    // covariance matching
    if (REG) {
        stage_in(Sf);
        jacobi_eigh_reg<kRegBlock>(lds_mats, V, cs, sg, pq, red);
        stage_out_a(Sf);
    } else if (local) {
        stage_in(Sf);
        jacobi_eigh(lds_mats, lds_mats + gg, g, cs, red);
        stage_out(Sf, V);
    } else {
        jacobi_eigh(Sf, V, g, cs, red);
    }
    eig_power(Sf, V, R1, g, false, w);
    if (REG) {
        stage_in(Sq);
        jacobi_eigh_reg<kRegBlock>(lds_mats, V, cs, sg, pq, red);
        stage_out_a(Sq);
    } else if (local) {
        stage_in(Sq);
        jacobi_eigh(lds_mats, lds_mats + gg, g, cs, red);
        stage_out(Sq, V);
    } else {
        jacobi_eigh(Sq, V, g, cs, red);
    }
    eig_power(Sq, V, R2, g, true, w);
    for (int e = tid; e < (int)gg; e += kCalThreads) {
        const int r = e / g, c = e % g;
        double s = 0.0;
        for (int k = 0; k < g; ++k) s = fma(R1[r * g + k], R2[k * g + c], s);
        G[e] = s;
    }
    __syncthreads();
    // singular value smoothing
    if (REG) {
        stage_in(G);
        jacobi_svd_reg<kRegBlock>(lds_mats, V, cs, sg, &flag);
        stage_out_a(G);
    } else if (local) {
        stage_in(G);
        jacobi_svd(lds_mats, lds_mats + gg, g, cs, &flag);
        stage_out(G, V);
    } else {
        jacobi_svd(G, V, g, cs, &flag);
    }
    for (int j = tid; j < g; j += kCalThreads) {
        double s = 0.0;
        for (int i = 0; i < g; ++i) s = fma(G[i * g + j], G[i * g + j], s);
        sig[j] = sqrt(s);
    }
    __syncthreads();
    double ssum = 0.0;
    for (int j = tid; j < g; j += kCalThreads) ssum += sig[j];
    const double sbar = wg_sum(ssum, red) / g;
    for (int j = tid; j < g; j += kCalThreads) {      // factor sigma'_j / sigma_j on column j of U Sigma
        const double s = sig[j];
        w[j] = s > 0.0 ? ((1.0 - eta) * s + eta * sbar) / s : 0.0;
    }
    __syncthreads();
    for (int e = tid; e < (int)gg; e += kCalThreads) {
        const int r = e / g, c = e % g;
        double s = 0.0;
        for (int k = 0; k < g; ++k) s = fma(G[r * g + k] * w[k], V[c * g + k], s);
        // identity shrinkage
        R1[e] = (1.0 - alpha) * s + (r == c ? alpha : 0.0);
    }
    __syncthreads();
    // bias, outputs
    for (int r = tid; r < g; r += kCalThreads) {
        double s = 0.0;
        for (int c = 0; c < g; ++c) s = fma(R1[r * g + c], mu_q[c], s);
        const double d = mu_f[r] - s;
        tac_d[b * g + r] = f64_to_f16(d);
        if (d64) d64[b * g + r] = d;
    }
    for (int e = tid; e < (int)gg; e += kCalThreads) {
        tac_M[(size_t)b * gg + e] = f64_to_f16(R1[e]);
        if (M64) M64[(size_t)b * gg + e] = R1[e];
    }
}

template <int G>
hipError_t launch_stats(const uint16_t* Zf, const uint16_t* Zq, int N, int C, int per, int chunks, double* part,
                        hipStream_t st) {
    constexpr int S = G > 64 ? G : 64;
    dim3 grid(C / S, chunks, 2);
    hipLaunchKernelGGL(tac_stats_kernel<G>, grid, dim3(kCalThreads), 0, st, Zf, Zq, N, C, per, chunks, part);
    return hipGetLastError();
}

// Token chunks: about 128 tokens each, at most 64, and at most what keeps the
// partial sums under 64 MB.
void calib_plan(int N, int C, int g, int& chunks, int& per) {
    const size_t per_chunk = 2 * ((size_t)C / g) * ((size_t)g * g + g) * sizeof(double);
    const size_t cap_bytes = (size_t)64 << 20;
    int cap = (int)(cap_bytes / per_chunk);
    cap = cap < 1 ? 1 : (cap > kMaxChunks ? kMaxChunks : cap);
    chunks = (N + kChunkTok - 1) / kChunkTok;
    chunks = chunks < 1 ? 1 : (chunks > cap ? cap : chunks);
    per = (N + chunks - 1) / chunks;
    chunks = (N + per - 1) / per;
}

}  // namespace

size_t tac_calib_workspace_bytes(int N, int C, int g) {
    if (N <= 0 || C <= 0 || g <= 0) return 0;
    int chunks, per;
    calib_plan(N, C, g, chunks, per);
    const size_t B = (size_t)C / g, gg = (size_t)g * g;
    const size_t part = 2 * (size_t)chunks * B * (gg + g) * sizeof(double);
    const size_t work = B * (6 * gg + 3 * g) * sizeof(double);
    return ((part + 255) / 256) * 256 + work;
}

hipError_t launch_tac_calib(const uint16_t* Zf, const uint16_t* Zq, int N, int C, int g, double rho, double eps,
                            double eta, double alpha, uint16_t* tac_M, uint16_t* tac_d, double* M64, double* d64,
                            void* ws, hipStream_t st) {
    int chunks, per;
    calib_plan(N, C, g, chunks, per);
    const size_t B = (size_t)C / g, gg = (size_t)g * g;
    double* part = static_cast<double*>(ws);
    const size_t part_bytes = 2 * (size_t)chunks * B * (gg + g) * sizeof(double);
    double* wk = reinterpret_cast<double*>(static_cast<uint8_t*>(ws) + ((part_bytes + 255) / 256) * 256);
    hipError_t e;
    switch (g) {
        case 1: e = launch_stats<1>(Zf, Zq, N, C, per, chunks, part, st); break;
        case 2: e = launch_stats<2>(Zf, Zq, N, C, per, chunks, part, st); break;
        case 4: e = launch_stats<4>(Zf, Zq, N, C, per, chunks, part, st); break;
        case 8: e = launch_stats<8>(Zf, Zq, N, C, per, chunks, part, st); break;
        case 16: e = launch_stats<16>(Zf, Zq, N, C, per, chunks, part, st); break;
        case 32: e = launch_stats<32>(Zf, Zq, N, C, per, chunks, part, st); break;
        case 64: e = launch_stats<64>(Zf, Zq, N, C, per, chunks, part, st); break;
        default: e = launch_stats<128>(Zf, Zq, N, C, per, chunks, part, st); break;
    }
    if (e != hipSuccess) return e;
    if (g == kRegBlock) {
        static std::atomic<int> lds_set[kMaxDevices];   // above the 64 KB default for dynamic LDS
        const hipError_t attr = allow_dynamic_lds(reinterpret_cast<const void*>(&tac_finalize_kernel<true>),
                                                  (int)(gg * sizeof(double)), lds_set);
        if (attr != hipSuccess) return attr;
        hipLaunchKernelGGL(tac_finalize_kernel<true>, dim3((unsigned)B), dim3(kCalThreads), gg * sizeof(double), st,
                           part, chunks, N, C, g, rho, eps, eta, alpha, wk, tac_M, tac_d, M64, d64);
        return hipGetLastError();
    }
    const size_t lds = g <= kLdsBlock ? 2 * gg * sizeof(double) : 0;
    hipLaunchKernelGGL(tac_finalize_kernel<false>, dim3((unsigned)B), dim3(kCalThreads), lds, st, part, chunks, N, C,
                       g, rho, eps, eta, alpha, wk, tac_M, tac_d, M64, d64);
    return hipGetLastError();
}

}  // namespace sq
