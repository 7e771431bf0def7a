// SGAT activation transform (Sec. 3.2, Eq. 11): x'_i = x_i P G_{s_i}, and the
// ungated weight-side product W P used by weight preparation (Eq. 12).
//
// Fixed evaluation order (part of the result, because the codes quantised from
// x' flip at rounding midpoints): output (i, j) accumulates k in chunks of 256,
// each chunk an fp32 fused multiply-add chain in ascending k from +0, and the
// chunk sums are added in ascending order to a +0 total.  That order is a
// plain register-tiled SGEMM on the VALU whose k loop is never split across
// threads; MFMA is not used because its internal summation order is not this
// one.
//
// Tiling: a 256-thread workgroup owns BM = 16*TM rows x 128 columns; each
// thread owns TM x 8 outputs (an accumulator and a chunk total for each), with
// X (converted fp16 -> fp32) and P staged through double-buffered LDS 16 k at a
// time and the next global tile prefetched into registers during compute.
#include "sq_internal.hpp"

namespace sq {
namespace {

constexpr int kThreads = 256;
constexpr int kBN = 128;
constexpr int kBK = 16;
constexpr int kTN = 8;

template <int TM>
__global__ __launch_bounds__(kThreads) void transform_kernel(
    const uint16_t* __restrict__ X, const uint8_t* __restrict__ state, const float* __restrict__ P,
    int M, int K, int dm, int du, float* __restrict__ Xp) {
    constexpr int BM = 16 * TM;
    constexpr int AP = BM + 4;                       // padded LDS row (k-major A tile)
    constexpr int BP = kBN + 4;
    __shared__ float As[2][kBK][AP];
    __shared__ float Bs[2][kBK][BP];

    const int tid = threadIdx.x;
    const int tx = tid % 16, ty = tid / 16;
    // up to 16 row tiles of a column tile of P run on one XCD at the same
    // time, so that XCD's L2 fetches the column tile once per group (all of a
    // 1024-token batch is one group) and the XCDs work on different columns
    int rt, ct;
    const int R = (M + BM - 1) / BM;
    xcd_tile(blockIdx.x, R, (K + kBN - 1) / kBN, R < 16 ? R : 16, rt, ct);
    const int row0 = rt * BM, col0 = ct * kBN;

    // global -> register prefetch slots
    // A: BM rows x 16 k fp16 = BM*2 16-byte vectors; thread t takes vectors t, t+256, ..
    constexpr int AV = (BM * 2 + kThreads - 1) / kThreads;
    uint4 ra[AV];
    // P: 16 rows x 128 cols fp32 = 512 float4; thread t takes t and t+256
    float4 rb[2];

    auto load_tiles = [&](int k0) {
#pragma unroll
        for (int v = 0; v < AV; ++v) {
            const int e = tid + v * kThreads;
            ra[v] = make_uint4(0, 0, 0, 0);
            if (e < BM * 2) {
                const int r = e >> 1, h = e & 1, row = row0 + r;
                if (row < M) ra[v] = *reinterpret_cast<const uint4*>(X + (size_t)row * K + k0 + h * 8);
            }
        }
#pragma unroll
        for (int v = 0; v < 2; ++v) {
            const int e = tid + v * kThreads;
            const int kr = e / 32, c4 = (e % 32) * 4;
            rb[v] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (col0 + c4 < K) rb[v] = *reinterpret_cast<const float4*>(P + (size_t)(k0 + kr) * K + col0 + c4);
        }
    };
    auto store_tiles = [&](int buf) {
#pragma unroll
        for (int v = 0; v < AV; ++v) {
            const int e = tid + v * kThreads;
            if (e < BM * 2) {
                const int r = e >> 1, h = e & 1;
                const uint16_t* hv = reinterpret_cast<const uint16_t*>(&ra[v]);
#pragma unroll
                for (int q = 0; q < 8; ++q) As[buf][h * 8 + q][r] = h2f(hv[q]);
            }
        }
#pragma unroll
        for (int v = 0; v < 2; ++v) {
            const int e = tid + v * kThreads;
            const int kr = e / 32, c4 = (e % 32) * 4;
            *reinterpret_cast<float4*>(&Bs[buf][kr][c4]) = rb[v];
        }
    };

    float acc[TM][kTN], tot[TM][kTN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < kTN; ++j) acc[i][j] = 0.0f, tot[i][j] = 0.0f;

    const int nk = K / kBK;
    load_tiles(0);
    store_tiles(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) load_tiles((kt + 1) * kBK);
#pragma unroll
        for (int kk = 0; kk < kBK; ++kk) {
            float a[TM], b[kTN];
#pragma unroll
            for (int i = 0; i < TM; i += 4) {
                const float4 t = *reinterpret_cast<const float4*>(&As[buf][kk][ty * TM + i]);
                a[i] = t.x, a[i + 1] = t.y, a[i + 2] = t.z, a[i + 3] = t.w;
            }
#pragma unroll
            for (int j = 0; j < kTN; j += 4) {
                const float4 t = *reinterpret_cast<const float4*>(&Bs[buf][kk][tx * kTN + j]);
                b[j] = t.x, b[j + 1] = t.y, b[j + 2] = t.z, b[j + 3] = t.w;
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < kTN; ++j) acc[i][j] = __builtin_fmaf(a[i], b[j], acc[i][j]);
        }
        const int kend = (kt + 1) * kBK;
        if (kend % kChunk == 0 || kend == K) {       // chunk boundary: fold into the total
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < kTN; ++j) tot[i][j] = tot[i][j] + acc[i][j], acc[i][j] = 0.0f;
        }
        if (kt + 1 < nk) {
            store_tiles(buf ^ 1);
            __syncthreads();
        }
    }

    const int cbase = col0 + tx * kTN;
    if (cbase >= K) return;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int row = row0 + ty * TM + i;
        if (row >= M) break;
        float o[kTN];
        if (state) {
            const bool masked = state[row] != 0;
#pragma unroll
            for (int j = 0; j < kTN; ++j) o[j] = kept(cbase + j, K, dm, du, masked) ? tot[i][j] : 0.0f;
        } else {
#pragma unroll
            for (int j = 0; j < kTN; ++j) o[j] = tot[i][j];
        }
        float4* dst = reinterpret_cast<float4*>(Xp + (size_t)row * K + cbase);
        dst[0] = make_float4(o[0], o[1], o[2], o[3]);
        dst[1] = make_float4(o[4], o[5], o[6], o[7]);
    }
}

// P == NULL: the input is already in the P basis; x' = x, then the gate.
__global__ __launch_bounds__(kThreads) void gate_copy_kernel(const uint16_t* __restrict__ X,
                                                             const uint8_t* __restrict__ state, int M,
                                                             int K, int dm, int du, float* __restrict__ Xp) {
    const size_t nvec = (size_t)M * K / 8;
    for (size_t v = (size_t)blockIdx.x * kThreads + threadIdx.x; v < nvec; v += (size_t)gridDim.x * kThreads) {
        const size_t e0 = v * 8;
        const int row = (int)(e0 / K), c0 = (int)(e0 % K);
        const uint4 raw = *reinterpret_cast<const uint4*>(X + e0);
        const uint16_t* h = reinterpret_cast<const uint16_t*>(&raw);
        const bool masked = state ? state[row] != 0 : false;
        float o[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) o[q] = (!state || kept(c0 + q, K, dm, du, masked)) ? h2f(h[q]) : 0.0f;
        float4* dst = reinterpret_cast<float4*>(Xp + e0);
        dst[0] = make_float4(o[0], o[1], o[2], o[3]);
        dst[1] = make_float4(o[4], o[5], o[6], o[7]);
    }
}

}  // namespace

hipError_t launch_transform(const uint16_t* X, const uint8_t* state, const float* P, int M, int K,
                            int dm, int du, float* Xp, hipStream_t st) {
    if (!P) {
        const size_t nvec = (size_t)M * K / 8;
        const int blocks = (int)((nvec + kThreads - 1) / kThreads < 8192 ? (nvec + kThreads - 1) / kThreads : 8192);
        hipLaunchKernelGGL(gate_copy_kernel, dim3(blocks), dim3(kThreads), 0, st, X, state, M, K, dm, du, Xp);
        return hipGetLastError();
    }
    const int ncol = (K + kBN - 1) / kBN;
    if ((size_t)((M + 63) / 64) * ncol > 0x7fffffffu) return hipErrorInvalidConfiguration;
    // enough workgroups to cover the 256 CUs at least twice, else the taller tile
    if ((size_t)ncol * ((M + 127) / 128) >= 512) {
        hipLaunchKernelGGL(transform_kernel<8>, dim3(((M + 127) / 128) * ncol), dim3(kThreads), 0, st, X, state, P,
                           M, K, dm, du, Xp);
    } else {
        hipLaunchKernelGGL(transform_kernel<4>, dim3(((M + 63) / 64) * ncol), dim3(kThreads), 0, st, X, state, P,
                           M, K, dm, du, Xp);
    }
    return hipGetLastError();
}

}  // namespace sq
