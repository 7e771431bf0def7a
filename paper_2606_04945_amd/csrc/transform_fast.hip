// Fast activation transform on the fp16 MFMA (x' = x P G_s, Eq. 11): the
// matrix-core alternative to the fixed-order fp32 transform.
//
// P (fp32, orthogonal, |P| <= 1) is split once, offline, into two fp16 parts of
// the scaled basis v = 2^14 P: hi = fp16(v), lo = fp16(v - hi), stored
// transposed and side by side as Ps [K][2K] (row j = column j of P: hi over k,
// then lo over k).  Then
//   2^14 x'_j = sum_k x_k hi_kj + sum_k x_k lo_kj + sum_k x_k delta_kj,
// |delta| <= 2^-22 |v| + 2^-25, and the first two sums are one fp16 GEMM of
// [x, x] (K doubled) against Ps with fp32 accumulation: the products of two
// fp16 values are exact in fp32, so the result differs from the exact x P by
// at most 2^-14 (sum_k |x_k| |delta_kj| + gamma_2K sum_k |x_k| (|hi_kj| + |lo_kj|)).
// Codes from x' match the fixed-order transform's except where a value lies
// within that bound of a rounding boundary; the fixed-order path is the one the
// codes are defined by, this one trades that for the matrix cores.
//
// The kernel is the GEMM's three-stage direct-to-LDS pipeline on fp16
// operands: 128 x 128 or 64 x 64 output tiles, four waves.  A stage
// holds one k step of 32 of x and the matching steps of both halves of Ps
// (hi and lo), so x is fetched and read from LDS once for both: two
// v_mfma_f32_16x16x32_f16 per 16 x 16 tile and step (hi then lo, into one
// accumulator), the gate applied in the epilogue, fp32 out.
#include "tile_common.hpp"

namespace sq {
namespace {

typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr float kBasisScale = 16384.0f;        // 2^14
constexpr float kBasisUnscale = 1.0f / 16384.0f;

// Ps[j][k] = hi(2^14 P[k][j]), Ps[j][K + k] = lo: 32 x 32 tiles through LDS.
__global__ __launch_bounds__(256) void split_basis_kernel(const float* __restrict__ P, int K,
                                                         uint16_t* __restrict__ Ps) {
    __shared__ float t[32][33];
    const int k0 = blockIdx.y * 32, j0 = blockIdx.x * 32;
    const int tx = threadIdx.x % 32, ty = threadIdx.x / 32;
    for (int r = ty; r < 32; r += 8) t[r][tx] = P[(size_t)(k0 + r) * K + j0 + tx];
    __syncthreads();
    for (int r = ty; r < 32; r += 8) {
        const float v = t[tx][r] * kBasisScale;                 // element (k0 + tx, j0 + r), exact
        const uint16_t hi = f2h(v);
        const uint16_t lo = f2h(v - h2f(hi));                    // v - hi is exact in fp32
        uint16_t* row = Ps + (size_t)(j0 + r) * (2 * (size_t)K);
        row[k0 + tx] = hi;
        row[K + k0 + tx] = lo;
    }
}

template <int WM, int WN, int TM, int TN>
__global__ __launch_bounds__(64 * WM * WN) void transform_mfma_kernel(const uint16_t* __restrict__ X,
                                                                     const uint8_t* __restrict__ state,
                                                                     const uint16_t* __restrict__ Ps, int M, int K,
                                                                     int dm, int du, float* __restrict__ Xp) {
    constexpr int NW = WM * WN;
    constexpr int BM = 16 * WM * TM, BN = 16 * WN * TN;
    constexpr int AB = BM * kKStep, BB = BN * kKStep;   // bytes of one stage: x, then Ps hi, then Ps lo
    constexpr int SB = AB + 2 * BB;
    constexpr int LA = AB / 1024 / NW, LB = BB / 1024 / NW;
    static_assert(LA * NW * 1024 == AB && LB * NW * 1024 == BB, "stage loads must divide evenly");
    __shared__ __attribute__((aligned(16))) uint8_t sm[3 * SB];

    const int tid = threadIdx.x;
    const int lane = tid % kWave, wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int wm = wave / WN, wn = wave % WN;
    int rt, ct;
    xcd_tile(blockIdx.x, (M + BM - 1) / BM, (K + BN - 1) / BN, 8, rt, ct);
    const int row0 = rt * BM, col0 = ct * BN;
    const uint32_t lda = (uint32_t)K * 2;                // X row bytes
    const uint32_t ldb = (uint32_t)K * 4;                // Ps row bytes (hi then lo)
    const int nk = (int)(lda / kKStep);                  // k steps (each with both halves of Ps)
    const uint32_t lo_off = lda;                         // byte offset of the lo half in a Ps row
    const u32x4 rA = sgpr_rsrc(X, (uint32_t)M * lda);
    const u32x4 rB = sgpr_rsrc(Ps, (uint32_t)K * ldb);
    auto swz = [](int r) { return (r >> 1) & 3; };

    uint32_t oa[LA], ob[LB];
#pragma unroll
    for (int u = 0; u < LA; ++u) {
        const int r = 16 * (wave * LA + u) + lane / 4;
        const uint32_t seg = 16 * ((lane % 4) ^ swz(r));
        oa[u] = row0 + r < M ? (uint32_t)(row0 + r) * lda + seg : kOOB;
    }
#pragma unroll
    for (int u = 0; u < LB; ++u) {
        const int r = 16 * (wave * LB + u) + lane / 4;
        const uint32_t seg = 16 * ((lane % 4) ^ swz(r));
        ob[u] = col0 + r < K ? (uint32_t)(col0 + r) * ldb + seg : kOOB;
    }
    auto issue = [&](int kt, int stage) {
        uint8_t* dA = sm + stage * SB;
        uint8_t* dB = dA + AB;
        const uint32_t ko = (uint32_t)kt * kKStep;
#pragma unroll
        for (int u = 0; u < LA; ++u) dma16(rA, lds_addr(dA + (wave * LA + u) * 1024), oa[u] == kOOB ? kOOB : oa[u] + ko);
#pragma unroll
        for (int u = 0; u < LB; ++u) {
            dma16(rB, lds_addr(dB + (wave * LB + u) * 1024), ob[u] == kOOB ? kOOB : ob[u] + ko);
            dma16(rB, lds_addr(dB + BB + (wave * LB + u) * 1024), ob[u] == kOOB ? kOOB : ob[u] + lo_off + ko);
        }
    };

    v4f acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
    const int lr = lane % 16, lg = lane / 16;
    const int fo = (lg ^ swz(lr)) * 16;
    const int offA = ((wm * TM) * 16 + lr) * kKStep + fo;
    const int offB = AB + ((wn * TN) * 16 + lr) * kKStep + fo;
    auto step = [&](int kt, int sc, int sn) {
        asm volatile("" ::: "memory");
        if (kt + 1 < nk)
            wait_vm<LA + 2 * LB>();
        else
            wait_vm<0>();
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        const uint8_t* st = sm + sc * SB;
        v8h fa[TM], fh[TN], fl[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) fa[i] = *reinterpret_cast<const v8h*>(st + offA + i * 16 * kKStep);
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            fh[j] = *reinterpret_cast<const v8h*>(st + offB + j * 16 * kKStep);
            fl[j] = *reinterpret_cast<const v8h*>(st + offB + BB + j * 16 * kKStep);
        }
        if (kt + 2 < nk) issue(kt + 2, sn);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {   // basis columns as the row operand: see the epilogue
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fh[j], fa[i], acc[i][j], 0, 0, 0);
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fl[j], fa[i], acc[i][j], 0, 0, 0);
            }
    };
    issue(0, 0);
    if (1 < nk) issue(1, 1);
    for (int kt = 0; kt < nk; kt += 3) {
        step(kt, 0, 2);
        if (kt + 1 < nk) step(kt + 1, 1, 0);
        if (kt + 2 < nk) step(kt + 2, 2, 1);
    }
    // acc[i][j]: token row lr of A block i, columns 4 lg .. 4 lg + 3 of basis block j
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int row = row0 + (wm * TM + i) * 16 + lr;
        if (row >= M) continue;
        const bool masked = state ? state[row] != 0 : false;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = col0 + (wn * TN + j) * 16 + lg * 4;
            if (col >= K) continue;
            float4 o;
            o.x = (!state || kept(col + 0, K, dm, du, masked)) ? acc[i][j][0] * kBasisUnscale : 0.0f;
            o.y = (!state || kept(col + 1, K, dm, du, masked)) ? acc[i][j][1] * kBasisUnscale : 0.0f;
            o.z = (!state || kept(col + 2, K, dm, du, masked)) ? acc[i][j][2] * kBasisUnscale : 0.0f;
            o.w = (!state || kept(col + 3, K, dm, du, masked)) ? acc[i][j][3] * kBasisUnscale : 0.0f;
            *reinterpret_cast<float4*>(Xp + (size_t)row * K + col) = o;
        }
    }
}

}  // namespace

hipError_t launch_split_basis(const float* P, int K, uint16_t* Ps, hipStream_t st) {
    hipLaunchKernelGGL(split_basis_kernel, dim3(K / 32, K / 32), dim3(256), 0, st, P, K, Ps);
    return hipGetLastError();
}

hipError_t launch_transform_fast(const uint16_t* X, const uint8_t* state, const uint16_t* Ps, int M, int K, int dm,
                                 int du, float* Xp, hipStream_t st) {
    const size_t t128 = (size_t)((M + 127) / 128) * (size_t)((K + 127) / 128);
    const size_t t64 = (size_t)((M + 63) / 64) * (size_t)((K + 63) / 64);
    if (t64 > 0x7fffffffu) return hipErrorInvalidConfiguration;
    // 128 x 128 tiles from one per CU on (1024 x 4096, 256 tiles: 73.6 us
    // against 99.8 us for 512 tiles of 64 x 128 and 111.6 us for 1024 of 64 x 64;
    // 1024 x 12288: 580 us against 862 and 1003)
    if (t128 >= 256) {
        hipLaunchKernelGGL((transform_mfma_kernel<2, 2, 4, 4>), dim3((unsigned)t128), dim3(256), 0, st, X, state, Ps,
                           M, K, dm, du, Xp);
    } else {
        hipLaunchKernelGGL((transform_mfma_kernel<2, 2, 2, 2>), dim3((unsigned)t64), dim3(256), 0, st, X, state, Ps,
                           M, K, dm, du, Xp);
    }
    return hipGetLastError();
}

}  // namespace sq
