// Exact W4A4 products on the FP6 matrix cores (the GEMM of Eq. 5 / Eq. 13).
//
// gfx950's f8f6f4 MFMA multiplies 6-bit floats; its 32 x 32 x 64 form does
// twice the work of the int8 32 x 32 x 32 form in about the same issue time.  In
// the e3m2 format (sign, 3 exponent bits with bias 3, 2 mantissa bits: OCP
// Microscaling Formats v1.0, FP6 E3M2) every int4 code -8..7 is exact, every
// product of two codes is an integer of magnitude at most 64, and every partial
// sum of at most 131072 such products is an integer below 2^24, so the fp32
// accumulation inside and across the MFMAs is exact in any order: the fp32
// result is the int32 dot product.  The epilogue is the W4A4 GEMM's.
//
// Operand layout (A and W alike).  Per row, the K codes, padded with zero codes
// to whole blocks of 128, take 96 bytes per block.  Chunk c of block b (codes
// 128 b + 32 c .. + 31, the k range of one MFMA lane group) is the 192-bit
// little-endian string with code j in bits 6 j .. 6 j + 5; its bytes 0..15 sit
// at 96 b + 16 c and its bytes 16..23 at 96 b + 64 + 8 c, so a lane fetches its
// fragment with one 16-byte and one 8-byte LDS read.
//
// Kernel: the W4A4 tile kernel's three-stage direct-to-LDS pipeline, a k step
// being one block of 128 codes (two 32 x 32 x 64 MFMAs per 32 x 32 block).  Per
// stage and operand the 16-byte parts form a [rows][64 B] tile XOR-swizzled by
// 16-byte chunk ((row >> 1) & 3) and the 8-byte parts a [rows][32 B] tile whose
// two 16-byte halves swap on every other group of 8 rows ((row >> 3) & 1); both
// make the fragment reads conflict-free.  No unpacking: the MFMA takes the
// fragments as they are.
#include "tile_common.hpp"

namespace sq {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kBlock = 128;          // codes per k step
constexpr int kBlockBytes = 96;
constexpr int kFmtE3M2 = 3;          // operand format selector of the f8f6f4 MFMA

// e3m2 pattern of a two's complement int4 nibble: |q| = 2^e (1 + m/4) with
// exponent field e + 3; zero is the all-zero pattern.
__device__ __forceinline__ uint32_t e3m2_of_nibble(uint32_t n) {
    const uint32_t neg = n >> 3;
    const uint32_t a = neg ? 16u - n : n;                 // 0..8
    if (a == 0) return 0;
    const uint32_t e = 31u - __builtin_clz(a);            // floor(log2 a)
    const uint32_t m = ((a << 2) >> e) & 3u;              // a = 2^e (4 + m) / 4
    return (neg << 5) | ((e + 3u) << 2) | m;
}

// One thread per (row, block, chunk): 32 packed codes in, 24 bytes out.
__global__ __launch_bounds__(256) void codes_to_fp6_kernel(const uint8_t* __restrict__ src, int R, int K,
                                                           uint8_t* __restrict__ dst) {
    const int nblk = (K + kBlock - 1) / kBlock;
    const size_t t = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= (size_t)R * nblk * 4) return;
    const int c = (int)(t % 4);
    const size_t rb = t / 4;
    const int b = (int)(rb % nblk);
    const size_t r = rb / nblk;
    const int k0 = b * kBlock + 32 * c;                   // K % 64 == 0: a chunk is all in or all out
    uint4 in = make_uint4(0, 0, 0, 0);
    if (k0 < K) in = *reinterpret_cast<const uint4*>(src + r * (size_t)(K / 2) + k0 / 2);
    const uint32_t w[4] = {in.x, in.y, in.z, in.w};
    uint32_t o[6] = {0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 32; ++j) {
        const uint32_t p = e3m2_of_nibble((w[j / 8] >> (4 * (j % 8))) & 15u);
        const int bit = 6 * j;
        o[bit / 32] |= p << (bit % 32);
        if (bit % 32 > 26) o[bit / 32 + 1] |= p >> (32 - bit % 32);
    }
    uint8_t* row = dst + r * (size_t)(nblk * kBlockBytes) + b * kBlockBytes;
    *reinterpret_cast<uint4*>(row + 16 * c) = make_uint4(o[0], o[1], o[2], o[3]);
    *reinterpret_cast<uint2*>(row + 64 + 8 * c) = make_uint2(o[4], o[5]);
}

template <int WM, int WN, int TM, int TN, int OCC>
__global__ __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(OCC))) void gemm_fp6_kernel(
    const uint8_t* __restrict__ A6, const float* __restrict__ s_a, const uint8_t* __restrict__ W6,
    const float* __restrict__ s_w, int M, int N, int K, uint16_t* __restrict__ Y, int32_t* __restrict__ acc_out) {
    constexpr int NW = WM * WN;
    constexpr int BM = 32 * WM * TM, BN = 32 * WN * TN;
    constexpr int PA = BM * 64, QA = BM * 32, PB = BN * 64, QB = BN * 32;   // bytes of one stage
    constexpr int SB = PA + QA + PB + QB;
    constexpr int LPA = PA / 1024 / NW, LQA = QA / 1024 / NW, LPB = PB / 1024 / NW, LQB = QB / 1024 / NW;
    static_assert(LPA * NW * 1024 == PA && LQA * NW * 1024 == QA && LPB * NW * 1024 == PB &&
                      LQB * NW * 1024 == QB && LQA > 0 && LQB > 0,
                  "stage loads must divide evenly");
    constexpr int LOADS = LPA + LQA + LPB + LQB;
    __shared__ __attribute__((aligned(16))) uint8_t sm[3 * SB];

    const int tid = threadIdx.x;
    const int lane = tid % kWave, wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int wm = wave / WN, wn = wave % WN;
    const int nk = (K + kBlock - 1) / kBlock;
    const uint32_t ldb = (uint32_t)nk * kBlockBytes;
    const u32x4 rA = sgpr_rsrc(A6, (uint32_t)M * ldb);
    const u32x4 rW = sgpr_rsrc(W6, (uint32_t)N * ldb);
    auto swz = [](int r) { return (r >> 1) & 3; };      // 16-byte chunk swizzle of a 64-byte row
    auto qsw = [](int r) { return (r >> 3) & 1; };      // half swap of a 32-byte row

    int rt, ct;
    xcd_tile(blockIdx.x, (M + BM - 1) / BM, (N + BN - 1) / BN, 8, rt, ct);
    const int row0 = rt * BM, col0 = ct * BN;

    // source offsets: a 16-byte-part load covers 16 rows x 4 chunks (tile row
    // 16 u' + lane / 4 takes, at slot lane % 4, chunk (lane % 4) ^ swz(row)); an
    // 8-byte-part load covers 32 rows x 2 halves (row 32 u' + lane / 2, slot
    // lane % 2 holds half (lane % 2) ^ qsw(row))
    uint32_t opa[LPA], oqa[LQA], opb[LPB], oqb[LQB];
#pragma unroll
    for (int u = 0; u < LPA; ++u) {
        const int r = 16 * (wave * LPA + u) + lane / 4;
        opa[u] = row0 + r < M ? (uint32_t)(row0 + r) * ldb + 16 * ((lane % 4) ^ swz(r)) : kOOB;
    }
#pragma unroll
    for (int u = 0; u < LQA; ++u) {
        const int r = 32 * (wave * LQA + u) + lane / 2;
        oqa[u] = row0 + r < M ? (uint32_t)(row0 + r) * ldb + 64 + 16 * ((lane % 2) ^ qsw(r)) : kOOB;
    }
#pragma unroll
    for (int u = 0; u < LPB; ++u) {
        const int r = 16 * (wave * LPB + u) + lane / 4;
        opb[u] = col0 + r < N ? (uint32_t)(col0 + r) * ldb + 16 * ((lane % 4) ^ swz(r)) : kOOB;
    }
#pragma unroll
    for (int u = 0; u < LQB; ++u) {
        const int r = 32 * (wave * LQB + u) + lane / 2;
        oqb[u] = col0 + r < N ? (uint32_t)(col0 + r) * ldb + 64 + 16 * ((lane % 2) ^ qsw(r)) : kOOB;
    }
    auto issue = [&](int kt, int stage) {
        uint8_t* s = sm + stage * SB;
        const uint32_t ko = (uint32_t)kt * kBlockBytes;
#pragma unroll
        for (int u = 0; u < LPA; ++u) dma16(rA, lds_addr(s + (wave * LPA + u) * 1024), opa[u] + ko);
#pragma unroll
        for (int u = 0; u < LQA; ++u) dma16(rA, lds_addr(s + PA + (wave * LQA + u) * 1024), oqa[u] + ko);
#pragma unroll
        for (int u = 0; u < LPB; ++u) dma16(rW, lds_addr(s + PA + QA + (wave * LPB + u) * 1024), opb[u] + ko);
#pragma unroll
        for (int u = 0; u < LQB; ++u)
            dma16(rW, lds_addr(s + PA + QA + PB + (wave * LQB + u) * 1024), oqb[u] + ko);
    };

    v16f acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    // lane (r, g) = (lane % 32, lane / 32) reads row r of each 32-row block, chunks
    // g and g + 2; MFMA s (K = 64) takes chunk g + 2 s, i.e. codes 64 s .. 64 s + 63
    const int lr = lane % 32, lg = lane / 32;
    int fp[2], fq[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int c = lg + 2 * s;
        fp[s] = (c ^ swz(lr)) * 16;
        fq[s] = 16 * ((c >> 1) ^ qsw(lr)) + 8 * (c & 1);
    }
    const int rowA = (wm * TM) * 32 + lr, rowB = (wn * TN) * 32 + lr;
    auto frag = [](const uint8_t* p16, const uint8_t* p8) {
        const v4i x = *reinterpret_cast<const v4i*>(p16);
        const int2 y = *reinterpret_cast<const int2*>(p8);
        return v8i{x[0], x[1], x[2], x[3], y.x, y.y, 0, 0};
    };
    auto mma = [&](const uint8_t* st) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            v8i fb[TN];
#pragma unroll
            for (int j = 0; j < TN; ++j)
                fb[j] = frag(st + PA + QA + (rowB + 32 * j) * 64 + fp[s], st + PA + QA + PB + (rowB + 32 * j) * 32 + fq[s]);
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const v8i fa = frag(st + (rowA + 32 * i) * 64 + fp[s], st + PA + (rowA + 32 * i) * 32 + fq[s]);
#pragma unroll
                for (int j = 0; j < TN; ++j)   // weights as the row operand, as in the int4 kernel
                    acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fb[j], fa, acc[i][j], kFmtE3M2,
                                                                                kFmtE3M2, 0, 0, 0, 0);
            }
        }
    };
    auto step = [&](int kt, int sc, int sn) {
        asm volatile("" ::: "memory");
        if (kt + 1 < nk)
            wait_vm<LOADS>();                            // this wave's loads of step kt are done
        else
            wait_vm<0>();
        __builtin_amdgcn_s_barrier();                    // ... and every wave's
        asm volatile("" ::: "memory");
        // the stage step kt - 1 used is free: every wave finished its reads of it
        // (they fed MFMAs issued before that wave reached the barrier above)
        if (kt + 2 < nk) issue(kt + 2, sn);
        mma(sm + sc * SB);
    };
    issue(0, 0);
    if (1 < nk) issue(1, 1);
    for (int kt = 0; kt < nk; kt += 3) {
        step(kt, 0, 2);
        if (kt + 1 < nk) step(kt + 1, 1, 0);
        if (kt + 2 < nk) step(kt + 2, 2, 1);
    }
    // acc[i][j] is the 32 x 32 block W_j A_i^T: element 4 q + e of this lane is
    // output column 8 q + 4 lg + e of W block j for token row lr of A block i.
    // All of the lane's row and weight scales are requested before any is used
    // (indices clamped into range, so no branch separates the loads).
    float sa[TM];
    float4 sw[TN][4];
    if (Y) {
#pragma unroll
        for (int i = 0; i < TM; ++i) sa[i] = s_a[min(row0 + (wm * TM + i) * 32 + lr, M - 1)];
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                sw[j][q] = *reinterpret_cast<const float4*>(
                    s_w + min(col0 + (wn * TN + j) * 32 + 8 * q + 4 * lg, N - 4));
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int row = row0 + (wm * TM + i) * 32 + lr;
        if (row >= M) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int col = col0 + (wn * TN + j) * 32 + 8 * q + 4 * lg;   // N % 8 == 0: all four or none
                if (col >= N) continue;
                // the fp32 sums are exact integers below 2^24 in magnitude
                const int v0 = (int)acc[i][j][4 * q], v1 = (int)acc[i][j][4 * q + 1];
                const int v2 = (int)acc[i][j][4 * q + 2], v3 = (int)acc[i][j][4 * q + 3];
                const size_t o = (size_t)row * N + col;
                if (acc_out) *reinterpret_cast<int4*>(acc_out + o) = make_int4(v0, v1, v2, v3);
                if (Y) {
                    const float4 w = sw[j][q];
                    const uint32_t y0 = f2h(((float)v0 * sa[i]) * w.x), y1 = f2h(((float)v1 * sa[i]) * w.y);
                    const uint32_t y2 = f2h(((float)v2 * sa[i]) * w.z), y3 = f2h(((float)v3 * sa[i]) * w.w);
                    *reinterpret_cast<uint2*>(Y + o) = make_uint2(y0 | (y1 << 16), y2 | (y3 << 16));
                }
            }
    }
}

template <int WM, int WN, int TM, int TN, int OCC>
hipError_t launch_fp6_tiled(const uint8_t* A6, const float* s_a, const uint8_t* W6, const float* s_w, int M, int N,
                            int K, uint16_t* Y, int32_t* acc, hipStream_t st) {
    constexpr int BM = 32 * WM * TM, BN = 32 * WN * TN;
    const size_t tiles = (size_t)((M + BM - 1) / BM) * (size_t)((N + BN - 1) / BN);
    if (tiles > 0x7fffffffu) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((gemm_fp6_kernel<WM, WN, TM, TN, OCC>), dim3((unsigned)tiles), dim3(64 * WM * WN), 0, st, A6,
                       s_a, W6, s_w, M, N, K, Y, acc);
    return hipGetLastError();
}

}  // namespace

size_t fp6_row_bytes(int K) { return (size_t)((K + kBlock - 1) / kBlock) * kBlockBytes; }

hipError_t launch_codes_to_fp6(const uint8_t* src, int R, int K, uint8_t* dst, hipStream_t st) {
    const size_t threads = (size_t)R * ((K + kBlock - 1) / kBlock) * 4;
    const size_t blocks = (threads + 255) / 256;
    if (blocks > 0x7fffffffu) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(codes_to_fp6_kernel, dim3((unsigned)blocks), dim3(256), 0, st, src, R, K, dst);
    return hipGetLastError();
}

// Plan: 256 x 256 tiles (eight waves of 64 x 128) when that gives >= 512 tiles,
// else 128 x 128 (four waves of 64 x 64).
hipError_t launch_gemm_fp6(const uint8_t* A6, const float* s_a, const uint8_t* W6, const float* s_w, int M, int N,
                           int K, uint16_t* Y, int32_t* acc, hipStream_t st) {
    const size_t t256 = (size_t)((M + 255) / 256) * (size_t)((N + 255) / 256);
    if (t256 >= 512) return launch_fp6_tiled<4, 2, 2, 4, 1>(A6, s_a, W6, s_w, M, N, K, Y, acc, st);
    return launch_fp6_tiled<2, 2, 2, 2, 2>(A6, s_a, W6, s_w, M, N, K, Y, acc, st);
}

}  // namespace sq
