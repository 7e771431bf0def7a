// W4A4 GEMM with dequantising epilogue (Eq. 13; Eq. 5):
//   acc[i][n] = sum_j qa[i][j] * qw[n][j]            (exact int32)
//   Y[i][n]   = fp16((float(acc) * s_a[i]) * s_w[n])
//
// gfx950 has no int4 matrix instruction, so packed nibbles feed the int8 MFMA
// v_mfma_i32_16x16x64_i8.  Unpacking keeps each nibble in the high half of a
// byte: for a packed dword w, (w << 4) & 0xF0F0F0F0 holds the even-k codes and
// w & 0xF0F0F0F0 the odd-k codes, each as the int8 value 16*q, with no sign
// extension step.  With both operands scaled by 16 the MFMA sums 256*qa*qw
// exactly (|sum| <= 256 * 64 * K < 2^31 for K <= 131072), and >> 8 recovers the
// integer dot product.  Even and odd k land in different registers; the same
// permutation is applied to A and W, and an integer sum does not depend on its
// order, so the result is the plain dot product.
//
// Tiling: a 256-thread workgroup owns a 128 x 128 output tile; its four waves
// each own 64 x 64 (4 x 4 MFMA tiles).  Packed int4 tiles (128 rows x 64 bytes
// per 128-k step) are staged through double-buffered LDS with the next tile
// prefetched into registers during compute, and unpacked to int8 operands as
// they leave LDS.  Short M splits K across workgroups; the int32 partial sums
// are then added exactly by a small epilogue kernel.
#include "sq_internal.hpp"

namespace sq {
namespace {

constexpr int kThreads = 256;
constexpr int kBM = 128, kBN = 128;
constexpr int kBKB = 64;                  // packed bytes per row per k step (128 codes)
constexpr int kRowB = kBKB + 16;          // padded LDS row

__device__ __forceinline__ v4i unpack_op(uint32_t w0, uint32_t w1) {
    v4i r;
    r[0] = (int)((w0 << 4) & 0xF0F0F0F0u);
    r[1] = (int)((w1 << 4) & 0xF0F0F0F0u);
    r[2] = (int)(w0 & 0xF0F0F0F0u);
    r[3] = (int)(w1 & 0xF0F0F0F0u);
    return r;
}

__device__ __forceinline__ void store_out(int row, int col, int v, const float* __restrict__ s_a,
                                          const float* __restrict__ s_w, uint16_t* __restrict__ Y,
                                          int32_t* __restrict__ acc, int N) {
    const size_t o = (size_t)row * N + col;
    if (acc) acc[o] = v;
    if (Y) Y[o] = f2h(((float)v * s_a[row]) * s_w[col]);
}

// SPLIT == false: full K, fused epilogue.  SPLIT == true: K range of blockIdx.z,
// raw int32 sums to part[z][M][N].
template <bool SPLIT>
__global__ __launch_bounds__(kThreads) void gemm_kernel(const uint8_t* __restrict__ Aq,
                                                        const float* __restrict__ s_a,
                                                        const uint8_t* __restrict__ Wq,
                                                        const float* __restrict__ s_w, int M, int N, int K,
                                                        int ktiles_per_split, uint16_t* __restrict__ Y,
                                                        int32_t* __restrict__ acc_out,
                                                        int32_t* __restrict__ part) {
    __shared__ __attribute__((aligned(16))) uint8_t sA[2][kBM * kRowB];
    __shared__ __attribute__((aligned(16))) uint8_t sB[2][kBN * kRowB];

    const int tid = threadIdx.x;
    const int lane = tid % kWave, wave = tid / kWave;
    const int wm = wave / 2, wn = wave % 2;
    const int row0 = blockIdx.y * kBM, col0 = blockIdx.x * kBN;
    const size_t ldb = (size_t)K / 2;         // bytes per packed row

    const int nk_total = (K + 2 * kBKB - 1) / (2 * kBKB);   // last step may be half full
    const int kt0 = SPLIT ? blockIdx.z * ktiles_per_split : 0;
    const int kt1 = SPLIT ? min(nk_total, kt0 + ktiles_per_split) : nk_total;

    // global -> register staging: each thread moves 2 x 16 B of A and of W per k step
    uint4 ra[2], rb[2];
    auto load = [&](int kt) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int e = tid + i * kThreads;
            const int r = e / 4, seg = e % 4;
            const size_t off = (size_t)kt * kBKB + seg * 16;
            ra[i] = make_uint4(0, 0, 0, 0);
            rb[i] = make_uint4(0, 0, 0, 0);
            if (off < ldb) {                  // K % 64 == 0: a 16-byte segment is all in or all out
                if (row0 + r < M) ra[i] = *reinterpret_cast<const uint4*>(Aq + (size_t)(row0 + r) * ldb + off);
                if (col0 + r < N) rb[i] = *reinterpret_cast<const uint4*>(Wq + (size_t)(col0 + r) * ldb + off);
            }
        }
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int e = tid + i * kThreads;
            const int r = e / 4, seg = e % 4;
            *reinterpret_cast<uint4*>(&sA[buf][r * kRowB + seg * 16]) = ra[i];
            *reinterpret_cast<uint4*>(&sB[buf][r * kRowB + seg * 16]) = rb[i];
        }
    };

    v4i acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    const int lr = lane % 16, lg = lane / 16;     // operand row within a 16-tile, k group
    if (kt0 < kt1) {
        load(kt0);
        stash(0);
        __syncthreads();
    }
    for (int kt = kt0; kt < kt1; ++kt) {
        const int buf = (kt - kt0) & 1;
        if (kt + 1 < kt1) load(kt + 1);
        // each lane reads 16 packed bytes (32 codes) per operand tile: its k group
        // holds bytes [16*lg, 16*lg + 16) of the 64-byte row slice
        uint4 fa[4], fb[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            fa[i] = *reinterpret_cast<const uint4*>(&sA[buf][(wm * 64 + i * 16 + lr) * kRowB + lg * 16]);
            fb[i] = *reinterpret_cast<const uint4*>(&sB[buf][(wn * 64 + i * 16 + lr) * kRowB + lg * 16]);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            v4i a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                a[i] = h ? unpack_op(fa[i].z, fa[i].w) : unpack_op(fa[i].x, fa[i].y);
                b[i] = h ? unpack_op(fb[i].z, fb[i].w) : unpack_op(fb[i].x, fb[i].y);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < kt1) {
            stash(buf ^ 1);
            __syncthreads();
        }
    }

    // D layout of the 16x16 tile: lane holds column (lane % 16), rows 4*(lane / 16) + r
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = col0 + wn * 64 + j * 16 + lr;
            if (col >= N) continue;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = row0 + wm * 64 + i * 16 + lg * 4 + r;
                if (row >= M) continue;
                const int v = acc[i][j][r] >> 8;
                if (SPLIT)
                    part[((size_t)blockIdx.z * M + row) * N + col] = v;
                else
                    store_out(row, col, v, s_a, s_w, Y, acc_out, N);
            }
        }
}

// Adds the split-K partial sums (exact int32) and applies the epilogue.
__global__ __launch_bounds__(kThreads) void splitk_epilogue(const int32_t* __restrict__ part, int splits,
                                                            const float* __restrict__ s_a,
                                                            const float* __restrict__ s_w, int M, int N,
                                                            uint16_t* __restrict__ Y, int32_t* __restrict__ acc) {
    const size_t total = (size_t)M * N;
    for (size_t e = (size_t)blockIdx.x * kThreads + threadIdx.x; e < total; e += (size_t)gridDim.x * kThreads) {
        int v = 0;
        for (int z = 0; z < splits; ++z) v += part[(size_t)z * total + e];
        store_out((int)(e / N), (int)(e % N), v, s_a, s_w, Y, acc, N);
    }
}

int choose_splits(int M, int N, int K) {
    const int tiles = ((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN);
    const int nk = (K + 2 * kBKB - 1) / (2 * kBKB);
    if (tiles >= 256) return 1;
    int s = (512 + tiles - 1) / tiles;
    s = s < nk ? s : nk;
    s = s < 32 ? s : 32;
    return s < 1 ? 1 : s;
}

}  // namespace

size_t gemm_workspace_bytes(int M, int N, int K) {
    const int s = choose_splits(M, N, K);
    return s > 1 ? (size_t)s * M * N * sizeof(int32_t) : 0;
}

hipError_t launch_gemm(const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w, int M, int N,
                       int K, uint16_t* Y, int32_t* acc, void* ws, hipStream_t st) {
    const int splits = choose_splits(M, N, K);
    const int nk = (K + 2 * kBKB - 1) / (2 * kBKB);
    dim3 grid((N + kBN - 1) / kBN, (M + kBM - 1) / kBM, 1);
    if (splits == 1) {
        hipLaunchKernelGGL(gemm_kernel<false>, grid, dim3(kThreads), 0, st, Aq, s_a, Wq, s_w, M, N, K, nk, Y, acc,
                           (int32_t*)nullptr);
        return hipGetLastError();
    }
    const int per = (nk + splits - 1) / splits;
    const int used = (nk + per - 1) / per;      // splits that own at least one k step
    grid.z = used;
    int32_t* part = static_cast<int32_t*>(ws);
    hipLaunchKernelGGL(gemm_kernel<true>, grid, dim3(kThreads), 0, st, Aq, s_a, Wq, s_w, M, N, K, per,
                       (uint16_t*)nullptr, (int32_t*)nullptr, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t total = (size_t)M * N;
    const int blocks = (int)((total + kThreads - 1) / kThreads < 4096 ? (total + kThreads - 1) / kThreads : 4096);
    hipLaunchKernelGGL(splitk_epilogue, dim3(blocks), dim3(kThreads), 0, st, part, used, s_a, s_w, M, N, Y, acc);
    return hipGetLastError();
}

}  // namespace sq
