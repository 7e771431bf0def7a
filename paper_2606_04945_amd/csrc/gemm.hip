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
// Tiling (template): WM x WN waves, each owning TM x TN MFMA tiles of 16 x 16, so
// a workgroup owns (16 WM TM) x (16 WN TN) outputs.  Per k step (128 codes) the
// workgroup reads 64 packed bytes of every row of both operands with raw buffer
// loads (out-of-range reads return 0, so no predicates in the loop), prefetching
// the next step into registers during compute, and stages them through
// double-buffered LDS.  UNPACK selects where nibbles become int8: when staged
// (LDS holds int8 rows, each tile unpacked once per workgroup) or as fragments
// leave LDS (LDS holds packed rows, each wave unpacks what it reads).  LDS rows
// are XOR-swizzled by 16-byte chunk so the row-wise fragment reads and the
// segment-wise stores are free of bank conflicts.  Short M splits K across
// workgroups; the int32 partial sums are then added exactly by a small kernel.
//
// BITS = 8 is the W8A8 variant (App. D): codes are int8 already, so the same
// tiles feed the MFMA straight from LDS with no unpacking and no scaling.
#include "sq_internal.hpp"

namespace sq {
namespace {

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

constexpr int kKB = 64;                              // bytes per row per k step (128 4-bit / 64 8-bit codes)

// MFMA operand for step h of a lane's 16-byte fragment: two int4 halves unpacked
// (4-bit) or the int8 codes themselves (8-bit, one step)
template <int BITS>
__device__ __forceinline__ v4i operand(const v4i& raw, int h) {
    if (BITS == 8) return raw;
    return h ? unpack_op(raw[2], raw[3]) : unpack_op(raw[0], raw[1]);
}
template <int BITS>
__device__ __forceinline__ int acc_value(int raw) {   // 4-bit operands carry a factor 16 each
    return BITS == 8 ? raw : raw >> 8;
}

template <int WM, int WN, int TM, int TN, bool UNPACK>
struct GemmCfg {
    static constexpr int NT = 64 * WM * WN;          // threads
    static constexpr int BM = 16 * WM * TM;          // rows of A per tile
    static constexpr int BN = 16 * WN * TN;          // rows of W (output columns) per tile
    static constexpr int SEG = kKB / 16;             // 16-byte packed segments per row per k step
    static constexpr int AV = BM * SEG / NT;         // segments per thread
    static constexpr int BV = BN * SEG / NT;
    static constexpr int RB = UNPACK ? 2 * kKB : kKB;   // LDS row bytes per k step
    static constexpr int CH = RB / 16;                  // 16-byte chunks per LDS row
    // chunk c of LDS row r sits at chunk (c ^ swz(r)), swz(r) = index of the
    // 128-byte line the row starts in, modulo the chunks per row: any eight
    // consecutive rows then touch distinct 16-byte bank groups
    static __device__ __forceinline__ int chunk(int r, int c) { return c ^ ((r / (128 / RB)) & (CH - 1)); }
};

// Raw buffer resource over [base, base + bytes): loads outside it return 0, which
// is how rows past M (or N) and the unused half of a last k step read as zeros.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

constexpr uint32_t kOOB = 0x80000000u;   // an offset past any buffer this kernel builds

// SPLIT == false: full K, fused epilogue.  SPLIT == true: K range of blockIdx.z,
// raw int32 sums to part[z][M][N].
template <int WM, int WN, int TM, int TN, bool UNPACK, bool SPLIT, int SCHED = 0, int BITS = 4>
__global__ __launch_bounds__(64 * WM * WN) void gemm_kernel(const uint8_t* __restrict__ Aq,
                                                           const float* __restrict__ s_a,
                                                           const uint8_t* __restrict__ Wq,
                                                           const float* __restrict__ s_w, int M, int N, int K,
                                                           int ksteps_per_split, uint16_t* __restrict__ Y,
                                                           int32_t* __restrict__ acc_out,
                                                           int32_t* __restrict__ part) {
    using C = GemmCfg<WM, WN, TM, TN, UNPACK>;
    static_assert(C::BM * C::SEG % C::NT == 0 && C::BN * C::SEG % C::NT == 0, "tile loads must divide evenly");
    static_assert(BITS == 4 || (BITS == 8 && !UNPACK && SCHED), "8-bit codes use the one-fragment loop");
    __shared__ __attribute__((aligned(16))) uint8_t sA[2][C::BM * C::RB];
    __shared__ __attribute__((aligned(16))) uint8_t sB[2][C::BN * C::RB];

    const int tid = threadIdx.x;
    const int lane = tid % kWave, wave = tid / kWave;
    const int wm = wave / WN, wn = wave % WN;
    const int row0 = blockIdx.y * C::BM, col0 = blockIdx.x * C::BN;
    const uint32_t ldb = (uint32_t)K * BITS / 8;         // bytes per row of codes

    const int nk_total = (int)((ldb + kKB - 1) / kKB);   // the last step may be half empty
    const int nk_full = (int)(ldb / kKB);                // steps with every byte in range
    const int kt0 = SPLIT ? blockIdx.z * ksteps_per_split : 0;
    const int kt1 = SPLIT ? min(nk_total, kt0 + ksteps_per_split) : nk_total;

    const __amdgpu_buffer_rsrc_t rA = make_rsrc(Aq, (uint32_t)M * ldb);
    const __amdgpu_buffer_rsrc_t rW = make_rsrc(Wq, (uint32_t)N * ldb);
    // this thread's 16-byte segments: tile row e / SEG, segment e % SEG
    uint32_t oa[C::AV], ow[C::BV];
#pragma unroll
    for (int i = 0; i < C::AV; ++i) {
        const int e = tid + i * C::NT, r = e / C::SEG;
        oa[i] = row0 + r < M ? (uint32_t)(row0 + r) * ldb + (e % C::SEG) * 16 : kOOB;
    }
#pragma unroll
    for (int i = 0; i < C::BV; ++i) {
        const int e = tid + i * C::NT, r = e / C::SEG;
        ow[i] = col0 + r < N ? (uint32_t)(col0 + r) * ldb + (e % C::SEG) * 16 : kOOB;
    }

    v4i ra[C::AV], rb[C::BV];
    auto load = [&](int kt, bool tail) {
        const uint32_t ko = (uint32_t)kt * kKB;
#pragma unroll
        for (int i = 0; i < C::AV; ++i) {
            const int seg = ((tid + i * C::NT) % C::SEG) * 16;
            const uint32_t o = (tail && ko + seg >= ldb) ? kOOB : oa[i] + ko;
            ra[i] = __builtin_amdgcn_raw_buffer_load_b128(rA, (int)o, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < C::BV; ++i) {
            const int seg = ((tid + i * C::NT) % C::SEG) * 16;
            const uint32_t o = (tail && ko + seg >= ldb) ? kOOB : ow[i] + ko;
            rb[i] = __builtin_amdgcn_raw_buffer_load_b128(rW, (int)o, 0, 0);
        }
    };
    auto load_step = [&](int kt) {
        if (kt < nk_full)
            load(kt, false);
        else
            load(kt, true);
    };
    // packed segment s of row r -> LDS; with UNPACK its two int8 halves (MFMA steps
    // h = 0, 1 of k group s) go to chunks 2s and 2s + 1
    auto put = [&](uint8_t* base, int e, const v4i& v) {
        const int r = e / C::SEG, s = e % C::SEG;
        uint8_t* row = base + r * C::RB;
        if (UNPACK) {
            *reinterpret_cast<v4i*>(row + C::chunk(r, 2 * s) * 16) = unpack_op(v[0], v[1]);
            *reinterpret_cast<v4i*>(row + C::chunk(r, 2 * s + 1) * 16) = unpack_op(v[2], v[3]);
        } else {
            *reinterpret_cast<v4i*>(row + C::chunk(r, s) * 16) = v;
        }
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int i = 0; i < C::AV; ++i) put(sA[buf], tid + i * C::NT, ra[i]);
#pragma unroll
        for (int i = 0; i < C::BV; ++i) put(sB[buf], tid + i * C::NT, rb[i]);
    };

    v4i acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    const int lr = lane % 16, lg = lane / 16;            // row within a 16-tile, k group
    // a lane's fragment rows differ by multiples of 16, so swz(row) == swz(lr)
    const int offA = ((wm * TM) * 16 + lr) * C::RB;
    const int offB = ((wn * TN) * 16 + lr) * C::RB;
    if (kt0 < kt1) {
        load_step(kt0);
        stash(0);
        __syncthreads();
    }
    for (int kt = kt0; kt < kt1; ++kt) {
        const int buf = (kt - kt0) & 1;
        if (kt + 1 < kt1) load_step(kt + 1);
        if (SCHED && !UNPACK) {
            // one 16-byte fragment per tile per k step; with 4-bit codes both MFMA
            // steps are unpacked and the scheduler interleaves the second step's
            // unpacking with the first step's MFMAs
            constexpr int SUBS = BITS == 4 ? 2 : 1;
            v4i fa[TM], fb[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                fa[i] = *reinterpret_cast<const v4i*>(&sA[buf][offA + i * 16 * C::RB + C::chunk(lr, lg) * 16]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                fb[j] = *reinterpret_cast<const v4i*>(&sB[buf][offB + j * 16 * C::RB + C::chunk(lr, lg) * 16]);
#pragma unroll
            for (int h = 0; h < SUBS; ++h) {
                v4i a[TM], b[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i) a[i] = operand<BITS>(fa[i], h);
#pragma unroll
                for (int j = 0; j < TN; ++j) b[j] = operand<BITS>(fb[j], h);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[i], b[j], acc[i][j], 0, 0, 0);
            }
            constexpr int nmma = TM * TN;
            __builtin_amdgcn_sched_group_barrier(0x100, TM + TN, 0);         // fragment reads
            if (BITS == 4) {
                constexpr int nvalu = 6 * (TM + TN);                         // one MFMA step's unpacking
                constexpr int per = (nvalu + nmma - 1) / nmma;
                __builtin_amdgcn_sched_group_barrier(0x002, nvalu, 0);       // step-0 unpack
#pragma unroll
                for (int q = 0; q < nmma; ++q) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);       // step-0 MFMA
                    __builtin_amdgcn_sched_group_barrier(0x002, per, 0);     // step-1 unpack
                }
            }
            __builtin_amdgcn_sched_group_barrier(0x008, nmma, 0);            // remaining MFMAs
        } else {
            // k group lg of a lane covers packed bytes [16 lg, 16 lg + 16) of the row
            // slice; MFMA step h uses 8 of them (same bytes for A and W)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                v4i a[TM], b[TN];
                if (UNPACK) {
#pragma unroll
                    for (int i = 0; i < TM; ++i)
                        a[i] = *reinterpret_cast<const v4i*>(&sA[buf][offA + i * 16 * C::RB +
                                                                       C::chunk(lr, 2 * lg + h) * 16]);
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        b[j] = *reinterpret_cast<const v4i*>(&sB[buf][offB + j * 16 * C::RB +
                                                                       C::chunk(lr, 2 * lg + h) * 16]);
                } else {
#pragma unroll
                    for (int i = 0; i < TM; ++i) {
                        const uint2 u = *reinterpret_cast<const uint2*>(&sA[buf][offA + i * 16 * C::RB +
                                                                                 C::chunk(lr, lg) * 16 + 8 * h]);
                        a[i] = unpack_op(u.x, u.y);
                    }
#pragma unroll
                    for (int j = 0; j < TN; ++j) {
                        const uint2 u = *reinterpret_cast<const uint2*>(&sB[buf][offB + j * 16 * C::RB +
                                                                                 C::chunk(lr, lg) * 16 + 8 * h]);
                        b[j] = unpack_op(u.x, u.y);
                    }
                }
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[i], b[j], acc[i][j], 0, 0, 0);
            }
        }
        if (kt + 1 < kt1) {
            stash(buf ^ 1);
            __syncthreads();
        }
    }

    // D layout of a 16x16 tile: lane holds column (lane % 16), rows 4*(lane / 16) + r
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = col0 + (wn * TN + j) * 16 + lr;
            if (col >= N) continue;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = row0 + (wm * TM + i) * 16 + lg * 4 + r;
                if (row >= M) continue;
                const int v = acc_value<BITS>(acc[i][j][r]);
                if (SPLIT)
                    part[((size_t)blockIdx.z * M + row) * N + col] = v;
                else
                    store_out(row, col, v, s_a, s_w, Y, acc_out, N);
            }
        }
}

// Short M (<= 64 tokens): the weights are streamed once and each is used by at
// most 64 rows, so the kernel is bound by HBM bandwidth, not by the MFMA.  No
// LDS and no barriers: each wave owns 16 output columns and walks its K range,
// loading its W rows and the (L2-resident) activation rows straight into MFMA
// operand registers with raw buffer loads, U k steps in flight per batch.  Lane
// (c, g) reads bytes [16 g, 16 g + 16) of the 64-byte slice of row c (W) or of
// the activation row, exactly as the tiled kernel's fragments.
template <int TM, int U, bool SPLIT, int BITS = 4>
__global__ __launch_bounds__(256) void gemm_skinny_kernel(const uint8_t* __restrict__ Aq,
                                                          const float* __restrict__ s_a,
                                                          const uint8_t* __restrict__ Wq,
                                                          const float* __restrict__ s_w, int M, int N, int K,
                                                          int ksteps_per_split, uint16_t* __restrict__ Y,
                                                          int32_t* __restrict__ acc_out,
                                                          int32_t* __restrict__ part) {
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int lr = lane % 16, lg = lane / 16;
    const int col0 = (blockIdx.x * 4 + wave) * 16;
    if (col0 >= N) return;                                   // whole wave past N: nothing to do
    const uint32_t ldb = (uint32_t)K * BITS / 8;
    const int nk_total = (int)((ldb + kKB - 1) / kKB);
    const int kt0 = SPLIT ? blockIdx.z * ksteps_per_split : 0;
    const int kt1 = SPLIT ? min(nk_total, kt0 + ksteps_per_split) : nk_total;
    const __amdgpu_buffer_rsrc_t rA = make_rsrc(Aq, (uint32_t)M * ldb);
    const __amdgpu_buffer_rsrc_t rW = make_rsrc(Wq, (uint32_t)N * ldb);
    const uint32_t seg = 16 * lg;
    const uint32_t ow = col0 + lr < N ? (uint32_t)(col0 + lr) * ldb + seg : kOOB;
    uint32_t oa[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) oa[i] = 16 * i + lr < M ? (uint32_t)(16 * i + lr) * ldb + seg : kOOB;

    v4i acc[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) acc[i] = v4i{0, 0, 0, 0};
    // two register batches of U k steps: batch b + 1 is in flight while batch b is
    // multiplied (steps past the split or the row read as zeros)
    auto issue = [&](int kb, v4i (&w)[U], v4i (&a)[U][TM]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t ko = (uint32_t)(kb + u) * kKB;
            const bool in = kb + u < kt1 && ko + seg < ldb;
            w[u] = __builtin_amdgcn_raw_buffer_load_b128(rW, (int)(in ? ow + ko : kOOB), 0, 0);
#pragma unroll
            for (int i = 0; i < TM; ++i)
                a[u][i] = __builtin_amdgcn_raw_buffer_load_b128(rA, (int)(in ? oa[i] + ko : kOOB), 0, 0);
        }
    };
    auto compute = [&](const v4i (&w)[U], const v4i (&a)[U][TM]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int h = 0; h < (BITS == 4 ? 2 : 1); ++h) {
                const v4i b = operand<BITS>(w[u], h);
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    acc[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(operand<BITS>(a[u][i], h), b, acc[i], 0, 0, 0);
            }
        }
    };
    v4i w0[U], a0[U][TM], w1[U], a1[U][TM];
    issue(kt0, w0, a0);
    for (int kb = kt0; kb < kt1; kb += 2 * U) {
        issue(kb + U, w1, a1);
        __builtin_amdgcn_sched_barrier(0);
        compute(w0, a0);
        if (kb + U >= kt1) break;
        issue(kb + 2 * U, w0, a0);
        __builtin_amdgcn_sched_barrier(0);
        compute(w1, a1);
    }
    const int col = col0 + lr;
    if (col >= N) return;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * i + 4 * lg + r;
            if (row >= M) continue;
            const int v = acc_value<BITS>(acc[i][r]);
            if (SPLIT)
                part[((size_t)blockIdx.z * M + row) * N + col] = v;
            else
                store_out(row, col, v, s_a, s_w, Y, acc_out, N);
        }
}

// Adds the split-K partial sums (exact int32) and applies the epilogue.
__global__ __launch_bounds__(256) void splitk_epilogue(const int32_t* __restrict__ part, int splits,
                                                       const float* __restrict__ s_a,
                                                       const float* __restrict__ s_w, int M, int N,
                                                       uint16_t* __restrict__ Y, int32_t* __restrict__ acc) {
    const size_t total = (size_t)M * N;
    for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (size_t)gridDim.x * 256) {
        int v = 0;
        for (int z = 0; z < splits; ++z) v += part[(size_t)z * total + e];
        store_out((int)(e / N), (int)(e % N), v, s_a, s_w, Y, acc, N);
    }
}

// A launch plan: tile shape and K split.
struct Plan {
    int cfg;       // 0: 128 x 128, 1: 64 x 128, 2: 64 x 64, 3: skinny (see launch_gemm)
    int bm, bn;
    int splits;    // K split count actually used (1 = fused epilogue)
    int per;       // k steps per split
};

Plan make_plan(int M, int N, int K, int bm, int bn, int want_splits, int bits = 4) {
    (void)M;
    (void)N;
    Plan p;
    p.cfg = -1;
    p.bm = bm;
    p.bn = bn;
    const int nk = (K * bits / 8 + kKB - 1) / kKB;
    const int s = want_splits < 1 ? 1 : (want_splits > nk ? nk : want_splits);
    p.per = (nk + s - 1) / s;
    p.splits = (nk + p.per - 1) / p.per;
    return p;
}

template <int TM, int U, int BITS = 4>
hipError_t launch_skinny(const Plan& p, const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w,
                         int M, int N, int K, uint16_t* Y, int32_t* acc, int32_t* part, hipStream_t st) {
    dim3 grid((N + 63) / 64, 1, p.splits);
    if (p.splits == 1) {
        hipLaunchKernelGGL((gemm_skinny_kernel<TM, U, false, BITS>), grid, dim3(256), 0, st, Aq, s_a, Wq, s_w, M, N, K,
                           p.per, Y, acc, (int32_t*)nullptr);
    } else {
        hipLaunchKernelGGL((gemm_skinny_kernel<TM, U, true, BITS>), grid, dim3(256), 0, st, Aq, s_a, Wq, s_w, M, N, K,
                           p.per, (uint16_t*)nullptr, (int32_t*)nullptr, part);
    }
    return hipGetLastError();
}

template <int WM, int WN, int TM, int TN, bool UNPACK, int SCHED = 0, int BITS = 4>
hipError_t launch_cfg(const Plan& p, const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w,
                      int M, int N, int K, uint16_t* Y, int32_t* acc, int32_t* part, hipStream_t st) {
    dim3 grid((N + p.bn - 1) / p.bn, (M + p.bm - 1) / p.bm, p.splits);
    dim3 block(64 * WM * WN);
    if (p.splits == 1) {
        hipLaunchKernelGGL((gemm_kernel<WM, WN, TM, TN, UNPACK, false, SCHED, BITS>), grid, block, 0, st, Aq, s_a, Wq, s_w, M,
                           N, K, p.per, Y, acc, (int32_t*)nullptr);
    } else {
        hipLaunchKernelGGL((gemm_kernel<WM, WN, TM, TN, UNPACK, true, SCHED, BITS>), grid, block, 0, st, Aq, s_a, Wq, s_w, M, N,
                           K, p.per, (uint16_t*)nullptr, (int32_t*)nullptr, part);
    }
    return hipGetLastError();
}

hipError_t finish_split(const Plan& p, int32_t* part, const float* s_a, const float* s_w, int M, int N, uint16_t* Y,
                        int32_t* acc, hipStream_t st) {
    if (p.splits == 1) return hipSuccess;
    const size_t total = (size_t)M * N;
    const int blocks = (int)((total + 255) / 256 < 4096 ? (total + 255) / 256 : 4096);
    hipLaunchKernelGGL(splitk_epilogue, dim3(blocks), dim3(256), 0, st, part, p.splits, s_a, s_w, M, N, Y, acc);
    return hipGetLastError();
}

// The production plan (from measured sweeps on MI355X):
//  - M <= 16: the skinny kernel (weight streaming, K split only for narrow N);
//  - M <= 64: 64 x 64 tiles and a K split up to ~512 workgroups;
//  - at least 512 tiles of 128 x 128: 128 x 128 (four waves of 64 x 64);
//  - otherwise 64 x 128 (four waves of 64 x 32), split along K below 512 tiles.
Plan choose_plan(int M, int N, int K, int bits) {
    const int nk = (K * bits / 8 + kKB - 1) / kKB;
    auto splits_for = [&](int tiles) {
        int s = tiles >= 512 ? 1 : (512 + tiles - 1) / tiles;
        const int cap = nk / 4 > 1 ? nk / 4 : 1;       // keep at least 4 k steps per split
        s = s < cap ? s : cap;
        return s < 32 ? s : 32;
    };
    Plan p;
    if (M <= 16) {
        // skinny kernel: one wave per 16 columns; split K only when there are few columns
        const int wgs = (N + 63) / 64;
        int s = wgs >= 128 ? 1 : (256 + wgs - 1) / wgs;
        const int cap = nk / 16 > 1 ? nk / 16 : 1;     // keep two batches of 8 k steps per split
        s = s < cap ? s : cap;
        p = make_plan(M, N, K, 16, 64, s, bits);
        p.cfg = 3;
    } else if (M <= 64) {
        const int tiles = ((M + 63) / 64) * ((N + 63) / 64);
        p = make_plan(M, N, K, 64, 64, splits_for(tiles), bits);
        p.cfg = 2;
    } else if (((M + 127) / 128) * ((N + 127) / 128) >= 512) {
        p = make_plan(M, N, K, 128, 128, 1, bits);
        p.cfg = 0;
    } else {
        const int tiles = ((M + 63) / 64) * ((N + 127) / 128);
        p = make_plan(M, N, K, 64, 128, splits_for(tiles), bits);
        p.cfg = 1;
    }
    return p;
}

}  // namespace

size_t gemm_workspace_bytes(int M, int N, int K, int bits) {
    const Plan p = choose_plan(M, N, K, bits);
    return p.splits > 1 ? (size_t)p.splits * M * N * sizeof(int32_t) : 0;
}

hipError_t launch_gemm(const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w, int M, int N,
                       int K, uint16_t* Y, int32_t* acc, void* ws, hipStream_t st, int bits) {
    const Plan p = choose_plan(M, N, K, bits);
    int32_t* part = static_cast<int32_t*>(ws);
    hipError_t e;
    const int sel = p.cfg + (bits == 8 ? 4 : 0);
    switch (sel) {
        case 3: e = launch_skinny<1, 8, 4>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
        case 2: e = launch_cfg<2, 2, 2, 2, false, 1, 4>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
        case 1: e = launch_cfg<1, 4, 4, 2, false, 1, 4>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
        case 0: e = launch_cfg<2, 2, 4, 4, false, 1, 4>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
        case 7: e = launch_skinny<1, 8, 8>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
        case 6: e = launch_cfg<2, 2, 2, 2, false, 1, 8>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
        case 5: e = launch_cfg<1, 4, 4, 2, false, 1, 8>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
        default: e = launch_cfg<2, 2, 4, 4, false, 1, 8>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
    }
    if (e != hipSuccess) return e;
    return finish_split(p, part, s_a, s_w, M, N, Y, acc, st);
}

}  // namespace sq
