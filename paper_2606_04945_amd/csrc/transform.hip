// SGAT activation transform (Sec. 3.2, Eq. 11): x'_i = x_i P G_{s_i}, and the
// ungated weight-side product W P used by weight preparation (Eq. 12).
//
// Fixed evaluation order (part of the result, because the codes quantised from
// x' flip at rounding midpoints): output (i, j) accumulates k in chunks of 256,
// each chunk an fp32 fused multiply-add chain in ascending k from +0, and the
// chunk sums are added in ascending order to a +0 total.
//
// Tiling: a 256-thread workgroup (four waves) owns a BM x BN tile of outputs
// (128 x 128, 64 x 128, or 32 x 256 for a few rows), each output with a chunk
// accumulator (in the matrix-core result registers) and a total.  X (converted
// fp16 -> fp32 on the way) and P are staged through double-buffered LDS 32 k at
// a time, the next global tile prefetched into registers during the multiply.
// The prefetch loads are unconditional (rows past M and columns past K read a
// valid address and are zeroed when staged), so that no wait for them sits
// before the multiply; the high fp16 of each loaded pair is converted in place
// (an SDWA word select) for the same reason.
//
// Rows grouped by state (the paper's split of the batch into masked and
// unmasked tokens, Eq. 7): when some 128-column tile lies wholly inside one of
// the two bands, row tiles are taken over the rows in the order "masked rows,
// then unmasked rows" (each group ascending).  A row tile whose rows all share
// one state then skips the column tiles of the band that state drops (they
// are +0, Eq. 10) instead of computing and discarding them; only the one row
// tile that straddles the two groups computes every column.  Each workgroup
// finds its rows itself from the state vector (a count of masked rows per
// thread, a workgroup scan, then the rows whose rank falls in its tile), so
// the call needs no workspace.  The order of the rows changes nothing in any
// row's result.
#include "sq_internal.hpp"

namespace sq {
namespace {

constexpr int kThreads = 256;
constexpr int kBK = 32;

// This workgroup's rows when rows are grouped by state: rowmap[i] is the row
// of rank rt * BM + i in the order (masked rows, then unmasked rows), or -1
// past the last row; returns the number of masked rows.
template <int BM>
__device__ int group_rows(const uint8_t* __restrict__ state, int M, int rt, int* rowmap, int* scan) {
    const int tid = threadIdx.x;
    const int per = (M + kThreads - 1) / kThreads;   // states per thread, in one contiguous run
    const int b = min(M, tid * per), e = min(M, b + per);
    int cnt = 0;
    for (int i = b; i < e; ++i) cnt += state[i] != 0;
    if (tid < BM) rowmap[tid] = -1;
    scan[tid] = cnt;
    __syncthreads();
    // inclusive scan of the per-thread counts (Hillis-Steele over 256 entries)
    for (int o = 1; o < kThreads; o <<= 1) {
        const int v = tid >= o ? scan[tid - o] : 0;
        __syncthreads();
        scan[tid] += v;
        __syncthreads();
    }
    const int nm = scan[kThreads - 1];
    int m_rank = scan[tid] - cnt;                    // masked rows before this run
    int u_rank = nm + (b - m_rank);                  // rank of its first unmasked row
    const int lo = rt * BM;
    for (int i = b; i < e; ++i) {
        const bool masked = state[i] != 0;
        const int rank = masked ? m_rank++ : u_rank++;
        if (rank >= lo && rank < lo + BM) rowmap[rank - lo] = i;
    }
    __syncthreads();
    return nm;
}

// fp16 pair -> two fp32 (exact), low half first; the asm keeps the conversion
// where the value is staged instead of next to its load.
__device__ __forceinline__ void h2f_pair(uint32_t w, float& lo, float& hi) {
    asm volatile("v_cvt_f32_f16_e32 %0, %2\n\tv_cvt_f32_f16_sdwa %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_1"
                 : "=&v"(lo), "=&v"(hi) : "v"(w));
}

typedef float f32x32 __attribute__((ext_vector_type(32)));

// The matrix-core form of the same fixed order.  v_mfma_f32_32x32x1_2b_f32
// multiplies one k at a time: each of its 2 x 32 x 32 outputs receives exactly
// one product per instruction, d = fma(a, b, c) with a single rounding,
// subnormals kept (checked bit for bit against fmaf chains, signed zeros and
// subnormal results included).  A chain of these instructions over ascending k
// from a zeroed accumulator is therefore the chunk chain itself, and the chunk
// totals are added on the VALU exactly as before.  The instruction's two
// blocks are the two 32-column halves of a wave's 64 columns (the A operand
// repeats the same 32 rows in both lane halves); TMI instructions per k cover
// 32 TMI rows.  A wave owns 32 TMI x 64 outputs, a workgroup WR x WC waves.
//
// Operand lane layout (block b = lane / 32): A lane 32 b + i holds row i, B
// lane 32 b + j holds column j; result register v of block b = v / 16 holds
// row 8 ((v % 16) / 4) + 4 (lane / 32) + v % 4, column lane % 32.
template <int TMI, int WR, int WC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void transform_kernel(
    const uint16_t* __restrict__ X, const uint8_t* __restrict__ state, const float* __restrict__ P,
    int M, int K, int dm, int du, int grouped, float* __restrict__ Xp) {
    static_assert(WR * WC * kWave == kThreads, "four waves");
    constexpr int BM = 32 * TMI * WR;
    constexpr int BN = 64 * WC;
    constexpr int AP = BM + 2;                       // padded LDS row (k-major A tile)
    __shared__ float As[2][kBK][AP];
    __shared__ float Bs[2][kBK][BN];
    __shared__ int rowmap[BM];
    __shared__ int scan[kThreads];

    const int tid = threadIdx.x;
    const int lane = tid % kWave, wave = tid / kWave;
    const int wr = wave / WC, wc = wave % WC;
    // up to 16 row tiles of a column tile of P run on one XCD at the same
    // time, so that XCD's L2 fetches the column tile once per group and the
    // XCDs work on different columns
    int rt, ct;
    const int R = (M + BM - 1) / BM;
    xcd_tile(blockIdx.x, R, (K + BN - 1) / BN, R < 16 ? R : 16, rt, ct);
    const int row0 = rt * BM, col0 = ct * BN;
    // rows of this tile: in order, or grouped by state (then a tile of one
    // state whose columns all lie in the band that state drops writes +0)
    if (grouped) {
        const int nm = group_rows<BM>(state, M, rt, rowmap, scan);
        const int rows_end = min(M, row0 + BM);
        const bool all_m = rows_end <= nm, all_u = row0 >= nm;
        const bool dropped = (all_m && col0 >= K - du) ||
                             (all_u && col0 >= K - dm - du && col0 + BN <= K - du);
        if (dropped) {
            const int ncol4 = min(BN, K - col0) / 4;
            for (int e = tid; e < BM * ncol4; e += kThreads) {
                const int r = rowmap[e / ncol4];
                if (r >= 0)
                    *reinterpret_cast<float4*>(Xp + (size_t)r * K + col0 + (e % ncol4) * 4) =
                        make_float4(0.f, 0.f, 0.f, 0.f);
            }
            return;
        }
    } else {
        if (tid < BM) rowmap[tid] = row0 + tid < M ? row0 + tid : -1;
        __syncthreads();
    }

    // global -> register prefetch slots
    // A: BM rows x 32 k fp16 = 4 16-byte vectors per row; thread t takes vectors t, t+256, ..
    constexpr int VPR = kBK / 8;
    constexpr int AV = (BM * VPR + kThreads - 1) / kThreads;
    uint4 ra[AV];
    // P: 32 rows x BN cols fp32 = 8 BN float4; thread t takes t, t+256, ..
    constexpr int NB = kBK * BN / 4 / kThreads;
    float4 rb[NB];

    // the rows and columns this thread loads, fixed for the whole k loop; a row
    // past M or a column past K reads row 0 / column 0 and is zeroed when staged
    int arow[AV];
    const uint16_t* aptr[AV];
#pragma unroll
    for (int v = 0; v < AV; ++v) {
        const int e = tid + v * kThreads;
        arow[v] = e < BM * VPR ? rowmap[e / VPR] : -1;
        aptr[v] = X + (size_t)(arow[v] >= 0 ? arow[v] : 0) * K + (e % VPR) * 8;
    }
    bool bok[NB];
    const float* bptr[NB];
#pragma unroll
    for (int v = 0; v < NB; ++v) {
        const int e = tid + v * kThreads;
        const int kr = e / (BN / 4), c4 = (e % (BN / 4)) * 4;
        bok[v] = col0 + c4 < K;
        bptr[v] = P + (size_t)kr * K + (bok[v] ? col0 + c4 : 0);
    }
    auto load_tiles = [&](int k0) {
#pragma unroll
        for (int v = 0; v < AV; ++v)
            if (BM * VPR >= (v + 1) * kThreads || tid + v * kThreads < BM * VPR)
                ra[v] = *reinterpret_cast<const uint4*>(aptr[v] + k0);
#pragma unroll
        for (int v = 0; v < NB; ++v) rb[v] = *reinterpret_cast<const float4*>(bptr[v] + (size_t)k0 * K);
    };
    auto store_tiles = [&](int buf) {
#pragma unroll
        for (int v = 0; v < AV; ++v) {
            const int e = tid + v * kThreads;
            if (e < BM * VPR) {
                const int r = e / VPR, h = e % VPR;
                const uint4 w = arow[v] >= 0 ? ra[v] : make_uint4(0, 0, 0, 0);
                const uint32_t wv[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float lo, hi;
                    h2f_pair(wv[q], lo, hi);
                    As[buf][h * 8 + 2 * q][r] = lo;
                    As[buf][h * 8 + 2 * q + 1][r] = hi;
                }
            }
        }
#pragma unroll
        for (int v = 0; v < NB; ++v) {
            const int e = tid + v * kThreads;
            const int kr = e / (BN / 4), c4 = (e % (BN / 4)) * 4;
            *reinterpret_cast<float4*>(&Bs[buf][kr][c4]) = bok[v] ? rb[v] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    };

    f32x32 acc[TMI], tot[TMI];
#pragma unroll
    for (int t = 0; t < TMI; ++t)
#pragma unroll
        for (int v = 0; v < 32; ++v) acc[t][v] = 0.0f, tot[t][v] = 0.0f;

    const int arow0 = wr * 32 * TMI + (lane & 31);   // A operand row of this lane (both lane halves)
    const int bcol = wc * 64 + lane;                 // B operand column of this lane
    const int nk = K / kBK;
    load_tiles(0);
    store_tiles(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) load_tiles((kt + 1) * kBK);
#pragma unroll
        for (int kk = 0; kk < kBK; ++kk) {
            const float b = Bs[buf][kk][bcol];
#pragma unroll
            for (int t = 0; t < TMI; ++t)
                acc[t] = __builtin_amdgcn_mfma_f32_32x32x1f32(As[buf][kk][arow0 + 32 * t], b, acc[t], 0, 0, 0);
        }
        const int kend = (kt + 1) * kBK;
        if (kend % kChunk == 0 || kend == K) {       // chunk boundary: fold into the total
#pragma unroll
            for (int t = 0; t < TMI; ++t)
#pragma unroll
                for (int v = 0; v < 32; ++v) tot[t][v] = tot[t][v] + acc[t][v], acc[t][v] = 0.0f;
        }
        if (kt + 1 < nk) {
            store_tiles(buf ^ 1);
            __syncthreads();
        }
    }

    // result register v of row group t: tile row 32 (WR-row) + 8 ((v % 16) / 4) + 4 (lane / 32) + v % 4,
    // tile column 64 wc + 32 (v / 16) + lane % 32; 32 lanes store 128 contiguous bytes of a row
#pragma unroll
    for (int t = 0; t < TMI; ++t)
#pragma unroll
        for (int v = 0; v < 32; ++v) {
            const int r = rowmap[wr * 32 * TMI + 32 * t + 8 * ((v % 16) / 4) + 4 * (lane / 32) + (v % 4)];
            const int col = col0 + wc * 64 + 32 * (v / 16) + (lane % 32);
            if (r < 0 || col >= K) continue;
            const bool keep = !state || kept(col, K, dm, du, state[r] != 0);
            Xp[(size_t)r * K + col] = keep ? tot[t][v] : 0.0f;
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
    // 128 x 128 tiles where they give at least two workgroups per CU, else 64 x 128,
    // and 32 x 256 for a few rows
    const int tiles128 = ((M + 127) / 128) * ((K + 127) / 128);
    const int BM = tiles128 >= 512 ? 128 : (M > 32 ? 64 : 32);
    const int BN = BM == 32 ? 256 : 128;
    const int ncol = (K + BN - 1) / BN;
    if ((size_t)((M + BM - 1) / BM) * ncol > 0x7fffffffu) return hipErrorInvalidConfiguration;
    // group rows by state only where a column tile lies wholly in a band
    const int u0 = K - du, m0 = K - dm - du;
    const bool band_tile = (u0 + BN - 1) / BN * BN < K ||            // a tile wholly in [u0, K)
                           (m0 + BN - 1) / BN * BN + BN <= u0;       // a tile wholly in [m0, u0)
    const int grouped = state != nullptr && band_tile ? 1 : 0;
    const dim3 grid(((M + BM - 1) / BM) * ncol);
    if (BM == 128)
        hipLaunchKernelGGL((transform_kernel<2, 2, 2>), grid, dim3(kThreads), 0, st, X, state, P, M, K, dm, du,
                           grouped, Xp);
    else if (BM == 64)
        hipLaunchKernelGGL((transform_kernel<1, 2, 2>), grid, dim3(kThreads), 0, st, X, state, P, M, K, dm, du,
                           grouped, Xp);
    else
        hipLaunchKernelGGL((transform_kernel<1, 1, 4>), grid, dim3(kThreads), 0, st, X, state, P, M, K, dm, du,
                           grouped, Xp);
    return hipGetLastError();
}

}  // namespace sq
