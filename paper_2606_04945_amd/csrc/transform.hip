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
// X (converted fp16 -> fp32) and P staged through double-buffered LDS 32 k at a
// time and the next global tile prefetched into registers during compute.  The
// fragments of step k + 1 are read from LDS while step k multiplies (two
// register sets), and the prefetch loads are unconditional (rows past M and
// columns past K read a valid address and are zeroed when staged), so that no
// wait for them sits before the multiply: with a conditional load the compiler
// split the fp16 pairs right after it and so waited for global memory at the
// top of every step.  The high fp16 of each loaded pair is converted in place
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
constexpr int kBN = 128;
constexpr int kBK = 32;
constexpr int kTN = 8;

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

template <int TM>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void transform_kernel(
    const uint16_t* __restrict__ X, const uint8_t* __restrict__ state, const float* __restrict__ P,
    int M, int K, int dm, int du, int grouped, float* __restrict__ Xp) {
    constexpr int BM = 16 * TM;
    constexpr int AP = BM + 4;                       // padded LDS row (k-major A tile)
    constexpr int BP = kBN + 4;
    __shared__ float As[2][kBK][AP];
    __shared__ float Bs[2][kBK][BP];
    __shared__ int rowmap[BM];
    __shared__ int scan[kThreads];

    const int tid = threadIdx.x;
    const int tx = tid % 16, ty = tid / 16;
    // up to 16 row tiles of a column tile of P run on one XCD at the same
    // time, so that XCD's L2 fetches the column tile once per group (all of a
    // 1024-token batch is one group) and the XCDs work on different columns
    int rt, ct;
    const int R = (M + BM - 1) / BM;
    xcd_tile(blockIdx.x, R, (K + kBN - 1) / kBN, R < 16 ? R : 16, rt, ct);
    const int row0 = rt * BM, col0 = ct * kBN;
    // rows of this tile: in order, or grouped by state (then a tile of one
    // state whose columns all lie in the band that state drops writes +0)
    if (grouped) {
        const int nm = group_rows<BM>(state, M, rt, rowmap, scan);
        const int rows_end = min(M, row0 + BM);
        const bool all_m = rows_end <= nm, all_u = row0 >= nm;
        const bool dropped = (all_m && col0 >= K - du) ||
                             (all_u && col0 >= K - dm - du && col0 + kBN <= K - du);
        if (dropped) {
            const int cbase = col0 + tx * kTN;
            if (cbase >= K) return;
            for (int i = 0; i < TM; ++i) {
                const int r = rowmap[ty * TM + i];
                if (r < 0) continue;
                float4* dst = reinterpret_cast<float4*>(Xp + (size_t)r * K + cbase);
                dst[0] = make_float4(0.f, 0.f, 0.f, 0.f);
                dst[1] = make_float4(0.f, 0.f, 0.f, 0.f);
            }
            return;
        }
    } else if (tid < BM) {
        rowmap[tid] = row0 + tid < M ? row0 + tid : -1;
    }
    if (!grouped) __syncthreads();

    // global -> register prefetch slots
    // A: BM rows x 32 k fp16 = 4 16-byte vectors per row; thread t takes vectors t, t+256, ..
    constexpr int VPR = kBK / 8;
    constexpr int AV = (BM * VPR + kThreads - 1) / kThreads;
    uint4 ra[AV];
    // P: 32 rows x 128 cols fp32 = 1024 float4; thread t takes t, t+256, t+512, t+768
    constexpr int NB = kBK * kBN / 4 / kThreads;
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
        const int kr = e / 32, c4 = (e % 32) * 4;
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
            const int kr = e / 32, c4 = (e % 32) * 4;
            *reinterpret_cast<float4*>(&Bs[buf][kr][c4]) = bok[v] ? rb[v] : make_float4(0.f, 0.f, 0.f, 0.f);
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
        float a[2][TM], b[2][kTN];
        auto frag = [&](int kk, float* aa, float* bb) {
#pragma unroll
            for (int i = 0; i < TM; i += 4) {
                const float4 t = *reinterpret_cast<const float4*>(&As[buf][kk][ty * TM + i]);
                aa[i] = t.x, aa[i + 1] = t.y, aa[i + 2] = t.z, aa[i + 3] = t.w;
            }
#pragma unroll
            for (int j = 0; j < kTN; j += 4) {
                const float4 t = *reinterpret_cast<const float4*>(&Bs[buf][kk][tx * 4 + (j / 4) * 64]);
                bb[j] = t.x, bb[j + 1] = t.y, bb[j + 2] = t.z, bb[j + 3] = t.w;
            }
        };
        frag(0, a[0], b[0]);
#pragma unroll
        for (int kk = 0; kk < kBK; ++kk) {
            if (kk + 1 < kBK) frag(kk + 1, a[(kk + 1) & 1], b[(kk + 1) & 1]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < kTN; ++j) acc[i][j] = __builtin_fmaf(a[kk & 1][i], b[kk & 1][j], acc[i][j]);
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

    // this thread's columns: col0 + 4 tx + {0..3} and col0 + 64 + 4 tx + {0..3}
    // (eight neighbouring lanes then read 128 contiguous bytes of a B row)
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int row = rowmap[ty * TM + i];
        if (row < 0) continue;
        const bool masked = state ? state[row] != 0 : false;
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            const int cb = col0 + hf * 64 + tx * 4;
            if (cb >= K) continue;
            float o[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) o[j] = (!state || kept(cb + j, K, dm, du, masked)) ? tot[i][hf * 4 + j] : 0.0f;
            *reinterpret_cast<float4*>(Xp + (size_t)row * K + cb) = make_float4(o[0], o[1], o[2], o[3]);
        }
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
    // group rows by state only where a column tile lies wholly in a band
    const int u0 = K - du, m0 = K - dm - du;
    const bool band_tile = (u0 + kBN - 1) / kBN * kBN < K ||            // a tile wholly in [u0, K)
                           (m0 + kBN - 1) / kBN * kBN + kBN <= u0;      // a tile wholly in [m0, u0)
    const int grouped = state != nullptr && band_tile ? 1 : 0;
    // enough workgroups to cover the 256 CUs at least twice, else the taller tile
    if ((size_t)ncol * ((M + 127) / 128) >= 512) {
        hipLaunchKernelGGL(transform_kernel<8>, dim3(((M + 127) / 128) * ncol), dim3(kThreads), 0, st, X, state, P,
                           M, K, dm, du, grouped, Xp);
    } else {
        hipLaunchKernelGGL(transform_kernel<4>, dim3(((M + 63) / 64) * ncol), dim3(kThreads), 0, st, X, state, P,
                           M, K, dm, du, grouped, Xp);
    }
    return hipGetLastError();
}

}  // namespace sq
