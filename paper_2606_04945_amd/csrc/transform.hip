// SGAT activation transform (Sec. 3.2, Eq. 11): x'_i = x_i P G_{s_i}, and the
// ungated weight-side product W P used by weight preparation (Eq. 12).
//
// Fixed evaluation order (part of the result, because the codes quantised from
// x' flip at rounding midpoints): output (i, j) accumulates k in chunks of 256,
// each chunk an fp32 fused multiply-add chain in ascending k from +0, and the
// chunk sums are added in ascending order to a +0 total.
//
// Matrix cores: v_mfma_f32_16x16x4_f32 computes each of its 16 x 16 outputs as
// c + a0 b0 + a1 b1 + a2 b2 + a3 b3 evaluated as a forward chain of four
// fused multiply-adds, k ascending, each rounded once, subnormals kept
// (checked bit for bit against fmaf chains, signed zeros and subnormal
// results included).  A chain of these instructions over ascending groups of
// four k, from a zeroed accumulator, is therefore exactly one chunk's chain;
// the chunk totals are added on the VALU.
//
// Tiling: a workgroup owns a BM x BN tile of outputs, a wave IB x JB blocks of
// 16 x 16, each output with a chunk accumulator (the instruction's result
// registers) and a total: 128 x 128 tiles of eight waves of 32 x 64 (four waves
// per SIMD at two workgroups per CU; four waves of 64 x 64 were 3-9 % slower),
// 64 x 128 tiles of four waves where 128-row tiles would leave CUs idle, and
// 32 x 256 for up to 32 rows.  Main kernel: both operand tiles go from HBM straight
// into LDS (buffer loads with the LDS destination, no staging registers)
// through a three-stage ring, two k steps of 32 in flight while a third is
// multiplied, one barrier per step; X stays fp16 in LDS and is widened as it is
// read.  Staging the tiles through registers instead (converting X on the way)
// ran at 0.75 of the speed on the 8 x 2048-token shapes; that form remains for
// batches of up to 32 rows.
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
#include "tile_common.hpp"

namespace sq {
namespace {

constexpr int kThreads = 256;
constexpr int kBK = 32;

// This workgroup's rows when rows are grouped by state: rowmap[i] is the row
// of rank rt * BM + i in the order (masked rows, then unmasked rows), or -1
// past the last row; returns the number of masked rows.
template <int BM, int NT = kThreads>
__device__ int group_rows(const uint8_t* __restrict__ state, int M, int rt, int* rowmap, int* scan) {
    const int tid = threadIdx.x;
    const int per = (M + NT - 1) / NT;               // states per thread, in one contiguous run
    const int b = min(M, tid * per), e = min(M, b + per);
    int cnt = 0;
    for (int i = b; i < e; ++i) cnt += state[i] != 0;
    if (tid < BM) rowmap[tid] = -1;
    scan[tid] = cnt;
    __syncthreads();
    // inclusive scan of the per-thread counts (Hillis-Steele over NT entries)
    for (int o = 1; o < NT; o <<= 1) {
        const int v = tid >= o ? scan[tid - o] : 0;
        __syncthreads();
        scan[tid] += v;
        __syncthreads();
    }
    const int nm = scan[NT - 1];
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

typedef float f32x4 __attribute__((ext_vector_type(4)));

// v_mfma_f32_16x16x4_f32: D = C + sum_k A[:, k] B[k, :] over its four k as a
// forward chain of single-rounding fused multiply-adds, k ascending (checked bit
// for bit against fmaf chains).  A chain of these over ascending groups of
// four k is the chunk chain itself.  Lane l supplies A[l % 16][l / 16] and
// B[l / 16][l % 16]; result register v holds row 4 (l / 16) + v, column l % 16.
// A wave owns IB x JB blocks of 16 x 16 outputs, a workgroup WR x WC waves.
template <int IB, int JB, int WR, int WC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void transform_kernel(
    const uint16_t* __restrict__ X, const uint8_t* __restrict__ state, const float* __restrict__ P,
    int M, int K, int dm, int du, int grouped, float* __restrict__ Xp) {
    static_assert(WR * WC * kWave == kThreads, "four waves");
    constexpr int BM = 16 * IB * WR;
    constexpr int BN = 16 * JB * WC;
    constexpr int AP = BM + 4;                       // padded LDS row (k-major A tile)
    constexpr int BP = BN + 4;
    __shared__ float As[2][kBK][AP];
    __shared__ float Bs[2][kBK][BP];
    __shared__ int rowmap[BM];
    __shared__ int scan[kThreads];

    const int tid = threadIdx.x;
    const int lane = tid % kWave, wave = tid / kWave;
    const int wr = wave / WC, wc = wave % WC;
    int rt, ct;
    const int R = (M + BM - 1) / BM;
    xcd_tile(blockIdx.x, R, (K + BN - 1) / BN, R < 16 ? R : 16, rt, ct);
    const int row0 = rt * BM, col0 = ct * BN;
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

    constexpr int VPR = kBK / 8;
    constexpr int AV = (BM * VPR + kThreads - 1) / kThreads;
    uint4 ra[AV];
    constexpr int NB = kBK * BN / 4 / kThreads;
    float4 rb[NB];
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

    f32x4 acc[IB][JB], tot[IB][JB];
#pragma unroll
    for (int i = 0; i < IB; ++i)
#pragma unroll
        for (int j = 0; j < JB; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) acc[i][j][v] = 0.0f, tot[i][j][v] = 0.0f;

    const int kl = lane / 16, il = lane % 16;
    const int arow0 = wr * 16 * IB + il;             // A operand row of this lane in block 0
    const int bcol0 = wc * 16 * JB + il;             // B operand column of this lane in block 0
    const int nk = K / kBK;
    load_tiles(0);
    store_tiles(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) load_tiles((kt + 1) * kBK);
#pragma unroll
        for (int s4 = 0; s4 < kBK / 4; ++s4) {
            const int kk = 4 * s4 + kl;
            float a[IB], b[JB];
#pragma unroll
            for (int i = 0; i < IB; ++i) a[i] = As[buf][kk][arow0 + 16 * i];
#pragma unroll
            for (int j = 0; j < JB; ++j) b[j] = Bs[buf][kk][bcol0 + 16 * j];
#pragma unroll
            for (int i = 0; i < IB; ++i)
#pragma unroll
                for (int j = 0; j < JB; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        const int kend = (kt + 1) * kBK;
        if (kend % kChunk == 0 || kend == K) {       // chunk boundary: fold into the total
#pragma unroll
            for (int i = 0; i < IB; ++i)
#pragma unroll
                for (int j = 0; j < JB; ++j)
#pragma unroll
                    for (int v = 0; v < 4; ++v) tot[i][j][v] = tot[i][j][v] + acc[i][j][v], acc[i][j][v] = 0.0f;
        }
        if (kt + 1 < nk) {
            store_tiles(buf ^ 1);
            __syncthreads();
        }
    }

    // result register v of block (i, j): tile row 16 (IB wr + i) + 4 (lane / 16) + v,
    // tile column 16 (JB wc + j) + lane % 16; 16 lanes store 64 contiguous bytes of a row
#pragma unroll
    for (int i = 0; i < IB; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int r = rowmap[wr * 16 * IB + 16 * i + 4 * kl + v];
            if (r < 0) continue;
            const bool masked = state ? state[r] != 0 : false;
#pragma unroll
            for (int j = 0; j < JB; ++j) {
                const int col = col0 + wc * 16 * JB + 16 * j + il;
                if (col >= K) continue;
                const bool keep = !state || kept(col, K, dm, du, masked);
                Xp[(size_t)r * K + col] = keep ? tot[i][j][v] : 0.0f;
            }
        }
}

// The same computation with both operand tiles copied from HBM straight into
// LDS (buffer loads with the LDS destination, no staging registers) through a
// three-stage ring: two k steps are in flight while a third is multiplied, one
// barrier per step.  X stays fp16 in LDS (64 bytes per row and step, its four
// 16-byte chunks XOR-swizzled by row) and is widened when read; P is staged
// as it is in HBM, 512 bytes per k row, its 16-byte chunks XOR-swizzled by k
// so that the four k of an instruction fall on different banks.
template <int IB, int JB, int WR, int WC, int NT = 64 * WR * WC>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(NT / 128))) void transform_dma_kernel(
    const uint16_t* __restrict__ X, const uint8_t* __restrict__ state, const float* __restrict__ P,
    int M, int K, int dm, int du, int grouped, float* __restrict__ Xp) {
    static_assert(WR * WC * kWave == NT, "wave count");
    constexpr int NW = WR * WC;
    constexpr int BM = 16 * IB * WR;
    constexpr int BN = 16 * JB * WC;
    constexpr int AB = BM * kBK * 2;                 // fp16 X tile bytes per stage
    constexpr int BB = kBK * BN * 4;                 // fp32 P tile bytes per stage
    constexpr int SB = AB + BB;
    constexpr int LA = AB / 1024 / NW, LB = BB / 1024 / NW;   // 1 KB loads per wave per stage
    static_assert(LA * NW * 1024 == AB && LB * NW * 1024 == BB, "stage loads must divide evenly");
    static_assert(BN == 128, "P rows of 32 16-byte chunks");
    __shared__ __attribute__((aligned(16))) uint8_t sm[3 * SB];
    __shared__ int rowmap[BM];
    __shared__ int scan[NT];

    const int tid = threadIdx.x;
    const int lane = tid % kWave, wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int wr = wave / WC, wc = wave % WC;
    int rt, ct;
    const int R = (M + BM - 1) / BM;
    xcd_tile(blockIdx.x, R, (K + BN - 1) / BN, R < 16 ? R : 16, rt, ct);
    const int row0 = rt * BM, col0 = ct * BN;
    if (grouped) {
        const int nm = group_rows<BM, NT>(state, M, rt, rowmap, scan);
        const int rows_end = min(M, row0 + BM);
        const bool all_m = rows_end <= nm, all_u = row0 >= nm;
        const bool dropped = (all_m && col0 >= K - du) ||
                             (all_u && col0 >= K - dm - du && col0 + BN <= K - du);
        if (dropped) {
            const int ncol4 = min(BN, K - col0) / 4;
            for (int e = tid; e < BM * ncol4; e += NT) {
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

    // X: tile row r's 64 bytes hold its chunks c at slot c ^ swa(r); P: k row k's
    // 512 bytes hold column chunk c at slot c ^ swb(k)
    auto swa = [](int r) { return (r >> 2) & 3; };
    auto swb = [](int k) { return 4 * (k & 3); };
    const u32x4 rX = sgpr_rsrc(X, (uint32_t)((size_t)M * K * 2));
    uint32_t oa[LA], ob[LB];
#pragma unroll
    for (int u = 0; u < LA; ++u) {
        const int r = 16 * (wave * LA + u) + lane / 4;
        const int tok = rowmap[r];
        oa[u] = tok >= 0 ? (uint32_t)tok * K * 2 + 16 * ((lane % 4) ^ swa(r)) : kOOB;
    }
#pragma unroll
    for (int u = 0; u < LB; ++u) {
        const int k = 2 * (wave * LB + u) + lane / 32;
        const int c = (lane % 32) ^ swb(k);
        ob[u] = col0 + 4 * c < K ? (uint32_t)k * K * 4 + (uint32_t)(col0 + 4 * c) * 4 : kOOB;
    }
    auto issue = [&](int kt, int stage) {
        uint8_t* dA = sm + stage * SB;
        uint8_t* dB = dA + AB;
        // P rows k0 .. k0 + 31 through a descriptor based at row k0 (offsets stay below 128 K bytes)
        const u32x4 rP = sgpr_rsrc(P + (size_t)kt * kBK * K, (uint32_t)kBK * K * 4);
#pragma unroll
        for (int u = 0; u < LA; ++u) dma16s(rX, lds_addr(dA + (wave * LA + u) * 1024), oa[u], (uint32_t)kt * kBK * 2);
#pragma unroll
        for (int u = 0; u < LB; ++u) dma16(rP, lds_addr(dB + (wave * LB + u) * 1024), ob[u]);
    };

    f32x4 acc[IB][JB], tot[IB][JB];
#pragma unroll
    for (int i = 0; i < IB; ++i)
#pragma unroll
        for (int j = 0; j < JB; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) acc[i][j][v] = 0.0f, tot[i][j][v] = 0.0f;

    const int kl = lane / 16, il = lane % 16;
    int aoff[IB];                                    // byte offset of this lane's A row in a stage
#pragma unroll
    for (int i = 0; i < IB; ++i) aoff[i] = (wr * 16 * IB + 16 * i + il) * 64;
    const int aswz = swa(il);                        // swa(r) depends on r % 16 only (rows of a block)
    int boff[JB];                                    // column chunk and position of this lane's B column
#pragma unroll
    for (int j = 0; j < JB; ++j) boff[j] = wc * 16 * JB + 16 * j + il;

    auto compute = [&](const uint8_t* sa) {
        const uint8_t* sbp = sa + AB;
#pragma unroll
        for (int s4 = 0; s4 < kBK / 4; ++s4) {
            const int kk = 4 * s4 + kl;
            float a[IB], b[JB];
#pragma unroll
            for (int i = 0; i < IB; ++i) {
                const uint16_t h = *reinterpret_cast<const uint16_t*>(sa + aoff[i] + 16 * ((kk / 8) ^ aswz) + 2 * (kk % 8));
                a[i] = h2f(h);
            }
#pragma unroll
            for (int j = 0; j < JB; ++j) {
                const int c = boff[j];
                b[j] = *reinterpret_cast<const float*>(sbp + kk * (BN * 4) + 16 * ((c / 4) ^ swb(kk)) + 4 * (c % 4));
            }
#pragma unroll
            for (int i = 0; i < IB; ++i)
#pragma unroll
                for (int j = 0; j < JB; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    };

    const int nk = K / kBK;
    auto step = [&](int kt, int sc, int sn) {
        asm volatile("" ::: "memory");
        if (kt + 1 < nk)
            wait_vm<LA + LB>();                          // this wave's loads of step kt are done
        else
            wait_vm<0>();
        __builtin_amdgcn_s_barrier();                    // ... and every wave's
        asm volatile("" ::: "memory");
        if (kt + 2 < nk) issue(kt + 2, sn);              // into the stage step kt - 1 used
        compute(sm + sc * SB);
        const int kend = (kt + 1) * kBK;
        if (kend % kChunk == 0 || kend == K) {           // chunk boundary: fold into the total
#pragma unroll
            for (int i = 0; i < IB; ++i)
#pragma unroll
                for (int j = 0; j < JB; ++j)
#pragma unroll
                    for (int v = 0; v < 4; ++v) tot[i][j][v] = tot[i][j][v] + acc[i][j][v], acc[i][j][v] = 0.0f;
        }
    };
    issue(0, 0);
    issue(1, 1);
    for (int kt = 0; kt < nk; kt += 3) {
        step(kt, 0, 2);
        if (kt + 1 < nk) step(kt + 1, 1, 0);
        if (kt + 2 < nk) step(kt + 2, 2, 1);
    }

#pragma unroll
    for (int i = 0; i < IB; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int r = rowmap[wr * 16 * IB + 16 * i + 4 * kl + v];
            if (r < 0) continue;
            const bool masked = state ? state[r] != 0 : false;
#pragma unroll
            for (int j = 0; j < JB; ++j) {
                const int col = col0 + wc * 16 * JB + 16 * j + il;
                if (col >= K) continue;
                const bool keep = !state || kept(col, K, dm, du, masked);
                Xp[(size_t)r * K + col] = keep ? tot[i][j][v] : 0.0f;
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
    // up to 32 rows: the register-staged kernel on 32 x 256 tiles
    if (M <= 32) {
        const int ncol = (K + 255) / 256;
        const int u0 = K - du, m0 = K - dm - du;
        const bool band_tile = (u0 + 255) / 256 * 256 < K || (m0 + 255) / 256 * 256 + 256 <= u0;
        const int grouped = state != nullptr && band_tile ? 1 : 0;
        hipLaunchKernelGGL((transform_kernel<2, 4, 1, 4>), dim3(ncol), dim3(kThreads), 0, st, X, state, P, M, K, dm,
                           du, grouped, Xp);
        return hipGetLastError();
    }
    // The pipelined kernel addresses X with 32-bit buffer offsets, so a call whose
    // X exceeds 2 GiB runs as independent chunks of rows (rows never interact).
    const int Mc = (int)(((size_t)0x7fffffff / ((size_t)K * 2)) / 128 * 128);
    for (int r0 = 0; r0 < M; r0 += Mc) {
        const int m = M - r0 < Mc ? M - r0 : Mc;
        const uint16_t* x = X + (size_t)r0 * K;
        const uint8_t* s = state ? state + r0 : nullptr;
        float* xp = Xp + (size_t)r0 * K;
        // 128 x 128 tiles where they give at least two workgroups per CU, else 64 x 128
        const int ncol = (K + 127) / 128;
        const int BM = (size_t)((m + 127) / 128) * ncol >= 512 ? 128 : 64;
        // group rows by state only where a column tile lies wholly in a band
        const int u0 = K - du, m0 = K - dm - du;
        const bool band_tile = (u0 + 127) / 128 * 128 < K ||           // a tile wholly in [u0, K)
                               (m0 + 127) / 128 * 128 + 128 <= u0;     // a tile wholly in [m0, u0)
        const int grouped = s != nullptr && band_tile ? 1 : 0;
        const dim3 grid((unsigned)(((m + BM - 1) / BM) * ncol));
        if (BM == 128)
            hipLaunchKernelGGL((transform_dma_kernel<2, 4, 4, 2>), grid, dim3(512), 0, st, x, s, P, m, K, dm, du,
                               grouped, xp);
        else
            hipLaunchKernelGGL((transform_dma_kernel<2, 4, 2, 2>), grid, dim3(kThreads), 0, st, x, s, P, m, K, dm, du,
                               grouped, xp);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipGetLastError();
}

}  // namespace sq
