// W4A4 GEMM with dequantising epilogue (Eq. 13; Eq. 5):
//   acc[i][n] = sum_j qa[i][j] * qw[n][j]            (exact int32)
//   Y[i][n]   = fp16((float(acc) * s_a[i]) * s_w[n])
//
// gfx950 has no int4 matrix instruction, so packed nibbles feed the int8 MFMA
// v_mfma_i32_16x16x64_i8.  Unpacking keeps each nibble in the high half of a
// byte: for a packed dword w, (w << 4) & 0xF0F0F0F0 holds the even-k codes and
// w & 0xF0F0F0F0 the odd-k codes, each as the int8 value 16*q, with no sign
// extension step.  With both operands scaled by 16 the MFMA sums 256*qa*qw
// exactly, and >> 8 recovers the integer dot product (see acc_value for the one
// sum, +2^23 at K = 131072, whose scaled value wraps).  Even and odd k land in different registers; the same
// permutation is applied to A and W, and an integer sum does not depend on its
// order, so the result is the plain dot product.
//
// Tiled kernel (template): WM x WN waves, each owning TM x TN MFMA tiles of
// 16 x 16, so a workgroup owns (16 WM TM) x (16 WN TN) outputs.  A k step is 64
// packed bytes (128 codes) of every row of both operands.  Operand tiles go from
// HBM straight into LDS with buffer_load ... lds (no staging registers), three
// LDS stages deep: two k steps are in flight while a third is multiplied, with
// one barrier per step.  LDS rows are XOR-swizzled by 16-byte chunk so the
// fragment reads are free of bank conflicts; each wave unpacks the fragments it
// reads.  Rows past M (or N) and the unused half of a last k step read as zero
// through the buffer descriptors' range check.  Few tiles (M of 17 to a few
// hundred) split K across workgroups; the int32 partial sums are then added
// exactly by a small kernel.
// M <= 48 has kernels of their own that stream the weights into registers.
//
// BITS = 8 is the W8A8 variant (App. D): codes are int8 already, so the same
// tiles feed the MFMA straight from LDS with no unpacking and no scaling.
#include "tile_common.hpp"

namespace sq {
namespace {

__device__ __forceinline__ v4i unpack_op(uint32_t w0, uint32_t w1) {
    // one 64-bit shift moves the low nibbles of both words up; the nibble that
    // crosses from w0 into w1 is cleared by the mask
    uint64_t t = ((uint64_t)w1 << 32) | w0;
    asm("v_lshlrev_b64 %0, 4, %1" : "=v"(t) : "v"(t));  // kept as one instruction
    v4i r;
    r[0] = (int)((uint32_t)t & 0xF0F0F0F0u);
    r[1] = (int)((uint32_t)(t >> 32) & 0xF0F0F0F0u);
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
    // 4-bit: the dot product lies in [-56 K, 64 K] (codes in [-8, 7]), so 256 x it
    // fits in int32 except at +2^31, reached only when every product is
    // (-8)(-8) at K = 131072; that wraps to INT_MIN, which no in-range sum
    // produces, and stands for +2^23
    return BITS == 8 ? raw : (raw == INT32_MIN ? (1 << 23) : raw >> 8);
}

// KG > 1: KG sets of WM x WN waves share the tile and split its k steps
// (set g multiplies steps g, g + KG, ...; a stage holds KG consecutive steps,
// one per set), so a workgroup that owns a whole tile has KG times the waves;
// the sets' partial sums meet in LDS (exact integer adds) before the epilogue.
template <int WM, int WN, int TM, int TN, bool SPLIT, int BITS, int OCC, bool WF = false, int KG = 1>
__global__ __launch_bounds__(64 * WM * WN * KG) __attribute__((amdgpu_waves_per_eu(OCC))) void gemm_tile_kernel(
    const uint8_t* __restrict__ Aq, const float* __restrict__ s_a, const uint8_t* __restrict__ Wq,
    const float* __restrict__ s_w, int M, int N, int K, int ksteps_per_split, uint16_t* __restrict__ Y,
    int32_t* __restrict__ acc_out, int32_t* __restrict__ part) {
    static_assert(KG == 1 || !SPLIT, "k groups replace the split across workgroups");
    constexpr int NW = WM * WN;                          // waves of one k group
    constexpr int BM = 16 * WM * TM, BN = 16 * WN * TN;
    constexpr int AB = BM * kKB, BB = BN * kKB;          // bytes of one k step
    constexpr int SG = AB + BB;
    constexpr int SB = KG * SG;                          // bytes of one stage
    constexpr int LA = AB / 1024 / NW, LB = BB / 1024 / NW;   // 1 KB loads per wave per stage
    static_assert(LA * NW * 1024 == AB && LB * NW * 1024 == BB, "stage loads must divide evenly");
    static_assert((KG - 1) * NW * TM * TN * kWave * 16 <= 3 * SB, "k-group partial sums fit in the stages");
    __shared__ __attribute__((aligned(16))) uint8_t sm[3 * SB];

    const int tid = threadIdx.x;
    const int lane = tid % kWave, wave_all = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int kg = wave_all / NW, wave = wave_all % NW;  // k group, wave within it
    const int wm = wave / WN, wn = wave % WN;
    const uint32_t ldb = (uint32_t)K * BITS / 8;
    const int nk_total = (int)((ldb + kKB - 1) / kKB);
    const int nk_full = (int)(ldb / kKB);
    const u32x4 rA = sgpr_rsrc(Aq, (uint32_t)M * ldb);
    const int ngrp = (N + 15) / 16;                     // WF: fragment-ordered weights, 16-row groups
    const u32x4 rW = sgpr_rsrc(Wq, WF ? (uint32_t)ngrp * nk_total * 1024 : (uint32_t)N * ldb);
    auto swz = [](int r) { return (r >> 1) & 3; };       // 16-byte chunk swizzle of a 64-byte LDS row

    // groups of 8 row tiles per XCD (see xcd_tile): the workgroups an XCD runs
    // together share 8 row tiles of A and a few column tiles of W in its L2
    int rt, ct;
    xcd_tile(blockIdx.x, (M + BM - 1) / BM, (N + BN - 1) / BN, 8, rt, ct);
    const int row0 = rt * BM, col0 = ct * BN;
    // stage indices: stage kt holds k steps KG kt .. KG kt + KG - 1
    const int kt0 = SPLIT ? blockIdx.z * ksteps_per_split : 0;
    const int kt1 = SPLIT ? min(nk_total, kt0 + ksteps_per_split) : (nk_total + KG - 1) / KG;

    // this lane's source segment for each of its loads: tile row r = 16 j + lane / 4
    // holds, at chunk slot lane % 4, segment (lane % 4) ^ swz(r)
    uint32_t oa[LA], ow[LB];
    int sa_[LA], sw_[LB];
#pragma unroll
    for (int u = 0; u < LA; ++u) {
        const int r = 16 * (wave * LA + u) + lane / 4;
        sa_[u] = 16 * ((lane % 4) ^ swz(r));
        oa[u] = row0 + r < M ? (uint32_t)(row0 + r) * ldb + sa_[u] : kOOB;
    }
#pragma unroll
    for (int u = 0; u < LB; ++u) {
        const int r = 16 * (wave * LB + u) + lane / 4;
        sw_[u] = 16 * ((lane % 4) ^ swz(r));
        if (WF) {   // one 1 KB block per k step, copied as it is: lane l fetches bytes 16 l .. 16 l + 15
            const int g = (col0 + r) / 16;
            ow[u] = g < ngrp ? (uint32_t)g * 1024 + (uint32_t)lane * 16 : kOOB;
        } else {
            ow[u] = col0 + r < N ? (uint32_t)(col0 + r) * ldb + sw_[u] : kOOB;
        }
    }
    auto issue = [&](int st_kt, int stage) {
        // this k group's step of the stage; a step past the end reads as zeros
        const int kt = KG * st_kt + kg;
        uint8_t* dA = sm + stage * SB + kg * SG;
        uint8_t* dB = dA + AB;
        const uint32_t ko = (uint32_t)kt * kKB;
        const bool tail = kt >= nk_full;
        if (WF && !tail) {
            // Whole k steps of fragment-ordered weights: the k offsets ride in
            // the scalar offset (no vector instruction per load).  Every access
            // of a row below M stays inside that row, and rows past M (and
            // weight groups past N) carry an out-of-range vector offset.
#pragma unroll
            for (int u = 0; u < LA; ++u) dma16s(rA, lds_addr(dA + (wave * LA + u) * 1024), oa[u], ko);
#pragma unroll
            for (int u = 0; u < LB; ++u)
                dma16s(rW, lds_addr(dB + (wave * LB + u) * 1024), ow[u], (uint32_t)kt * ngrp * 1024);
            return;
        }
#pragma unroll
        for (int u = 0; u < LA; ++u) {
            const uint32_t o = (tail && ko + sa_[u] >= ldb) ? kOOB : oa[u] + ko;
            dma16(rA, lds_addr(dA + (wave * LA + u) * 1024), o);
        }
#pragma unroll
        for (int u = 0; u < LB; ++u) {
            // fragment-ordered weights are zero-padded to whole k steps
            const uint32_t o = WF ? ow[u] + (uint32_t)kt * ngrp * 1024 : (tail && ko + sw_[u] >= ldb) ? kOOB : ow[u] + ko;
            dma16(rW, lds_addr(dB + (wave * LB + u) * 1024), o);
        }
    };

    v4i acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = v4i{0, 0, 0, 0};
    const int lr = lane % 16, lg = lane / 16;
    const int fo = (lg ^ swz(lr)) * 16;                  // this lane's fragment slot in a row
    const int offA = ((wm * TM) * 16 + lr) * kKB + fo;
    // fragment-ordered weights sit in LDS in fragment order: lane l's 16 bytes at 16 l
    const int offB = WF ? AB + (wn * TN) * 1024 + lane * 16 : AB + ((wn * TN) * 16 + lr) * kKB + fo;
    v4i fa[TM], fb[TN];
    auto frags = [&](const uint8_t* st) {
#pragma unroll
        for (int i = 0; i < TM; ++i) fa[i] = *reinterpret_cast<const v4i*>(st + offA + i * 16 * kKB);
#pragma unroll
        for (int j = 0; j < TN; ++j) fb[j] = *reinterpret_cast<const v4i*>(st + offB + j * 16 * kKB);
    };
    // B operands of one half are expanded once; each A operand just before
    // its row of MFMAs, so that its expansion overlaps the previous row
    auto mma = [&]() {
        constexpr int SUBS = BITS == 4 ? 2 : 1;
#pragma unroll
        for (int h = 0; h < SUBS; ++h) {
            v4i b[TN];
#pragma unroll
            for (int j = 0; j < TN; ++j) b[j] = operand<BITS>(fb[j], h);
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const v4i a = operand<BITS>(fa[i], h);
#pragma unroll
                for (int j = 0; j < TN; ++j)   // weights as the row operand: see the epilogue
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b[j], a, acc[i][j], 0, 0, 0);
            }
        }
    };
    // acc[i][j] is the 16 x 16 block W_j A_i^T: this lane holds token row
    // lr of A block i and the four consecutive output columns 4 lg .. 4 lg + 3
    // of W block j, so each store is one contiguous 8-byte (fp16) or 16-byte
    // (int32) run and the weight scales come in as one float4.
    // The dequantisation scales of all of this lane's rows and columns are
    // requested together before any is used (indices clamped into range, so no
    // branch separates the loads): one memory round trip per tile rather than
    // one per 16 x 16 block.  Below K = 131072 the scaled sum 256 x dot cannot
    // wrap, so the shift alone recovers the dot product (acc_value's special
    // case is only needed at the largest K).
    auto epilogue = [&](auto NOWRAP) {
        float sa[TM];
        float4 sw[TN];
        if (!SPLIT && Y) {
#pragma unroll
            for (int i = 0; i < TM; ++i) sa[i] = s_a[min(row0 + (wm * TM + i) * 16 + lr, M - 1)];
#pragma unroll
            for (int j = 0; j < TN; ++j)
                sw[j] = *reinterpret_cast<const float4*>(s_w + min(col0 + (wn * TN + j) * 16 + lg * 4, N - 4));
        }
        auto value = [](int raw) { return decltype(NOWRAP)::value && BITS == 4 ? raw >> 8 : acc_value<BITS>(raw); };
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int row = row0 + (wm * TM + i) * 16 + lr;
            if (row >= M) continue;
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int col = col0 + (wn * TN + j) * 16 + lg * 4;   // N % 8 == 0: all four in range or none
                if (col >= N) continue;
                const int v0 = value(acc[i][j][0]), v1 = value(acc[i][j][1]);
                const int v2 = value(acc[i][j][2]), v3 = value(acc[i][j][3]);
                if (SPLIT) {
                    *reinterpret_cast<int4*>(part + ((size_t)blockIdx.z * M + row) * N + col) = make_int4(v0, v1, v2, v3);
                    continue;
                }
                const size_t o = (size_t)row * N + col;
                if (acc_out) *reinterpret_cast<int4*>(acc_out + o) = make_int4(v0, v1, v2, v3);
                if (Y) {
                    const uint32_t y0 = f2h(((float)v0 * sa[i]) * sw[j].x), y1 = f2h(((float)v1 * sa[i]) * sw[j].y);
                    const uint32_t y2 = f2h(((float)v2 * sa[i]) * sw[j].z), y3 = f2h(((float)v3 * sa[i]) * sw[j].w);
                    *reinterpret_cast<uint2*>(Y + o) = make_uint2(y0 | (y1 << 16), y2 | (y3 << 16));
                }
            }
        }
    };

    // step kt lives in stage (kt - kt0) % 3.  At each step the loads of the
    // step itself and of the next one are in flight; after the wait and the
    // barrier the stage of the previous step is free for the step after next.
    auto step = [&](int kt, int sc, int sn) {
        asm volatile("" ::: "memory");
        if (kt + 1 < kt1)
            wait_vm<LA + LB>();                          // this wave's loads of step kt are done
        else
            wait_vm<0>();
        // ... and every wave's.  A bare s_barrier: the workgroup fence of
        // __syncthreads would also wait for the loads still in flight, which
        // is the overlap this pipeline exists for.
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        frags(sm + sc * SB + kg * SG);
        if (kt + 2 < kt1) issue(kt + 2, sn);             // into the stage step kt - 1 used
        mma();
    };
    if (kt0 < kt1) issue(kt0, 0);
    if (kt0 + 1 < kt1) issue(kt0 + 1, 1);
    for (int kt = kt0; kt < kt1; kt += 3) {
        step(kt, 0, 2);
        if (kt + 1 < kt1) step(kt + 1, 1, 0);
        if (kt + 2 < kt1) step(kt + 2, 2, 1);
    }
    if constexpr (KG > 1) {
        // every wave is past its last fragment read: the stages take the partial sums
        __syncthreads();
        v4i* red = reinterpret_cast<v4i*>(sm);           // [KG - 1][NW][TM][TN][lane]
        if (kg > 0) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) red[((((kg - 1) * NW + wave) * TM + i) * TN + j) * kWave + lane] = acc[i][j];
        }
        __syncthreads();
        if (kg > 0) return;
#pragma unroll
        for (int g = 0; g < KG - 1; ++g)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] += red[(((g * NW + wave) * TM + i) * TN + j) * kWave + lane];
    }
    if (K < 131072)
        epilogue(std::true_type{});
    else
        epilogue(std::false_type{});
}

// Short M (<= 16 tokens): every weight is used by at most 16 rows, so these
// kernels are bound by streaming the weights from HBM, not by the MFMA.  One
// 16-row MFMA tile covers all the tokens; each wave owns 16 output columns and
// loads its weight fragments straight into registers (lane (c, g) reads bytes
// [16 g, 16 g + 16) of the 64-byte slice of row c, the tiled kernel's fragment
// order).  The k offset of a load rides in the scalar offset, so issuing a load
// costs no vector instruction; a ring of D batches of U k steps keeps D - 1
// batches in flight while one is multiplied.  There is no branch between a
// batch's loads and their use: a conditional exit there lets the compiler sink
// the loads past the other batch's multiply, which serialises memory and MFMA.
//
// Zeros: k steps past the row read as zero weights (in-range row offset plus an
// out-of-range scalar offset), and the activation bytes past the end of a row
// (the second half of a last, half-filled k step) read as zero activations, so
// a product that mixes in a neighbouring row's bytes is always a product with
// zero.  Rows past M and columns past N are clamped to the last valid one and
// their outputs are not stored.  The dequantisation scales are fetched while
// the weights stream, so the epilogue waits on no load.

// Scalar offset of k step kt: past the last step, one that no buffer reaches.
__device__ __forceinline__ int step_offset(int kt, int nk) { return kt < nk ? kt * kKB : (int)kOOB; }

// Epilogue of the short-M kernels: lane (c, g) holds rows row0 + 4 g .. + 3 of
// output column col.
template <int BITS>
__device__ __forceinline__ void skinny_store(const v4i& acc, int row0, int lg, int col, int M, int N,
                                             const float (&sav)[4], float swv, uint16_t* __restrict__ Y,
                                             int32_t* __restrict__ acc_out) {
    if (col >= N) return;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int row = row0 + 4 * lg + r;
        if (row >= M) continue;
        const int v = acc_value<BITS>(acc[r]);
        const size_t o = (size_t)row * N + col;
        if (acc_out) acc_out[o] = v;
        if (Y) Y[o] = f2h(((float)v * sav[r]) * swv);
    }
}

// Short-M kernels cover M <= 16 TM tokens with TM row tiles of 16, TM <= 3: at
// four row tiles the activation unpacking outweighs what the kernels save over
// the tiled one.
constexpr int kShortMaxTiles = 3;

// KW waves share one group of 16 columns and take turns over k, batch by batch
// (wave w multiplies batches w, w + KW, ...); their partial sums meet in LDS.
// Activation fragments come from global memory (they stay in L2: every
// workgroup reads the same M x K codes).  The K split gives narrow layers
// enough waves to keep HBM busy.
template <int U, int KW, int TM, int BITS>
__global__ __launch_bounds__(64 * KW) void gemm_skinny_kernel(const uint8_t* __restrict__ Aq,
                                                              const float* __restrict__ s_a,
                                                              const uint8_t* __restrict__ Wq,
                                                              const float* __restrict__ s_w, int M, int N, int K,
                                                              uint16_t* __restrict__ Y, int32_t* __restrict__ acc_out) {
    constexpr int D = 2;
    __shared__ v4i red[KW > 1 ? KW - 1 : 1][TM][kWave];
    const int lane = threadIdx.x % kWave, wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lr = lane % 16, lg = lane / 16;
    const int col = blockIdx.x * 16 + lr;
    const uint32_t ldb = (uint32_t)K * BITS / 8;
    const int nk = (int)((ldb + kKB - 1) / kKB);
    const int nb = (nk + U - 1) / U;
    const __amdgpu_buffer_rsrc_t rA = make_rsrc(Aq, (uint32_t)M * ldb);
    const __amdgpu_buffer_rsrc_t rW = make_rsrc(Wq, (uint32_t)N * ldb);
    const uint32_t seg = 16 * lg;
    const uint32_t ow = (uint32_t)min(col, N - 1) * ldb + seg;
    uint32_t oa[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) oa[i] = (uint32_t)min(16 * i + lr, M - 1) * ldb + seg;
    const uint32_t alim = ldb > seg ? ldb - seg : 0;   // this lane's activation bytes end here
    auto issue = [&](int b, v4i (&w)[U], v4i (&a)[U][TM]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kt = b * U + u;
            const int so = step_offset(kt, nk);
            const bool in = (uint32_t)kt * kKB < alim;
            w[u] = __builtin_amdgcn_raw_buffer_load_b128(rW, (int)ow, so, 0);
#pragma unroll
            for (int i = 0; i < TM; ++i)
                a[u][i] = __builtin_amdgcn_raw_buffer_load_b128(rA, in ? (int)oa[i] : (int)kOOB, so, 0);
        }
    };
    v4i acc[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) acc[i] = v4i{0, 0, 0, 0};
    auto compute = [&](const v4i (&w)[U], const v4i (&a)[U][TM]) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int h = 0; h < (BITS == 4 ? 2 : 1); ++h) {
                const v4i wop = operand<BITS>(w[u], h);
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    acc[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(operand<BITS>(a[u][i], h), wop, acc[i], 0, 0, 0);
            }
    };
    v4i w[D][U], a[D][U][TM];
    issue(wave, w[0], a[0]);
    float sav[TM][4];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) sav[i][r] = s_a[min(16 * i + 4 * lg + r, M - 1)];
    const float swv = s_w[min(col, N - 1)];
    int b = wave;
    do {
        issue(b + KW, w[1], a[1]);
        __builtin_amdgcn_sched_barrier(0);
        compute(w[0], a[0]);
        __builtin_amdgcn_sched_barrier(0);
        issue(b + 2 * KW, w[0], a[0]);
        __builtin_amdgcn_sched_barrier(0);
        compute(w[1], a[1]);
        __builtin_amdgcn_sched_barrier(0);
        b += 2 * KW;
    } while (b < nb);
    if (KW > 1) {
        if (wave > 0) {
#pragma unroll
            for (int i = 0; i < TM; ++i) red[wave - 1][i][lane] = acc[i];
        }
        __syncthreads();
        if (wave > 0) return;
#pragma unroll
        for (int r = 0; r < KW - 1; ++r)
#pragma unroll
            for (int i = 0; i < TM; ++i) acc[i] += red[r][i][lane];
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) skinny_store<BITS>(acc[i], 16 * i, lg, col, M, N, sav[i], swv, Y, acc_out);
}

// Wide layers, 4-bit codes: the workgroup's waves (blockDim.x / 64 of them)
// each stream their own 16 columns, and the M x K activation codes are staged
// once per workgroup in LDS by a direct-to-LDS copy (zero past M and K), instead
// of being fetched by every wave.  With one row tile (M <= 16) they are then
// expanded once, by all waves together, to MFMA operands ([k step][half][lane]
// [16 B]); with more row tiles each wave expands its fragments as it multiplies
// (the expanded copy would not fit).  The weight ring is issued before the copy
// is waited on, so the first batches are already in flight.
constexpr int kSharedU = 2, kSharedD = 4;
constexpr int kSharedMaxSteps = 32;                 // one row tile, K <= 4096: 96 KB of LDS
constexpr int kSharedMaxTileSteps = 128;            // more row tiles: row tiles x k steps <= 128 (128 KB)
constexpr int kSharedMaxWaves = 16;

template <int TM>
__global__ __launch_bounds__(64 * kSharedMaxWaves) void gemm_skinny_shared_kernel(
    const uint8_t* __restrict__ Aq, const float* __restrict__ s_a, const uint8_t* __restrict__ Wq,
    const float* __restrict__ s_w, int M, int N, int K, uint16_t* __restrict__ Y, int32_t* __restrict__ acc_out) {
    constexpr int U = kSharedU, D = kSharedD;
    constexpr bool kExpand = TM == 1;
    extern __shared__ __attribute__((aligned(16))) uint8_t sm[];
    const int nw = blockDim.x / kWave;
    const int lane = threadIdx.x % kWave, wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lr = lane % 16, lg = lane / 16;
    const int col = (blockIdx.x * nw + wave) * 16 + lr;
    const uint32_t ldb = (uint32_t)K / 2;
    const int nk = (int)((ldb + kKB - 1) / kKB);
    const int nb = (nk + U - 1) / U;
    uint8_t* raw = sm;                   // [TM][nk] x 1 KB: packed activation fragments
    uint8_t* ops = sm + nk * 1024;       // one row tile: nk x 2 KB of expanded operands
    const u32x4 rA = sgpr_rsrc(Aq, (uint32_t)M * ldb);
    const __amdgpu_buffer_rsrc_t rW = make_rsrc(Wq, (uint32_t)N * ldb);
    const uint32_t seg = 16 * lg;
    for (int p = wave; p < TM * nk; p += nw) {
        const int row = 16 * (p / nk) + lr;
        const uint32_t ko = (uint32_t)(p % nk) * kKB;
        dma16(rA, lds_addr(raw + p * 1024), (row < M && ko + seg < ldb) ? (uint32_t)row * ldb + ko + seg : kOOB);
    }
    const uint32_t ow = (uint32_t)min(col, N - 1) * ldb + seg;
    auto issue = [&](int b, v4i (&w)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u)
            w[u] = __builtin_amdgcn_raw_buffer_load_b128(rW, (int)ow, step_offset(b * U + u, nk), 0);
    };
    v4i w[D][U];
#pragma unroll
    for (int d = 0; d < D - 1; ++d) issue(d, w[d]);
    wait_vm<(D - 1) * U>();              // this wave's copies have landed (its weight loads may not have)
    __builtin_amdgcn_s_barrier();        // ... and every wave's
    asm volatile("" ::: "memory");
    if (kExpand) {
        for (int s = wave; s < nk; s += nw) {
            const v4i r = *reinterpret_cast<const v4i*>(raw + s * 1024 + lane * 16);
            *reinterpret_cast<v4i*>(ops + (2 * s) * 1024 + lane * 16) = operand<4>(r, 0);
            *reinterpret_cast<v4i*>(ops + (2 * s + 1) * 1024 + lane * 16) = operand<4>(r, 1);
        }
        __syncthreads();
    }
    float sav[TM][4];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) sav[i][r] = s_a[min(16 * i + 4 * lg + r, M - 1)];
    const float swv = s_w[min(col, N - 1)];
    v4i acc[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) acc[i] = v4i{0, 0, 0, 0};
    auto compute = [&](int b, const v4i (&wb)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kt = min(b * U + u, nk - 1);      // past the end the weights read as zero
            v4i ar[TM];
            if (!kExpand) {
#pragma unroll
                for (int i = 0; i < TM; ++i) ar[i] = *reinterpret_cast<const v4i*>(raw + (i * nk + kt) * 1024 + lane * 16);
            }
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const v4i wop = operand<4>(wb[u], h);
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    const v4i x = kExpand ? *reinterpret_cast<const v4i*>(ops + (2 * kt + h) * 1024 + lane * 16)
                                          : operand<4>(ar[i], h);
                    acc[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(x, wop, acc[i], 0, 0, 0);
                }
            }
        }
    };
    int b = 0;
    do {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            issue(b + d + D - 1, w[(d + D - 1) % D]);
            __builtin_amdgcn_sched_barrier(0);
            compute(b + d, w[d]);
            __builtin_amdgcn_sched_barrier(0);
        }
        b += D;
    } while (b < nb);
#pragma unroll
    for (int i = 0; i < TM; ++i) skinny_store<4>(acc[i], 16 * i, lg, col, M, N, sav[i], swv, Y, acc_out);
}

// Short M on fragment-ordered weights.  The weights of 16 columns at one k step
// are one 1 KB block in the MFMA fragment order (lane l's 16 bytes at 16 l), the
// blocks of one k step side by side, so every weight load of a wave reads 1 KB
// of consecutive bytes and neighbouring waves read neighbouring blocks
// (row-major weights give 16 runs of 64 bytes per load, which the memory system
// serves markedly slower), with the non-temporal hint, as nothing reuses them.  A workgroup holds CG column groups
// times KW waves that take turns over k (wave w of a group multiplies batches
// w, w + KW, ...; partial sums meet in LDS).  Activation fragments are staged
// once per workgroup in LDS (ALDS) or, for narrow layers whose few column
// groups leave each workgroup little weight to stream, read from L2 by each
// wave, which does not wait for a whole-workgroup copy before its first
// multiply.  A ring of D batches of U k steps keeps D - 1 batches in flight;
// zero handling and epilogue as in the kernels above; the weights past K and
// past N read as zero from the layout's own padding.
constexpr int kFragNT = 2;                             // buffer-load cache policy: non-temporal
constexpr size_t kFragMaxLds = 160 * 1024;

template <int TM, int KW, bool ALDS, int U, int D, int BITS = 4>
__global__ __launch_bounds__(ALDS ? 1024 : 512) void gemm_short_frag_kernel(
    const uint8_t* __restrict__ Aq, const float* __restrict__ s_a, const uint8_t* __restrict__ Wf,
    const float* __restrict__ s_w, int M, int N, int K, uint16_t* __restrict__ Y, int32_t* __restrict__ acc_out) {
    extern __shared__ __attribute__((aligned(16))) uint8_t sm[];
    const int CG = blockDim.x / kWave / KW;
    const int lane = threadIdx.x % kWave, wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int cgi = wave % CG, kw = wave / CG;
    const int lr = lane % 16, lg = lane / 16;
    const int ngrp = (N + 15) / 16;
    const int grp = blockIdx.x * CG + cgi;
    const int col = grp * 16 + lr;
    const uint32_t ldb = (uint32_t)K * BITS / 8;
    const int nk = (int)((ldb + kKB - 1) / kKB);
    const int nb = (nk + U - 1) / U;
    const uint32_t seg = 16 * lg;
    uint8_t* raw = sm;                                         // ALDS: [TM][nk] x 1 KB of activation fragments
    v4i* red = reinterpret_cast<v4i*>(sm + (ALDS ? (size_t)TM * nk * 1024 : 0));   // [KW - 1][CG][TM][lane]
    const __amdgpu_buffer_rsrc_t rW = make_rsrc(Wf, (uint32_t)ngrp * nk * 1024);
    const __amdgpu_buffer_rsrc_t rA = make_rsrc(Aq, (uint32_t)M * ldb);
    if (ALDS) {
        const u32x4 rAs = sgpr_rsrc(Aq, (uint32_t)M * ldb);
        for (int p = wave; p < TM * nk; p += blockDim.x / kWave) {
            const int row = 16 * (p / nk) + lr;
            const uint32_t ko = (uint32_t)(p % nk) * kKB;
            dma16(rAs, lds_addr(raw + p * 1024), (row < M && ko + seg < ldb) ? (uint32_t)row * ldb + ko + seg : kOOB);
        }
    }
    uint32_t oa[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) oa[i] = (uint32_t)min(16 * i + lr, M - 1) * ldb + seg;
    const uint32_t alim = ldb > seg ? ldb - seg : 0;   // this lane's activation bytes end here
    const uint32_t ow = (uint32_t)min(grp, ngrp - 1) * 1024 + lane * 16;
    const int kstride = ngrp * 1024;                   // bytes from one k step to the next
    auto issue = [&](int b, v4i (&w)[U], v4i (&a)[U][TM]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kt = b * U + u;
            w[u] = __builtin_amdgcn_raw_buffer_load_b128(rW, (int)ow, kt < nk ? kt * kstride : (int)kOOB, kFragNT);
            if (!ALDS) {
                const bool in = (uint32_t)kt * kKB < alim;
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    a[u][i] = __builtin_amdgcn_raw_buffer_load_b128(rA, in ? (int)oa[i] : (int)kOOB, step_offset(kt, nk), 0);
            }
        }
    };
    v4i w[D][U];
    v4i a[ALDS ? 1 : D][U][TM];
#pragma unroll
    for (int d = 0; d < D - 1; ++d) issue(kw + d * KW, w[d], a[ALDS ? 0 : d]);
    if (ALDS) {
        wait_vm<(D - 1) * U>();          // this wave's copies have landed (its weight loads may not have)
        __builtin_amdgcn_s_barrier();    // ... and every wave's
        asm volatile("" ::: "memory");
    }
    float sav[TM][4];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) sav[i][r] = s_a[min(16 * i + 4 * lg + r, M - 1)];
    const float swv = s_w[min(col, N - 1)];
    v4i acc[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) acc[i] = v4i{0, 0, 0, 0};
    auto compute = [&](int b, const v4i (&wb)[U], const v4i (&ab)[U][TM]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kt = min(b * U + u, nk - 1);      // past the end the weights read as zero
            v4i ar[TM];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                ar[i] = ALDS ? *reinterpret_cast<const v4i*>(raw + (i * nk + kt) * 1024 + lane * 16) : ab[u][i];
#pragma unroll
            for (int h = 0; h < (BITS == 4 ? 2 : 1); ++h) {
                const v4i wop = operand<BITS>(wb[u], h);
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    acc[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(operand<BITS>(ar[i], h), wop, acc[i], 0, 0, 0);
            }
        }
    };
    int b = kw;
    do {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            issue(b + (d + D - 1) * KW, w[(d + D - 1) % D], a[ALDS ? 0 : (d + D - 1) % D]);
            __builtin_amdgcn_sched_barrier(0);
            compute(b + d * KW, w[d], a[ALDS ? 0 : d]);
            __builtin_amdgcn_sched_barrier(0);
        }
        b += D * KW;
    } while (b < nb);
    if (KW > 1) {
        if (kw > 0) {
#pragma unroll
            for (int i = 0; i < TM; ++i) red[(((kw - 1) * CG + cgi) * TM + i) * kWave + lane] = acc[i];
        }
        __syncthreads();
        if (kw > 0) return;
#pragma unroll
        for (int r = 0; r < KW - 1; ++r)
#pragma unroll
            for (int i = 0; i < TM; ++i) acc[i] += red[((r * CG + cgi) * TM + i) * kWave + lane];
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) skinny_store<BITS>(acc[i], 16 * i, lg, col, M, N, sav[i], swv, Y, acc_out);
}

// Packed int4 weights [N][K/2] -> fragment order: one thread per 16-byte unit
// (k step t, group g, lane l) = bytes 64 t + 16 (l / 16) .. + 15 of row
// 16 g + l % 16, zero past N and past the row.
__global__ __launch_bounds__(256) void weights_to_frag_kernel(const uint8_t* __restrict__ Wq, int N, int K,
                                                              uint8_t* __restrict__ Wf) {
    const uint32_t ldb = (uint32_t)K / 2;
    const uint32_t nk = (ldb + kKB - 1) / kKB;
    const uint32_t ngrp = (uint32_t)(N + 15) / 16;
    const size_t units = (size_t)ngrp * nk * kWave;
    for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < units; e += (size_t)gridDim.x * 256) {
        const uint32_t l = (uint32_t)(e % kWave);
        const size_t tg = e / kWave;
        const uint32_t g = (uint32_t)(tg % ngrp), t = (uint32_t)(tg / ngrp);
        const uint32_t row = 16 * g + l % 16, byte = t * kKB + 16 * (l / 16);
        v4i v = v4i{0, 0, 0, 0};
        if (row < (uint32_t)N && byte < ldb) v = *reinterpret_cast<const v4i*>(Wq + (size_t)row * ldb + byte);
        *reinterpret_cast<v4i*>(Wf + e * 16) = v;
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
    int cfg;       // 0: 256 x 128, 1: 128 x 128, 2: 64 x 64, 4: 64 x 128, 7: 128 x 256 (8-bit), 8: 128 x 128
                   // in two waves of 128 x 64 (8-bit), 9: 128 x 128 in two k groups of four waves,
                   // 3: short M, K split in the
                   // workgroup, 5: short M, activations shared in LDS (see launch_gemm), 6: short M on
                   // fragment-ordered weights (see launch_gemm_frag)
    int bm, bn;
    int splits;    // K split count across workgroups actually used (1 = fused epilogue)
    int per;       // k steps per split
    int waves;     // cfg 3: waves sharing a column group over k; cfg 5: waves per workgroup;
                   // cfg 6: column groups per workgroup
    int kw;        // cfg 6: waves per column group, taking turns over k
    bool alds;     // cfg 6: activation fragments staged in LDS (else read from L2)
    int u, d;      // cfg 6: k steps per batch, batches in the register ring
};

Plan make_plan(int M, int N, int K, int bm, int bn, int want_splits, int bits = 4) {
    (void)M;
    (void)N;
    Plan p;
    p.cfg = -1;
    p.waves = 1;
    p.kw = 1;
    p.alds = false;
    p.u = 2;
    p.d = 4;
    p.bm = bm;
    p.bn = bn;
    const int nk = (K * bits / 8 + kKB - 1) / kKB;
    const int s = want_splits < 1 ? 1 : (want_splits > nk ? nk : want_splits);
    p.per = (nk + s - 1) / s;
    p.splits = (nk + p.per - 1) / p.per;
    return p;
}

template <int U, int KW, int TM, int BITS>
hipError_t launch_skinny(const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w, int M, int N,
                         int K, uint16_t* Y, int32_t* acc, hipStream_t st) {
    hipLaunchKernelGGL((gemm_skinny_kernel<U, KW, TM, BITS>), dim3((N + 15) / 16), dim3(64 * KW), 0, st, Aq, s_a, Wq,
                       s_w, M, N, K, Y, acc);
    return hipGetLastError();
}

// Bytes of dynamic LDS the shared-activation kernel needs, 0 if it cannot run.
size_t shared_lds_bytes(int tiles, int nk) {
    if (tiles == 1) return nk <= kSharedMaxSteps ? (size_t)nk * 3 * 1024 : 0;
    return tiles * nk <= kSharedMaxTileSteps ? (size_t)tiles * nk * 1024 : 0;
}

template <int TM>
hipError_t launch_skinny_shared_tm(int waves, const uint8_t* Aq, const float* s_a, const uint8_t* Wq,
                                   const float* s_w, int M, int N, int K, uint16_t* Y, int32_t* acc, hipStream_t st) {
    const int nk = (K / 2 + kKB - 1) / kKB;
    const size_t lds = shared_lds_bytes(TM, nk);
    static std::atomic<int> lds_set[kMaxDevices];   // above the 64 KB default for dynamic LDS
    const hipError_t attr =
        allow_dynamic_lds(reinterpret_cast<const void*>(&gemm_skinny_shared_kernel<TM>),
                          (int)(TM == 1 ? kSharedMaxSteps * 3 * 1024 : kSharedMaxTileSteps * 1024), lds_set);
    if (attr != hipSuccess) return attr;
    if (lds == 0 || waves < 1 || waves > kSharedMaxWaves) return hipErrorInvalidConfiguration;
    const int groups = (N + 15) / 16;
    hipLaunchKernelGGL((gemm_skinny_shared_kernel<TM>), dim3((groups + waves - 1) / waves), dim3(64 * waves), lds,
                       st, Aq, s_a, Wq, s_w, M, N, K, Y, acc);
    return hipGetLastError();
}

hipError_t launch_skinny_shared(int waves, const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w,
                                int M, int N, int K, uint16_t* Y, int32_t* acc, hipStream_t st) {
    switch ((M + 15) / 16) {
        case 1: return launch_skinny_shared_tm<1>(waves, Aq, s_a, Wq, s_w, M, N, K, Y, acc, st);
        case 2: return launch_skinny_shared_tm<2>(waves, Aq, s_a, Wq, s_w, M, N, K, Y, acc, st);
        case 3: return launch_skinny_shared_tm<3>(waves, Aq, s_a, Wq, s_w, M, N, K, Y, acc, st);
        default: return hipErrorInvalidConfiguration;
    }
}

template <int WM, int WN, int TM, int TN, int BITS = 4, int OCC = 1, bool WF = false, int KG = 1>
hipError_t launch_tiled(const Plan& p, const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w,
                       int M, int N, int K, uint16_t* Y, int32_t* acc, int32_t* part, hipStream_t st) {
    const size_t tiles = (size_t)((N + p.bn - 1) / p.bn) * (size_t)((M + p.bm - 1) / p.bm);
    if (tiles > 0x7fffffffu) return hipErrorInvalidConfiguration;
    dim3 grid((unsigned)tiles, 1, p.splits);
    dim3 block(64 * WM * WN * KG);
    if (p.splits == 1) {
        hipLaunchKernelGGL((gemm_tile_kernel<WM, WN, TM, TN, false, BITS, OCC, WF, KG>), grid, block, 0, st, Aq, s_a,
                           Wq, s_w, M, N, K, p.per, Y, acc, (int32_t*)nullptr);
    } else if constexpr (KG == 1) {
        hipLaunchKernelGGL((gemm_tile_kernel<WM, WN, TM, TN, true, BITS, OCC, WF>), grid, block, 0, st, Aq, s_a, Wq,
                           s_w, M, N, K, p.per, (uint16_t*)nullptr, (int32_t*)nullptr, part);
    } else {
        return hipErrorInvalidConfiguration;
    }
    return hipGetLastError();
}

// Dynamic LDS of the fragment-ordered short-M kernel.
size_t frag_lds_bytes(int tm, int nk, int kw, int cg, bool alds) {
    return (alds ? (size_t)tm * nk * 1024 : 0) + (kw > 1 ? (size_t)(kw - 1) * cg * tm * 1024 : 0);
}

template <int TM, int KW, bool ALDS, int U, int D, int BITS>
hipError_t launch_short_frag_t(const Plan& p, const uint8_t* Aq, const float* s_a, const uint8_t* Wf,
                               const float* s_w, int M, int N, int K, uint16_t* Y, int32_t* acc, hipStream_t st) {
    const int nk = (K * BITS / 8 + kKB - 1) / kKB;
    const size_t lds = frag_lds_bytes(TM, nk, KW, p.waves, ALDS);
    static std::atomic<int> lds_set[kMaxDevices];   // above the 64 KB default for dynamic LDS
    const hipError_t attr = allow_dynamic_lds(
        reinterpret_cast<const void*>(&gemm_short_frag_kernel<TM, KW, ALDS, U, D, BITS>), (int)kFragMaxLds, lds_set);
    if (attr != hipSuccess) return attr;
    if (lds > kFragMaxLds || p.waves < 1 || p.waves * KW > (ALDS ? 16 : 8)) return hipErrorInvalidConfiguration;
    const int groups = (N + 15) / 16;
    hipLaunchKernelGGL((gemm_short_frag_kernel<TM, KW, ALDS, U, D, BITS>), dim3((groups + p.waves - 1) / p.waves),
                       dim3(64 * p.waves * KW), lds, st, Aq, s_a, Wf, s_w, M, N, K, Y, acc);
    return hipGetLastError();
}

// The (waves per group, activation staging, batch, ring) combinations the plan uses.
template <int TM, int BITS>
hipError_t launch_short_frag_tm(const Plan& p, const uint8_t* Aq, const float* s_a, const uint8_t* Wf,
                                const float* s_w, int M, int N, int K, uint16_t* Y, int32_t* acc, hipStream_t st) {
    if (p.alds) {
        if (p.d != 4) return hipErrorInvalidConfiguration;
        switch (p.kw * 4 + p.u) {
            case 5: return launch_short_frag_t<TM, 1, true, 1, 4, BITS>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
            case 6: return launch_short_frag_t<TM, 1, true, 2, 4, BITS>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
            case 9: return launch_short_frag_t<TM, 2, true, 1, 4, BITS>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
            case 10: return launch_short_frag_t<TM, 2, true, 2, 4, BITS>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
            default: return hipErrorInvalidConfiguration;
        }
    }
    if (p.u != 2) return hipErrorInvalidConfiguration;
    switch (p.kw * 8 + p.d) {
        case 12: return launch_short_frag_t<TM, 1, false, 2, 4, BITS>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
        case 20: return launch_short_frag_t<TM, 2, false, 2, 4, BITS>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
        case 34: return launch_short_frag_t<TM, 4, false, 2, 2, BITS>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
        case 36: return launch_short_frag_t<TM, 4, false, 2, 4, BITS>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
        default: return hipErrorInvalidConfiguration;
    }
}

template <int BITS>
hipError_t launch_short_frag_bits(const Plan& p, const uint8_t* Aq, const float* s_a, const uint8_t* Wf,
                                  const float* s_w, int M, int N, int K, uint16_t* Y, int32_t* acc, hipStream_t st) {
    switch ((M + 15) / 16) {
        case 1: return launch_short_frag_tm<1, BITS>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
        case 2: return launch_short_frag_tm<2, BITS>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
        case 3: return launch_short_frag_tm<3, BITS>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
        case 4:   // four row tiles only for 4-bit codes (frag_four_tiles)
            if constexpr (BITS == 4) return launch_short_frag_tm<4, BITS>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
            return hipErrorInvalidConfiguration;
        default: return hipErrorInvalidConfiguration;
    }
}

hipError_t launch_short_frag(const Plan& p, const uint8_t* Aq, const float* s_a, const uint8_t* Wf, const float* s_w,
                             int M, int N, int K, uint16_t* Y, int32_t* acc, hipStream_t st, int bits) {
    return bits == 8 ? launch_short_frag_bits<8>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st)
                     : launch_short_frag_bits<4>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, st);
}

// Fragment-ordered weights at 49 ... 64 tokens: the short-M kernel with four
// row tiles where it beats the tiled plan (its K split and separate reduction),
// measured at 64 tokens: layers up to 12288 wide with K <= 4096 (LLaDA QKV 15.9
// -> 12.8 us, O 10.2 -> 8.5; Dream QKV 10.5 -> 10.0, O 9.8 -> 8.0).  Wider or
// deeper layers stay tiled (gate+up 17.1 against 19.3 us, down 14.9 against
// 17.6): there each wave's expansion of four activation fragments per weight
// fragment costs more than the tiled plan loses.
bool frag_four_tiles(int M, int N, int K) { return M > 48 && M <= 64 && N <= 12288 && K <= 4096; }

template <int TM, int BITS>
hipError_t skinny_kw_tm(int kw, const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w, int M, int N,
                        int K, uint16_t* Y, int32_t* acc, hipStream_t st) {
    // two register batches of U k steps in flight: 8 steps per batch for one row
    // tile and up to two waves per column group, 4 for four or eight waves, 2 for
    // more row tiles (each step holds TM + 1 fragments)
    constexpr int U1 = TM == 1 ? 8 : 2, U4 = TM == 1 ? 4 : 2;
    switch (kw) {
        case 1: return launch_skinny<U1, 1, TM, BITS>(Aq, s_a, Wq, s_w, M, N, K, Y, acc, st);
        case 2: return launch_skinny<U1, 2, TM, BITS>(Aq, s_a, Wq, s_w, M, N, K, Y, acc, st);
        case 4: return launch_skinny<U4, 4, TM, BITS>(Aq, s_a, Wq, s_w, M, N, K, Y, acc, st);
        default: return launch_skinny<U4, 8, TM, BITS>(Aq, s_a, Wq, s_w, M, N, K, Y, acc, st);
    }
}

template <int BITS>
hipError_t skinny_kw(int kw, const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w, int M, int N,
                     int K, uint16_t* Y, int32_t* acc, hipStream_t st) {
    switch ((M + 15) / 16) {
        case 1: return skinny_kw_tm<1, BITS>(kw, Aq, s_a, Wq, s_w, M, N, K, Y, acc, st);
        case 2: return skinny_kw_tm<2, BITS>(kw, Aq, s_a, Wq, s_w, M, N, K, Y, acc, st);
        case 3: return skinny_kw_tm<3, BITS>(kw, Aq, s_a, Wq, s_w, M, N, K, Y, acc, st);
        default: return hipErrorInvalidConfiguration;
    }
}

hipError_t finish_split(const Plan& p, int32_t* part, const float* s_a, const float* s_w, int M, int N, uint16_t* Y,
                        int32_t* acc, hipStream_t st) {
    if (p.splits == 1) return hipSuccess;
    const size_t total = (size_t)M * N;
    const int blocks = (int)((total + 255) / 256 < 4096 ? (total + 255) / 256 : 4096);
    hipLaunchKernelGGL(splitk_epilogue, dim3(blocks), dim3(256), 0, st, part, p.splits, s_a, s_w, M, N, Y, acc);
    return hipGetLastError();
}

// The production plan (from measured sweeps on MI355X, graph-replayed with
// rotating weights):
//  - M <= 48: the short-M kernels (weight streaming; activations shared in LDS
//    for wide 4-bit layers, K split inside the workgroup otherwise);
//  - 4-bit codes with at least 448 tiles of 256 x 128 or of 128 x 128:
//    256 x 128 (eight waves of 64 x 64) at 448 ... 512 tiles of it, else
//    128 x 128 (four waves of 64 x 64) (see below);
//  - 8-bit codes (one MFMA per 64-byte k step, so operand reads from LDS weigh
//    twice as much per MFMA as for 4-bit codes): larger wave tiles.  128 x 256
//    (four waves of 64 x 128, two workgroups per CU; each wave reads 12
//    fragments per 32 MFMAs where 64 x 64 reads 8 per 16) from 512 of its
//    tiles; else 128 x 128 in two waves of 128 x 64 from 640 of its tiles
//    (three workgroups per CU fill the chip at 768); else 128 x 256 from 192
//    of its tiles; else 128 x 128 (four waves) from 192 of its tiles;
//  - 129 ... 256 tiles of 128 x 128 and at least 128 k steps (64 for 8-bit
//    codes): 128 x 128 with two k groups of four waves (see below);
//  - at least 512 tiles of 64 x 128: 64 x 128 (four waves of 64 x 32);
//  - otherwise 64 x 64 (four waves of 32 x 32), with K split below 256 tiles
//    (twice as deep for K >= 8192) and kept at 8 k steps or more per split.
Plan choose_plan(int M, int N, int K, int bits) {
    const int nk = (K * bits / 8 + kKB - 1) / kKB;
    auto tiles = [&](int bm, int bn) { return ((M + bm - 1) / bm) * ((N + bn - 1) / bn); };
    auto splits_for = [&](int t) {
        int s = t >= 256 ? 1 : (256 + t - 1) / t;
        if (K >= 8192 && t <= 256) s *= 2;
        const int cap = nk / 8 > 1 ? nk / 8 : 1;
        s = s < cap ? s : cap;
        return s < 32 ? s : 32;
    };
    Plan p;
    if (M <= 16 * kShortMaxTiles) {
        // one wave per 16 columns, all M <= 48 tokens in its MFMA row tiles.  Wide
        // 4-bit layers whose activation codes fit in LDS share them among
        // ceil(groups / 256) waves per workgroup (one workgroup per CU); the rest
        // split K inside the workgroup, the more ways the fewer column groups
        // there are, keeping two batches per wave
        const int groups = (N + 15) / 16;
        const int tm = (M + 15) / 16;
        p = make_plan(M, N, K, 16 * tm, 16, 1, bits);
        if (bits == 4 && groups >= 768 && shared_lds_bytes(tm, nk) > 0) {
            p.cfg = 5;
            p.waves = (groups + 255) / 256 < kSharedMaxWaves ? (groups + 255) / 256 : kSharedMaxWaves;
        } else {
            const int u1 = tm == 1 ? 8 : 2, u4 = tm == 1 ? 4 : 2;
            int kw = groups >= 1024 ? 1 : groups >= 256 ? 2 : groups >= 128 ? 4 : 8;
            while (kw > 1 && (nk + (kw <= 2 ? u1 : u4) - 1) / (kw <= 2 ? u1 : u4) < 2 * kw) kw /= 2;
            p.cfg = 3;
            p.waves = kw;
        }
    } else if (tiles(128, 128) > 128 && tiles(128, 128) <= 256 && nk >= (bits == 8 ? 64 : 128)) {
        // at most one 128 x 128 tile per CU and a deep K: two k groups of four
        // waves per tile (interleaved timings with rotating weights against the
        // plans below: 8-bit 1024 x 4096 x 4096 13 % faster, 1024 x 4096 x 12288
        // 15 %, 256 x 12288 x 4096 9 %, 1024 x 3584 x 18944 18 %; 4-bit
        // 1024 x 3584 x 18944 17 %, but 4 % slower at 1024 x 4096 x 12288 (96
        // k steps) and 6 % at 768 x 4096 x 12288, hence 128 k steps for 4-bit)
        p = make_plan(M, N, K, 128, 128, 1, bits);
        p.cfg = 9;
    } else if (bits == 4 && (tiles(256, 128) >= 448 || tiles(128, 128) >= 448)) {
        // 4-bit codes, from interleaved graph-replayed timings of both plans on
        // the layer-set shapes at 512 ... 16384 tokens: 256 x 128 wins only when
        // its 448 ... 512 tiles fill one round of two workgroups per CU (4096
        // tokens of the 3584- and 4096-wide layers, by 2-7 %); everywhere else
        // 128 x 128 (three workgroups per CU) is as fast or faster, by up to
        // 16 % where the 256 x 128 tiles leave a partly filled last round
        // (16384 x 4608: 6 % ; 4096 x 4608: 16 %) and 10 % over 64 x 128 at
        // 448 ... 511 tiles of 128 x 128
        const bool big = tiles(256, 128) >= 448 && tiles(256, 128) <= 512;
        p = make_plan(M, N, K, big ? 256 : 128, 128, 1, bits);
        p.cfg = big ? 0 : 1;
    } else if (bits == 8 && tiles(128, 256) >= 512) {
        // 8-bit codes, from timings with rotating weights of the LLaDA-shaped
        // layers at 128 ... 4096 tokens: 128 x 256 from 512 of its tiles 2-14 %
        // faster than 256 x 128 in eight waves; 768 tiles of 128 x 128 in two
        // waves (512 x 24576, 1024 x 12288) 12-15 % faster than four waves or
        // 128 x 256; 128 x 256 at 192 ... 511 of its tiles 9-16 % faster than
        // 128 x 128; below that 128 x 128 in four waves (1024 tokens of the
        // 4096-wide layers: 11-39 % faster than the larger tiles)
        p = make_plan(M, N, K, 128, 256, 1, bits);
        p.cfg = 7;
    } else if (bits == 8 && tiles(128, 128) >= 640) {
        p = make_plan(M, N, K, 128, 128, 1, bits);
        p.cfg = 8;
    } else if (bits == 8 && tiles(128, 256) >= 192) {
        p = make_plan(M, N, K, 128, 256, 1, bits);
        p.cfg = 7;
    } else if (bits == 8 && tiles(128, 128) >= 192) {
        p = make_plan(M, N, K, 128, 128, 1, bits);
        p.cfg = 1;
    } else if (tiles(128, 128) >= 512) {
        p = make_plan(M, N, K, 128, 128, 1, bits);
        p.cfg = 1;
    } else if (tiles(64, 128) >= 512) {
        p = make_plan(M, N, K, 64, 128, 1, bits);
        p.cfg = 4;
    } else {
        p = make_plan(M, N, K, 64, 64, splits_for(tiles(64, 64)), bits);
        p.cfg = 2;
    }
    return p;
}

// Fragment-ordered weights, M <= 48 (from graph-replayed sweeps with rotating
// weights): at most about one workgroup per CU.  Wide layers (>= 1024 column
// groups): one wave per column group, activations in LDS; mid-width (>= 384):
// two waves per column group, activations in LDS; 257-383 groups: two waves per
// group, two groups per workgroup, activations in LDS (one group per workgroup
// would leave some CUs twice the work of the rest); up to 256: four waves per
// column group, one group per workgroup, activations from L2, a ring of two
// batches from 17 tokens on.  Batches of two k steps, or of one where that
// leaves fewer zero-weight k steps in the last pass of the ring.  At least two
// batches per wave.
Plan choose_frag_short(int M, int N, int K, int bits) {
    const int nk = (K * bits / 8 + kKB - 1) / kKB, nb = (nk + 1) / 2;
    const int groups = (N + 15) / 16, tm = (M + 15) / 16;
    Plan p = make_plan(M, N, K, 16 * tm, 16, 1, bits);
    p.cfg = 6;
    int kw, cg;
    bool alds;
    if (groups >= 1024) {
        kw = 1, cg = (groups + 255) / 256, alds = true;
    } else if (groups >= 384) {
        kw = 2, cg = tm == 1 ? (groups + 255) / 256 : (groups + 191) / 192, alds = true;
    } else if (groups > 256) {
        kw = 2, cg = 2, alds = true;
    } else {
        kw = 4, cg = 1, alds = false;
    }
    while (kw > 1 && nb < 2 * kw) kw /= 2;
    const int cg0 = cg;
    if (alds) {   // staged activations that do not fit in LDS are read from L2 instead
        cg = cg < 16 / kw ? cg : 16 / kw;
        while (cg > 1 && frag_lds_bytes(tm, nk, kw, cg, true) > kFragMaxLds) --cg;
        alds = frag_lds_bytes(tm, nk, kw, cg, true) <= kFragMaxLds;
    }
    if (!alds) cg = cg0 < 8 / kw ? cg0 : 8 / kw;
    p.waves = cg;
    p.kw = kw;
    p.alds = alds;
    p.d = !alds && kw == 4 && tm > 1 ? 2 : 4;
    // k steps a wave multiplies past the end: its batches rounded up to whole passes of the ring
    auto waste = [&](int u) {
        const int batches = (nk + u - 1) / u, per_wave = (batches + kw - 1) / kw;
        return (((per_wave + p.d - 1) / p.d) * p.d * kw - batches) * u;
    };
    p.u = alds && waste(1) < waste(2) ? 1 : 2;
    return p;
}

}  // namespace

size_t frag_weight_bytes(int N, int K) {
    return (size_t)((N + 15) / 16) * (size_t)((K / 2 + kKB - 1) / kKB) * 1024;
}

hipError_t launch_weights_to_frag(const uint8_t* Wq, int N, int K, uint8_t* Wf, hipStream_t st) {
    const size_t units = frag_weight_bytes(N, K) / 16;
    const size_t blocks = (units + 255) / 256;
    hipLaunchKernelGGL(weights_to_frag_kernel, dim3((unsigned)(blocks < 16384 ? blocks : 16384)), dim3(256), 0, st, Wq,
                       N, K, Wf);
    return hipGetLastError();
}

hipError_t launch_gemm_frag(const uint8_t* Aq, const float* s_a, const uint8_t* Wf, const float* s_w, int M, int N,
                            int K, uint16_t* Y, int32_t* acc, void* ws, hipStream_t st, int bits) {
    if (M <= 16 * kShortMaxTiles || (bits == 4 && frag_four_tiles(M, N, K)))
        return launch_short_frag(choose_frag_short(M, N, K, bits), Aq, s_a, Wf, s_w, M, N, K, Y, acc, st, bits);
    const Plan p = choose_plan(M, N, K, bits);   // the tiled plans of row-major weights
    int32_t* part = static_cast<int32_t*>(ws);
    hipError_t e;
    if (bits == 8) {
        switch (p.cfg) {
            case 7: e = launch_tiled<2, 2, 4, 8, 8, 2, true>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, part, st); break;
            case 9: e = launch_tiled<2, 2, 4, 4, 8, 2, true, 2>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, part, st); break;
            case 8: e = launch_tiled<1, 2, 8, 4, 8, 2, true>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, part, st); break;
            case 1: e = launch_tiled<2, 2, 4, 4, 8, 3, true>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, part, st); break;
            case 2: e = launch_tiled<2, 2, 2, 2, 8, 4, true>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, part, st); break;
            default: e = launch_tiled<1, 4, 4, 2, 8, 4, true>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, part, st); break;
        }
    } else {
        switch (p.cfg) {
            case 0: e = launch_tiled<4, 2, 4, 4, 4, 2, true>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, part, st); break;
            case 9: e = launch_tiled<2, 2, 4, 4, 4, 2, true, 2>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, part, st); break;
            case 1: e = launch_tiled<2, 2, 4, 4, 4, 3, true>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, part, st); break;
            case 2: e = launch_tiled<2, 2, 2, 2, 4, 4, true>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, part, st); break;
            default: e = launch_tiled<1, 4, 4, 2, 4, 4, true>(p, Aq, s_a, Wf, s_w, M, N, K, Y, acc, part, st); break;
        }
    }
    if (e != hipSuccess) return e;
    return finish_split(p, part, s_a, s_w, M, N, Y, acc, st);
}

size_t gemm_workspace_bytes(int M, int N, int K, int bits) {
    const Plan p = choose_plan(M, N, K, bits);
    return p.splits > 1 ? (size_t)p.splits * M * N * sizeof(int32_t) : 0;
}

hipError_t launch_gemm(const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w, int M, int N,
                       int K, uint16_t* Y, int32_t* acc, void* ws, hipStream_t st, int bits) {
    const Plan p = choose_plan(M, N, K, bits);
    int32_t* part = static_cast<int32_t*>(ws);
    hipError_t e;
    if (bits == 8) {
        switch (p.cfg) {
            case 3: e = skinny_kw<8>(p.waves, Aq, s_a, Wq, s_w, M, N, K, Y, acc, st); break;
            case 7: e = launch_tiled<2, 2, 4, 8, 8, 2>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
            case 9: e = launch_tiled<2, 2, 4, 4, 8, 2, false, 2>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
            case 8: e = launch_tiled<1, 2, 8, 4, 8, 2>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
            case 1: e = launch_tiled<2, 2, 4, 4, 8, 3>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
            case 2: e = launch_tiled<2, 2, 2, 2, 8, 4>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
            default: e = launch_tiled<1, 4, 4, 2, 8, 4>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
        }
    } else {
        switch (p.cfg) {
            case 3: e = skinny_kw<4>(p.waves, Aq, s_a, Wq, s_w, M, N, K, Y, acc, st); break;
            case 5: e = launch_skinny_shared(p.waves, Aq, s_a, Wq, s_w, M, N, K, Y, acc, st); break;
            case 0: e = launch_tiled<4, 2, 4, 4, 4, 2>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
            case 9: e = launch_tiled<2, 2, 4, 4, 4, 2, false, 2>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
            case 1: e = launch_tiled<2, 2, 4, 4, 4, 3>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
            case 2: e = launch_tiled<2, 2, 2, 2, 4, 4>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
            default: e = launch_tiled<1, 4, 4, 2, 4, 4>(p, Aq, s_a, Wq, s_w, M, N, K, Y, acc, part, st); break;
        }
    }
    if (e != hipSuccess) return e;
    return finish_split(p, part, s_a, s_w, M, N, Y, acc, st);
}

}  // namespace sq
