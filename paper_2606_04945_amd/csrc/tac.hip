// Temporal Attention Compensation (Sec. 3.3, Eq. 17; App. C): per token and per
// block b of g channels, z'_{bg+r} = fp16( sum_c M_b[r][c] z_{bg+c} + d_{bg+r} ),
// each sum an fp32 fused multiply-add chain in ascending c from +0, bias last.
//
// The map is a batch of small [tokens x g] x [g x g] products, one per block.
// For widths that are a multiple of 128 channels it runs on the matrix cores
// (tac_mfma_kernel, below), whose fp32 instruction reproduces that chain bit
// for bit.  Other widths take tac_kernel, a register-tiled batched SGEMM on the
// VALU: a workgroup owns TT tokens x CW channels (CW = max(g, 64) so a span
// holds whole blocks), stages the span's block matrices and the token tile
// through LDS as fp32, and each thread keeps 8 tokens x 8 channels of
// accumulators (8 x 4 when g < 8), so each pair of LDS reads feeds 64 (32)
// fused multiply-adds.
#include "tile_common.hpp"

namespace sq {
namespace {

constexpr int kThreads = 256;
constexpr int kTPT = 8;   // tokens per thread

// CPT channels per thread (8, or 4 for g < 8); CC block-matrix columns staged per pass
template <int CW, int CPT>
__global__ __launch_bounds__(kThreads) void tac_kernel(const uint16_t* __restrict__ Z,
                                                       const uint16_t* __restrict__ Mb,
                                                       const uint16_t* __restrict__ d, int M, int C,
                                                       int g, uint16_t* __restrict__ out) {
    constexpr int kCPT = CPT;
    constexpr int kCC = CW == 128 ? 8 : 16;
    constexpr int MPT = CW * kCC / kThreads; // block-matrix values each thread stages per pass
    constexpr int CG = CW / kCPT;            // channel groups per span
    constexpr int TG = kThreads / CG;        // token groups
    constexpr int TT = TG * kTPT;            // tokens per tile
    constexpr int ZP = TT + 4;               // padded row of the transposed token tile
    constexpr int MP = CW + 4;               // padded row of the transposed block tile
    extern __shared__ float smem[];
    float* zsT = smem;                       // [CW][ZP]   zsT[ch][tok]
    float* msT = smem + CW * ZP;             // [2][kCC][MP]  msT[c-c0][ch] = M_{blk(ch)}[ch%g][c]

    const int tid = threadIdx.x;
    const int span0 = blockIdx.x * CW;       // first channel of this span
    const int tok0 = blockIdx.y * TT;

    // stage the token tile, 8 channels (16 B) per load
    for (int e = tid; e < TT * (CW / 8); e += kThreads) {
        const int t = e / (CW / 8), v = e % (CW / 8);
        const int tok = tok0 + t;
        uint4 raw = make_uint4(0, 0, 0, 0);
        if (tok < M) raw = *reinterpret_cast<const uint4*>(Z + (size_t)tok * C + span0 + v * 8);
        const uint16_t* h = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
        for (int q = 0; q < 8; ++q) zsT[(v * 8 + q) * ZP + t] = h2f(h[q]);
    }

    const int cg = tid % CG, tg = tid / CG;
    const int ch0 = cg * kCPT;               // first of this thread's channels (span-local)
    float acc[kTPT][kCPT];
#pragma unroll
    for (int t = 0; t < kTPT; ++t)
#pragma unroll
        for (int q = 0; q < kCPT; ++q) acc[t][q] = 0.0f;

    // the block matrices are staged kCC columns c at a time, double-buffered:
    // the next pass's values are loaded into registers while this pass
    // computes; every accumulator still sees c in ascending order
    const int cc = g < kCC ? g : kCC;
    const int npass = g / cc;
    uint16_t pre[MPT];
    auto load_pass = [&](int c0) {
#pragma unroll
        for (int i = 0; i < MPT; ++i) {
            const int e = tid + i * kThreads;
            const int ch = e / cc, c = e % cc;
            // tac_M is [C/g][g][g] == [C][g]: row (span0 + ch), column c0 + c
            pre[i] = e < CW * cc ? Mb[(size_t)(span0 + ch) * g + c0 + c] : (uint16_t)0;
        }
    };
    auto store_pass = [&](float* buf) {
#pragma unroll
        for (int i = 0; i < MPT; ++i) {
            const int e = tid + i * kThreads;
            if (e < CW * cc) buf[(e % cc) * MP + e / cc] = h2f(pre[i]);
        }
    };
    load_pass(0);
    store_pass(msT);
    __syncthreads();                         // token tile and first pass staged
    for (int p = 0; p < npass; ++p) {
        const int c0 = p * cc;
        const float* ms = msT + (p & 1) * kCC * MP;
        if (p + 1 < npass) load_pass(c0 + cc);
        if (CPT == 8 || g >= kCPT) {         // CPT == 8 is launched for g >= 8 only
            const int base = (ch0 / g) * g;  // block start, shared by the thread's channels
            // column c: the thread's kCPT block-matrix values and kTPT inputs
            auto fetch = [&](int c, float4 (&r)[4]) {
                r[0] = *reinterpret_cast<const float4*>(ms + c * MP + ch0);
                r[1] = *reinterpret_cast<const float4*>(ms + c * MP + ch0 + 4);
                const float* zr = zsT + (base + c0 + c) * ZP + tg * kTPT;
                r[2] = *reinterpret_cast<const float4*>(zr);
                r[3] = *reinterpret_cast<const float4*>(zr + 4);
            };
            auto madd = [&](const float4 (&r)[4]) {
                const float m[8] = {r[0].x, r[0].y, r[0].z, r[0].w, r[1].x, r[1].y, r[1].z, r[1].w};
                const float zv[8] = {r[2].x, r[2].y, r[2].z, r[2].w, r[3].x, r[3].y, r[3].z, r[3].w};
#pragma unroll
                for (int t = 0; t < kTPT; ++t)
#pragma unroll
                    for (int q = 0; q < kCPT; ++q) acc[t][q] = __builtin_fmaf(m[q], zv[t], acc[t][q]);
            };
            if (cc == kCC) {
                // a full pass (g >= kCC), unrolled with the next column's LDS
                // reads issued ahead of this column's multiply-adds
                float4 r[2][4];
                fetch(0, r[0]);
#pragma unroll
                for (int c = 0; c < kCC; ++c) {
                    if (c + 1 < kCC) fetch(c + 1, r[(c + 1) & 1]);
                    madd(r[c & 1]);
                }
            } else {
                for (int c = 0; c < cc; ++c) {
                    float4 r[4];
                    fetch(c, r);
                    madd(r);
                }
            }
        } else if constexpr (CPT == 4) {
            // g in {1, 2}: the thread's channels lie in different blocks
#pragma unroll
            for (int q = 0; q < kCPT; ++q) {
                const int ch = ch0 + q, base = (ch / g) * g;
                for (int c = 0; c < cc; ++c) {
                    const float m = ms[c * MP + ch];
#pragma unroll
                    for (int t = 0; t < kTPT; ++t)
                        acc[t][q] = __builtin_fmaf(m, zsT[(base + c0 + c) * ZP + tg * kTPT + t], acc[t][q]);
                }
            }
        }
        if (p + 1 < npass) store_pass(msT + ((p + 1) & 1) * kCC * MP);
        __syncthreads();                     // next buffer filled; this one free for p + 2
    }

    float dv[kCPT];
#pragma unroll
    for (int q = 0; q < kCPT; ++q) dv[q] = h2f(d[span0 + ch0 + q]);
#pragma unroll
    for (int t = 0; t < kTPT; ++t) {
        const int tok = tok0 + tg * kTPT + t;
        if (tok >= M) break;
#pragma unroll
        for (int q = 0; q < kCPT; q += 4) {
            ushort4 o;
            o.x = f2h(acc[t][q] + dv[q]);
            o.y = f2h(acc[t][q + 1] + dv[q + 1]);
            o.z = f2h(acc[t][q + 2] + dv[q + 2]);
            o.w = f2h(acc[t][q + 3] + dv[q + 3]);
            *reinterpret_cast<ushort4*>(out + (size_t)tok * C + span0 + ch0 + q) = o;
        }
    }
}

// The matrix-core form, for C a multiple of 128.  v_mfma_f32_16x16x4_f32
// evaluates its four products as a forward chain of single-rounding fused
// multiply-adds, k ascending (subnormals kept), so a chain of these
// instructions over ascending groups of four c is exactly the fixed chain
// above.  Outputs are taken 16 channels at a time: for g >= 16 the chain of a
// 16-channel group runs over the g inputs of its block; for g < 16 it runs over
// the group's own 16 inputs against a block-diagonal 16 x 16 operand whose
// off-block entries are zero.  A zero product leaves a running sum unchanged
// (the chain starts at +0 and never reaches -0), so the result is the same chain
// over the block's g inputs.  A workgroup (eight waves) owns 128 tokens x 128
// channels: the token tile and the 128 rows of the block matrices are staged
// in LDS as fp16 (widened as they are read), each wave multiplies 16 tokens x
// 128 channels, and the fp16 results leave through LDS in 16-byte stores
// (eight waves of 16 tokens were 5-18 % faster than four waves of 32).
typedef float f32x4 __attribute__((ext_vector_type(4)));
constexpr int kTacTile = 128;

constexpr int kTacWaves = kTacTile / 16;          // one wave per 16 tokens of the tile
constexpr int kTacThreads = 64 * kTacWaves;

template <int G>
__global__ __launch_bounds__(kTacThreads) __attribute__((amdgpu_waves_per_eu(kTacWaves / 2))) void tac_mfma_kernel(
    const uint16_t* __restrict__ Z, const uint16_t* __restrict__ Mb, const uint16_t* __restrict__ d, int M, int C,
    uint16_t* __restrict__ out) {
    constexpr int TR = kTacTile, CW = kTacTile, NT = kTacThreads;
    constexpr int L = G < 16 ? 16 : G;               // chain length of a 16-channel output group
    constexpr int ZP = CW + 8;                       // fp16 row of the token tile: 16-byte aligned, rows 4 banks apart
    constexpr int MP = G >= 8 ? G + 8 : G;           // fp16 row of the block-matrix tile
    __shared__ __attribute__((aligned(16))) uint16_t zs[TR * ZP];
    __shared__ __attribute__((aligned(16))) uint16_t ms[CW * MP];

    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const int span0 = blockIdx.x * CW, tok0 = blockIdx.y * TR;

    // token tile: 16 16-byte vectors per row; rows past M read as zero
#pragma unroll
    for (int v = 0; v < TR * CW / 8 / NT; ++v) {
        const int e = tid + v * NT, r = e / (CW / 8), q = e % (CW / 8);
        uint4 w = make_uint4(0, 0, 0, 0);
        if (tok0 + r < M) w = *reinterpret_cast<const uint4*>(Z + (size_t)(tok0 + r) * C + span0 + 8 * q);
        *reinterpret_cast<uint4*>(zs + r * ZP + 8 * q) = w;
    }
    // block-matrix rows of the span's channels: tac_M viewed as [C][G], rows span0 .. span0 + 127
    {
        const uint16_t* src = Mb + (size_t)span0 * G;
        for (int e = tid; e < CW * G / 8; e += NT) {
            const uint4 w = *reinterpret_cast<const uint4*>(src + 8 * e);
            if (G >= 8) {
                const int r = 8 * e / G, c = 8 * e % G;
                *reinterpret_cast<uint4*>(ms + r * MP + c) = w;
            } else {
                *reinterpret_cast<uint4*>(ms + 8 * e) = w;
            }
        }
    }
    __syncthreads();

    const int il = lane % 16, kl = lane / 16;
    f32x4 acc[CW / 16];
#pragma unroll
    for (int og = 0; og < CW / 16; ++og)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[og][v] = 0.0f;

    const uint16_t* za = zs + (16 * wave + il) * ZP;   // this lane's token row
    if constexpr (G < 32) {
        // one 16-channel group per chain input range
#pragma unroll
        for (int og = 0; og < CW / 16; ++og) {
            const int in0 = G < 16 ? 16 * og : (16 * og / G) * G;   // first input channel of the chain
            const int mrow = 16 * og + il;                   // block-matrix row (output channel) of this lane
#pragma unroll
            for (int s4 = 0; s4 < L / 4; ++s4) {
                const int c = 4 * s4 + kl;                   // position in the chain
                const float b = G >= 16 ? h2f(ms[mrow * MP + c])
                                        : (c / G == il / G ? h2f(ms[mrow * MP + c % G]) : 0.0f);
                const float a = h2f(za[in0 + c]);
                acc[og] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[og], 0, 0, 0);
            }
        }
    } else {
        // the G / 16 groups of a block share their inputs: each token value read feeds all of them
        constexpr int NG = G / 16;
#pragma unroll
        for (int blk = 0; blk < CW / G; ++blk) {
#pragma unroll 4
            for (int s4 = 0; s4 < G / 4; ++s4) {
                const int c = 4 * s4 + kl;
                const float a = h2f(za[blk * G + c]);
#pragma unroll
                for (int q = 0; q < NG; ++q) {
                    const int og = blk * NG + q;
                    const float b = h2f(ms[(16 * og + il) * MP + c]);
                    acc[og] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[og], 0, 0, 0);
                }
            }
        }
    }

    // z' = fp16(sum + d), through LDS (the token tile is no longer read) to 16-byte stores
    float dv[CW / 16];
#pragma unroll
    for (int og = 0; og < CW / 16; ++og) dv[og] = h2f(d[span0 + 16 * og + il]);
    __syncthreads();
#pragma unroll
    for (int og = 0; og < CW / 16; ++og)
#pragma unroll
        for (int v = 0; v < 4; ++v) zs[(16 * wave + 4 * kl + v) * ZP + 16 * og + il] = f2h(acc[og][v] + dv[og]);
    __syncthreads();
#pragma unroll
    for (int v = 0; v < TR * CW / 8 / NT; ++v) {
        const int e = tid + v * NT, r = e / (CW / 8), q = e % (CW / 8);
        if (tok0 + r < M)
            *reinterpret_cast<uint4*>(out + (size_t)(tok0 + r) * C + span0 + 8 * q) =
                *reinterpret_cast<const uint4*>(zs + r * ZP + 8 * q);
    }
}

template <int CW, int CPT>
hipError_t launch_cw(const uint16_t* Z, const uint16_t* Mb, const uint16_t* d, int M, int C, int g,
                     uint16_t* out, hipStream_t st) {
    constexpr int CG = CW / CPT, TT = (kThreads / CG) * kTPT;
    constexpr int CC = CW == 128 ? 8 : 16;
    const size_t lds = sizeof(float) * ((size_t)CW * (TT + 4) + 2 * (size_t)CC * (CW + 4));
    static std::atomic<int> lds_set[kMaxDevices];   // above the 64 KB default for dynamic LDS
    const hipError_t attr = allow_dynamic_lds(reinterpret_cast<const void*>(&tac_kernel<CW, CPT>), (int)lds, lds_set);
    if (attr != hipSuccess) return attr;
    dim3 grid(C / CW, (M + TT - 1) / TT);
    hipLaunchKernelGGL((tac_kernel<CW, CPT>), grid, dim3(kThreads), lds, st, Z, Mb, d, M, C, g, out);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_tac(const uint16_t* Z, const uint16_t* Mb, const uint16_t* d, int M, int C, int g,
                      uint16_t* out, hipStream_t st) {
    if (C % kTacTile == 0) {
        const dim3 grid(C / kTacTile, (M + kTacTile - 1) / kTacTile);
        switch (g) {
#define SQ_TM(G)                                                                                              \
    case G:                                                                                                   \
        hipLaunchKernelGGL(tac_mfma_kernel<G>, grid, dim3(kTacThreads), 0, st, Z, Mb, d, M, C, out);     \
        return hipGetLastError();
            SQ_TM(1) SQ_TM(2) SQ_TM(4) SQ_TM(8) SQ_TM(16) SQ_TM(32) SQ_TM(64) SQ_TM(128)
#undef SQ_TM
            default:
                return hipErrorInvalidValue;
        }
    }
    if (g < 8) return launch_cw<64, 4>(Z, Mb, d, M, C, g, out, st);
    if (g <= 64) return launch_cw<64, 8>(Z, Mb, d, M, C, g, out, st);
    return launch_cw<128, 8>(Z, Mb, d, M, C, g, out, st);
}

}  // namespace sq

// ---------------------------------------------------------------------------
// TAC fused with the gate and the per-token quantiser, for g <= 16 and an
// input already in the P basis (no dense transform): z -> fp16(M_b z_b + d_b)
// -> G_s -> absmax -> codes, without materialising z'.
//
// A workgroup owns a run of token rows.  Its consumer waves cover the row's
// channels, 8 per thread (K / 8 active threads), each thread keeping the block
// rows (8 x g fp16) and biases of its channels in registers for the whole run.
// One more wave, the producer, only moves data: it copies each row of the run
// from HBM straight into a ring of D row slots in LDS (buffer loads with the
// LDS destination), D - 1 rows ahead of the consumers.  So the consumers never
// load from memory inside the loop (their only memory operations there are
// the code stores), and the producer never stores, so its counter waits count
// its own loads exactly.  One workgroup barrier per row does three jobs: the
// row has landed in its slot, every wave has written its partial max of the
// previous row, and the slot read two rows back is free again.  After it the
// consumers finish the previous row (block max, codes, store) and compute the
// current one (g fused multiply-adds per output in the order and rounding of
// tac_kernel, the gate, the wave max), so a row's two halves sit on either side
// of one barrier.
namespace sq {
namespace {

constexpr int kTqMaxConsumerWaves = 8;       // K <= 4096
constexpr int kTqRing = 6;                   // row slots in the LDS ring
constexpr int kTqMaxRows = 64;               // rows per workgroup (their states live in LDS)
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

// Producer: wait until at most `n` of this wave's ring loads are in flight
// (n = consumer waves x rows still ahead; the immediate must be a constant).
__device__ __forceinline__ void wait_ring(int n) {
    switch (n) {
#define SQ_W(N) case N: wait_vm<N>(); break;
        SQ_W(0) SQ_W(1) SQ_W(2) SQ_W(3) SQ_W(4) SQ_W(5) SQ_W(6) SQ_W(7) SQ_W(8) SQ_W(9) SQ_W(10) SQ_W(11)
        SQ_W(12) SQ_W(14) SQ_W(15) SQ_W(16) SQ_W(18) SQ_W(20) SQ_W(21) SQ_W(24) SQ_W(25) SQ_W(28) SQ_W(30)
        SQ_W(32) SQ_W(35) SQ_W(40)
#undef SQ_W
        default: wait_vm<0>(); break;
    }
}

// Max over the wave of non-negative values, through DPP lane moves (no LDS):
// quads, then halves of 16-lane rows, rows, then rows 0-1 into row 1, 2-3 into
// row 3 and row 1 into row 3; lane 63 ends with the maximum.  Non-negative
// floats order as their bit patterns do as integers.
__device__ __forceinline__ float wave_max_dpp(float v) {
    int x = __float_as_int(v);
    x = max(x, __builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false));    // quad_perm [1, 0, 3, 2]
    x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false));    // quad_perm [2, 3, 0, 1]
    x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x141, 0xF, 0xF, false));   // row_half_mirror
    x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x140, 0xF, 0xF, false));   // row_mirror
    x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x142, 0xA, 0xF, false));   // row_bcast:15
    x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x143, 0xC, 0xF, false));   // row_bcast:31
    return __int_as_float(__builtin_amdgcn_readlane(x, 63));
}

// LDS writes of this wave are complete, then the workgroup barrier (a bare
// s_barrier: __syncthreads would also wait for the producer's loads in flight)
__device__ __forceinline__ void ring_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (0 << 8) | (3 << 14));   // lgkmcnt(0), vmcnt untouched
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <int G, int BITS>
__global__ __launch_bounds__(64 * (kTqMaxConsumerWaves + 1)) void tac_quant_kernel(
    const uint16_t* __restrict__ Z, const uint16_t* __restrict__ Mb, const uint16_t* __restrict__ d,
    const uint8_t* __restrict__ state, int M, int K, int dm, int du, int rows_per_wg, uint8_t* __restrict__ Aq,
    float* __restrict__ s_out) {
    constexpr int ZW = G > 8 ? G : 8;                   // input channels a thread reads (whole blocks)
    extern __shared__ __attribute__((aligned(16))) float tq_smem[];
    uint8_t* smem = reinterpret_cast<uint8_t*>(tq_smem);
    const int cw = (K / 8 + kWave - 1) / kWave;         // consumer waves
    const int slot_bytes = cw * 1024;                   // one row: 16 bytes per consumer thread
    uint8_t* ring = smem;
    float* red = reinterpret_cast<float*>(smem + kTqRing * slot_bytes);        // [2][kTqMaxConsumerWaves]
    uint8_t* st_lds = reinterpret_cast<uint8_t*>(red + 2 * kTqMaxConsumerWaves); // [rows_per_wg]

    const int t = threadIdx.x, lane = t % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(t / kWave);
    const bool producer = wave == cw;
    const bool active = !producer && 8 * t < K;
    const int c0 = 8 * t;                               // first output channel of this thread
    const int z0 = (c0 / ZW) * ZW;                      // first input channel it reads
    const int row_begin = blockIdx.x * rows_per_wg;
    const int nrows = min(M, row_begin + rows_per_wg) - row_begin;
    const bool gated = state != nullptr;

    if (t < nrows) st_lds[t] = gated ? state[row_begin + t] : 0;

    // tac_M viewed as [K][G]: this thread's rows c0 .. c0 + 7 are 8 G fp16
    // values, held as G vectors of 8 (element r G + c of the run = row r,
    // column c), widened by the mixed-precision multiply-adds
    v8h mh[G];
    float dv[8];
    const int cm = active ? c0 : 0;                     // other threads read the first rows, unused
    if constexpr (G >= 4) {
        // A thread's rows are PB = 16 G contiguous bytes at PB t, so loaded
        // directly the lanes of one 16-byte load would touch up to 64 cache
        // lines.  Instead each consumer wave loads the runs of TPP of its
        // threads at a time with whole-wave contiguous 16-byte loads, writes
        // them to per-thread slots padded by 16 bytes (in the ring, not yet in
        // use), so the 16-byte reads back are free of bank conflicts, and those
        // threads read their slots.  A wave's LDS accesses are performed in
        // order, so only the compiler has to be kept from reordering them.
        constexpr int PB = 16 * G, NC = PB / 16, SLOT = PB + 16;
        constexpr int TPP = G == 16 ? 16 : (G == 8 ? 32 : 64);   // at most 5 KB per wave per pass
        constexpr int PASSES = kWave / TPP;
        constexpr int LOADS = TPP * NC / kWave;         // 16-byte loads per lane per pass
        static_assert(TPP * SLOT <= 1024 * kTqRing, "parameter staging fits in a wave's share of the ring");
        if (!producer) {
            uint8_t* stage = ring + wave * (TPP * SLOT);
            const __amdgpu_buffer_rsrc_t rM = make_rsrc(Mb, (uint32_t)K * G * 2);
            const int slab = wave * kWave * NC;         // first chunk of this wave's runs
            auto wave_sync = [] {
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            };
#pragma unroll
            for (int p = 0; p < PASSES; ++p) {
                v4i ch[LOADS];
#pragma unroll
                for (int i = 0; i < LOADS; ++i)
                    ch[i] = __builtin_amdgcn_raw_buffer_load_b128(rM, (slab + p * TPP * NC + i * kWave + lane) * 16,
                                                                  0, 0);
#pragma unroll
                for (int i = 0; i < LOADS; ++i) {
                    const int c = i * kWave + lane;     // chunk of this pass: thread c / NC, piece c % NC
                    *reinterpret_cast<v4i*>(stage + (c / NC) * SLOT + (c % NC) * 16) = ch[i];
                }
                wave_sync();
                if (lane / TPP == p) {
#pragma unroll
                    for (int j = 0; j < NC; ++j)
                        mh[j] = *reinterpret_cast<const v8h*>(stage + (lane - p * TPP) * SLOT + j * 16);
                }
                wave_sync();
            }
        }
    } else {
        // runs of 16 or 32 bytes: the lanes of a load already cover whole lines
#pragma unroll
        for (int j = 0; j < G; ++j) mh[j] = *reinterpret_cast<const v8h*>(Mb + (size_t)cm * G + 8 * j);
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) dv[r] = h2f(d[cm + r]);
    __syncthreads();                                    // parameters read; states in LDS; the ring is free

    // producer: row r of the run into slot r % kTqRing, one 1 KB load per consumer wave
    if (producer) {
        auto issue = [&](int r) {
            const u32x4 rz = sgpr_rsrc(Z + (size_t)(row_begin + r) * K, (uint32_t)K * 2);
            uint8_t* dst = ring + (r % kTqRing) * slot_bytes;
            for (int j = 0; j < cw; ++j) dma16(rz, lds_addr(dst + j * 1024), (uint32_t)(j * kWave + lane) * 16);
        };
        for (int r = 0; r < kTqRing - 1 && r < nrows; ++r) issue(r);
        for (int i = 0; i <= nrows; ++i) {
            if (i < nrows) wait_ring(min(kTqRing - 2, nrows - 1 - i) * cw);   // row i has landed
            ring_barrier();
            if (i + kTqRing - 1 < nrows) issue(i + kTqRing - 1);             // into the slot row i - 1 used
        }
        return;
    }

    // consumers: the same number of barriers, each row split around one of them.
    // The gate keeps or drops this thread's 8 channels together unless a band
    // edge falls inside them (then it is applied channel by channel).
    const bool keep_m = kept(c0, K, dm, du, true), keep_u = kept(c0, K, dm, du, false);
    bool edge = false;
#pragma unroll
    for (int r = 1; r < 8; ++r)
        edge |= kept(c0 + r, K, dm, du, true) != keep_m || kept(c0 + r, K, dm, du, false) != keep_u;
    float op[8];                                        // the row being carried across the barrier
    constexpr float kQmax = BITS == 4 ? 7.0f : 127.0f;
    auto compute = [&](int i) {                         // row i: TAC, gate, partial max
        float amax = 0.0f;
        if (active) {
            const uint8_t* src = ring + (i % kTqRing) * slot_bytes + z0 * 2;
            v8h zh[ZW / 8];
#pragma unroll
            for (int v = 0; v < ZW / 8; ++v) zh[v] = *reinterpret_cast<const v8h*>(src + 16 * v);
            const bool masked = st_lds[i] != 0;
#pragma unroll
            for (int j = 0; j < G; ++j) asm volatile("" : "+v"(mh[j]));
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                // block start within zh: c0 is a multiple of 8, so for g = 16 the
                // thread's 8 outputs lie in one block whose inputs are all of zh,
                // and for g <= 8 the block of output r starts at (r / g) g
                const int base = G == 16 ? 0 : (r / G) * G;
                float acc = 0.0f;
#pragma unroll
                for (int c = 0; c < G; ++c) {
                    const int e = r * G + c, zi = base + c;
                    acc = __builtin_fmaf((float)mh[e / 8][e % 8], (float)zh[zi / 8][zi % 8], acc);
                }
                op[r] = h2f(f2h(acc + dv[r]));             // TAC output, materialised as fp16
            }
            if (gated) {
                if (__builtin_expect(edge, 0)) {
#pragma unroll
                    for (int r = 0; r < 8; ++r) op[r] = kept(c0 + r, K, dm, du, masked) ? op[r] : 0.0f;
                } else {
                    const bool keep = masked ? keep_m : keep_u;
#pragma unroll
                    for (int r = 0; r < 8; ++r) op[r] = keep ? op[r] : 0.0f;
                }
            }
#pragma unroll
            for (int r = 0; r < 8; ++r) amax = fmaxf(amax, fabsf(op[r]));
        }
        amax = wave_max_dpp(amax);
        if (lane == 0) red[(i & 1) * kTqMaxConsumerWaves + wave] = amax;
    };
    auto finish = [&](int i) {                          // row i: block max, codes, store
        // partial maxima of absent waves are never written: only the first cw count
        const float4* rp = reinterpret_cast<const float4*>(red + (i & 1) * kTqMaxConsumerWaves);
        const float4 r0 = rp[0], r1 = rp[1];
        const float rv[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
        float a = rv[0];
#pragma unroll
        for (int w = 1; w < kTqMaxConsumerWaves; ++w) a = w < cw ? fmaxf(a, rv[w]) : a;
        const float s = a / kQmax;
        const float y = s != 0.0f ? 1.0f / s : 0.0f;
        const int row = row_begin + i;
        if (t == 0) s_out[row] = s;
        if (!active) return;
        if (BITS == 4) {
            uint32_t w4 = 0;
            if (s != 0.0f) {
                int c[8];
                quant_codes8<7>(op, s, y, c);
#pragma unroll
                for (int q = 0; q < 8; ++q) w4 |= (uint32_t)(c[q] & 15) << (4 * q);
            }
            *reinterpret_cast<uint32_t*>(Aq + (size_t)row * (K / 2) + 4 * t) = w4;
        } else {
            uint32_t lo = 0, hi = 0;
            if (s != 0.0f) {
                int c[8];
                quant_codes8<127>(op, s, y, c);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    lo |= (uint32_t)(c[q] & 255) << (8 * q);
                    hi |= (uint32_t)(c[4 + q] & 255) << (8 * q);
                }
            }
            *reinterpret_cast<uint2*>(Aq + (size_t)row * K + 8 * t) = make_uint2(lo, hi);
        }
    };
    ring_barrier();
    compute(0);
    for (int i = 1; i < nrows; ++i) {
        ring_barrier();
        finish(i - 1);
        compute(i);
    }
    ring_barrier();
    finish(nrows - 1);
}


// ---------------------------------------------------------------------------
// The same fused pass on the matrix cores for g = 16, for rows of four to eight
// parts of 16 NG = 512 channels (hidden size 3584 takes seven waves, 4096
// eight).  A workgroup walks 16-token tiles; each of its waves owns
// 16 NG consecutive channels of every row.  Per tile a wave:
//   * takes its z values straight from HBM, 16 bytes per lane (8 channels of
//     one token), half a tile of loads ahead in a register ring;
//   * rearranges them with two rounds of cross-row lane swaps into the operand
//     the fp32 MFMA wants (lane (t, k) needs channels k, k + 4, k + 8, k + 12 of
//     a 16-channel group for token t);
//   * runs z'^T = M_b z^T for each 16-channel block (g = 16) as a chain of four
//     v_mfma_f32_16x16x4_f32 over ascending c (the TAC chain of tac_kernel bit
//     for bit, as in tac_mfma_kernel), adds the bias, applies the gate, rounds
//     to fp16 and parks the result in its own LDS tile (each lane holds four
//     consecutive channels of one token per block: one 8-byte write);
//   * tracks the token's absmax, combines it over the wave and posts it.
// One workgroup barrier per tile publishes the partial maxima.  Then each wave
// forms the 16 token scales, reads its tile back as runs of 8 channels of one
// token, codes them (quant_codes8, the rule of every quantiser here) and
// stores the codes.  The block-matrix operands (four values per lane and
// group, packed fp16) stay in registers for the whole walk, which is why a
// wave takes many channels and a CU runs one workgroup of up to eight waves.
constexpr int kTqmTok = 16;
constexpr int kTqmMaxWaves = 8;

// Lanes 16 r + k (row r = 0..3 of the wave, k = 0..15) hold x_0 .. x_3; on
// return lane 16 r + k holds in x_p what lane 16 p + k held in x_r.  Two
// rounds of lane-half / lane-row swaps.
__device__ __forceinline__ void transpose_rows4(uint32_t& x0, uint32_t& x1, uint32_t& x2, uint32_t& x3) {
    auto s02 = __builtin_amdgcn_permlane32_swap(x0, x2, false, false);
    auto s13 = __builtin_amdgcn_permlane32_swap(x1, x3, false, false);
    x0 = s02[0], x2 = s02[1], x1 = s13[0], x3 = s13[1];
    auto s01 = __builtin_amdgcn_permlane16_swap(x0, x1, false, false);
    auto s23 = __builtin_amdgcn_permlane16_swap(x2, x3, false, false);
    x0 = s01[0], x1 = s01[1], x2 = s23[0], x3 = s23[1];
}

__device__ __forceinline__ float lo_h(uint32_t x) { return h2f((uint16_t)(x & 0xFFFFu)); }
__device__ __forceinline__ float hi_h(uint32_t x) { return h2f((uint16_t)(x >> 16)); }

template <int NG>
struct TqmShape {
    static constexpr int kCWV = 16 * NG;                        // channels per wave
    static constexpr int kRS = 2 * kCWV + 16;                   // fp16 row of a wave's output tile (banks spread)
    static constexpr int kStage = kCWV * 32;                    // block-matrix rows of a wave, staged once
    static constexpr int kRegion = kStage > kTqmTok * kRS ? kStage : kTqmTok * kRS;
    static size_t lds_bytes(int K) {
        return (size_t)K * 4 + 2 * kTqmTok * kTqmMaxWaves * 4 + (size_t)(K / kCWV) * kRegion;
    }
};

template <int BITS, int NG>
__global__ __launch_bounds__(64 * kTqmMaxWaves) void tac_quant_mfma_kernel(
    const uint16_t* __restrict__ Z, const uint16_t* __restrict__ Mb, const uint16_t* __restrict__ d,
    const uint8_t* __restrict__ state, int M, int K, int dm, int du, uint8_t* __restrict__ Aq,
    float* __restrict__ s_out) {
    using S = TqmShape<NG>;
    constexpr int CWV = S::kCWV, NC = NG / 2, D = NC / 2;       // D: chunk loads in flight per lane
    constexpr float kQmax = BITS == 4 ? 7.0f : 127.0f;
    constexpr int VPL = CWV / 32;                               // 8-channel runs per lane in the coding pass
    static_assert(NC % D == 0 && VPL % 2 == 0 && CWV % kWave == 0, "static ring slots; runs coded in pairs");
    extern __shared__ __attribute__((aligned(16))) float tqm_smem[];
    const int lane = threadIdx.x % kWave, wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int il = lane % 16, kl = lane / 16;
    const int W = K / CWV, ch0 = wave * CWV;
    float* bias = tqm_smem;                                     // [K] fp32
    float* red = bias + K;                                      // [2][16 tokens][8 waves]
    uint8_t* region = reinterpret_cast<uint8_t*>(red + 2 * kTqmTok * kTqmMaxWaves) + wave * S::kRegion;
    auto wave_sync = [] {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };

    // biases of this wave's channels, widened (only this wave reads them); all
    // loads are issued before the first is used
    {
        uint16_t bh[CWV / kWave];
#pragma unroll
        for (int i = 0; i < CWV / kWave; ++i) bh[i] = d[ch0 + lane + i * kWave];
#pragma unroll
        for (int i = 0; i < CWV / kWave; ++i) bias[ch0 + lane + i * kWave] = h2f(bh[i]);
    }

    // Block-matrix operands.  Row r of the wave's range is staged as 8 dwords,
    // dword 2 m + h = (M[r][8 h + m], M[r][8 h + m + 4]) with M[r] the 16 block-
    // matrix entries of channel r, so lane (t, k) reads its four values
    // M[16 b + t][k + 4 s], s = 0..3, as dwords 2 k and 2 k + 1 of row 16 b + t.
    // Task = (row, half); every lane's loads are issued before the first is used.
    constexpr int TPL = 2 * CWV / kWave;                        // tasks per lane
    uint16_t v[TPL][8];
#pragma unroll
    for (int it = 0; it < TPL; ++it) {
        const int task = lane + it * kWave, r = task / 2, h = task % 2, ch = ch0 + r;
        const uint4 w = *reinterpret_cast<const uint4*>(Mb + (size_t)ch * 16 + 8 * h);
        const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int i = 0; i < 8; ++i) v[it][i] = (uint16_t)(wd[i / 2] >> (16 * (i % 2)));
    }
#pragma unroll
    for (int it = 0; it < TPL; ++it) {
        const int task = lane + it * kWave, r = task / 2, h = task % 2;
#pragma unroll
        for (int m = 0; m < 4; ++m)
            *reinterpret_cast<uint32_t*>(region + r * 32 + (2 * m + h) * 4) =
                (uint32_t)v[it][m] | ((uint32_t)v[it][m + 4] << 16);
    }
    wave_sync();
    uint32_t mp[NG][2];
#pragma unroll
    for (int b = 0; b < NG; ++b) {
        const uint2 w = *reinterpret_cast<const uint2*>(region + (16 * b + il) * 32 + 8 * kl);
        mp[b][0] = w.x;
        mp[b][1] = w.y;
    }
    wave_sync();   // the region now holds this wave's output tile

    const int ntiles = (M + kTqmTok - 1) / kTqmTok;
    const __amdgpu_buffer_rsrc_t rz = make_rsrc(Z, (uint32_t)((size_t)M * K * 2));
    // byte offset of this lane's first 16 bytes of tile n (chunk j adds 64 j); past M reads zero
    auto tile_base = [&](int n) -> uint32_t {
        return n < ntiles ? (uint32_t)(((size_t)(n * kTqmTok + il) * K + ch0 + 8 * kl) * 2) : kOOB;
    };
    const int m_lo = K - dm - du, u_lo = K - du;
    const bool gated = state != nullptr && dm + du > 0;
    // bit b: group b of this wave meets the bands [m_lo, K) (one scalar word,
    // tested per group, instead of a precomputed condition per group)
    const int bgate = !gated ? NG : (m_lo <= ch0 ? 0 : ((m_lo - ch0) / 16 < NG ? (m_lo - ch0) / 16 : NG));
    const uint32_t gmask = __builtin_amdgcn_readfirstlane(bgate >= 32 ? 0u : ~0u << bgate);
    // States, codes and scales go through range-checked buffer accesses (reads
    // past the end give 0, writes past it are dropped), so the loop has no
    // branch around a memory access and the compiler can count the loads in
    // flight exactly (a guessed count would make it wait for all of them).
    const __amdgpu_buffer_rsrc_t rS = make_rsrc(state ? (const void*)state : (const void*)Z, state ? (uint32_t)M : 0u);
    auto state_of = [&](int n) -> int {                         // nonzero: masked
        return __builtin_amdgcn_raw_buffer_load_b8(rS, n < ntiles ? (uint32_t)(n * kTqmTok + il) : kOOB, 0, 0);
    };
    const uint32_t row_bytes = (uint32_t)K * BITS / 8;
    const __amdgpu_buffer_rsrc_t rA = make_rsrc(Aq, (uint32_t)M * row_bytes);
    const __amdgpu_buffer_rsrc_t rSo = make_rsrc(s_out, (uint32_t)M * 4);
    const int rr = lane / 4, pp = lane % 4;                     // coding pass: token rr, runs 8 j + 2 pp, 8 j + 2 pp + 1

    int n = blockIdx.x;
    int st_cur = state_of(n);                                   // issued ahead of the ring, as in the loop
    uint32_t zb = tile_base(n);
    v4i zr[D];
#pragma unroll
    for (int q = 0; q < D; ++q) zr[q] = __builtin_amdgcn_raw_buffer_load_b128(rz, zb + 64 * q, 0, 0);
    for (int par = 0; n < ntiles; n += gridDim.x, par ^= 1) {
        const int t0 = n * kTqmTok;
        const uint32_t zn = tile_base(n + gridDim.x);
        const int st_next = state_of(n + gridDim.x);            // needed one tile later
        // the other state's band is dropped: [u_lo, K) for masked tokens, [m_lo, u_lo) otherwise
        const bool masked = gated && st_cur != 0;
        int drop_rel = 4 * kl - (masked ? u_lo : m_lo);         // channel gc + q of this lane is gc + q + 4 k
        const int drop_n = masked ? K - u_lo : u_lo - m_lo;
        asm volatile("" : "+v"(drop_rel));                      // (kept whole, not folded into per-group constants)

        float amax = 0.0f;
#pragma unroll
        for (int j = 0; j < NC; ++j) {
            const v4i z = zr[j % D];
            zr[j % D] = j + D < NC ? __builtin_amdgcn_raw_buffer_load_b128(rz, zb + 64 * (j + D), 0, 0)
                                   : __builtin_amdgcn_raw_buffer_load_b128(rz, zn + 64 * (j + D - NC), 0, 0);
            // (c, c + 4) pairs of this lane's 8 channels, then across the four rows:
            // x_p ends as (channel 8 p + k, 8 p + k + 4) of the 32-channel chunk
            uint32_t x0 = __builtin_amdgcn_perm((uint32_t)z.z, (uint32_t)z.x, 0x05040100u);
            uint32_t x1 = __builtin_amdgcn_perm((uint32_t)z.z, (uint32_t)z.x, 0x07060302u);
            uint32_t x2 = __builtin_amdgcn_perm((uint32_t)z.w, (uint32_t)z.y, 0x05040100u);
            uint32_t x3 = __builtin_amdgcn_perm((uint32_t)z.w, (uint32_t)z.y, 0x07060302u);
            transpose_rows4(x0, x1, x2, x3);
            // the chunk's two groups (2 j, 2 j + 1): their MFMA chains interleaved, so
            // one's latency covers the other's; then the two epilogues
            const int b0 = 2 * j;
            asm volatile("" : "+v"(mp[b0][0]), "+v"(mp[b0][1]), "+v"(mp[b0 + 1][0]), "+v"(mp[b0 + 1][1]));
            f32x4 acc[2] = {{0.0f, 0.0f, 0.0f, 0.0f}, {0.0f, 0.0f, 0.0f, 0.0f}};
            // (widening the block-matrix operands only here: converted ahead, or
            // hoisted out of the tile loop, they would double their registers)
            acc[0] = __builtin_amdgcn_mfma_f32_16x16x4f32(lo_h(mp[b0][0]), lo_h(x0), acc[0], 0, 0, 0);
            acc[1] = __builtin_amdgcn_mfma_f32_16x16x4f32(lo_h(mp[b0 + 1][0]), lo_h(x2), acc[1], 0, 0, 0);
            acc[0] = __builtin_amdgcn_mfma_f32_16x16x4f32(hi_h(mp[b0][0]), hi_h(x0), acc[0], 0, 0, 0);
            acc[1] = __builtin_amdgcn_mfma_f32_16x16x4f32(hi_h(mp[b0 + 1][0]), hi_h(x2), acc[1], 0, 0, 0);
            acc[0] = __builtin_amdgcn_mfma_f32_16x16x4f32(lo_h(mp[b0][1]), lo_h(x1), acc[0], 0, 0, 0);
            acc[1] = __builtin_amdgcn_mfma_f32_16x16x4f32(lo_h(mp[b0 + 1][1]), lo_h(x3), acc[1], 0, 0, 0);
            acc[0] = __builtin_amdgcn_mfma_f32_16x16x4f32(hi_h(mp[b0][1]), hi_h(x1), acc[0], 0, 0, 0);
            acc[1] = __builtin_amdgcn_mfma_f32_16x16x4f32(hi_h(mp[b0 + 1][1]), hi_h(x3), acc[1], 0, 0, 0);
#pragma unroll
            for (int gg = 0; gg < 2; ++gg) {
                const int b = b0 + gg;
                // this lane: channels gc + 4 k + v of token t; the gate (exact zeros)
                // and the maximum act on the fp32 sums, whose fp16 rounding is monotone
                const int gc = ch0 + 16 * b;
                const float4 bv = *reinterpret_cast<const float4*>(bias + gc + 4 * kl);
                float v[4] = {acc[gg][0] + bv.x, acc[gg][1] + bv.y, acc[gg][2] + bv.z, acc[gg][3] + bv.w};
                if (gmask & (1u << b)) {                        // the group meets a band
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        v[q] = (unsigned)(drop_rel + (gc + q)) < (unsigned)drop_n ? 0.0f : v[q];
                }
                amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
                uint16_t h[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) h[q] = f2h(v[q]);
                *reinterpret_cast<uint2*>(region + il * S::kRS + 2 * (16 * b + 4 * kl)) =
                    make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
            }
            // chunk by chunk: a chain of four dependent MFMAs already keeps the matrix
            // pipe busy, and running further ahead only raises register pressure
            __builtin_amdgcn_sched_barrier(0);
        }
        // the token's maximum over this wave (lanes t, t + 16, t + 32, t + 48), rounded
        // to fp16 as the values are (rounding is monotone: the max of the rounded values)
        amax = fmaxf(amax, __shfl_xor(amax, 16, kWave));
        amax = fmaxf(amax, __shfl_xor(amax, 32, kWave));
        amax = h2f(f2h(amax));
        if (kl == 0) red[(par * kTqmTok + il) * kTqmMaxWaves + wave] = amax;
        ring_barrier();   // every wave's maxima and this wave's output tile are in LDS

        // coding pass: lane -> token rr and, in each group of 8 runs of 8 channels of
        // the wave's range, runs 2 pp and 2 pp + 1 (the four lanes of a token read 64
        // consecutive LDS bytes per read, not runs 256 bytes apart in one bank)
        const float4* rp = reinterpret_cast<const float4*>(red + (par * kTqmTok + rr) * kTqmMaxWaves);
        const float4 r0 = rp[0], r1 = rp[1];
        const float rv[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
        float a = rv[0];
#pragma unroll
        for (int w = 1; w < kTqmMaxWaves; ++w) a = w < W ? fmaxf(a, rv[w]) : a;
        const float s = a / kQmax;
        const float y = s != 0.0f ? 1.0f / s : 0.0f;   // s = 0: every value is 0 and codes 0
        if (wave == 0)
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(s), rSo, pp == 0 ? (uint32_t)(t0 + rr) * 4 : kOOB, 0, 0);
        const uint8_t* src = region + rr * S::kRS + 32 * pp;
        const uint32_t dst = (uint32_t)(t0 + rr) * row_bytes + (uint32_t)(ch0 + 16 * pp) * BITS / 8;
#pragma unroll
        for (int i0 = 0; i0 < VPL; i0 += 2) {
            uint32_t wv[BITS == 4 ? 2 : 4];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const v4i hv = *reinterpret_cast<const v4i*>(src + 16 * (4 * i0 + i));
                const float x[8] = {lo_h(hv.x), hi_h(hv.x), lo_h(hv.y), hi_h(hv.y),
                                    lo_h(hv.z), hi_h(hv.z), lo_h(hv.w), hi_h(hv.w)};
                int c[8];
                quant_codes8<BITS == 4 ? 7 : 127>(x, s, y, c);
                if (BITS == 4) {
                    uint32_t w4 = 0;
#pragma unroll
                    for (int q = 0; q < 8; ++q) w4 |= (uint32_t)(c[q] & 15) << (4 * q);
                    wv[i] = w4;
                } else {
                    uint32_t lo = 0, hi = 0;
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        lo |= (uint32_t)(c[q] & 255) << (8 * q);
                        hi |= (uint32_t)(c[4 + q] & 255) << (8 * q);
                    }
                    wv[2 * i] = lo, wv[2 * i + 1] = hi;
                }
            }
            if (BITS == 4) {
                typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
                __builtin_amdgcn_raw_buffer_store_b64(u32x2{wv[0], wv[1]}, rA, dst + 16 * i0, 0, 0);
            } else {
                __builtin_amdgcn_raw_buffer_store_b128(u32x4{wv[0], wv[1], wv[2], wv[3]}, rA, dst + 32 * i0, 0, 0);
            }
        }
        wave_sync();   // this wave's tile is rewritten by its next tile
        zb = zn;
        st_cur = st_next;
    }
}

// The matrix-core form (measured against tac_quant_kernel, interleaved on one
// box): g = 16 only (at g <= 8 the VALU kernel multiplies g, not 16, values per
// output and is faster), rows of four to eight 512-channel parts (hidden sizes
// 2048 ... 4096, 3584 among them),
// operands under 2 GiB, and at least 4096 tokens (256 tiles: one per CU; at
// 2048 tokens the row-streaming kernel is faster).
constexpr int kTqmMaxGroups = 256;                  // one workgroup per CU
constexpr int kTqmMinRows = 4096;
bool tac_quant_mfma_usable(int M, int K, int g) {
    return g == 16 && M >= kTqmMinRows && (size_t)M * K * 2 <= ((size_t)1 << 31) && K % 512 == 0 && K / 512 >= 4 &&
           K / 512 <= kTqmMaxWaves;
}

template <int BITS, int NG>
hipError_t launch_tqm(int M, const uint16_t* Z, const uint16_t* Mb, const uint16_t* d, const uint8_t* state, int K,
                      int dm, int du, uint8_t* Aq, float* s, hipStream_t st) {
    using S = TqmShape<NG>;
    static std::atomic<int> lds_set[kMaxDevices];   // above the 64 KB default for dynamic LDS
    const hipError_t attr = allow_dynamic_lds(reinterpret_cast<const void*>(&tac_quant_mfma_kernel<BITS, NG>),
                                              (int)S::lds_bytes(S::kCWV * kTqmMaxWaves), lds_set);
    if (attr != hipSuccess) return attr;
    const int ntiles = (M + kTqmTok - 1) / kTqmTok;
    const dim3 grid(ntiles < kTqmMaxGroups ? ntiles : kTqmMaxGroups), block(64 * (K / S::kCWV));
    hipLaunchKernelGGL((tac_quant_mfma_kernel<BITS, NG>), grid, block, S::lds_bytes(K), st, Z, Mb, d, state, M, K, dm,
                       du, Aq, s);
    return hipGetLastError();
}

}  // namespace

bool tac_quant_fusable(int K, int g) { return g <= 16 && K % 16 == 0 && K / 8 <= 64 * kTqMaxConsumerWaves; }

hipError_t launch_tac_quant(const uint16_t* Z, const uint16_t* Mb, const uint16_t* d, const uint8_t* state, int M,
                            int K, int g, int dm, int du, uint8_t* Aq, float* s, hipStream_t st, int bits) {
    if (tac_quant_mfma_usable(M, K, g))
        return bits == 8 ? launch_tqm<8, 32>(M, Z, Mb, d, state, K, dm, du, Aq, s, st)
                         : launch_tqm<4, 32>(M, Z, Mb, d, state, K, dm, du, Aq, s, st);
    const int cw = (K / 8 + kWave - 1) / kWave;
    const int threads = (cw + 1) * kWave;
    // about two workgroups per CU, each streaming a run of up to 64 rows
    int rows = (M + 511) / 512;
    rows = rows < 1 ? 1 : (rows > kTqMaxRows ? kTqMaxRows : rows);
    const dim3 grid((M + rows - 1) / rows);
    // at most 6 x 8 KB + 128 bytes (K <= 4096): inside the default 64 KB dynamic-LDS limit
    const size_t lds = (size_t)kTqRing * cw * 1024 + 2 * kTqMaxConsumerWaves * sizeof(float) + kTqMaxRows;
    switch (g * (bits == 8 ? -1 : 1)) {
#define SQ_TQ(G)                                                                                                  \
    case G:                                                                                                       \
        hipLaunchKernelGGL((tac_quant_kernel<G, 4>), grid, dim3(threads), lds, st, Z, Mb, d, state, M, K, dm, du, \
                           rows, Aq, s);                                                                          \
        break;                                                                                                    \
    case -G:                                                                                                      \
        hipLaunchKernelGGL((tac_quant_kernel<G, 8>), grid, dim3(threads), lds, st, Z, Mb, d, state, M, K, dm, du, \
                           rows, Aq, s);                                                                          \
        break;
        SQ_TQ(1)
        SQ_TQ(2)
        SQ_TQ(4)
        SQ_TQ(8)
        SQ_TQ(16)
#undef SQ_TQ
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace sq
