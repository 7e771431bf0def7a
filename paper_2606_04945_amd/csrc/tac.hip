// Temporal Attention Compensation (Sec. 3.3, Eq. 17; App. C): per token and per
// block b of g channels, z'_{bg+r} = fp16( sum_c M_b[r][c] z_{bg+c} + d_{bg+r} ),
// each sum an fp32 fused multiply-add chain in ascending c from +0, bias last.
//
// The map is a batch of small [tokens x g] x [g x g] products, one per block.
// It runs on the VALU because the fixed FMA order is part of the result; the
// kernel is a register-tiled batched SGEMM: a workgroup owns TT tokens x CW
// channels (CW = max(g, 64) so a span holds whole blocks), stages the span's
// block matrices and the token tile through LDS as fp32, and each thread keeps
// 8 tokens x 8 channels of accumulators (8 x 4 when g < 8), so each pair of
// LDS reads feeds 64 (32) fused multiply-adds.
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
    if (g < 8) return launch_cw<64, 4>(Z, Mb, d, M, C, g, out, st);
    if (g <= 64) return launch_cw<64, 8>(Z, Mb, d, M, C, g, out, st);
    return launch_cw<128, 8>(Z, Mb, d, M, C, g, out, st);
}

}  // namespace sq

// ---------------------------------------------------------------------------
// TAC fused with the gate and the per-token int4 quantiser, for g <= 16 and an
// input already in the P basis (no dense transform): z -> fp16(M_b z_b + d_b)
// -> G_s -> absmax -> codes, without materialising z'.  Thread t owns channels
// [8t, 8t + 8) of every token row (K / 8 active threads), keeps those channels'
// block-matrix rows (8 x g) and biases in registers, and walks the workgroup's
// tokens one row at a time: 8 outputs of g fused multiply-adds each (same order
// and rounding as tac_kernel), the gate, a block max, then the 8 codes packed
// into 4 bytes.
namespace sq {
namespace {

constexpr int kFusedThreads = 512;
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float block_max_db(float v, float (*red)[kFusedThreads / kWave], int parity) {
    v = wave_max(v);
    const int w = threadIdx.x / kWave, l = threadIdx.x % kWave;
    if (l == 0) red[parity][w] = v;
    __syncthreads();
    float r = 0.0f;
    const int nw = (int)(blockDim.x + kWave - 1) / kWave;
    for (int i = 0; i < nw; ++i) r = fmaxf(r, red[parity][i]);
    return r;
}

template <int G, int BITS>
__global__ __launch_bounds__(kFusedThreads) void tac_quant_kernel(const uint16_t* __restrict__ Z,
                                                                  const uint16_t* __restrict__ Mb,
                                                                  const uint16_t* __restrict__ d,
                                                                  const uint8_t* __restrict__ state, int M, int K,
                                                                  int dm, int du, int rows_per_wg,
                                                                  uint8_t* __restrict__ Aq,
                                                                  float* __restrict__ s_out) {
    constexpr int ZW = G > 8 ? G : 8;                   // input channels a thread reads (whole blocks)
    __shared__ float red[2][kFusedThreads / kWave];
    // staging of the block-matrix rows (G >= 4): per wave, TPP slots of 16 G + 16 bytes
    constexpr int kStage = G >= 4 ? (G == 16 ? 32 : 64) * (16 * G + 16) : 16;
    __shared__ __attribute__((aligned(16))) uint8_t pstage[kFusedThreads / kWave * kStage];
    const int t = threadIdx.x;
    const bool active = 8 * t < K;
    const int c0 = 8 * t;                               // first output channel of this thread
    const int z0 = (c0 / ZW) * ZW;                      // first input channel it reads
    const int row_begin = blockIdx.x * rows_per_wg;
    const int row_end = min(M, row_begin + rows_per_wg);
    // A row's inputs (its activations and state byte) are requested before the
    // previous row's work, the first row's around the block parameters, so these
    // fetches overlap instead of following one another.  Buffer loads: inactive
    // threads and a call without states read zeros, with no branch.
    const bool gated = state != nullptr;
    const __amdgpu_buffer_rsrc_t rS = make_rsrc(state, gated ? (uint32_t)M : 0u);
    v4i zr[ZW / 8];
    uint32_t sb = 0;
    auto fetch_z = [&](int row) {
        const __amdgpu_buffer_rsrc_t rz = make_rsrc(Z + (size_t)row * K, (uint32_t)K * 2);
#pragma unroll
        for (int v = 0; v < ZW / 8; ++v)
            zr[v] = __builtin_amdgcn_raw_buffer_load_b128(rz, active ? (z0 + 8 * v) * 2 : (int)kOOB, 0, 0);
    };
    auto fetch_s = [&](int row) { sb = __builtin_amdgcn_raw_buffer_load_b8(rS, row, 0, 0); };
    if (row_begin < row_end) fetch_z(row_begin);
    // tac_M viewed as [K][G]: this thread's rows c0 .. c0 + 7 are 8 G fp16
    // values, held as G vectors of 8 (element r G + c of the run = row r,
    // column c) and widened to fp32 where they are used
    v8h mh[G];
    float dv[8];
    const int cm = active ? c0 : 0;                     // inactive threads read the first rows, unused
    if constexpr (G >= 4) {
        // A thread's rows are PB = 16 G contiguous bytes at PB t, so loaded
        // directly the lanes of one 16-byte load would touch up to 64 cache
        // lines.  Instead each wave loads its 64 runs with whole-wave
        // contiguous 16-byte loads, writes them to per-thread LDS slots padded
        // by 16 bytes (so the 16-byte reads below are free of bank conflicts),
        // and each thread reads its own slot back; for G = 16 in two passes of
        // 32 threads, one after the other so that only one pass's loads hold
        // registers.  A wave's LDS accesses are performed in order, so only
        // the compiler has to be kept from reordering them (the fences).
        constexpr int PB = 16 * G, NC = PB / 16, SLOT = PB + 16;
        constexpr int TPP = G == 16 ? 32 : 64;          // threads per pass
        constexpr int PASSES = kWave / TPP;
        constexpr int LOADS = TPP * NC / kWave;         // 16-byte loads per lane per pass
        const int wave = t / kWave, lane = t % kWave;
        uint8_t* stage = pstage + wave * (TPP * SLOT);
        const __amdgpu_buffer_rsrc_t rM = make_rsrc(Mb, (uint32_t)K * G * 2);
        const int slab = wave * kWave * NC;             // first chunk of this wave's runs
        auto load_pass = [&](int p, v4i* ch) {
#pragma unroll
            for (int i = 0; i < LOADS; ++i)
                ch[i] = __builtin_amdgcn_raw_buffer_load_b128(rM, (slab + p * TPP * NC + i * kWave + lane) * 16, 0, 0);
        };
        auto wave_sync = [] {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        };
#pragma unroll
        for (int p = 0; p < PASSES; ++p) {
            v4i ch[LOADS];
            load_pass(p, ch);
#pragma unroll
            for (int i = 0; i < LOADS; ++i) {
                const int c = i * kWave + lane;         // chunk of this pass: thread c / NC, piece c % NC
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
    } else {
        // runs of 16 or 32 bytes: the lanes of a load already cover whole lines
#pragma unroll
        for (int j = 0; j < G; ++j) mh[j] = *reinterpret_cast<const v8h*>(Mb + (size_t)cm * G + 8 * j);
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) dv[r] = h2f(d[cm + r]);
    if (row_begin < row_end) fetch_s(row_begin);
    for (int row = row_begin; row < row_end; ++row) {
        // keeps the block rows packed as fp16 (the multiply-adds widen them):
        // hoisting their conversion out of the loop would hold 8 G fp32
        // registers and leave room for fewer waves
#pragma unroll
        for (int j = 0; j < G; ++j) asm volatile("" : "+v"(mh[j]));
        float o[8];
        float amax = 0.0f;
        float z[ZW];
#pragma unroll
        for (int v = 0; v < ZW / 8; ++v) {
            const uint16_t* h = reinterpret_cast<const uint16_t*>(&zr[v]);
#pragma unroll
            for (int i = 0; i < 8; ++i) z[8 * v + i] = h2f(h[i]);
        }
        const bool masked = sb != 0;
        if (row + 1 < row_end) {
            fetch_z(row + 1);
            fetch_s(row + 1);
        }
        if (active) {
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const int base = ((c0 - z0 + r) / G) * G;   // block start within z[]
                float acc = 0.0f;
#pragma unroll
                for (int c = 0; c < G; ++c) {
                    const int e = r * G + c;
                    acc = __builtin_fmaf((float)mh[e / 8][e % 8], z[base + c], acc);
                }
                const float v = h2f(f2h(acc + dv[r]));  // TAC output, materialised as fp16
                o[r] = (!gated | kept_sel(c0 + r, K, dm, du, masked)) ? v : 0.0f;
                amax = fmaxf(amax, fabsf(o[r]));
            }
        }
        const float s = block_max_db(amax, red, row & 1) / (BITS == 4 ? 7.0f : 127.0f);
        const float y = s != 0.0f ? 1.0f / s : 0.0f;
        if (t == 0) s_out[row] = s;
        if (active) {
            if (BITS == 4) {
                uint32_t w = 0;
                if (s != 0.0f) {
                    int c[8];
                    quant_codes8<7>(o, s, y, c);
#pragma unroll
                    for (int q = 0; q < 8; ++q) w |= (uint32_t)(c[q] & 15) << (4 * q);
                }
                *reinterpret_cast<uint32_t*>(Aq + (size_t)row * (K / 2) + 4 * t) = w;
            } else {
                uint32_t lo = 0, hi = 0;
                if (s != 0.0f) {
                    int c[8];
                    quant_codes8<127>(o, s, y, c);
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        lo |= (uint32_t)(c[q] & 255) << (8 * q);
                        hi |= (uint32_t)(c[4 + q] & 255) << (8 * q);
                    }
                }
                *reinterpret_cast<uint2*>(Aq + (size_t)row * K + 8 * t) = make_uint2(lo, hi);
            }
        }
    }
}

}  // namespace

bool tac_quant_fusable(int K, int g) { return g <= 16 && K % 16 == 0 && K / 8 <= kFusedThreads; }

hipError_t launch_tac_quant(const uint16_t* Z, const uint16_t* Mb, const uint16_t* d, const uint8_t* state, int M,
                            int K, int g, int dm, int du, uint8_t* Aq, float* s, hipStream_t st, int bits) {
    const int threads = ((K / 8 + kWave - 1) / kWave) * kWave;
    // enough workgroups to fill the chip, each reusing its parameters over several rows
    int rows = M / 512;
    rows = rows < 1 ? 1 : (rows > 16 ? 16 : rows);
    const dim3 grid((M + rows - 1) / rows);
    switch (g * (bits == 8 ? -1 : 1)) {
#define SQ_TQ(G)                                                                                                  \
    case G:                                                                                                       \
        hipLaunchKernelGGL((tac_quant_kernel<G, 4>), grid, dim3(threads), 0, st, Z, Mb, d, state, M, K, dm, du,  \
                           rows, Aq, s);                                                                          \
        break;                                                                                                    \
    case -G:                                                                                                      \
        hipLaunchKernelGGL((tac_quant_kernel<G, 8>), grid, dim3(threads), 0, st, Z, Mb, d, state, M, K, dm, du,  \
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
