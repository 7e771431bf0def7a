// Per-token symmetric quantisation (Sec. 3.1, Eq. 2 with zero point 0 and
// Eq. 5: per-token activations, per-output-channel weights), at BITS = 4:
//   a = max_j |x_j|,  s = a / 7 (fp32, correctly rounded),
//   q_j = clamp(rint(x_j / s), -8, 7)  (0 when s == 0),
//   byte t = (q_{2t} & 15) | (q_{2t+1} & 15) << 4;
// and at BITS = 8 (the W8A8 variant of App. D): s = a / 127, q_j =
// clamp(rint(x_j / s), -128, 127), one signed byte per code.
//
// One 256-thread workgroup per row: coalesced 16-byte loads held in registers,
// all issued before the first is used (buffer loads, whose range check reads
// past the row, and the state of a call without one, as zero, so no branch
// separates them and a row costs one memory round trip however long it is), a
// wavefront max reduction plus one LDS exchange across the four waves, then
// quantise-and-pack straight from the registers.  Two input forms:
//   quant_f16: fp16 rows already in the P basis, with the SGAT gate applied on
//              the fly (state select, Eq. 9-11) -- the folded-basis hot path;
//   quant_f32: fp32 rows from the dense transform (already gated).
// Rows longer than NV*256 vectors are read twice instead of held.
//
// Few rows (decode-sized batches) would leave most of the chip idle with one
// workgroup per row, and each lane's chain of NV vectors then sets the time.
// There the quantisers run `slices` workgroups per row: each reads the whole row
// and forms the same absmax (max is exact and order-free, so every slice
// derives the identical s), and quantises only its own vector of each lane.
#include "tile_common.hpp"

namespace sq {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float block_max(float v, float* red) {
    v = wave_max(v);
    const int w = threadIdx.x / kWave, l = threadIdx.x % kWave;
    if (l == 0) red[w] = v;
    __syncthreads();
    float r = red[0];
#pragma unroll
    for (int i = 1; i < kThreads / kWave; ++i) r = fmaxf(r, red[i]);
    return r;
}

// 8 values -> their codes, stored at code index 8v of the row: 4 bytes (4-bit)
// or 8 bytes (8-bit)
// (y = 1 / s, see quant_codes8)
template <int BITS>
__device__ __forceinline__ void store8(uint8_t* row, int v, const float* x, float s, float y) {
    if (BITS == 4) {
        uint32_t out = 0;
        if (s != 0.0f) {
            int c[8];
            quant_codes8<7>(x, s, y, c);
#pragma unroll
            for (int q = 0; q < 8; ++q) out |= (uint32_t)(c[q] & 15) << (4 * q);
        }
        reinterpret_cast<uint32_t*>(row)[v] = out;
    } else {
        uint32_t lo = 0, hi = 0;
        if (s != 0.0f) {
            int c[8];
            quant_codes8<127>(x, s, y, c);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                lo |= (uint32_t)(c[q] & 255) << (8 * q);
                hi |= (uint32_t)(c[4 + q] & 255) << (8 * q);
            }
        }
        reinterpret_cast<uint2*>(row)[v] = make_uint2(lo, hi);
    }
}

template <int BITS>
__device__ __forceinline__ float qmaxf() { return BITS == 4 ? 7.0f : 127.0f; }

__device__ __forceinline__ void load_f16x8(const uint16_t* p, const uint8_t* state, int row, int c0, int K,
                                           int dm, int du, float* x) {
    const uint4 raw = *reinterpret_cast<const uint4*>(p);
    const uint16_t* h = reinterpret_cast<const uint16_t*>(&raw);
    const bool masked = state ? state[row] != 0 : false;
#pragma unroll
    for (int q = 0; q < 8; ++q) x[q] = (!state || kept(c0 + q, K, dm, du, masked)) ? h2f(h[q]) : 0.0f;
}

// fp16 input; NV vectors of 8 per thread held in registers (NV == 0: reload).
template <int NV, int BITS>
__global__ __launch_bounds__(kThreads) void quant_f16_kernel(const uint16_t* __restrict__ X,
                                                             const uint8_t* __restrict__ state, int K, int dm,
                                                             int du, int slices, uint8_t* __restrict__ Aq,
                                                             float* __restrict__ s_out) {
    __shared__ float red[kThreads / kWave];
    const int row = blockIdx.x / slices, slice = blockIdx.x % slices;
    const int nvec = K / 8;
    const uint16_t* xr = X + (size_t)row * K;
    uint8_t* qr = Aq + (size_t)row * (K * BITS / 8);
    float amax = 0.0f;
    if constexpr (NV > 0) {
        const bool gated = state != nullptr;
        const __amdgpu_buffer_rsrc_t rX = make_rsrc(xr, (uint32_t)K * 2);
        const __amdgpu_buffer_rsrc_t rS = make_rsrc(state, gated ? (uint32_t)row + 1 : 0u);
        v4i raw[NV];
#pragma unroll
        for (int i = 0; i < NV; ++i)
            raw[i] = __builtin_amdgcn_raw_buffer_load_b128(rX, ((int)threadIdx.x + i * kThreads) * 16, 0, 0);
        const bool masked = __builtin_amdgcn_raw_buffer_load_b8(rS, row, 0, 0) != 0;
        // The gate keeps columns [0, lim0) and [lim1, K) of this row (a masked
        // row drops its u-band, an unmasked one its m-band), so nearly every
        // vector of 8 is kept or dropped whole; only a vector that straddles a
        // band edge is gated column by column.
        const int lim0 = gated ? (masked ? K - du : K - dm - du) : K;
        const int lim1 = masked ? K : K - du;
        float x[NV][8];
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int v = threadIdx.x + i * kThreads;
            const int lo = v * 8;
            const uint16_t* h = reinterpret_cast<const uint16_t*>(&raw[i]);
            if ((lo + 8 <= lim0) | (lo >= lim1)) {
#pragma unroll
                for (int q = 0; q < 8; ++q) x[i][q] = h2f(h[q]);
            } else if ((lo >= lim0) & (lo + 8 <= lim1)) {
#pragma unroll
                for (int q = 0; q < 8; ++q) x[i][q] = 0.0f;
            } else {
#pragma unroll
                for (int q = 0; q < 8; ++q) x[i][q] = (lo + q < lim0) | (lo + q >= lim1) ? h2f(h[q]) : 0.0f;
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) amax = fmaxf(amax, fabsf(x[i][q]));
        }
        const float s = block_max(amax, red) / qmaxf<BITS>();
        const float y = s != 0.0f ? 1.0f / s : 0.0f;
        if (threadIdx.x == 0 && slice == 0) s_out[row] = s;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int v = threadIdx.x + i * kThreads;
            if ((slices == 1 || i == slice) && v < nvec) store8<BITS>(qr, v, x[i], s, y);
        }
    } else {
        float x[8];
        for (int v = threadIdx.x; v < nvec; v += kThreads) {
            load_f16x8(xr + v * 8, state, row, v * 8, K, dm, du, x);
#pragma unroll
            for (int q = 0; q < 8; ++q) amax = fmaxf(amax, fabsf(x[q]));
        }
        const float s = block_max(amax, red) / qmaxf<BITS>();
        const float y = s != 0.0f ? 1.0f / s : 0.0f;
        if (threadIdx.x == 0) s_out[row] = s;
        for (int v = threadIdx.x; v < nvec; v += kThreads) {
            load_f16x8(xr + v * 8, state, row, v * 8, K, dm, du, x);
            store8<BITS>(qr, v, x, s, y);
        }
    }
}

// fp32 input (already gated); NV vectors of 8 floats per thread (NV == 0: reload).
template <int NV, int BITS>
__global__ __launch_bounds__(kThreads) void quant_f32_kernel(const float* __restrict__ X, int K, int slices,
                                                             uint8_t* __restrict__ Aq, float* __restrict__ s_out) {
    __shared__ float red[kThreads / kWave];
    const int row = blockIdx.x / slices, slice = blockIdx.x % slices;
    const int nvec = K / 8;
    const float* xr = X + (size_t)row * K;
    uint8_t* qr = Aq + (size_t)row * (K * BITS / 8);
    float amax = 0.0f;
    auto ld = [&](int v, float* x) {
        const float4 a = *reinterpret_cast<const float4*>(xr + v * 8);
        const float4 b = *reinterpret_cast<const float4*>(xr + v * 8 + 4);
        x[0] = a.x, x[1] = a.y, x[2] = a.z, x[3] = a.w, x[4] = b.x, x[5] = b.y, x[6] = b.z, x[7] = b.w;
    };
    if constexpr (NV > 0) {
        const __amdgpu_buffer_rsrc_t rX = make_rsrc(xr, (uint32_t)K * 4);
        v4i raw[NV][2];
#pragma unroll
        for (int i = 0; i < NV; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                raw[i][j] = __builtin_amdgcn_raw_buffer_load_b128(rX, ((int)threadIdx.x + i * kThreads) * 32 + 16 * j,
                                                                  0, 0);
        float x[NV][8];
#pragma unroll
        for (int i = 0; i < NV; ++i)
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int b = raw[i][q / 4][q % 4];   // copied out first: a bit cast of a vector element reads element 0
                x[i][q] = __builtin_bit_cast(float, b);
                amax = fmaxf(amax, fabsf(x[i][q]));
            }
        const float s = block_max(amax, red) / qmaxf<BITS>();
        const float y = s != 0.0f ? 1.0f / s : 0.0f;
        if (threadIdx.x == 0 && slice == 0) s_out[row] = s;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int v = threadIdx.x + i * kThreads;
            if ((slices == 1 || i == slice) && v < nvec) store8<BITS>(qr, v, x[i], s, y);
        }
    } else {
        float x[8];
        for (int v = threadIdx.x; v < nvec; v += kThreads) {
            ld(v, x);
#pragma unroll
            for (int q = 0; q < 8; ++q) amax = fmaxf(amax, fabsf(x[q]));
        }
        const float s = block_max(amax, red) / qmaxf<BITS>();
        const float y = s != 0.0f ? 1.0f / s : 0.0f;
        if (threadIdx.x == 0) s_out[row] = s;
        for (int v = threadIdx.x; v < nvec; v += kThreads) {
            ld(v, x);
            store8<BITS>(qr, v, x, s, y);
        }
    }
}

template <template <int, int> class Launch, int BITS, typename... A>
hipError_t by_nv(int K, A... args) {
    const int per = (K / 8 + kThreads - 1) / kThreads;   // vectors per thread
    if (per <= 1) return Launch<1, BITS>::run(args...);
    if (per <= 2) return Launch<2, BITS>::run(args...);
    if (per <= 4) return Launch<4, BITS>::run(args...);
    if (per <= 6) return Launch<6, BITS>::run(args...);
    if (per <= 8) return Launch<8, BITS>::run(args...);
    if (per <= 12) return Launch<12, BITS>::run(args...);
    return Launch<0, BITS>::run(args...);
}

// The quantisers split each row over one workgroup per vector of a lane while
// that gives at most this many workgroups (M x slices); past it the repeated
// reads of each row cost more than the shorter chains gain
constexpr long kSplitWorkgroups = 768;

template <int NV, int BITS>
struct LaunchF16 {
    static hipError_t run(const uint16_t* x, const uint8_t* state, int M, int K, int dm, int du, uint8_t* q,
                          float* s, hipStream_t st) {
        const int per = (K / 8 + kThreads - 1) / kThreads;
        const int slices = NV > 1 && (long)M * per <= kSplitWorkgroups ? per : 1;
        hipLaunchKernelGGL((quant_f16_kernel<NV, BITS>), dim3(M * slices), dim3(kThreads), 0, st, x, state, K, dm,
                           du, slices, q, s);
        return hipGetLastError();
    }
};

template <int NV, int BITS>
struct LaunchF32 {
    static hipError_t run(const float* x, int M, int K, uint8_t* q, float* s, hipStream_t st) {
        const int per = (K / 8 + kThreads - 1) / kThreads;
        const int slices = NV > 1 && (long)M * per <= kSplitWorkgroups ? per : 1;
        hipLaunchKernelGGL((quant_f32_kernel<NV, BITS>), dim3(M * slices), dim3(kThreads), 0, st, x, K, slices, q, s);
        return hipGetLastError();
    }
};

}  // namespace

hipError_t launch_quant_f16(const uint16_t* x, const uint8_t* state, int M, int K, int dm, int du, uint8_t* q,
                            float* s, hipStream_t st, int bits) {
    if (bits == 8) return by_nv<LaunchF16, 8>(K, x, state, M, K, dm, du, q, s, st);
    return by_nv<LaunchF16, 4>(K, x, state, M, K, dm, du, q, s, st);
}

hipError_t launch_quant_f32(const float* x, int M, int K, uint8_t* q, float* s, hipStream_t st, int bits) {
    if (bits == 8) return by_nv<LaunchF32, 8>(K, x, M, K, q, s, st);
    return by_nv<LaunchF32, 4>(K, x, M, K, q, s, st);
}

}  // namespace sq
