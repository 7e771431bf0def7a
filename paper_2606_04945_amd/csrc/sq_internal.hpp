// Internal declarations shared by the HIP translation units of libstarquant.
// gfx950 (CDNA4) only: wave64, int8 MFMA, 160 KB LDS per CU.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>

namespace sq {

constexpr int kWave = 64;
constexpr int kChunk = 256;          // transform k-chunk (fixed evaluation order)
constexpr int kXcds = 8;             // accelerator complex dies, each with its own L2

// Tile order for a one-dimensional grid of T = R x C output tiles.  Workgroup
// dispatch goes round-robin over the XCDs (dispatch index L runs on XCD L % 8),
// so the tiles are first split into 8 contiguous ranges, one per XCD, and
// within a range they are visited in groups of G row tiles, row tile fastest:
// the workgroups an XCD runs at the same time then share G row tiles and a few
// column tiles, which its L2 serves after the first fetch.  A bijection on
// [0, T) for any dispatch order, so only locality depends on the assumption.
__device__ __forceinline__ void xcd_tile(int L, int R, int C, int G, int& r, int& c) {
    const int T = R * C;
    const int base = T / kXcds, rem = T % kXcds;
    const int x = L % kXcds, local = L / kXcds;
    const int v = x * base + (x < rem ? x : rem) + local;
    const int per_group = G * C;
    const int first = (v / per_group) * G;
    const int gsz = R - first < G ? R - first : G;
    r = first + (v % per_group) % gsz;
    c = (v % per_group) / gsz;
}

typedef int v4i __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float h2f(uint16_t h) {
    return (float)__builtin_bit_cast(_Float16, h);
}
// fp32 -> fp16, round to nearest even, from a materialised fp32 value.  The
// empty asm keeps the compiler from folding the multiply or add that produced f
// into a mixed-precision v_fma_mix*_f16, which would round the exact result once
// to fp16 instead of rounding to fp32 first (and ignores -ffp-contract=off).
__device__ __forceinline__ uint16_t f2h(float f) {
    asm volatile("" : "+v"(f));
    return __builtin_bit_cast(uint16_t, (_Float16)f);
}

// Column j of a transformed row is kept for this state (gate G_s, Eq. 9).
__device__ __forceinline__ bool kept(int j, int K, int dm, int du, bool masked) {
    const int m_lo = K - dm - du, u_lo = K - du;
    return j < m_lo || (j < u_lo ? masked : !masked);
}

// The same without control flow (bitwise on the comparisons), for use between
// loads that must all be in flight together.
__device__ __forceinline__ bool kept_sel(int j, int K, int dm, int du, bool masked) {
    return (j < K - dm - du) | ((j < K - du) == masked);
}

// Symmetric int4 code of x for scale s (s > 0): clamp(rint(x / s), -8, 7).
// `/` is the correctly rounded fp32 divide (built without fast-math).
__device__ __forceinline__ int quant4(float x, float s) {
    float r = __builtin_rintf(x / s);
    r = r < -8.0f ? -8.0f : (r > 7.0f ? 7.0f : r);
    return (int)r;
}

// Symmetric int8 code of x for scale s (s > 0): clamp(rint(x / s), -128, 127).
__device__ __forceinline__ int quant8(float x, float s) {
    float r = __builtin_rintf(x / s);
    r = r < -128.0f ? -128.0f : (r > 127.0f ? 127.0f : r);
    return (int)r;
}

// The same code as quant4 (QMAX = 7) or quant8 (QMAX = 127), given also
// y = 1 / s correctly rounded, with a multiply in place of most divides.  y and
// the product x y each round once, and fl(x / s) once, so x y is within
// 3 2^-24 |x / s| of fl(x / s).  Where the clamp does not decide the code,
// |x / s| < QMAX + 2, so the two are less than half of kNear (2^-18, resp.
// 2^-14) apart; when x y is farther than kNear from every half-integer both lie
// between the same two half-integers and rint gives the same integer.  Where
// the clamp decides it, both roundings land beyond the same end of the range.
// Only the remaining x take the divide, and so do NaN and infinite products
// (the comparison is written to be false for NaN), which covers y = inf from a
// subnormal s and non-finite inputs.  Eight codes at a time, with one (rarely
// taken) branch for the group.
template <int QMAX>
__device__ __forceinline__ void quant_codes8(const float* x, float s, float y, int* code) {
    constexpr float kNear = QMAX == 7 ? 0x1p-18f : 0x1p-14f;
    static_assert(QMAX == 7 || QMAX == 127, "4- or 8-bit codes");
    float r[8];
    bool near = false;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const float q0 = x[q] * y;
        r[q] = __builtin_rintf(q0);
        near |= !(fabsf(q0 - r[q]) < 0.5f - kNear);
    }
    if (__builtin_expect(near, 0)) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const float q0 = x[q] * y;
            if (!(fabsf(q0 - r[q]) < 0.5f - kNear)) r[q] = __builtin_rintf(x[q] / s);
        }
    }
    // clamp with one median-of-three (identical to the two-sided clamp for
    // every finite value; it also maps a NaN from non-finite input to a code)
    constexpr float lo = -(QMAX + 1.0f), hi = (float)QMAX;
#pragma unroll
    for (int q = 0; q < 8; ++q) code[q] = (int)__builtin_amdgcn_fmed3f(r[q], lo, hi);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

// Raises kernel `fn`'s dynamic-LDS limit to `bytes` on the current device, once
// per device.  The attribute belongs to the device that is current when it is
// set, so a process that drives several GPUs needs it on each; `done` is the
// caller's per-device flag array (static storage, kMaxDevices entries).  A
// failed call is not remembered: the next launch tries again.
constexpr int kMaxDevices = 64;
inline hipError_t allow_dynamic_lds(const void* fn, int bytes, std::atomic<int>* done) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    if (done[dev].load(std::memory_order_acquire)) return hipSuccess;
    e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e == hipSuccess) done[dev].store(1, std::memory_order_release);
    return e;
}

// ---- launchers (each returns hipError_t of the launch) ----
hipError_t launch_tac(const uint16_t* Z, const uint16_t* Mb, const uint16_t* d,
                      int M, int C, int g, uint16_t* out, hipStream_t st);

// TAC fused with gate + int4 quantisation (P = NULL); valid when tac_quant_fusable.
// bits = 4 (packed int4 codes) or 8 (int8 codes, the W8A8 variant) here and below.
bool tac_quant_fusable(int K, int g);
hipError_t launch_tac_quant(const uint16_t* Z, const uint16_t* Mb, const uint16_t* d, const uint8_t* state, int M,
                            int K, int g, int dm, int du, uint8_t* Aq, float* s, hipStream_t st, int bits);

hipError_t launch_transform(const uint16_t* X, const uint8_t* state, const float* P,
                            int M, int K, int dm, int du, float* Xp, hipStream_t st);

hipError_t launch_quant_f32(const float* x, int M, int K, uint8_t* q, float* s, hipStream_t st, int bits);

hipError_t launch_quant_f16(const uint16_t* x, const uint8_t* state, int M, int K, int dm, int du,
                            uint8_t* q, float* s, hipStream_t st, int bits);

size_t gemm_workspace_bytes(int M, int N, int K, int bits);
hipError_t launch_gemm(const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w,
                       int M, int N, int K, uint16_t* Y, int32_t* acc, void* ws, hipStream_t st, int bits);

// TAC closed-form calibration (tac_calib.hip)
size_t tac_calib_workspace_bytes(int N, int C, int g);
hipError_t launch_tac_calib(const uint16_t* Zf, const uint16_t* Zq, int N, int C, int g, double rho, double eps,
                            double eta, double alpha, uint16_t* tac_M, uint16_t* tac_d, double* M64, double* d64,
                            void* ws, hipStream_t st);

// Fast transform on the fp16 MFMA (transform_fast.hip)
hipError_t launch_split_basis(const float* P, int K, uint16_t* Ps, hipStream_t st);
hipError_t launch_transform_fast(const uint16_t* X, const uint8_t* state, const uint16_t* Ps, int M, int K, int dm,
                                 int du, float* Xp, hipStream_t st);

// GEMM on fragment-ordered weights (gemm.hip), 4- or 8-bit codes; workspace as
// gemm_workspace_bytes(M, N, K, bits).  frag_weight_bytes and weights_to_frag
// count a row in int4 codes (K / 2 bytes): 8-bit rows of K bytes pass 2 K.
size_t frag_weight_bytes(int N, int K);
hipError_t launch_weights_to_frag(const uint8_t* Wq, int N, int K, uint8_t* Wf, hipStream_t st);
hipError_t launch_gemm_frag(const uint8_t* Aq, const float* s_a, const uint8_t* Wf, const float* s_w, int M, int N,
                            int K, uint16_t* Y, int32_t* acc, void* ws, hipStream_t st, int bits);

// int4 codes on the FP6 matrix cores (fp6.hip)
size_t fp6_row_bytes(int K);
hipError_t launch_codes_to_fp6(const uint8_t* src, int R, int K, uint8_t* dst, hipStream_t st);
hipError_t launch_gemm_fp6(const uint8_t* A6, const float* s_a, const uint8_t* W6, const float* s_w, int M, int N,
                           int K, uint16_t* Y, int32_t* acc, hipStream_t st);

}  // namespace sq
