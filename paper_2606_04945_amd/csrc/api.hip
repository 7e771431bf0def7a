// C ABI of libstarquant: argument checks, workspace layout and kernel dispatch.
// Every argument is checked before the first launch; on failure nothing is
// enqueued and the reason is kept in a thread-local message.
#include <stdarg.h>
#include <stdlib.h>
#include <stdio.h>

#include <atomic>
#include <mutex>

#include "../../include/starquant.h"
#include "sq_internal.hpp"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

// SQ_DEBUG_SYNC set to anything but "" or "0" (read once, at the first call):
// every launch is followed by a device-wide synchronisation and an error
// check, so an asynchronous fault is reported by the call whose kernel raised
// it, named in the message.  For debugging only: it serialises the device and
// cannot be used under stream capture.
bool debug_sync() {
    static const bool on = [] {
        const char* v = getenv("SQ_DEBUG_SYNC");
        return v != nullptr && v[0] != '\0' && !(v[0] == '0' && v[1] == '\0');
    }();
    return on;
}

int hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess && debug_sync()) {
        e = hipDeviceSynchronize();
        if (e == hipSuccess) e = hipGetLastError();
    }
    if (e == hipSuccess) return SQ_OK;
    return fail(SQ_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Row-tiled launches put row tiles (at least 64 rows each) on the second grid
// axis, which holds at most 65535 workgroups.
constexpr int32_t kMaxTiledRows = 65535 * 64;

constexpr size_t kAlign = 256;
size_t round_up(size_t n) { return (n + kAlign - 1) / kAlign * kAlign; }

int check_K(int32_t K) {
    if (K < 64 || K > 131072 || K % 64)
        return fail(SQ_ERR_SHAPE, "K=%d: need 64 <= K <= 131072 and K %% 64 == 0", K);
    return SQ_OK;
}

int check_band(int32_t K, int32_t dm, int32_t du) {
    if (dm < 0 || du < 0 || (int64_t)dm + du >= K)
        return fail(SQ_ERR_SHAPE, "bands d_m=%d d_u=%d: need d_m, d_u >= 0 and d_m + d_u < K=%d", dm, du, K);
    return SQ_OK;
}

int check_tac(int32_t C, int32_t g) {
    if (g < 1 || g > 128 || (g & (g - 1)) || C % g)
        return fail(SQ_ERR_SHAPE, "TAC block g=%d: need a power of two in [1, 128] dividing C=%d", g, C);
    return SQ_OK;
}

#define SQ_REQUIRE(cond, code, ...) \
    do {                            \
        if (!(cond)) return fail(code, __VA_ARGS__); \
    } while (0)

#define SQ_TRY(expr)                 \
    do {                             \
        int _rc = (expr);            \
        if (_rc != SQ_OK) return _rc; \
    } while (0)

}  // namespace

extern "C" {

const char* sq_last_error(void) { return g_err; }

const char* sq_version(void) { return "starquant 0.1 gfx950"; }

int32_t sq_tac_default_block(int32_t C) {
    if (C <= 0) return 0;
    for (int g = 16; g > 1; --g)
        if (C % g == 0) return g;
    return 1;
}

size_t sq_quant_act_workspace_bytes(int32_t M, int32_t K, int32_t has_P, int32_t has_tac) {
    if (M <= 0 || K <= 0) return 0;
    size_t n = 0;
    if (has_tac) n += round_up((size_t)M * K * sizeof(uint16_t));
    if (has_P) n += round_up((size_t)M * K * sizeof(float));
    return n;
}

size_t sq_prepare_weights_workspace_bytes(int32_t N, int32_t K, int32_t has_P) {
    if (N <= 0 || K <= 0 || !has_P) return 0;
    return round_up((size_t)N * K * sizeof(float));
}

size_t sq_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K) {
    if (M <= 0 || N <= 0 || K <= 0) return 0;
    return round_up(sq::gemm_workspace_bytes(M, N, K, 4));
}

size_t sq_gemm_w8_workspace_bytes(int32_t M, int32_t N, int32_t K) {
    if (M <= 0 || N <= 0 || K <= 0) return 0;
    return round_up(sq::gemm_workspace_bytes(M, N, K, 8));
}

}  // extern "C"

namespace {

int prepare_weights(const uint16_t* W, const float* P, int32_t N, int32_t K, uint8_t* Wq, float* s_w, void* ws,
                    size_t ws_bytes, void* stream, int bits, const char* name) {
    SQ_TRY(check_K(K));
    SQ_REQUIRE(N >= 0, SQ_ERR_SHAPE, "N=%d < 0", N);
    if (N == 0) return SQ_OK;
    SQ_REQUIRE(W && Wq && s_w, SQ_ERR_NULL, "%s: W, Wq and s_w are required", name);
    SQ_REQUIRE(aligned16(W) && aligned16(Wq) && aligned16(s_w) && aligned16(P) && aligned16(ws), SQ_ERR_ALIGN,
               "%s: pointers must be 16-byte aligned", name);
    const size_t need = sq_prepare_weights_workspace_bytes(N, K, P != nullptr);
    SQ_REQUIRE(ws_bytes >= need && (need == 0 || ws), SQ_ERR_WORKSPACE, "%s: workspace %zu B < %zu B", name,
               ws_bytes, need);
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (!P) return hip_status(sq::launch_quant_f16(W, nullptr, N, K, 0, 0, Wq, s_w, st, bits), "quant_f16");
    float* wp = static_cast<float*>(ws);
    SQ_TRY(hip_status(sq::launch_transform(W, nullptr, P, N, K, 0, 0, wp, st), "transform"));
    return hip_status(sq::launch_quant_f32(wp, N, K, Wq, s_w, st, bits), "quant_f32");
}

int quantize(const float* Xp, int32_t M, int32_t K, uint8_t* Aq, float* s, void* stream, int bits,
             const char* name) {
    SQ_TRY(check_K(K));
    SQ_REQUIRE(M >= 0, SQ_ERR_SHAPE, "M=%d < 0", M);
    if (M == 0) return SQ_OK;
    SQ_REQUIRE(Xp && Aq && s, SQ_ERR_NULL, "%s: Xp, Aq and s are required", name);
    SQ_REQUIRE(aligned16(Xp) && aligned16(Aq) && aligned16(s), SQ_ERR_ALIGN, "%s: pointers must be 16-byte aligned",
               name);
    return hip_status(sq::launch_quant_f32(Xp, M, K, Aq, s, static_cast<hipStream_t>(stream), bits), "quant_f32");
}

int quant_act(const uint16_t* X, const uint8_t* state, const float* P, int32_t M, int32_t K, int32_t d_m,
              int32_t d_u, const uint16_t* tac_M, const uint16_t* tac_d, int32_t g, uint8_t* Aq, float* s_a,
              void* ws, size_t ws_bytes, void* stream, int bits, const char* name) {
    SQ_TRY(check_K(K));
    SQ_TRY(check_band(K, d_m, d_u));
    SQ_REQUIRE(M >= 0, SQ_ERR_SHAPE, "M=%d < 0", M);
    if (tac_M) {
        SQ_REQUIRE(tac_d, SQ_ERR_NULL, "%s: tac_d is required with tac_M", name);
        SQ_TRY(check_tac(K, g));
        SQ_REQUIRE(M <= kMaxTiledRows, SQ_ERR_SHAPE, "%s: M=%d: at most %d rows per call with TAC", name, M,
                   kMaxTiledRows);
    }
    if (M == 0) return SQ_OK;
    SQ_REQUIRE(X && Aq && s_a, SQ_ERR_NULL, "%s: X, Aq and s_a are required", name);
    SQ_REQUIRE(aligned16(X) && aligned16(Aq) && aligned16(s_a) && aligned16(P) && aligned16(ws) &&
                   aligned16(tac_M) && aligned16(tac_d),
               SQ_ERR_ALIGN, "%s: pointers must be 16-byte aligned", name);
    const size_t need = sq_quant_act_workspace_bytes(M, K, P != nullptr, tac_M != nullptr);
    SQ_REQUIRE(ws_bytes >= need && (need == 0 || ws), SQ_ERR_WORKSPACE, "%s: workspace %zu B < %zu B", name,
               ws_bytes, need);
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (tac_M && !P && sq::tac_quant_fusable(K, g))
        return hip_status(sq::launch_tac_quant(X, tac_M, tac_d, state, M, K, g, d_m, d_u, Aq, s_a, st, bits),
                          "tac_quant");
    uint8_t* wsb = static_cast<uint8_t*>(ws);
    const uint16_t* src = X;
    if (tac_M) {
        uint16_t* z = reinterpret_cast<uint16_t*>(wsb);
        SQ_TRY(hip_status(sq::launch_tac(X, tac_M, tac_d, M, K, g, z, st), "tac"));
        src = z;
        wsb += round_up((size_t)M * K * sizeof(uint16_t));
    }
    if (!P) return hip_status(sq::launch_quant_f16(src, state, M, K, d_m, d_u, Aq, s_a, st, bits), "quant_f16");
    float* xp = reinterpret_cast<float*>(wsb);
    SQ_TRY(hip_status(sq::launch_transform(src, state, P, M, K, d_m, d_u, xp, st), "transform"));
    return hip_status(sq::launch_quant_f32(xp, M, K, Aq, s_a, st, bits), "quant_f32");
}

int gemm(const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w, int32_t M, int32_t N, int32_t K,
         uint16_t* Y, int32_t* acc, void* ws, size_t ws_bytes, void* stream, int bits, const char* name) {
    SQ_TRY(check_K(K));
    SQ_REQUIRE(bits == 4 || K <= 65536, SQ_ERR_SHAPE, "%s: K=%d: 8-bit codes need K <= 65536", name, K);
    SQ_REQUIRE(M >= 0 && N >= 0, SQ_ERR_SHAPE, "M=%d N=%d: need >= 0", M, N);
    SQ_REQUIRE(M <= kMaxTiledRows, SQ_ERR_SHAPE, "%s: M=%d: at most %d rows per call", name, M, kMaxTiledRows);
    SQ_REQUIRE(N % 8 == 0, SQ_ERR_SHAPE, "N=%d: need N %% 8 == 0", N);
    // operand rows are addressed with 32-bit buffer offsets
    const size_t row_bytes = (size_t)K * bits / 8;
    SQ_REQUIRE((size_t)M * row_bytes < (1u << 31) && (size_t)N * row_bytes < (1u << 31), SQ_ERR_SHAPE,
               "%s: each operand must be under 2 GiB (M=%d N=%d K=%d)", name, M, N, K);
    if (M == 0 || N == 0) return SQ_OK;
    SQ_REQUIRE(Aq && s_a && Wq && s_w && (Y || acc), SQ_ERR_NULL,
               "%s: Aq, s_a, Wq, s_w and one of Y / acc are required", name);
    SQ_REQUIRE(aligned16(Aq) && aligned16(s_a) && aligned16(Wq) && aligned16(s_w) && aligned16(Y) &&
                   aligned16(acc) && aligned16(ws),
               SQ_ERR_ALIGN, "%s: pointers must be 16-byte aligned", name);
    const size_t need = bits == 8 ? sq_gemm_w8_workspace_bytes(M, N, K) : sq_gemm_workspace_bytes(M, N, K);
    SQ_REQUIRE(ws_bytes >= need && (need == 0 || ws), SQ_ERR_WORKSPACE, "%s: workspace %zu B < %zu B", name,
               ws_bytes, need);
    return hip_status(
        sq::launch_gemm(Aq, s_a, Wq, s_w, M, N, K, Y, acc, ws, static_cast<hipStream_t>(stream), bits), "gemm");
}

// Shared argument checks of the fragment-ordered GEMM entry points; *done is
// set when there is nothing to compute (M == 0 or N == 0).
int check_gemm_frag(const uint8_t* Aq, const float* s_a, const uint8_t* Wf, const float* s_w, int32_t M, int32_t N,
                    int32_t K, uint16_t* Y, int32_t* acc, int bits, const char* name, int* done) {
    SQ_TRY(check_K(K));
    SQ_REQUIRE(bits == 4 || K <= 65536, SQ_ERR_SHAPE, "%s: K=%d: 8-bit codes need K <= 65536", name, K);
    SQ_REQUIRE(M >= 0 && N >= 0, SQ_ERR_SHAPE, "M=%d N=%d: need >= 0", M, N);
    SQ_REQUIRE(M <= kMaxTiledRows, SQ_ERR_SHAPE, "%s: M=%d: at most %d rows per call", name, M, kMaxTiledRows);
    SQ_REQUIRE(N % 8 == 0, SQ_ERR_SHAPE, "N=%d: need N %% 8 == 0", N);
    // the fragment layout counts a row in int4 codes: an 8-bit row of K bytes is 2 K of them
    SQ_REQUIRE((size_t)M * K * bits / 8 < (1u << 31) && sq::frag_weight_bytes(N, K * bits / 4) < (1u << 31),
               SQ_ERR_SHAPE, "%s: each operand must be under 2 GiB (M=%d N=%d K=%d)", name, M, N, K);
    *done = M == 0 || N == 0;
    if (*done) return SQ_OK;
    SQ_REQUIRE(Aq && s_a && Wf && s_w && (Y || acc), SQ_ERR_NULL,
               "%s: Aq, s_a, Wf, s_w and one of Y / acc are required", name);
    SQ_REQUIRE(aligned16(Aq) && aligned16(s_a) && aligned16(Wf) && aligned16(s_w) && aligned16(Y) && aligned16(acc),
               SQ_ERR_ALIGN, "%s: pointers must be 16-byte aligned", name);
    return SQ_OK;
}

// Scratch of w4a4_gemm_frag_noalloc: a file-scope device array, which every
// GPU the library runs on holds (its own copy) until the process ends.  It
// takes the K-split partial sums, the only scratch the GEMM uses; those are
// written in full before they are read, so nothing has to start at zero.
// Host code never passes the array's name to a kernel: it stands for a host
// symbol there.  The device address comes from hipGetSymbolAddress, once per
// device, on the first call that needs it with that device current.
constexpr size_t kNoallocScratchBytes = SQ_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) uint8_t scratch[kNoallocScratchBytes];
std::atomic<void*> g_scratch_ptr[sq::kMaxDevices];
std::mutex g_scratch_mu;

int scratch_for(void* stream, void** out) {
    int dev = -1;
    SQ_TRY(hip_status(hipGetDevice(&dev), "hipGetDevice"));
    SQ_REQUIRE(dev >= 0 && dev < sq::kMaxDevices, SQ_ERR_HIP, "device %d out of range", dev);
    if (stream) {   // the address belongs to the current device, so the stream must too
        hipDevice_t sdev = -1;
        SQ_TRY(hip_status(hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev), "hipStreamGetDevice"));
        SQ_REQUIRE(sdev == dev, SQ_ERR_SHAPE, "the stream belongs to device %d, not the current device %d",
                   (int)sdev, dev);
    }
    void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
        if (!p) {
            SQ_TRY(hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)"));
            SQ_REQUIRE(p, SQ_ERR_HIP, "hipGetSymbolAddress(scratch) gave a null address");
            g_scratch_ptr[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return SQ_OK;
}

}  // namespace

extern "C" {

int sgat_prepare_weights(const uint16_t* W, const float* P, int32_t N, int32_t K, uint8_t* Wq, float* s_w,
                         void* ws, size_t ws_bytes, void* stream) {
    return prepare_weights(W, P, N, K, Wq, s_w, ws, ws_bytes, stream, 4, "sgat_prepare_weights");
}

int sgat_prepare_weights_w8(const uint16_t* W, const float* P, int32_t N, int32_t K, int8_t* Wq, float* s_w,
                            void* ws, size_t ws_bytes, void* stream) {
    return prepare_weights(W, P, N, K, reinterpret_cast<uint8_t*>(Wq), s_w, ws, ws_bytes, stream, 8,
                           "sgat_prepare_weights_w8");
}

int sgat_transform(const uint16_t* X, const uint8_t* state, const float* P, int32_t M, int32_t K, int32_t d_m,
                   int32_t d_u, float* Xp, void* stream) {
    SQ_TRY(check_K(K));
    SQ_TRY(check_band(K, d_m, d_u));
    SQ_REQUIRE(M >= 0, SQ_ERR_SHAPE, "M=%d < 0", M);
    if (M == 0) return SQ_OK;
    SQ_REQUIRE(X && Xp, SQ_ERR_NULL, "sgat_transform: X and Xp are required");
    SQ_REQUIRE(aligned16(X) && aligned16(Xp) && aligned16(P), SQ_ERR_ALIGN,
               "sgat_transform: X, P and Xp must be 16-byte aligned");
    return hip_status(sq::launch_transform(X, state, P, M, K, d_m, d_u, Xp, static_cast<hipStream_t>(stream)),
                      "transform");
}

int sgat_quantize(const float* Xp, int32_t M, int32_t K, uint8_t* Aq, float* s, void* stream) {
    return quantize(Xp, M, K, Aq, s, stream, 4, "sgat_quantize");
}

int sgat_quantize_w8(const float* Xp, int32_t M, int32_t K, int8_t* Aq, float* s, void* stream) {
    return quantize(Xp, M, K, reinterpret_cast<uint8_t*>(Aq), s, stream, 8, "sgat_quantize_w8");
}

int sgat_quant_act(const uint16_t* X, const uint8_t* state, const float* P, int32_t M, int32_t K, int32_t d_m,
                   int32_t d_u, const uint16_t* tac_M, const uint16_t* tac_d, int32_t g, uint8_t* Aq, float* s_a,
                   void* ws, size_t ws_bytes, void* stream) {
    return quant_act(X, state, P, M, K, d_m, d_u, tac_M, tac_d, g, Aq, s_a, ws, ws_bytes, stream, 4,
                     "sgat_quant_act");
}

int sgat_quant_act_w8(const uint16_t* X, const uint8_t* state, const float* P, int32_t M, int32_t K, int32_t d_m,
                      int32_t d_u, const uint16_t* tac_M, const uint16_t* tac_d, int32_t g, int8_t* Aq,
                      float* s_a, void* ws, size_t ws_bytes, void* stream) {
    return quant_act(X, state, P, M, K, d_m, d_u, tac_M, tac_d, g, reinterpret_cast<uint8_t*>(Aq), s_a, ws,
                     ws_bytes, stream, 8, "sgat_quant_act_w8");
}

int w4a4_gemm(const uint8_t* Aq, const float* s_a, const uint8_t* Wq, const float* s_w, int32_t M, int32_t N,
              int32_t K, uint16_t* Y, int32_t* acc, void* ws, size_t ws_bytes, void* stream) {
    return gemm(Aq, s_a, Wq, s_w, M, N, K, Y, acc, ws, ws_bytes, stream, 4, "w4a4_gemm");
}

int w8a8_gemm(const int8_t* Aq, const float* s_a, const int8_t* Wq, const float* s_w, int32_t M, int32_t N,
              int32_t K, uint16_t* Y, int32_t* acc, void* ws, size_t ws_bytes, void* stream) {
    return gemm(reinterpret_cast<const uint8_t*>(Aq), s_a, reinterpret_cast<const uint8_t*>(Wq), s_w, M, N, K, Y,
                acc, ws, ws_bytes, stream, 8, "w8a8_gemm");
}

int tac_apply(const uint16_t* Z, const uint16_t* tac_M, const uint16_t* tac_d, int32_t M, int32_t C, int32_t g,
              uint16_t* Z_out, void* stream) {
    SQ_TRY(check_K(C));
    SQ_TRY(check_tac(C, g));
    SQ_REQUIRE(M >= 0, SQ_ERR_SHAPE, "M=%d < 0", M);
    SQ_REQUIRE(M <= kMaxTiledRows, SQ_ERR_SHAPE, "tac_apply: M=%d: at most %d rows per call", M, kMaxTiledRows);
    if (M == 0) return SQ_OK;
    SQ_REQUIRE(Z && tac_M && tac_d && Z_out, SQ_ERR_NULL, "tac_apply: Z, tac_M, tac_d and Z_out are required");
    SQ_REQUIRE(aligned16(Z) && aligned16(tac_M) && aligned16(tac_d) && aligned16(Z_out), SQ_ERR_ALIGN,
               "tac_apply: pointers must be 16-byte aligned");
    const uintptr_t a0 = (uintptr_t)Z, a1 = a0 + (size_t)M * C * 2;
    const uintptr_t b0 = (uintptr_t)Z_out, b1 = b0 + (size_t)M * C * 2;
    SQ_REQUIRE(a1 <= b0 || b1 <= a0, SQ_ERR_SHAPE, "tac_apply: Z_out overlaps Z");
    return hip_status(sq::launch_tac(Z, tac_M, tac_d, M, C, g, Z_out, static_cast<hipStream_t>(stream)), "tac");
}

size_t sq_fp6_row_bytes(int32_t K) {
    if (K < 64 || K > 131072 || K % 64) return 0;
    return sq::fp6_row_bytes(K);
}

int sq_codes_to_fp6(const uint8_t* codes, int32_t R, int32_t K, uint8_t* out, void* stream) {
    SQ_TRY(check_K(K));
    SQ_REQUIRE(R >= 0, SQ_ERR_SHAPE, "sq_codes_to_fp6: R=%d < 0", R);
    SQ_REQUIRE((size_t)R * sq::fp6_row_bytes(K) < (1u << 31), SQ_ERR_SHAPE,
               "sq_codes_to_fp6: the FP6 operand must be under 2 GiB (R=%d K=%d)", R, K);
    if (R == 0) return SQ_OK;
    SQ_REQUIRE(codes && out, SQ_ERR_NULL, "sq_codes_to_fp6: codes and out are required");
    SQ_REQUIRE(aligned16(codes) && aligned16(out), SQ_ERR_ALIGN, "sq_codes_to_fp6: pointers must be 16-byte aligned");
    const uintptr_t a0 = (uintptr_t)codes, a1 = a0 + (size_t)R * K / 2;
    const uintptr_t b0 = (uintptr_t)out, b1 = b0 + (size_t)R * sq::fp6_row_bytes(K);
    SQ_REQUIRE(a1 <= b0 || b1 <= a0, SQ_ERR_SHAPE, "sq_codes_to_fp6: out overlaps codes");
    return hip_status(sq::launch_codes_to_fp6(codes, R, K, out, static_cast<hipStream_t>(stream)), "codes_to_fp6");
}

int w4a4_gemm_fp6(const uint8_t* A6, const float* s_a, const uint8_t* W6, const float* s_w, int32_t M, int32_t N,
                  int32_t K, uint16_t* Y, int32_t* acc, void* stream) {
    SQ_TRY(check_K(K));
    SQ_REQUIRE(M >= 0 && N >= 0, SQ_ERR_SHAPE, "M=%d N=%d: need >= 0", M, N);
    SQ_REQUIRE(N % 8 == 0, SQ_ERR_SHAPE, "N=%d: need N %% 8 == 0", N);
    const size_t rb = sq::fp6_row_bytes(K);
    SQ_REQUIRE((size_t)M * rb < (1u << 31) && (size_t)N * rb < (1u << 31), SQ_ERR_SHAPE,
               "w4a4_gemm_fp6: each operand must be under 2 GiB (M=%d N=%d K=%d)", M, N, K);
    if (M == 0 || N == 0) return SQ_OK;
    SQ_REQUIRE(A6 && s_a && W6 && s_w && (Y || acc), SQ_ERR_NULL,
               "w4a4_gemm_fp6: A6, s_a, W6, s_w and one of Y / acc are required");
    SQ_REQUIRE(aligned16(A6) && aligned16(s_a) && aligned16(W6) && aligned16(s_w) && aligned16(Y) &&
                   aligned16(acc),
               SQ_ERR_ALIGN, "w4a4_gemm_fp6: pointers must be 16-byte aligned");
    return hip_status(sq::launch_gemm_fp6(A6, s_a, W6, s_w, M, N, K, Y, acc, static_cast<hipStream_t>(stream)),
                      "gemm_fp6");
}

size_t sq_frag_weight_bytes(int32_t N, int32_t K) {
    if (N < 0 || K < 64 || K > 131072 || K % 64) return 0;
    return sq::frag_weight_bytes(N, K);
}

int sq_weights_to_frag(const uint8_t* Wq, int32_t N, int32_t K, uint8_t* Wf, void* stream) {
    SQ_TRY(check_K(K));
    SQ_REQUIRE(N >= 0, SQ_ERR_SHAPE, "sq_weights_to_frag: N=%d < 0", N);
    SQ_REQUIRE(sq::frag_weight_bytes(N, K) < (1u << 31), SQ_ERR_SHAPE,
               "sq_weights_to_frag: the fragment-ordered weights must be under 2 GiB (N=%d K=%d)", N, K);
    if (N == 0) return SQ_OK;
    SQ_REQUIRE(Wq && Wf, SQ_ERR_NULL, "sq_weights_to_frag: Wq and Wf are required");
    SQ_REQUIRE(aligned16(Wq) && aligned16(Wf), SQ_ERR_ALIGN, "sq_weights_to_frag: pointers must be 16-byte aligned");
    const uintptr_t a0 = (uintptr_t)Wq, a1 = a0 + (size_t)N * K / 2;
    const uintptr_t b0 = (uintptr_t)Wf, b1 = b0 + sq::frag_weight_bytes(N, K);
    SQ_REQUIRE(a1 <= b0 || b1 <= a0, SQ_ERR_SHAPE, "sq_weights_to_frag: Wf overlaps Wq");
    return hip_status(sq::launch_weights_to_frag(Wq, N, K, Wf, static_cast<hipStream_t>(stream)), "weights_to_frag");
}

int w4a4_gemm_frag(const uint8_t* Aq, const float* s_a, const uint8_t* Wf, const float* s_w, int32_t M, int32_t N,
                   int32_t K, uint16_t* Y, int32_t* acc, void* ws, size_t ws_bytes, void* stream) {
    int done = 0;
    SQ_TRY(check_gemm_frag(Aq, s_a, Wf, s_w, M, N, K, Y, acc, 4, "w4a4_gemm_frag", &done));
    if (done) return SQ_OK;
    SQ_REQUIRE(aligned16(ws), SQ_ERR_ALIGN, "w4a4_gemm_frag: pointers must be 16-byte aligned");
    const size_t need = sq_gemm_workspace_bytes(M, N, K);
    SQ_REQUIRE(ws_bytes >= need && (need == 0 || ws), SQ_ERR_WORKSPACE, "w4a4_gemm_frag: workspace %zu B < %zu B",
               ws_bytes, need);
    return hip_status(
        sq::launch_gemm_frag(Aq, s_a, Wf, s_w, M, N, K, Y, acc, ws, static_cast<hipStream_t>(stream), 4),
        "gemm_frag");
}

size_t sq_frag_weight_w8_bytes(int32_t N, int32_t K) {
    if (K < 64 || K > 65536 || K % 64) return 0;
    return sq_frag_weight_bytes(N, 2 * K);
}

int sq_weights_to_frag_w8(const int8_t* Wq, int32_t N, int32_t K, uint8_t* Wf, void* stream) {
    SQ_REQUIRE(K <= 65536, SQ_ERR_SHAPE, "sq_weights_to_frag_w8: K=%d: 8-bit codes need K <= 65536", K);
    SQ_TRY(check_K(K));
    // a row of K int8 codes is reordered as a row of 2 K int4 codes: the same K bytes
    return sq_weights_to_frag(reinterpret_cast<const uint8_t*>(Wq), N, 2 * K, Wf, stream);
}

int w8a8_gemm_frag(const int8_t* Aq, const float* s_a, const uint8_t* Wf, const float* s_w, int32_t M, int32_t N,
                   int32_t K, uint16_t* Y, int32_t* acc, void* ws, size_t ws_bytes, void* stream) {
    int done = 0;
    const uint8_t* A8 = reinterpret_cast<const uint8_t*>(Aq);
    SQ_TRY(check_gemm_frag(A8, s_a, Wf, s_w, M, N, K, Y, acc, 8, "w8a8_gemm_frag", &done));
    if (done) return SQ_OK;
    SQ_REQUIRE(aligned16(ws), SQ_ERR_ALIGN, "w8a8_gemm_frag: pointers must be 16-byte aligned");
    const size_t need = sq_gemm_w8_workspace_bytes(M, N, K);
    SQ_REQUIRE(ws_bytes >= need && (need == 0 || ws), SQ_ERR_WORKSPACE, "w8a8_gemm_frag: workspace %zu B < %zu B",
               ws_bytes, need);
    return hip_status(
        sq::launch_gemm_frag(A8, s_a, Wf, s_w, M, N, K, Y, acc, ws, static_cast<hipStream_t>(stream), 8),
        "gemm_frag_w8");
}

int w4a4_gemm_frag_noalloc(const uint8_t* Aq, const float* s_a, const uint8_t* Wf, const float* s_w, int32_t M,
                           int32_t N, int32_t K, uint16_t* Y, int32_t* acc, void* stream) {
    int done = 0;
    SQ_TRY(check_gemm_frag(Aq, s_a, Wf, s_w, M, N, K, Y, acc, 4, "w4a4_gemm_frag_noalloc", &done));
    if (done) return SQ_OK;
    const size_t need = sq_gemm_workspace_bytes(M, N, K);
    SQ_REQUIRE(need <= kNoallocScratchBytes, SQ_ERR_WORKSPACE,
               "w4a4_gemm_frag_noalloc: this shape needs %zu B of scratch, above the %zu B the library holds "
               "(M=%d N=%d K=%d)", need, kNoallocScratchBytes, M, N, K);
    void* ws = nullptr;
    if (need > 0) SQ_TRY(scratch_for(stream, &ws));
    return hip_status(
        sq::launch_gemm_frag(Aq, s_a, Wf, s_w, M, N, K, Y, acc, ws, static_cast<hipStream_t>(stream), 4),
        "gemm_frag_noalloc");
}

size_t sq_tac_calibrate_workspace_bytes(int32_t N, int32_t C, int32_t g) {
    if (N <= 0 || C < 64 || C % 64 || g < 1 || g > 128 || (g & (g - 1)) || C % g) return 0;
    return sq::tac_calib_workspace_bytes(N, C, g);
}

int tac_calibrate(const uint16_t* Z_fp, const uint16_t* Z_q, int32_t N, int32_t C, int32_t g, double rho,
                  double eps, double eta, double alpha, uint16_t* tac_M, uint16_t* tac_d, double* M64,
                  double* d64, void* ws, size_t ws_bytes, void* stream) {
    SQ_TRY(check_K(C));
    SQ_TRY(check_tac(C, g));
    SQ_REQUIRE(N >= 1, SQ_ERR_SHAPE, "tac_calibrate: N=%d: need at least one token", N);
    SQ_REQUIRE(rho >= 0.0 && eps >= 0.0 && eta >= 0.0 && eta <= 1.0 && alpha >= 0.0 && alpha <= 1.0 &&
                   rho < 1e300 && eps < 1e300,
               SQ_ERR_SHAPE, "tac_calibrate: need rho, eps >= 0 (finite) and eta, alpha in [0, 1]");
    SQ_REQUIRE(Z_fp && Z_q && tac_M && tac_d && ws, SQ_ERR_NULL,
               "tac_calibrate: Z_fp, Z_q, tac_M, tac_d and ws are required");
    SQ_REQUIRE(aligned16(Z_fp) && aligned16(Z_q) && aligned16(tac_M) && aligned16(tac_d) && aligned16(M64) &&
                   aligned16(d64) && aligned16(ws),
               SQ_ERR_ALIGN, "tac_calibrate: pointers must be 16-byte aligned");
    const size_t need = sq::tac_calib_workspace_bytes(N, C, g);
    SQ_REQUIRE(ws_bytes >= need, SQ_ERR_WORKSPACE, "tac_calibrate: workspace %zu B < %zu B", ws_bytes, need);
    return hip_status(sq::launch_tac_calib(Z_fp, Z_q, N, C, g, rho, eps, eta, alpha, tac_M, tac_d, M64, d64, ws,
                                           static_cast<hipStream_t>(stream)),
                      "tac_calibrate");
}

int sgat_split_basis(const float* P, int32_t K, uint16_t* Ps, void* stream) {
    SQ_TRY(check_K(K));
    SQ_REQUIRE((size_t)K * K * 4 < (1u << 31), SQ_ERR_SHAPE,
               "sgat_split_basis: K=%d: the split basis (4 K^2 bytes) must be under 2 GiB", K);
    SQ_REQUIRE(P && Ps, SQ_ERR_NULL, "sgat_split_basis: P and Ps are required");
    SQ_REQUIRE(aligned16(P) && aligned16(Ps), SQ_ERR_ALIGN, "sgat_split_basis: pointers must be 16-byte aligned");
    return hip_status(sq::launch_split_basis(P, K, Ps, static_cast<hipStream_t>(stream)), "split_basis");
}

int sgat_transform_fast(const uint16_t* X, const uint8_t* state, const uint16_t* Ps, int32_t M, int32_t K,
                        int32_t d_m, int32_t d_u, float* Xp, void* stream) {
    SQ_TRY(check_K(K));
    SQ_TRY(check_band(K, d_m, d_u));
    SQ_REQUIRE(M >= 0, SQ_ERR_SHAPE, "M=%d < 0", M);
    SQ_REQUIRE((size_t)K * K * 4 < (1u << 31), SQ_ERR_SHAPE,
               "sgat_transform_fast: K=%d: the split basis (4 K^2 bytes) must be under 2 GiB", K);
    SQ_REQUIRE((size_t)M * K * 2 < (1u << 31), SQ_ERR_SHAPE,
               "sgat_transform_fast: X must be under 2 GiB (M=%d K=%d)", M, K);
    if (M == 0) return SQ_OK;
    SQ_REQUIRE(X && Ps && Xp, SQ_ERR_NULL, "sgat_transform_fast: X, Ps and Xp are required");
    SQ_REQUIRE(aligned16(X) && aligned16(Ps) && aligned16(Xp), SQ_ERR_ALIGN,
               "sgat_transform_fast: X, Ps and Xp must be 16-byte aligned");
    return hip_status(sq::launch_transform_fast(X, state, Ps, M, K, d_m, d_u, Xp, static_cast<hipStream_t>(stream)),
                      "transform_fast");
}

}  // extern "C"
