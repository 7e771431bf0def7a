// Building blocks shared by the MFMA tile kernels (the W4A4 / W8A8 GEMM and the
// MFMA transform) and the quantisers: buffer descriptors whose range check turns
// out-of-range reads into zeros, direct global-to-LDS loads, and the counter
// wait the three-stage pipelines use.
#pragma once
#include "sq_internal.hpp"

namespace sq {
namespace {

// Raw buffer resource over [base, base + bytes): loads outside it return 0, which
// is how rows past M (or N) and the unused half of a last k step read as zeros.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

constexpr uint32_t kOOB = 0x80000000u;   // an offset past any buffer this kernel builds
constexpr int kKStep = 64;               // bytes per operand row per pipeline step

// Direct loads into LDS: lane i of a buffer_load ... lds lands at LDS base +
// 16 i, so each lane fetches the 16-byte segment that belongs at its swizzled
// slot.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Buffer descriptor in scalar registers: base, stride 0, size in bytes, raw
// (untyped) buffer; offsets at or past `bytes` read as zero.
__device__ __forceinline__ u32x4 sgpr_rsrc(const void* base, uint32_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    return u32x4{(uint32_t)a, (uint32_t)(a >> 32) & 0xFFFFu, bytes, 0x00020000u};
}

// 16 bytes per lane from buffer offset `voff` straight into LDS: lane i's bytes
// land at LDS address `lds` + 16 i.  Issued as inline assembly so that the
// compiler's automatic counter waits (which cannot tell the pipeline stages
// apart and would wait for every load in flight) stay out of the loop; the
// kernel waits for these loads itself with wait_vm.
__device__ __forceinline__ void dma16(const u32x4& rsrc, uint32_t lds, uint32_t voff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(rsrc)
                 : "memory", "m0");
}

// The same with a wave-uniform offset `soff` in the scalar-offset field, added
// to voff, so a k-step offset costs no vector instruction.  Callers keep every
// in-range lane's voff + soff inside the buffer and put the out-of-range lanes'
// voff itself past it, so the result does not depend on whether the range
// check counts soff.
__device__ __forceinline__ void dma16s(const u32x4& rsrc, uint32_t lds, uint32_t voff, uint32_t soff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(rsrc),
                   "s"(__builtin_amdgcn_readfirstlane(soff))
                 : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

// vmcnt <= N and lgkmcnt == 0: this wave's loads older than its last N have
// landed in LDS, and its own LDS reads are complete
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}

}  // namespace
}  // namespace sq
