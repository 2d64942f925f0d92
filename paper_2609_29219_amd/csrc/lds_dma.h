// Global-to-LDS tile loads for gfx950 that the compiler does not track.
//
// A buffer load with the LDS bit (buffer_load_dwordx4 ... lds) copies 16
// bytes per lane from a buffer straight into LDS: lane i writes the 16 bytes
// at M0 + 16*i.  Issued through the compiler builtin, such a load makes the
// compiler's wait-count pass hold back later LDS reads until every
// outstanding LDS load has completed, because it cannot tell which LDS bytes
// the load writes; a tile that is being read would then wait for the next
// tile's loads, which serialises the load/compute pipeline.  Issued from
// inline assembly the loads are invisible to that pass, so the kernel states
// the waits itself: before the barrier that publishes a tile, every wave
// waits (vmcnt) until its own loads of that tile have landed, and the
// barrier then makes all waves' loads of it visible.
//
// Also the compile-time loop with which the kernels unroll their
// hand-scheduled MFMA slots.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace attn {

typedef uint32_t dma_rsrc_t __attribute__((ext_vector_type(4)));

// Raw buffer resource over [base, base + bytes): no stride, no swizzle,
// reads at or past `bytes` return 0.  Built from wave-uniform values.
__device__ __forceinline__ dma_rsrc_t make_dma_rsrc(const void* base, uint32_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    dma_rsrc_t r;
    r[0] = __builtin_amdgcn_readfirstlane((uint32_t)a);
    r[1] = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32) & 0xffffu);
    r[2] = __builtin_amdgcn_readfirstlane(bytes);
    r[3] = 0x00020000u;  // raw 32-bit buffer, gfx9 family
    return r;
}

// LDS byte address of a pointer into __shared__ memory (wave-uniform).
__device__ __forceinline__ uint32_t lds_address(const void* p) {
    return __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p);
}

// One wave instruction: lane i loads 16 bytes at byte offset soffset +
// voffset of the buffer into LDS at lds_base + 16*i.  (M0 takes the LDS
// base; one wait state separates the M0 write from the load.)
// M0 is a reserved register: the clobber tells the compiler it changes, which
// it otherwise only warns about (these kernels make no other use of M0).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_dma16(dma_rsrc_t rsrc, uint32_t lds_base, int voffset,
                                          int soffset) {
    // the scalar operands are wave-uniform; readfirstlane puts them in SGPRs
    // even where the compiler holds a uniform value in a VGPR
    rsrc[0] = __builtin_amdgcn_readfirstlane(rsrc[0]);
    rsrc[1] = __builtin_amdgcn_readfirstlane(rsrc[1]);
    rsrc[2] = __builtin_amdgcn_readfirstlane(rsrc[2]);
    rsrc[3] = __builtin_amdgcn_readfirstlane(rsrc[3]);
    lds_base = __builtin_amdgcn_readfirstlane(lds_base);
    soffset = __builtin_amdgcn_readfirstlane(soffset);
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, %3 offen lds"
        :
        : "s"(lds_base), "v"(voffset), "s"(rsrc), "s"(soffset)
        : "memory", "m0");
}
#pragma clang diagnostic pop

// Wait until at most N of this wave's vector-memory loads are outstanding
// and all its LDS operations have completed, then barrier: after it, every
// wave's loads older than its newest N are visible to the whole workgroup.
template <int N>
__device__ __forceinline__ void publish_barrier() {
    static_assert(N >= 0 && N < 64, "vmcnt holds 6 bits");
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" : : "n"(N) : "memory");
}

// Compile-time loop: f(std::integral_constant<int, I>{}) for I in [B, E).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

}  // namespace attn
