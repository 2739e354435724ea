// Global -> LDS tile DMA for gfx950, issued as inline assembly.
//
// buffer_load_dwordx4 ... lds moves 16 bytes per lane from a buffer straight
// into LDS (lane l's bytes land at the wave-uniform LDS address in M0 plus
// 16 l).  Issued through the compiler's builtin, such a load is tracked by the
// compiler's wait-count pass, which then drains every load in flight before
// each workgroup barrier and cannot keep tiles in flight across barriers.
// Issued here as inline assembly it is not tracked: the kernel waits for its
// tiles itself with wait_vmcnt, and its only other vector-memory operations
// must be ones the compiler waits for conservatively (loads issued after the
// tile DMAs, stores after the last wait).
#ifndef TILEATTN_LDS_DMA_H
#define TILEATTN_LDS_DMA_H

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tileattn_dma {

typedef uint32_t u32x4s __attribute__((ext_vector_type(4)));

// word 3 of a raw (unswizzled, stride 0) buffer resource on CDNA: 32-bit data
// format; loads past num_records return zero
constexpr uint32_t RSRC_WORD3 = 0x00020000;

// A raw buffer resource over `bytes` bytes from `base`, in scalar registers.
__device__ __forceinline__ u32x4s buffer_rsrc(const void *base, uint32_t bytes)
{
    const uint64_t a = (uint64_t)(uintptr_t)base;
    return u32x4s{(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a),
                  (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32) & 0xFFFFu),
                  (uint32_t)__builtin_amdgcn_readfirstlane(bytes), RSRC_WORD3};
}

// Lane l's 16 bytes at byte `voff` of the buffer land at LDS address
// `lds` + 16 l (`lds` wave-uniform).  M0 is an operand of the statement, so
// the compiler sets it (and keeps any value of its own) around the load.
// NT: the load carries the non-temporal cache policy, for data that no other
// workgroup reads again.
template <bool NT = false>
__device__ __forceinline__ void dma16(uint32_t lds, uint32_t voff, u32x4s rsrc)
{
    if constexpr (NT)
        asm volatile("s_nop 0\n\t"   // one wait state between the M0 write and the load
                     "buffer_load_dwordx4 %0, %1, 0 offen nt lds"
                     :
                     : "v"(voff), "s"(rsrc), "{m0}"(__builtin_amdgcn_readfirstlane(lds))
                     : "memory");
    else
        asm volatile("s_nop 0\n\t"
                     "buffer_load_dwordx4 %0, %1, 0 offen lds"
                     :
                     : "v"(voff), "s"(rsrc), "{m0}"(__builtin_amdgcn_readfirstlane(lds))
                     : "memory");
}

// The same with a wave-uniform byte offset `soff` (a scalar register) added to
// the lane's `voff`.
template <bool NT = false>
__device__ __forceinline__ void dma16_soff(uint32_t lds, uint32_t voff, uint32_t soff,
                                           u32x4s rsrc)
{
    if constexpr (NT)
        asm volatile("s_nop 0\n\t"
                     "buffer_load_dwordx4 %0, %1, %2 offen nt lds"
                     :
                     : "v"(voff), "s"(rsrc), "s"(soff),
                       "{m0}"(__builtin_amdgcn_readfirstlane(lds))
                     : "memory");
    else
        asm volatile("s_nop 0\n\t"
                     "buffer_load_dwordx4 %0, %1, %2 offen lds"
                     :
                     : "v"(voff), "s"(rsrc), "s"(soff),
                       "{m0}"(__builtin_amdgcn_readfirstlane(lds))
                     : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void *p)
{
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}

// s_waitcnt vmcnt(N), expcnt and lgkmcnt left at their maxima (N < 64)
template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

}  // namespace tileattn_dma

#endif  // TILEATTN_LDS_DMA_H
