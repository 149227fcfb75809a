// Buffer descriptors and LDS-DMA loads shared by the linear-layer kernels.
//
// An LDS-DMA load moves global memory straight into LDS without a vector
// register destination, so the compiler tracks no dependence for it: every
// kernel that issues these loads waits for them itself with an explicit
// s_waitcnt vmcnt(n), counting on vector-memory loads completing in the
// order they were issued.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rrq_detail {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kRsrcWord3 = 0x00020000u;
// Offset added to a load that must not touch memory: past every buffer
// these kernels address (all below 2^31 bytes), so it reads zeros.
constexpr uint32_t kSkip = 0x80000000u;

// Raw buffer descriptor (gfx9 family): accesses at or beyond bytes read zero.
__device__ __forceinline__ u32x4 make_desc(const void *base, uint32_t bytes)
{
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    u32x4 d;
    d[0] = (uint32_t)a;
    d[1] = (uint32_t)(a >> 32) & 0xFFFFu;
    d[2] = bytes;
    d[3] = kRsrcWord3;
    return d;
}

// LDS-DMA loads: every lane reads from the buffer at byte offset
// soff + voff (both range-checked against the descriptor's size) and the
// wave writes LDS at lds + lane * 16 (dwordx4) or lds + lane * 4 (dword,
// ushort). lds is a wave-uniform LDS byte address. m0, which carries it, is
// restored. The wait states the compiler cannot see inside the block are
// explicit: 5 before the load reads SGPRs that a VALU instruction may have
// just written, 1 after writing m0.
__device__ __forceinline__ void dma_x4(const u32x4 &desc, uint32_t soff, uint32_t lds,
                                       uint32_t voff)
{
    uint32_t m0;
    asm volatile("s_nop 4\n\t"
                 "s_mov_b32 %0, m0\n\t"
                 "s_mov_b32 m0, %2\n\t"
                 "s_nop 0\n\t"
                 "buffer_load_dwordx4 %1, %3, %4 offen lds\n\t"
                 "s_mov_b32 m0, %0"
                 : "=&s"(m0) : "v"(voff), "s"(lds), "s"(desc), "s"(soff) : "memory");
}

__device__ __forceinline__ void dma_dword(const u32x4 &desc, uint32_t soff, uint32_t lds,
                                          uint32_t voff)
{
    uint32_t m0;
    asm volatile("s_nop 4\n\t"
                 "s_mov_b32 %0, m0\n\t"
                 "s_mov_b32 m0, %2\n\t"
                 "s_nop 0\n\t"
                 "buffer_load_dword %1, %3, %4 offen lds\n\t"
                 "s_mov_b32 m0, %0"
                 : "=&s"(m0) : "v"(voff), "s"(lds), "s"(desc), "s"(soff) : "memory");
}

__device__ __forceinline__ void dma_ushort(const u32x4 &desc, uint32_t soff, uint32_t lds,
                                           uint32_t voff)
{
    uint32_t m0;
    asm volatile("s_nop 4\n\t"
                 "s_mov_b32 %0, m0\n\t"
                 "s_mov_b32 m0, %2\n\t"
                 "s_nop 0\n\t"
                 "buffer_load_ushort %1, %3, %4 offen lds\n\t"
                 "s_mov_b32 m0, %0"
                 : "=&s"(m0) : "v"(voff), "s"(lds), "s"(desc), "s"(soff) : "memory");
}

// Wait until at most N of the wave's vector-memory instructions are in
// flight.
template <int N>
__device__ __forceinline__ void wait_vm()
{
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}

// LDS byte address of a shared-memory object (for the DMA loads' m0).
template <typename T>
__device__ __forceinline__ uint32_t lds_address(T *p)
{
    return (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) T *)p);
}

}  // namespace
}  // namespace rrq_detail
