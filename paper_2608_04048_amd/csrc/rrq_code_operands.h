// Matrix-core B operands from packed 2-bit codes, shared by the linear-layer
// kernels.
//
// A code word holds 16 codes, code e at bits 2e, 2e + 1. The bfloat16
// 4 + Q has the bit pattern 0x4080 | Q << 5 (the code in the top two
// mantissa bits of 4), so one shift, one AND with 0x00600060 and one OR with
// 0x40804080 turn a word into a register holding two such values: register
// q of a word gets codes q and q + 8 (one per 16-bit half) from the word
// shifted so that code q lands on bits 5, 6.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rrq_detail {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// B operands of the four MFMA blocks of a lane's two code words w0, w1:
// b[v][h] is word v, block h; register r of block h holds codes 4 h + r and
// 4 h + r + 8 of the word. mask and four hold 0x00600060 and 0x40804080 in
// registers. The two words are shifted together by 64-bit shifts (a shift
// carries at most 9 bits from one word into the other, which land outside
// the mask); they are written as inline assembly because the compiler
// splits a 64-bit shift into two funnel shifts, twice the instructions.
__device__ __forceinline__ void code_operands_pair(uint32_t w0, uint32_t w1, uint32_t mask,
                                                   uint32_t four, u32x4 (&b)[2][2])
{
    const uint64_t w = ((uint64_t)w1 << 32) | w0;
    uint64_t s[8];
    asm("v_lshlrev_b64 %0, 5, %1" : "=v"(s[0]) : "v"(w));
    asm("v_lshlrev_b64 %0, 3, %1" : "=v"(s[1]) : "v"(w));
    asm("v_lshlrev_b64 %0, 1, %1" : "=v"(s[2]) : "v"(w));
    asm("v_lshrrev_b64 %0, 1, %1" : "=v"(s[3]) : "v"(w));
    asm("v_lshrrev_b64 %0, 3, %1" : "=v"(s[4]) : "v"(w));
    asm("v_lshrrev_b64 %0, 5, %1" : "=v"(s[5]) : "v"(w));
    asm("v_lshrrev_b64 %0, 7, %1" : "=v"(s[6]) : "v"(w));
    asm("v_lshrrev_b64 %0, 9, %1" : "=v"(s[7]) : "v"(w));
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        b[0][q >> 2][q & 3] = ((uint32_t)s[q] & mask) | four;
        b[1][q >> 2][q & 3] = ((uint32_t)(s[q] >> 32) & mask) | four;
    }
}

}  // namespace
}  // namespace rrq_detail
