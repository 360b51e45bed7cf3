// Device helpers shared by the gfx950 kernels of the binary-delta matmul.
//
// MFMA operand conventions used throughout (CDNA3/CDNA4 matrix cores, wave64):
//   v_mfma_f32_16x16x32_bf16  D[16x16] += A[16x32] * B[32x16]
//     lane l holds A row (l % 16) and B column (l % 16), eight consecutive
//     contraction slots 8*(l / 16) .. +7 of each; D element (4*(l/16) + r, l % 16)
//     sits in accumulator register r (r = 0..3).
//   v_mfma_f32_32x32x16_bf16  D[32x32] += A[32x16] * B[16x32]
//     lane l holds A row (l % 32) and B column (l % 32), slots 8*(l / 32) .. +7;
//     D element (8*(r/4) + 4*(l/32) + (r%4), l % 32) sits in register r (0..15).
// Both operands of one instruction use the same lane -> slot assignment, so a
// contraction is correct whatever physical k a slot stands for, as long as A
// and B agree on it.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bitdelta {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

// bf16 pair (-1, -1): 0xBF80 in each half.  Clearing a half's sign bit (bit 15
// or bit 31) turns that half into +1 (0x3F80).
constexpr uint32_t kMinusOnePair = 0xBF80BF80u;
constexpr uint32_t kSignBits = 0x80008000u;

__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Eight sign bits (bit i <-> slot i, bit 1 = +1) -> eight bf16 +1/-1 in slot order.
// The byte is first duplicated 15 bits higher, so one left shift brings bit 2j
// to position 15 and bit 2j+1 to position 31 at once; one 3-input bit op then
// flips the sign bits of the packed (-1, -1) constant: two values per two ops.
__device__ __forceinline__ u32x4 decode_signs8(uint32_t byte) {
    const uint32_t s = byte | (byte << 15);
    u32x4 r;
    r[0] = kMinusOnePair ^ ((s << 15) & kSignBits);
    r[1] = kMinusOnePair ^ ((s << 13) & kSignBits);
    r[2] = kMinusOnePair ^ ((s << 11) & kSignBits);
    r[3] = kMinusOnePair ^ ((s << 9) & kSignBits);
    return r;
}

// Eight bf16 weights (slot order, two per dword) and their eight sign bits ->
// bf16(w + (bit ? alpha : -alpha)), computed in fp32 and rounded to nearest even.
// neg_alpha_bits holds the fp32 bit pattern of -alpha: a set bit moved to
// position 31 flips it to +alpha.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi);

__device__ __forceinline__ u32x4 fuse_weights8(u32x4 w, uint32_t byte, uint32_t neg_alpha_bits) {
    u32x4 r;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const float lo = __builtin_bit_cast(float, w[j] << 16);
        const float hi = __builtin_bit_cast(float, w[j] & 0xFFFF0000u);
        const float a_lo = __builtin_bit_cast(float, neg_alpha_bits ^ ((byte << (31 - 2 * j)) & 0x80000000u));
        const float a_hi = __builtin_bit_cast(float, neg_alpha_bits ^ ((byte << (30 - 2 * j)) & 0x80000000u));
        r[j] = pack_bf16x2(lo + a_lo, hi + a_hi);
    }
    return r;
}

// fp32 -> bf16 round-to-nearest-even (quiet NaN stays NaN).
__device__ __forceinline__ uint16_t to_bf16(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return (uint32_t)to_bf16(lo) | ((uint32_t)to_bf16(hi) << 16);
}

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
    return *reinterpret_cast<const u32x4*>(p);
}

}  // namespace bitdelta
