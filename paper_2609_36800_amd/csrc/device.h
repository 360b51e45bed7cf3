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

#include <utility>

#include "internal.h"

namespace bitdelta {

// Calls f(integral_constant<int, i>) for i = 0 .. N-1 (indices usable as
// compile-time register-array subscripts).
template <typename Fn, int... Is>
__device__ __forceinline__ void static_for_impl(Fn&& f, std::integer_sequence<int, Is...>) {
    (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename Fn>
__device__ __forceinline__ void static_for(Fn&& f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Kernels templated on ET (the 16-bit element type of x and W: kBF16 or
// kF16) use the matching matrix instruction, +-1 constant and rounding.
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

// Pair (-1, -1) of the element type: 0xBF80 (bf16) or 0xBC00 (fp16) in each
// half.  Clearing a half's sign bit (bit 15 or bit 31) turns it into +1.
template <int ET>
constexpr uint32_t kMinusOnePair = ET == kF16 ? 0xBC00BC00u : 0xBF80BF80u;
constexpr uint32_t kSignBits = 0x80008000u;

template <int ET>
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
    if constexpr (ET == kF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

template <int ET>
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
    if constexpr (ET == kF16)
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Eight sign bits (bit i <-> slot i, bit 1 = +1) -> eight +1/-1 in slot order.
// The byte is first duplicated 15 bits higher, so one left shift brings bit 2j
// to position 15 and bit 2j+1 to position 31 at once; one 3-input bit op then
// flips the sign bits of the packed (-1, -1) constant: two values per two ops.
// Hides a value from the optimiser so that the shift-and-mask sequences built
// on it are emitted as written (left alone, it folds byte | byte << 15 and the
// following shifts into quarter-rate integer multiplies).
__device__ __forceinline__ uint32_t opaque_u32(uint32_t v) {
    asm("" : "+v"(v));
    return v;
}

template <int ET>
__device__ __forceinline__ u32x4 decode_signs8(uint32_t byte) {
    const uint32_t s = opaque_u32(byte | (byte << 15));
    u32x4 r;
    r[0] = kMinusOnePair<ET> ^ ((s << 15) & kSignBits);
    r[1] = kMinusOnePair<ET> ^ ((s << 13) & kSignBits);
    r[2] = kMinusOnePair<ET> ^ ((s << 11) & kSignBits);
    r[3] = kMinusOnePair<ET> ^ ((s << 9) & kSignBits);
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

// fp16 flavour: the pair (-a, -a) holds fp16(-alpha) twice; a set bit flips a
// half's sign to +a, and one packed fp16 add (nearest even) gives
// fp16(w + (bit ? a : -a)) for two weights at once.
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t add_f16x2(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, a) + __builtin_bit_cast(f16x2, b));
}

__device__ __forceinline__ u32x4 fuse_weights8_f16(u32x4 w, uint32_t byte, uint32_t neg_alpha_pair) {
    const uint32_t s = opaque_u32(byte | (byte << 15));
    u32x4 r;
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = add_f16x2(w[j], neg_alpha_pair ^ ((s << (15 - 2 * j)) & kSignBits));
    return r;
}

// fp32 -> bf16 round-to-nearest-even (quiet NaN stays NaN).
__device__ __forceinline__ uint16_t to_bf16(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// fp32 -> fp16 round-to-nearest-even (overflow to inf, NaN stays NaN).
__device__ __forceinline__ uint16_t to_f16(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f));
}

template <int ET>
__device__ __forceinline__ uint16_t to_half(float f) {
    if constexpr (ET == kF16) return to_f16(f);
    else return to_bf16(f);
}

// Output element m*N+n of a y of dtype y_dtype (kF32, or the 16-bit ET).
template <int ET>
__device__ __forceinline__ void store_y(void* y, size_t i, float v, int y_dtype) {
    if (y_dtype == kF32) reinterpret_cast<float*>(y)[i] = v;
    else reinterpret_cast<uint16_t*>(y)[i] = to_half<ET>(v);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return (uint32_t)to_bf16(lo) | ((uint32_t)to_bf16(hi) << 16);
}

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
    return *reinterpret_cast<const u32x4*>(p);
}

}  // namespace bitdelta
