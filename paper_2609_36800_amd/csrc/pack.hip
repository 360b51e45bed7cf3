// Pack and unpack kernels for the one-bit sign storage of the binary delta.
//
// Format: bit i of word j of a row <-> element k = 32*j + i, bit 1 = +1 and
// bit 0 = -1 (the 2b-1 decode of the BitDelta kernel, Appendix A.2).  With
// K a multiple of 32 every word belongs to one row, so both kernels run over
// the flat element range.
//
// Mapping: a thread owns four consecutive elements (one 16/8/4-byte load or
// store), eight neighbouring lanes own one 32-bit word.  Pack ORs the eight
// nibbles with three xor-shuffles; loads and stores are fully coalesced.
#include "device.h"
#include "internal.h"

namespace bitdelta {
namespace {

constexpr int kThreads = 256;

template <int DT>
__device__ __forceinline__ uint32_t sign_nibble(const void* src, int64_t quad) {
    if constexpr (DT == kF32) {
        const u32x4 v = reinterpret_cast<const u32x4*>(src)[quad];
        return ((~v[0] >> 31) & 1u) | (((~v[1] >> 31) & 1u) << 1) |
               (((~v[2] >> 31) & 1u) << 2) | (((~v[3] >> 31) & 1u) << 3);
    } else if constexpr (DT == kBF16) {
        const uint2 v = reinterpret_cast<const uint2*>(src)[quad];
        return ((~v.x >> 15) & 1u) | (((~v.x >> 31) & 1u) << 1) |
               (((~v.y >> 15) & 1u) << 2) | (((~v.y >> 31) & 1u) << 3);
    } else {
        const uint32_t v = reinterpret_cast<const uint32_t*>(src)[quad];
        return ((~v >> 7) & 1u) | (((~v >> 15) & 1u) << 1) |
               (((~v >> 23) & 1u) << 2) | (((~v >> 31) & 1u) << 3);
    }
}

template <int DT>
__global__ __launch_bounds__(kThreads) void pack_kernel(const void* __restrict__ src,
                                                        int64_t quads,
                                                        uint32_t* __restrict__ packed) {
    const int sub = threadIdx.x & 7;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    // The loop bound is uniform over the block, so every lane takes part in
    // the shuffles; only in-range lanes load and store.
    for (int64_t base = (int64_t)blockIdx.x * kThreads; base < quads; base += stride) {
        const int64_t q = base + threadIdx.x;
        uint32_t part = 0;
        if (q < quads) part = sign_nibble<DT>(src, q) << (4 * sub);
        part |= __shfl_xor(part, 1);
        part |= __shfl_xor(part, 2);
        part |= __shfl_xor(part, 4);
        if (q < quads && sub == 0) packed[q >> 3] = part;
    }
}

template <int DT>
__global__ __launch_bounds__(kThreads) void unpack_kernel(const uint32_t* __restrict__ packed,
                                                          int64_t quads,
                                                          void* __restrict__ dst) {
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t q = (int64_t)blockIdx.x * kThreads + threadIdx.x; q < quads; q += stride) {
        const uint32_t nib = (packed[q >> 3] >> (4 * (q & 7))) & 0xFu;
        if constexpr (DT == kF32) {
            u32x4 v;
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = ((nib >> i) & 1u) ? 0x3F800000u : 0xBF800000u;
            reinterpret_cast<u32x4*>(dst)[q] = v;
        } else if constexpr (DT == kBF16 || DT == kF16) {
            constexpr uint32_t kPlus = DT == kF16 ? 0x3C00u : 0x3F80u;
            constexpr uint32_t kMinus = kPlus | 0x8000u;
            uint2 v;
            v.x = (((nib >> 0) & 1u) ? kPlus : kMinus) | ((((nib >> 1) & 1u) ? kPlus : kMinus) << 16);
            v.y = (((nib >> 2) & 1u) ? kPlus : kMinus) | ((((nib >> 3) & 1u) ? kPlus : kMinus) << 16);
            reinterpret_cast<uint2*>(dst)[q] = v;
        } else {
            uint32_t v = 0;
#pragma unroll
            for (int i = 0; i < 4; ++i) v |= (((nib >> i) & 1u) ? 0x01u : 0xFFu) << (8 * i);
            reinterpret_cast<uint32_t*>(dst)[q] = v;
        }
    }
}

int grid_for(int64_t quads) {
    // Enough blocks to fill 256 CUs several times over; the loops stride the rest.
    const int64_t want = (quads + kThreads - 1) / kThreads;
    return (int)(want < 16384 ? want : 16384);
}

}  // namespace

hipError_t launch_pack(const void* signs, int dtype, int64_t elems, uint32_t* packed,
                       hipStream_t stream) {
    const int64_t quads = elems / 4;
    const int grid = grid_for(quads);
    if (dtype == kF32)
        pack_kernel<kF32><<<grid, kThreads, 0, stream>>>(signs, quads, packed);
    else if (dtype == kBF16)
        pack_kernel<kBF16><<<grid, kThreads, 0, stream>>>(signs, quads, packed);
    else
        pack_kernel<kI8><<<grid, kThreads, 0, stream>>>(signs, quads, packed);
    return hipGetLastError();
}

hipError_t launch_unpack(const uint32_t* packed, int64_t elems, void* signs, int dtype,
                         hipStream_t stream) {
    const int64_t quads = elems / 4;
    const int grid = grid_for(quads);
    if (dtype == kF32)
        unpack_kernel<kF32><<<grid, kThreads, 0, stream>>>(packed, quads, signs);
    else if (dtype == kBF16)
        unpack_kernel<kBF16><<<grid, kThreads, 0, stream>>>(packed, quads, signs);
    else if (dtype == kF16)
        unpack_kernel<kF16><<<grid, kThreads, 0, stream>>>(packed, quads, signs);
    else
        unpack_kernel<kI8><<<grid, kThreads, 0, stream>>>(packed, quads, signs);
    return hipGetLastError();
}

}  // namespace bitdelta
