// Compression of a fine-tuned weight into the binary-delta form the matmul
// kernels decode (packed signs, one scale; storage format of Appendix A.2):
//
//   delta[n][k] = W_fine[n][k] - W_base[n][k]                 (fp32)
//   bit (n, k)  = 1 where delta's sign bit is clear, else 0    (same rule as pack)
//   row_abs[n]  = sum_k |delta[n][k]|                          (fp32, fixed order)
//   alpha       = sum_n row_abs[n] / (rows * K)                (fp64 sum, fp32 result)
//
// alpha is the least-squares scale for those signs: with s fixed, the a that
// minimises sum (delta - a s)^2 satisfies sum s (delta - a s) = 0, and
// s * s = 1, s * delta = |delta| give a = mean |delta|.
//
// The difference of two bf16 (or fp16) values has the exact sign in fp32 (a
// nonzero difference is at least 2^-133 (2^-24) in magnitude, above fp32's
// smallest subnormal), and is exact itself unless the exponents differ by more
// than 15 (12 for fp16): the two significands then span more than 24 bits.
//
// compress_kernel streams both weights once (HBM-bound: 4 bytes read per
// element, 1/8 written).  One 4-wave workgroup per row; wave w takes the
// 512-element chunks w, w+4, ..., lane l the 8 consecutive elements 8l..8l+7
// of a chunk, so its 8 sign bits are byte l of the chunk's packed words and a
// wave's byte stores cover 64 contiguous bytes.  Up to four chunks per wave are
// loaded before any is used.  Per-lane sums are added in a fixed butterfly and
// the four wave sums in wave order, so the result does not depend on
// scheduling.  mean_kernel (one workgroup) then reduces the per-row sums in a
// fixed order.
#include "device.h"
#include "internal.h"

namespace bitdelta {
namespace {

constexpr int kWaves = 4;
constexpr int kChunk = 512;  // elements per wave-wide 16-byte load
constexpr int kUnroll = 4;

// The two 16-bit values of a dword as fp32 (exact).
template <int ET>
__device__ __forceinline__ float lo_f32(uint32_t v) {
    if constexpr (ET == kF16) return (float)__builtin_bit_cast(f16x2, v)[0];
    else return __builtin_bit_cast(float, v << 16);
}
template <int ET>
__device__ __forceinline__ float hi_f32(uint32_t v) {
    if constexpr (ET == kF16) return (float)__builtin_bit_cast(f16x2, v)[1];
    else return __builtin_bit_cast(float, v & 0xFFFF0000u);
}

template <int ET>
__global__ __launch_bounds__(kWaves * 64) void compress_kernel(
    const uint16_t* __restrict__ fine, const uint16_t* __restrict__ base, int K,
    uint32_t* __restrict__ packed, float* __restrict__ row_abs) {
    __shared__ float wave_sum[kWaves];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int row = blockIdx.x;
    const uint16_t* f = fine + (size_t)row * K;
    const uint16_t* b = base + (size_t)row * K;
    uint8_t* out = reinterpret_cast<uint8_t*>(packed + (size_t)row * (K / 32));

    float acc = 0.f;
    for (int k0 = kChunk * wv; k0 < K; k0 += kChunk * kWaves * kUnroll) {
        u32x4 fv[kUnroll], bv[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int k = k0 + kChunk * kWaves * u + 8 * lane;
            if (k < K) {
                fv[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(f + k));
                bv[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(b + k));
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int k = k0 + kChunk * kWaves * u + 8 * lane;
            if (k >= K) continue;
            uint32_t byte = 0;
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                const float dl = lo_f32<ET>(fv[u][p]) - lo_f32<ET>(bv[u][p]);
                const float dh = hi_f32<ET>(fv[u][p]) - hi_f32<ET>(bv[u][p]);
                byte |= ((~__builtin_bit_cast(uint32_t, dl)) >> 31) << (2 * p);
                byte |= ((~__builtin_bit_cast(uint32_t, dh)) >> 31) << (2 * p + 1);
                acc += __builtin_fabsf(dl);
                acc += __builtin_fabsf(dh);
            }
            out[k >> 3] = (uint8_t)byte;
        }
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) acc += __shfl_xor(acc, d);
    if (lane == 0) wave_sum[wv] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        float s = wave_sum[0];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) s += wave_sum[w];
        row_abs[row] = s;
    }
}

constexpr int kMeanThreads = 1024;
constexpr int kMeanUnroll = 16;         // rows <= 16384 in a single round of loads

__global__ __launch_bounds__(kMeanThreads) void mean_kernel(const float* __restrict__ row_abs,
                                                            int rows, double count,
                                                            float* __restrict__ alpha) {
    __shared__ double wave_part[kMeanThreads / 64];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    double s = 0.0;
    for (int i0 = 0; i0 < rows; i0 += kMeanThreads * kMeanUnroll) {
        float v[kMeanUnroll];
#pragma unroll
        for (int u = 0; u < kMeanUnroll; ++u) {
            const int i = i0 + kMeanThreads * u + (int)threadIdx.x;
            v[u] = i < rows ? row_abs[i] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kMeanUnroll; ++u) s += (double)v[u];
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) s += __shfl_xor(s, d);
    if (lane == 0) wave_part[wv] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = wave_part[0];
        for (int w = 1; w < kMeanThreads / 64; ++w) t += wave_part[w];
        alpha[0] = (float)(t / count);
    }
}

}  // namespace

hipError_t launch_compress(const uint16_t* fine, const uint16_t* base, int rows, int K, int et,
                           uint32_t* packed, float* row_abs, float* alpha, hipStream_t stream) {
    if (et == kF16)
        compress_kernel<kF16><<<rows, kWaves * 64, 0, stream>>>(fine, base, K, packed, row_abs);
    else
        compress_kernel<kBF16><<<rows, kWaves * 64, 0, stream>>>(fine, base, K, packed, row_abs);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || alpha == nullptr) return e;
    mean_kernel<<<1, kMeanThreads, 0, stream>>>(row_abs, rows, (double)rows * (double)K, alpha);
    return hipGetLastError();
}

}  // namespace bitdelta
