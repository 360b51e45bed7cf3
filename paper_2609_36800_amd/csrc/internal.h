// Host-side launchers of the gfx950 kernels (one translation unit each).
// Arguments are validated by the C-ABI layer before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bitdelta {

// Element dtype codes (same values as the public bitdelta_dtype).  The matmul
// launchers take `et`, the 16-bit type of x and W (kBF16 or kF16); a 16-bit
// y has that same type.
constexpr int kF32 = 0;
constexpr int kBF16 = 1;
constexpr int kI8 = 2;
constexpr int kF16 = 3;

// Pack / unpack over a flat run of `elems` elements (a multiple of 32): the
// packed words of consecutive rows are contiguous, so rows need no special care.
hipError_t launch_pack(const void* signs, int dtype, int64_t elems, uint32_t* packed,
                       hipStream_t stream);
hipError_t launch_unpack(const uint32_t* packed, int64_t elems, void* signs, int dtype,
                         hipStream_t stream);

// Binary delta of a fine-tuned weight: packed signs of W_fine - W_base, the
// per-row sums of |delta| and (when alpha is not null) their mean.
hipError_t launch_compress(const uint16_t* fine, const uint16_t* base, int rows, int K, int et,
                           uint32_t* packed, float* row_abs, float* alpha, hipStream_t stream);

// Single-tenant decode matmul for at most 16 rows (signs and x staged via LDS).
hipError_t launch_decode(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                         const uint32_t* packed, const float* alpha, void* y, int y_dtype,
                         int et, hipStream_t stream);

// Batched (multi-tenant) matmul for at most 64 rows, operands staged in LDS by
// global->LDS copies; needs K a positive multiple of 128 (multi_supported).
bool multi_supported(int K);
hipError_t launch_multi(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                        const uint32_t* packed, const float* alpha, const int32_t* tenant_ids,
                        int T, void* y, int y_dtype, int et, hipStream_t stream);

// Batched matmul for up to 64 rows and at most 16 distinct tenants, K a
// multiple of 128: each tenant's rows gathered into 16-row fragments, one sign
// decode per tenant and k-block.  batched_supported says where the dispatcher
// uses it (17 to 64 rows when N <= 4096 and K is a multiple of 256; above
// 4096 features also 8 to 16 rows over at most 8 tenants).
bool batched_supported(int M, int N, int K, int T);
hipError_t launch_batched(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                          const uint32_t* packed, const float* alpha, const int32_t* tenant_ids,
                          int T, void* y, int y_dtype, int et, hipStream_t stream);

// Decode-shaped matmul for at most 64 rows (any number of tenants).
hipError_t launch_skinny(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                         const uint32_t* packed, const float* alpha,
                         const int32_t* tenant_ids, int T, void* y, int y_dtype, int et,
                         hipStream_t stream);

// Prefill-shaped single-tenant matmul: one bf16 GEMM over W + alpha*s.
bool prefill_stream_supported(int M, int N, int K);
hipError_t launch_prefill(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                          const uint32_t* packed, const float* alpha, void* y, int y_dtype,
                          int et, hipStream_t stream);

// Prefill-shaped batched matmul: one fused GEMM per tenant over its rows,
// routed on the device; needs prefill_grouped_supported.  With more than 256
// output tiles the leftover tiles are split along K over the idle CUs when
// `scratch` (scratch_bytes, at least prefill_split_bytes() for the full split)
// can hold their fp32 partial sums and per-tile counters; the counters must be
// zero on entry and are left zero.  scratch may be null (no split).
size_t prefill_split_bytes();
// prefill_split_bytes() as a constant: 256 chunks of 256 x 256 fp32 partial
// sums and the split record (4 ints, then 260 per leftover tile)
constexpr size_t kPrefillSplitBytes = (size_t)256 * 256 * 256 * 4 + (4 + (size_t)256 * (256 + 4)) * 4;
bool prefill_grouped_supported(int M, int N, int K, int T);
hipError_t launch_prefill_grouped(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                                  const uint32_t* packed, const float* alpha,
                                  const int32_t* tenant_ids, int T, void* y, int y_dtype,
                                  int et, hipStream_t stream, void* scratch, size_t scratch_bytes);

// Batched matmul, wide form (wide.hip): 17 to 64 rows, at most 16 distinct
// tenants, K a multiple of 128, 48 or 64 features per workgroup, where those
// feature groups fill the CUs (wide_supported).
bool wide_supported(int M, int N, int K, int T);
hipError_t launch_wide(const uint16_t* x, int M, int K, const uint16_t* w, int N, const uint32_t* packed,
                       const float* alpha, const int32_t* tenant_ids, int T, void* y, int y_dtype, int et,
                       hipStream_t stream);

}  // namespace bitdelta
