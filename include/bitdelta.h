/*
 * bitdelta.h -- C ABI of the MI355X (gfx950) binary-delta matmul library.
 *
 * The operator is the BitDelta GEMM that the paper evaluates as a "standard"
 * and a "batched" kernel (Section 4.4; kernel description in Appendix A.2,
 * "BitDelta" paragraph): a fine-tuned weight is a shared base weight plus a
 * per-tenant scale times a matrix of signs stored one bit per weight,
 *
 *     y[m][n] = sum_k x[m][k] * W_base[n][k]
 *             + alpha[t] * sum_k x[m][k] * s_t[n][k],     t = tenant of row m,
 *
 * with the sign decoded from its packed bit b as s = 2b - 1 (Appendix A.2).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All array arguments are DEVICE pointers owned by the caller; the library
 *    never frees or retains them.  Arrays are dense and row-major.  The only
 *    memory the library allocates is the grouped prefill's workspace (see
 *    bitdelta_matmul_noalloc); calls on different streams are independent.
 *  - Work is enqueued asynchronously on `stream` (0 = the null stream); the
 *    functions return once the kernels are launched.
 *  - Arguments are checked on the host before anything is launched; a
 *    negative status means nothing was enqueued and no memory was touched.
 *  - Packed sign layout: uint32 words [rows][K/32]; bit i (LSB = bit 0) of word
 *    j of a row holds element k = 32*j + i; bit 1 means +1, bit 0 means -1.
 *    K must be a multiple of 32, so no word is partially used.
 *  - bf16 data is passed as its 16-bit patterns (uint16_t).
 *  - Paths are deterministic: the same inputs give bitwise-identical outputs.
 */
#ifndef BITDELTA_H
#define BITDELTA_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BITDELTA_OK = 0,
    BITDELTA_ERR_NULL = -1,        /* a required pointer is NULL                 */
    BITDELTA_ERR_SHAPE = -2,       /* negative size, K % 32 != 0, T < 1, ...     */
    BITDELTA_ERR_ALIGN = -3,       /* a pointer is not aligned as required       */
    BITDELTA_ERR_DTYPE = -4,       /* dtype code not accepted by this argument   */
    BITDELTA_ERR_UNSUPPORTED = -5, /* valid request this path cannot serve       */
    BITDELTA_ERR_HIP = -6,         /* the HIP runtime reported a launch failure  */
    BITDELTA_ERR_ALIAS = -7,       /* the output overlaps an input               */
    BITDELTA_ERR_TENANT = -8       /* a tenant id is outside [0, T) (reported in
                                      validation mode only, see bitdelta_matmul) */
} bitdelta_status;

typedef enum {
    BITDELTA_F32 = 0,   /* IEEE binary32                  */
    BITDELTA_BF16 = 1,  /* bfloat16 bit patterns          */
    BITDELTA_I8 = 2,    /* signed 8-bit integers          */
    BITDELTA_F16 = 3    /* IEEE binary16 bit patterns     */
} bitdelta_dtype;

/* Kernel paths of bitdelta_matmul (see bitdelta_matmul_path). */
typedef enum {
    BITDELTA_PATH_AUTO = 0,
    BITDELTA_PATH_SKINNY = 1,   /* M <= 64, any tenants: HBM-bound decode path   */
    BITDELTA_PATH_PREFILL = 2   /* fused (W + alpha_t*s_t) GEMM per tenant      */
} bitdelta_path;

/*
 * Pack signs into bits (the storage format of the binary delta, Appendix A.2).
 *
 *   signs     [rows][K] of in_dtype (F32, BF16, F16 or I8); alignment 4 * element size
 *   packed    [rows][K/32] uint32, 4-byte aligned
 *
 * Bit = 1 exactly when the element's sign bit is clear: +1 -> 1, -1 -> 0, and
 * for other values +0/+inf/positive NaN -> 1, -0/-inf/negative NaN -> 0,
 * int8 v >= 0 -> 1.  rows == 0 or K == 0 is a no-op.
 * Errors: NULL, SHAPE (rows < 0, K < 0, K % 32), ALIGN, DTYPE, HIP.
 */
int bitdelta_pack(const void* signs, int in_dtype, int64_t rows, int64_t K,
                  uint32_t* packed, hipStream_t stream);

/*
 * Decode packed bits into +1 / -1 (s = 2b - 1, Appendix A.2).
 *
 *   packed    [rows][K/32] uint32, 4-byte aligned
 *   signs     [rows][K] of out_dtype (F32, BF16, F16 or I8); alignment 4 * element size
 *
 * Errors: NULL, SHAPE, ALIGN, DTYPE, HIP.
 */
int bitdelta_unpack(const uint32_t* packed, int64_t rows, int64_t K,
                    void* signs, int out_dtype, hipStream_t stream);

/*
 * Compress a fine-tuned weight against its base into the binary-delta form
 * the matmul consumes (the packed signs of Appendix A.2 and one scale):
 *
 *   delta[n][k]     = w_fine[n][k] - w_base[n][k], computed in fp32 (its
 *                     sign is always exact)
 *   packed          bit set where delta's sign bit is clear (delta = +0
 *                   gives +1), by the same rule as bitdelta_pack
 *   row_abs_sum[n]  = sum_k |delta[n][k]| (fp32, fixed summation order)
 *   alpha[0]        = sum_n row_abs_sum[n] / (rows * K), summed in fp64
 *
 * alpha is the least-squares scale for these signs: it minimises
 * ||delta - a * s||_F over a (the derivative vanishes at a = mean |delta|).
 *
 *   w_fine, w_base  [rows][K] of in_dtype (BF16 or F16), 16-byte aligned
 *   packed          [rows][K/32] uint32 output, 4-byte aligned
 *   row_abs_sum     [rows] fp32 output, 4-byte aligned (also holds the
 *                   partial sums of the alpha reduction)
 *   alpha           [1] fp32 output, or NULL to skip the mean
 *
 * Inputs are expected finite and free of subnormals.  rows == 0 or K == 0
 * is a no-op.  Outputs must not overlap inputs or each other.
 * Errors: NULL, SHAPE (rows < 0, K < 0, K % 32), ALIGN, DTYPE, ALIAS, HIP.
 */
int bitdelta_compress(const uint16_t* w_fine, const uint16_t* w_base,
                      int64_t rows, int64_t K, int in_dtype, uint32_t* packed,
                      float* row_abs_sum, float* alpha, hipStream_t stream);

/*
 * Binary-delta matmul, standard and batched (multi-tenant) forms (Section 4.4).
 *
 *   x           [M][K] bf16, 16-byte aligned
 *   w_base      [N][K] bf16, 16-byte aligned
 *   packed_s    [T][N][K/32] uint32 sign bits, 4-byte aligned
 *   alpha       [T] fp32 scales (device memory), 4-byte aligned
 *   tenant_ids  [M] int32 (device memory): row m uses tenant tenant_ids[m];
 *               NULL means every row uses tenant 0 (the standard form)
 *   T           number of tenants held in packed_s / alpha, >= 1
 *   y           [M][N] of y_dtype (F32 or BF16), 16-byte aligned; must not
 *               overlap any input
 *
 * Accumulation is fp32; a bf16 output is rounded to nearest-even once at the
 * end.  The fused path (single tenant with M > 64, batched with M >= 256)
 * rounds the effective weight W_base + alpha_t*s_t to bf16 before its one
 * matrix-core GEMM; the decode-shaped path keeps the two sums apart and
 * never rounds the weight.
 * A row whose tenant id is outside [0, T) is written as quiet NaN (ids live in
 * device memory, so they are not checked on the host).  Validation mode: with
 * the environment variable BITDELTA_VALIDATE set to a value other than "0",
 * a batched call first reads the ids back (a device-to-host copy on `stream`
 * and a synchronisation of `stream`, so not under graph capture) and returns
 * BITDELTA_ERR_TENANT, launching nothing, if any id is outside [0, T); a
 * failure of that read-back returns BITDELTA_ERR_HIP.  Meant for debugging.
 * M == 0 or N == 0 is a no-op; K == 0 writes zeros.
 * Batched requests with M >= 256, K a multiple of 64 and T <= 2048 run one
 * fused GEMM per tenant over that tenant's rows (grouped on the device);
 * other batched requests with M > 64 are served 64 rows at a time.
 * Errors: NULL, SHAPE, ALIGN, DTYPE, ALIAS, HIP; TENANT in validation mode.
 */
int bitdelta_matmul(const uint16_t* x, int64_t M, int64_t K,
                    const uint16_t* w_base, int64_t N,
                    const uint32_t* packed_s, const float* alpha,
                    const int32_t* tenant_ids, int32_t T,
                    void* y, int y_dtype, hipStream_t stream);

/*
 * Same as bitdelta_matmul with the kernel path chosen by the caller (tests
 * exercise each path on the same inputs).  BITDELTA_PATH_PREFILL with
 * tenant_ids != NULL needs K a multiple of 64, T <= 2048 and M*K, N*K below
 * 2^30, else it returns BITDELTA_ERR_UNSUPPORTED; BITDELTA_PATH_SKINNY accepts
 * any M (64 rows per launch).
 */
int bitdelta_matmul_with_path(const uint16_t* x, int64_t M, int64_t K,
                              const uint16_t* w_base, int64_t N,
                              const uint32_t* packed_s, const float* alpha,
                              const int32_t* tenant_ids, int32_t T,
                              void* y, int y_dtype, int path, hipStream_t stream);

/*
 * The matmul with x and w_base of 16-bit type in_dtype: BITDELTA_BF16 (as
 * bitdelta_matmul_with_path) or BITDELTA_F16, the paper's own precision for
 * BitDelta (Appendix A.2).  y_dtype is F32 or in_dtype.  Everything else is
 * as in bitdelta_matmul_with_path; for F16 the fused path's effective weight
 * is fp16_rne(W_base + fp16_rne(+-alpha_t)), formed with packed fp16 adds.
 * Errors: as bitdelta_matmul, DTYPE for any other in_dtype / y_dtype pair.
 */
int bitdelta_matmul_typed(const uint16_t* x, int64_t M, int64_t K,
                          const uint16_t* w_base, int64_t N,
                          const uint32_t* packed_s, const float* alpha,
                          const int32_t* tenant_ids, int32_t T, int in_dtype,
                          void* y, int y_dtype, int path, hipStream_t stream);

/*
 * Allocation-free form of bitdelta_matmul_typed, for callers that cannot
 * allocate device memory: code under graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Arguments, results and errors are those
 * of bitdelta_matmul_typed; the outputs are bitwise identical to its.
 *
 * bitdelta_matmul_typed may allocate, once per (device, stream), the grouped
 * prefill's partial-sum workspace (the fp32 partial sums of output tiles split
 * along K when there are more tiles than compute units).  This form never
 * calls hipMalloc or any allocating routine: it uses a fixed array of
 * 67,375,120 bytes in the library's device memory (64 MiB of partial sums and
 * 266,256 bytes of split record), which each GPU the library runs on holds
 * until the process ends.  That size covers the largest split, so no request
 * is refused for its size; the only limits are bitdelta_matmul_typed's.  On
 * its first call on a device the address of that device's array is looked up
 * (hipGetSymbolAddress); BITDELTA_ERR_HIP if the runtime cannot give it.
 *
 * All calls of this form on one GPU share the array: calls that overlap in
 * time on one GPU (different streams, or different host threads) race and
 * may produce wrong results.  Calls in order on one stream are safe.  The
 * array keeps the last call's contents; every call writes what it reads.
 */
int bitdelta_matmul_noalloc(const uint16_t* x, int64_t M, int64_t K,
                            const uint16_t* w_base, int64_t N,
                            const uint32_t* packed_s, const float* alpha,
                            const int32_t* tenant_ids, int32_t T, int in_dtype,
                            void* y, int y_dtype, int path, hipStream_t stream);

/* The path bitdelta_matmul picks for these sizes (no side effects). */
int bitdelta_matmul_path(int64_t M, int64_t N, int64_t K, int32_t T, int has_tenant_ids);

/* Static, NUL-terminated description of a status code. */
const char* bitdelta_status_string(int status);

/* Library ABI version (major * 100 + minor). */
int bitdelta_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BITDELTA_H */
