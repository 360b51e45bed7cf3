/*
 * Reference oracle for the binary-delta matmul: TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the CPU-baseline leg of the
 * benchmark may load this library.  The product path (the HIP library under
 * paper_2609_36800_amd/) never calls it and shares no source with it.
 *
 * What it computes (plain definitions, fp64, k in ascending order):
 *
 *   sign decode   s[n][k] = 2*b - 1 where b is bit (k mod 32) of packed word
 *                 (k div 32) of row n (little-endian bit order inside a word).
 *                 The 2b-1 decode is the one the paper states for its BitDelta
 *                 kernel (Appendix A.2, "BitDelta" paragraph); the packing
 *                 axis and bit order are this library's stated format.
 *   pack          bit = 1 exactly when the input's IEEE / two's-complement
 *                 sign bit is clear (so +1 -> 1, -1 -> 0).
 *   inputs        x and W are bf16 or IEEE fp16 bit patterns, both decoded
 *                 exactly to double.
 *   compress      delta = W_fine - W_base; packed = pack(delta); the scale is
 *                 the mean of |delta| (the least-squares scale for the signs).
 *   matmul        y[m][n] = sum_k x[m][k] W[n][k]
 *                         + alpha[t] * sum_k x[m][k] s_t[n][k],  t = tenant(m)
 *                 i.e. the standard (single-tenant) and batched (per-row
 *                 tenant) BitDelta GEMMs evaluated in Section 4.4.  A tenant
 *                 id outside [0, T) yields a quiet-NaN output row.
 *
 * Acceptance of the GPU path against this oracle is tolerance based, as in the
 * paper's correctness criterion (Section 3.1, Eq. 1).
 *
 * Everything is a plain loop: no blocking, no reordering.  bf16 and fp32
 * inputs convert exactly to double, so the only roundings are the fp64
 * additions and multiplications in k order.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* bf16 bit pattern -> double (exact: bf16 is the top half of an fp32). */
static double bf16_to_double(uint16_t h) {
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* IEEE binary16 bit pattern -> double (exact): sign, 5-bit exponent with
 * bias 15, 10-bit fraction; exponent 0 holds the subnormals f * 2^-24. */
static double f16_to_double(uint16_t h) {
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1F;
    int f = h & 0x3FF;
    double v;
    if (e == 0) v = ldexp((double)f, -24);
    else if (e == 31) v = f ? NAN : INFINITY;
    else v = ldexp((double)(1024 + f), e - 25);
    return sign ? -v : v;
}

/* 16-bit element -> double for element type code dt (1 = bf16, 3 = fp16). */
static double elem_to_double(uint16_t h, int dt) {
    return dt == 3 ? f16_to_double(h) : bf16_to_double(h);
}

/* Sign of weight (n, k) from the packed rows: +1 when the bit is set, else -1. */
static double sign_at(const uint32_t* packed_row, int64_t k) {
    uint32_t word = packed_row[k / 32];
    uint32_t bit = (word >> (uint32_t)(k % 32)) & 1u;
    return bit ? 1.0 : -1.0;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ---- pack: one bit per element, bit set when the sign bit is clear ------ */

static void pack_bits(const uint8_t* signbit, int64_t rows, int64_t K, uint32_t* packed) {
    int64_t words = K / 32;
    for (int64_t r = 0; r < rows; ++r) {
        for (int64_t j = 0; j < words; ++j) {
            uint32_t w = 0;
            for (int64_t i = 0; i < 32; ++i) {
                int64_t k = 32 * j + i;
                if (!signbit[r * K + k]) w |= (1u << i);
            }
            packed[r * words + j] = w;
        }
    }
}

/* The sign bits are first extracted into a byte array, then packed. */
int oracle_pack_f32(const float* v, int64_t rows, int64_t K, uint32_t* packed) {
    if (K % 32 != 0 || rows < 0 || K < 0) return -2;
    int64_t n = rows * K;
    uint8_t* sb = (uint8_t*)malloc((size_t)(n > 0 ? n : 1));
    if (!sb) return -7;
    for (int64_t e = 0; e < n; ++e) {
        uint32_t u;
        memcpy(&u, &v[e], sizeof u);
        sb[e] = (uint8_t)(u >> 31);
    }
    pack_bits(sb, rows, K, packed);
    free(sb);
    return 0;
}

int oracle_pack_bf16(const uint16_t* v, int64_t rows, int64_t K, uint32_t* packed) {
    if (K % 32 != 0 || rows < 0 || K < 0) return -2;
    int64_t n = rows * K;
    uint8_t* sb = (uint8_t*)malloc((size_t)(n > 0 ? n : 1));
    if (!sb) return -7;
    for (int64_t e = 0; e < n; ++e) sb[e] = (uint8_t)(v[e] >> 15);
    pack_bits(sb, rows, K, packed);
    free(sb);
    return 0;
}

int oracle_pack_i8(const int8_t* v, int64_t rows, int64_t K, uint32_t* packed) {
    if (K % 32 != 0 || rows < 0 || K < 0) return -2;
    int64_t n = rows * K;
    uint8_t* sb = (uint8_t*)malloc((size_t)(n > 0 ? n : 1));
    if (!sb) return -7;
    for (int64_t e = 0; e < n; ++e) sb[e] = (uint8_t)(v[e] < 0 ? 1 : 0);
    pack_bits(sb, rows, K, packed);
    free(sb);
    return 0;
}

/* ---- unpack: s = 2b - 1 ------------------------------------------------- */

int oracle_unpack_f64(const uint32_t* packed, int64_t rows, int64_t K, double* out) {
    if (K % 32 != 0 || rows < 0 || K < 0) return -2;
    int64_t words = K / 32;
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t k = 0; k < K; ++k)
            out[r * K + k] = sign_at(packed + r * words, k);
    return 0;
}

/* ---- compress: sign of the delta and its least-squares scale ------------
 *
 *   delta[n][k] = W_fine[n][k] - W_base[n][k]   (fp64; exact unless the two
 *                 exponents differ by more than 45, and its sign always is)
 *   packed      = the pack rule applied to delta (bit set when delta's sign
 *                 bit is clear, so delta = +0 gives +1)
 *   row_abs[n]  = sum_k |delta[n][k]|           (k ascending)
 *   alpha       = sum_n row_abs[n] / (rows * K)
 *
 * With the sign matrix s fixed to the signs of delta, the scale a minimising
 * sum (delta - a s)^2 makes the derivative -2 sum s (delta - a s) vanish;
 * s*s = 1 and s*delta = |delta| turn that into a = sum |delta| / (rows * K).
 * The binary delta the paper's kernel decodes (Appendix A.2) is this pair.
 */
int oracle_compress(const uint16_t* fine, const uint16_t* base, int64_t rows, int64_t K,
                    int dt, uint32_t* packed, double* row_abs, double* alpha) {
    if (K % 32 != 0 || rows < 0 || K < 0) return -2;
    if (dt != 1 && dt != 3) return -4;
    int64_t n = rows * K;
    uint8_t* sb = (uint8_t*)malloc((size_t)(n > 0 ? n : 1));
    if (!sb) return -7;
    double total = 0.0;
    for (int64_t r = 0; r < rows; ++r) {
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            double d = elem_to_double(fine[r * K + k], dt) - elem_to_double(base[r * K + k], dt);
            sb[r * K + k] = (uint8_t)(signbit(d) ? 1 : 0);
            acc += fabs(d);
        }
        if (row_abs) row_abs[r] = acc;
        total += acc;
    }
    pack_bits(sb, rows, K, packed);
    free(sb);
    if (alpha) *alpha = n > 0 ? total / (double)n : 0.0;
    return 0;
}

/* ---- matmul ------------------------------------------------------------- */

/*
 * Evaluates the output at rows m in [0, M) and at the n_count output features
 * listed in n_idx (all of [0, N) when n_idx == NULL, with n_count == N).
 *
 *   x         16-bit bits [M][K]         W     16-bit bits [N][K]
 *   dt        element type of x and W: 1 = bf16, 3 = fp16 (IEEE binary16)
 *   packed    uint32 [T][N][K/32]        alpha fp32 [T]
 *   tenant    int32 [M] or NULL (every row uses tenant 0)
 *   base_out  optional fp64 [M][n_count]: sum_k x W
 *   delta_out optional fp64 [M][n_count]: sum_k x s   (before alpha)
 *   y_out     optional fp64 [M][n_count]: base + alpha * delta
 */
int oracle_matmul_parts(const uint16_t* x, int64_t M, int64_t K,
                        const uint16_t* W, int64_t N,
                        const uint32_t* packed, const float* alpha,
                        const int32_t* tenant, int32_t T,
                        const int64_t* n_idx, int64_t n_count, int dt,
                        double* base_out, double* delta_out, double* y_out) {
    if (K % 32 != 0 || M < 0 || N < 0 || K < 0 || T < 1 || n_count < 0) return -2;
    if (dt != 1 && dt != 3) return -4;
    if (n_idx == NULL && n_count != N) return -2;
    int64_t words = K / 32;
    int64_t j;
#pragma omp parallel for schedule(static)
    for (j = 0; j < n_count; ++j) {
        int64_t n = n_idx ? n_idx[j] : j;
        for (int64_t m = 0; m < M; ++m) {
            int32_t t = tenant ? tenant[m] : 0;
            int64_t o = m * n_count + j;
            if (n < 0 || n >= N || t < 0 || t >= T) {
                if (base_out) base_out[o] = NAN;
                if (delta_out) delta_out[o] = NAN;
                if (y_out) y_out[o] = NAN;
                continue;
            }
            const uint32_t* srow = packed + ((int64_t)t * N + n) * words;
            double base = 0.0, delta = 0.0;
            for (int64_t k = 0; k < K; ++k) {
                double xv = elem_to_double(x[m * K + k], dt);
                base += xv * elem_to_double(W[n * K + k], dt);
                delta += xv * sign_at(srow, k);
            }
            if (base_out) base_out[o] = base;
            if (delta_out) delta_out[o] = delta;
            if (y_out) y_out[o] = base + (double)alpha[t] * delta;
        }
    }
    return 0;
}
