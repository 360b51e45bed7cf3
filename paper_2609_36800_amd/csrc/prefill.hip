// Prefill-shaped binary-delta matmul (one tenant, many rows): one bf16 GEMM
//
//   y = x * W_eff^T,   W_eff[n][k] = bf16_rne( W[n][k] + (b ? alpha : -alpha) )
//
// At M = N = K = 4096 the work is bound by the matrix cores, so the two sums of
// the definition are fused into one contraction over the effective weight, the
// form the standard BitDelta GEMM takes once the decoded signs are fed straight
// to the matrix unit (Appendix A.2).  The price is one bf16 rounding of the
// effective weight (alpha is tiny next to |W|, so it shifts W by a few ulps).
//
// Tiling for gfx950: a 256-thread workgroup (4 waves, 2x2) owns a 256x256
// output tile; each wave owns 128x128 = 4x4 v_mfma_f32_32x32x16_bf16 tiles
// (256 fp32 accumulators per lane).  K advances in 64-wide tiles staged in LDS
// (double-buffered, 64 KB per stage).  Each thread moves eight 16-byte chunks
// of x and eight of W per tile with coalesced 128-bit loads plus the matching
// sign bytes; W chunks are fused with alpha*s in registers on their way to LDS,
// so every element of W_eff is decoded once per workgroup, not once per wave.
// LDS rows are 128 bytes; chunk c of row r is stored at slot c ^ (r & 7) so
// that the fragment reads of eight consecutive rows hit distinct banks.
//
// Workgroups are renumbered so that the 32 resident on one XCD (the hardware
// deals workgroups round-robin over the 8 XCDs) cover a 4 x 8 block of tiles
// and share their x and W panels in that XCD's L2.
#include "device.h"
#include "internal.h"

namespace bitdelta {
namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kThreads = 256;
constexpr int kChunks = BM * BK / 8 / kThreads;  // 16-byte chunks per thread per operand = 8
constexpr int kGroupM = 4;

struct PrefillLds {
    uint16_t a[2][BM * BK];
    uint16_t b[2][BN * BK];
};

__device__ __forceinline__ int lds_off(int row, int chunk) {
    return row * BK + ((chunk ^ (row & 7)) << 3);
}

__global__ __launch_bounds__(kThreads, 1) void prefill_kernel(
    const uint16_t* __restrict__ x, int M, int K, const uint16_t* __restrict__ w, int N,
    const uint32_t* __restrict__ packed, const float* __restrict__ alpha,
    void* __restrict__ y, int y_dtype, int tiles_m, int tiles_n) {
    __shared__ PrefillLds lds;

    // ---- tile assignment (XCD-aware) ----
    const int nwg = tiles_m * tiles_n;
    int bid = blockIdx.x;
    if ((nwg & 7) == 0) bid = (bid & 7) * (nwg >> 3) + (bid >> 3);
    const int group = bid / (kGroupM * tiles_n);
    const int first_m = group * kGroupM;
    const int gm = min(tiles_m - first_m, kGroupM);
    const int local = bid - group * kGroupM * tiles_n;
    const int tile_m = first_m + local % gm;
    const int tile_n = local / gm;
    const int m0 = tile_m * BM, n0 = tile_n * BN;

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int wm = wv >> 1, wn = wv & 1;
    const int KW = K >> 5;
    const int KT = (K + BK - 1) / BK;
    const uint32_t neg_alpha = __builtin_bit_cast(uint32_t, -alpha[0]);

    // ---- global -> register staging assignment ----
    const int q = tid & 7, r0 = tid >> 3;
    const uint16_t* pa[kChunks];
    const uint16_t* pb[kChunks];
    const uint32_t* ps[kChunks];
    bool va[kChunks], vb[kChunks];
#pragma unroll
    for (int i = 0; i < kChunks; ++i) {
        const int row = r0 + 32 * i;
        va[i] = m0 + row < M;
        vb[i] = n0 + row < N;
        pa[i] = x + (size_t)(va[i] ? m0 + row : 0) * K + 8 * q;
        pb[i] = w + (size_t)(vb[i] ? n0 + row : 0) * K + 8 * q;
        ps[i] = packed + (size_t)(vb[i] ? n0 + row : 0) * KW + (q >> 2);
    }
    const u32x4 zero = {0u, 0u, 0u, 0u};
    u32x4 ra[kChunks], rb[kChunks];
    uint32_t rs[kChunks];

    auto gload = [&](int kt) {
        const bool kv = kt * BK + 8 * q < K;
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            ra[i] = (va[i] && kv) ? load16(pa[i] + kt * BK) : zero;
            rb[i] = (vb[i] && kv) ? load16(pb[i] + kt * BK) : zero;
            rs[i] = (vb[i] && kv) ? ps[i][kt * 2] : 0u;
        }
    };
    auto lstore = [&](int buf, int kt) {
        const bool kv = kt * BK + 8 * q < K;
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            const int row = r0 + 32 * i;
            const int off = lds_off(row, q);
            *reinterpret_cast<u32x4*>(&lds.a[buf][off]) = ra[i];
            const u32x4 fused = fuse_weights8(rb[i], (rs[i] >> (8 * (q & 3))) & 0xFFu, neg_alpha);
            *reinterpret_cast<u32x4*>(&lds.b[buf][off]) = (vb[i] && kv) ? fused : zero;
        }
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    auto compute = [&](int buf) {
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
            const int c = kk * 2 + (lane >> 5);
            u32x4 af[4], bf[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = wm * 128 + i * 32 + (lane & 31);
                af[i] = *reinterpret_cast<const u32x4*>(&lds.a[buf][lds_off(row, c)]);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int col = wn * 128 + j * 32 + (lane & 31);
                bf[j] = *reinterpret_cast<const u32x4*>(&lds.b[buf][lds_off(col, c)]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = mfma32(af[i], bf[j], acc[i][j]);
        }
    };

    if (KT > 0) {
        gload(0);
        lstore(0, 0);
        __syncthreads();
        for (int kt = 0; kt < KT; ++kt) {
            const int buf = kt & 1;
            if (kt + 1 < KT) gload(kt + 1);
            compute(buf);
            if (kt + 1 < KT) lstore(buf ^ 1, kt + 1);
            __syncthreads();
        }
    }

    // ---- epilogue: lane holds column (lane & 31) of each 32x32 tile ----
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = n0 + wn * 128 + j * 32 + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                if (row < M && col < N) {
                    if (y_dtype == kF32)
                        reinterpret_cast<float*>(y)[(size_t)row * N + col] = acc[i][j][r];
                    else
                        reinterpret_cast<uint16_t*>(y)[(size_t)row * N + col] = to_bf16(acc[i][j][r]);
                }
            }
        }
}

}  // namespace

hipError_t launch_prefill(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                          const uint32_t* packed, const float* alpha, void* y, int y_dtype,
                          hipStream_t stream) {
    const int tiles_m = (M + BM - 1) / BM;
    const int tiles_n = (N + BN - 1) / BN;
    prefill_kernel<<<tiles_m * tiles_n, kThreads, 0, stream>>>(x, M, K, w, N, packed, alpha, y,
                                                               y_dtype, tiles_m, tiles_n);
    return hipGetLastError();
}

}  // namespace bitdelta
