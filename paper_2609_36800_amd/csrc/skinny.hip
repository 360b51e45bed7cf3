// Decode-shaped binary-delta matmul: at most 64 token rows, any number of tenants.
//
//   y[m][n] = sum_k x[m][k] W[n][k] + alpha[t(m)] * sum_k x[m][k] s_t(m)[n][k]
//
// (the standard and batched BitDelta GEMMs of Section 4.4).  At these shapes
// the kernel is bound by HBM: every byte of W and of the sign bits of the
// tenants present is read once, x stays in cache.
//
// Work split: a workgroup owns 16 output features and all rows; its waves
// split the contraction into contiguous runs of 32-wide k-blocks.  Per k-block
// a lane issues one 16-byte load of W (8 consecutive k of one feature, the MFMA
// B operand as stored), one 32-bit load of the sign word, and 16-byte loads of
// x.  Signs are decoded in registers into bf16 +1/-1 operands
// (decode_signs8) and both sums run on v_mfma_f32_16x16x32_bf16 with fp32
// accumulation: x*W^T into one accumulator, x*S^T into another.  The two are
// combined only in the epilogue, so the effective weight W + alpha*s is never
// rounded.  This is the MI355X form of "decode packed bits straight into
// matrix-core operands" (Appendix A.2): there is no LDS round trip of the
// decoded signs at all.
//
// Tenants (batched form): wave 0 groups the rows by tenant id with ballots
// (one ballot per distinct tenant present, no host round trip) and cuts each
// group into blocks of up to 16 rows.  A block's x rows are gathered into the
// MFMA A operand, its tenant's sign words are decoded into the B operand.
// Blocks are processed SBP at a time; only the first pass also streams W.
//
// Partial sums of the waves are combined in a fixed order through LDS, so the
// result is bitwise deterministic (no atomics).
#include "device.h"
#include "internal.h"

namespace bitdelta {
namespace {

constexpr int kRowsMax = 64;
constexpr int kFeat = 16;  // output features per workgroup

template <int MB, int NW>
struct SkinnyLds {
    float red_base[NW][MB * 16][kFeat];
    float red_sign[NW][MB * 16][kFeat];
    int row_tenant[kRowsMax];          // tenant of row m; -1: id out of range
    int blk_rows[kRowsMax][16];        // gathered row of each block slot, -1 = empty
    int blk_tenant[kRowsMax];
    int nblk;
};

__device__ __forceinline__ uint32_t sign_byte(uint32_t word, int group) {
    return (word >> (8 * group)) & 0xFFu;
}

// Contiguous share [kb0, kb1) of the 32-wide k-blocks for wave wv.
__device__ __forceinline__ void wave_range(int KB, int wv, int nw, int& kb0, int& kb1) {
    const int per = (KB + nw - 1) / nw;
    kb0 = min(KB, wv * per);
    kb1 = min(KB, kb0 + per);
}

// Single tenant.  Each wave streams a contiguous run of k-blocks through a
// ring of D register stages: the loads of block i+D are issued right after
// block i is consumed, so up to D blocks per lane stay in flight.  Loads are
// never predicated: rows beyond M or N are clamped onto the last valid row
// (they only feed output rows/columns that are not stored), which keeps the
// loads free of branches and lets the compiler wait on the oldest stage only.
template <int ET, int MB, int NW, int D>
__global__ __launch_bounds__(NW * 64) void skinny_single_kernel(
    const uint16_t* __restrict__ x, int M, int K, const uint16_t* __restrict__ w, int N,
    const uint32_t* __restrict__ packed, const float* __restrict__ alpha,
    void* __restrict__ y, int y_dtype) {
    __shared__ SkinnyLds<MB, NW> sh;
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
    const int nl = lane & 15, g = lane >> 4;
    const int n0 = blockIdx.x * kFeat;
    const int KB = K >> 5, KW = K >> 5;

    const int n = min(n0 + nl, N - 1);
    const uint16_t* wp = w + (size_t)n * K + 8 * g;
    // byte g of each sign word holds the signs of this lane's eight k
    const uint8_t* sp = reinterpret_cast<const uint8_t*>(packed + (size_t)n * KW) + g;
    const uint16_t* xp[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) xp[mb] = x + (size_t)min(mb * 16 + nl, M - 1) * K + 8 * g;

    f32x4 accb[MB], accs[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
        accb[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
        accs[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    int kb0, kb1;
    wave_range(KB, wv, NW, kb0, kb1);
    const int cnt = kb1 - kb0;
    if (cnt > 0) {
        u32x4 wf[D];
        uint32_t sb[D];
        u32x4 xf[D][MB];
        auto issue = [&](int slot, int kb) {
            wf[slot] = load16(wp + kb * 32);
            sb[slot] = sp[kb * 4];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) xf[slot][mb] = load16(xp[mb] + kb * 32);
            // keep stages in issue order: the oldest stage must complete first
            __builtin_amdgcn_sched_barrier(0);
        };
        auto consume = [&](int slot) {
            const u32x4 sf = decode_signs8<ET>(sb[slot]);
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                accb[mb] = mfma16<ET>(xf[slot][mb], wf[slot], accb[mb]);
                accs[mb] = mfma16<ET>(xf[slot][mb], sf, accs[mb]);
            }
        };
        // Rounds of D blocks: all D loads of a round are issued back to back
        // (in order), then consumed oldest first, each block waiting only for
        // its own stage.  A wave's whole share is one round when K <= 32*D*NW.
        for (int base = 0; base < cnt; base += D) {
            const int c = min(D, cnt - base);
#pragma unroll
            for (int j = 0; j < D; ++j) issue(j, kb0 + base + min(j, c - 1));
            if (c == D) {
                // full round: no guards, so no load can be sunk past its successors
#pragma unroll
                for (int j = 0; j < D; ++j) consume(j);
            } else {
#pragma unroll
                for (int j = 0; j < D; ++j)
                    if (j < c) consume(j);
            }
        }
    }

    // lane holds D(row 4g + r, feature nl) of each 16-row block
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            sh.red_base[wv][mb * 16 + 4 * g + r][nl] = accb[mb][r];
            sh.red_sign[wv][mb * 16 + 4 * g + r][nl] = accs[mb][r];
        }
    __syncthreads();

    const float a = alpha[0];
    for (int idx = threadIdx.x; idx < MB * 16 * kFeat; idx += NW * 64) {
        const int m = idx / kFeat, f = idx % kFeat;
        const int nn = n0 + f;
        if (m >= M || nn >= N) continue;
        float b = 0.f, s = 0.f;
#pragma unroll
        for (int v = 0; v < NW; ++v) {
            b += sh.red_base[v][m][f];
            s += sh.red_sign[v][m][f];
        }
        const float out = __builtin_fmaf(a, s, b);
        store_y<ET>(y, (size_t)m * N + nn, out, y_dtype);
    }
}

template <int ET, int MB, int NW, int U, int SBP>
__global__ __launch_bounds__(NW * 64) void skinny_multi_kernel(
    const uint16_t* __restrict__ x, int M, int K, const uint16_t* __restrict__ w, int N,
    const uint32_t* __restrict__ packed, const float* __restrict__ alpha,
    const int32_t* __restrict__ tenant_ids, int T, void* __restrict__ y, int y_dtype) {
    __shared__ SkinnyLds<MB, NW> sh;
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
    const int nl = lane & 15, g = lane >> 4;
    const int n0 = blockIdx.x * kFeat;
    const int n = n0 + nl;
    const bool nvalid = n < N;
    const int KB = K >> 5, KW = K >> 5;

    // ---- group rows by tenant (wave 0) ----
    if (wv == 0) {
        int t = -2;
        if (lane < M) {
            t = tenant_ids[lane];
            if (t < 0 || t >= T) t = -1;
        }
        sh.row_tenant[lane] = t;
#pragma unroll
        for (int i = 0; i < 16; ++i) sh.blk_rows[lane][i] = -1;
        unsigned long long remaining = __ballot(t >= 0);
        int nb = 0;
        while (remaining) {
            const int leader = __ffsll((long long)remaining) - 1;
            const int tl = __shfl(t, leader);
            const unsigned long long grp = __ballot(t == tl) & remaining;
            remaining &= ~grp;
            if ((grp >> lane) & 1ull) {
                const int rank = __popcll(grp & ((1ull << lane) - 1ull));
                sh.blk_rows[nb + rank / 16][rank % 16] = lane;
                if (rank % 16 == 0) sh.blk_tenant[nb + rank / 16] = tl;
            }
            nb += (__popcll(grp) + 15) / 16;
        }
        if (lane == 0) sh.nblk = nb;
    }
    __syncthreads();
    const int nblk = sh.nblk;

    const uint16_t* wrow = w + (size_t)(nvalid ? n : 0) * K + 8 * g;
    const uint16_t* xrow[MB];
    bool xvalid[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
        const int m = mb * 16 + nl;
        xvalid[mb] = m < M;
        xrow[mb] = x + (size_t)(xvalid[mb] ? m : 0) * K + 8 * g;
    }
    int kb0, kb1;
    wave_range(KB, wv, NW, kb0, kb1);
    const u32x4 zero = {0u, 0u, 0u, 0u};

    for (int p0 = 0; p0 == 0 || p0 < nblk; p0 += SBP) {
        const bool do_base = (p0 == 0);
        f32x4 accb[MB], accs[SBP];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) accb[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int b = 0; b < SBP; ++b) accs[b] = f32x4{0.f, 0.f, 0.f, 0.f};

        bool bact[SBP], gv[SBP];
        const uint32_t* sp[SBP];
        const uint16_t* gp[SBP];
#pragma unroll
        for (int b = 0; b < SBP; ++b) {
            const int blk = p0 + b;
            bact[b] = blk < nblk;
            const int t = bact[b] ? sh.blk_tenant[blk] : 0;
            const int row = bact[b] ? sh.blk_rows[blk][nl] : -1;
            gv[b] = row >= 0;
            gp[b] = x + (size_t)(gv[b] ? row : 0) * K + 8 * g;
            sp[b] = packed + ((size_t)t * N + (nvalid ? n : 0)) * KW;
        }

        auto run = [&](int kb, auto unroll_tag) {
            constexpr int UU = decltype(unroll_tag)::value;
            u32x4 wf[UU];
            u32x4 xf[UU][MB];
            uint32_t sw[UU][SBP];
            u32x4 gf[UU][SBP];
#pragma unroll
            for (int u = 0; u < UU; ++u) {
                const int k = (kb + u) * 32;
                if (do_base) {
                    wf[u] = nvalid ? load16(wrow + k) : zero;
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) xf[u][mb] = xvalid[mb] ? load16(xrow[mb] + k) : zero;
                }
#pragma unroll
                for (int b = 0; b < SBP; ++b) {
                    if (bact[b]) {
                        sw[u][b] = nvalid ? sp[b][kb + u] : 0u;
                        gf[u][b] = gv[b] ? load16(gp[b] + k) : zero;
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < UU; ++u) {
                if (do_base) {
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) accb[mb] = mfma16<ET>(xf[u][mb], wf[u], accb[mb]);
                }
#pragma unroll
                for (int b = 0; b < SBP; ++b) {
                    if (bact[b]) {
                        const u32x4 sf = decode_signs8<ET>(sign_byte(sw[u][b], g));
                        accs[b] = mfma16<ET>(gf[u][b], sf, accs[b]);
                    }
                }
            }
        };
        int kb = kb0;
        for (; kb + U <= kb1; kb += U) run(kb, std::integral_constant<int, U>{});
        for (; kb < kb1; ++kb) run(kb, std::integral_constant<int, 1>{});

        if (do_base) {
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int r = 0; r < 4; ++r) sh.red_base[wv][mb * 16 + 4 * g + r][nl] = accb[mb][r];
        }
#pragma unroll
        for (int b = 0; b < SBP; ++b) {
            if (!bact[b]) continue;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = sh.blk_rows[p0 + b][4 * g + r];
                if (row >= 0) sh.red_sign[wv][row][nl] = accs[b][r];
            }
        }
    }
    __syncthreads();

    for (int idx = threadIdx.x; idx < MB * 16 * kFeat; idx += NW * 64) {
        const int m = idx / kFeat, f = idx % kFeat;
        const int nn = n0 + f;
        if (m >= M || nn >= N) continue;
        const int t = sh.row_tenant[m];
        float out;
        if (t < 0) {
            out = __builtin_nanf("");
        } else {
            float b = 0.f, s = 0.f;
#pragma unroll
            for (int v = 0; v < NW; ++v) {
                b += sh.red_base[v][m][f];
                s += sh.red_sign[v][m][f];
            }
            out = __builtin_fmaf(alpha[t], s, b);
        }
        store_y<ET>(y, (size_t)m * N + nn, out, y_dtype);
    }
}

constexpr int kWaves = 8;

template <int ET, int MB>
hipError_t launch_single_mb(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                            const uint32_t* packed, const float* alpha, void* y, int y_dtype,
                            hipStream_t stream) {
    const int grid = (N + kFeat - 1) / kFeat;
    constexpr int D = MB == 1 ? 16 : (MB == 2 ? 12 : 8);
    skinny_single_kernel<ET, MB, kWaves, D><<<grid, kWaves * 64, 0, stream>>>(
        x, M, K, w, N, packed, alpha, y, y_dtype);
    return hipGetLastError();
}

template <int ET, int MB>
hipError_t launch_multi_mb(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                           const uint32_t* packed, const float* alpha, const int32_t* tenant_ids,
                           int T, void* y, int y_dtype, hipStream_t stream) {
    const int grid = (N + kFeat - 1) / kFeat;
    skinny_multi_kernel<ET, MB, kWaves, 2, 8><<<grid, kWaves * 64, 0, stream>>>(
        x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype);
    return hipGetLastError();
}

template <int ET>
hipError_t launch_skinny_et(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                            const uint32_t* packed, const float* alpha,
                            const int32_t* tenant_ids, int T, void* y, int y_dtype,
                            hipStream_t stream) {
    const int mb = (M + 15) / 16;
    if (tenant_ids == nullptr) {
        if (M <= 16) return launch_decode(x, M, K, w, N, packed, alpha, y, y_dtype, ET, stream);
        switch (mb) {
            case 1: return launch_single_mb<ET, 1>(x, M, K, w, N, packed, alpha, y, y_dtype, stream);
            case 2: return launch_single_mb<ET, 2>(x, M, K, w, N, packed, alpha, y, y_dtype, stream);
            case 3: return launch_single_mb<ET, 3>(x, M, K, w, N, packed, alpha, y, y_dtype, stream);
            default: return launch_single_mb<ET, 4>(x, M, K, w, N, packed, alpha, y, y_dtype, stream);
        }
    }
    if (wide_supported(M, N, K, T))
        return launch_wide(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, ET, stream);
    if (batched_supported(M, N, K, T))
        return launch_batched(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, ET, stream);
    if (multi_supported(K))
        return launch_multi(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, ET, stream);
    switch (mb) {
        case 1: return launch_multi_mb<ET, 1>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
        case 2: return launch_multi_mb<ET, 2>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
        case 3: return launch_multi_mb<ET, 3>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
        default: return launch_multi_mb<ET, 4>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
    }
}

}  // namespace

hipError_t launch_skinny(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                         const uint32_t* packed, const float* alpha,
                         const int32_t* tenant_ids, int T, void* y, int y_dtype, int et,
                         hipStream_t stream) {
    if (et == kF16)
        return launch_skinny_et<kF16>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
    return launch_skinny_et<kBF16>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
}

}  // namespace bitdelta
