// Batched (multi-tenant) binary-delta matmul for at most 64 token rows:
//
//   y[m][n] = sum_k x[m][k] W[n][k] + alpha[t(m)] * sum_k x[m][k] s_t(m)[n][k]
//
// (the batched BitDelta GEMM of Section 4.4).  Row m selects its tenant's
// sign matrix by id; every W byte and the sign bytes of each tenant present
// are read once from HBM.
//
// Work split: a 512-thread workgroup owns 16 output features.  The
// contraction runs in tiles of 8 k-blocks (256 k); in each tile wave w owns
// k-block w.  All three operand streams of a tile
//   W      16 features x 256 k  bf16       8 KB
//   signs  16 tenant slots x 16 features x 8 words  8 KB
//   x      16*MB rows x 256 k    bf16      8 KB per 16 rows
// are copied global -> LDS with global_load_lds_dwordx4 (no register staging)
// into a ring of NB tile buffers, NB-1 tiles ahead of the tile being
// computed.  Every wave issues the same number of copies per tile in a fixed
// order, so one s_waitcnt vmcnt((NB-2)*ops_per_tile) plus a barrier makes a
// tile visible without draining the copies still in flight (the memory
// counter retires loads in issue order).  MFMA operands are then read from
// LDS: W as B for x*W^T (A = 16-row blocks of x), and for each tenant block
// the sign bytes are decoded in registers into bf16 +1/-1 B operands
// against its rows of x gathered as A (decode_signs8).
//
// Tenant routing: wave 0 groups the rows by tenant id with ballots (one per
// distinct tenant) into blocks of up to 16 rows, 16 blocks per pass; a pass
// covering more than 16 blocks re-streams x and signs (rare: > 16 blocks needs
// more than 16 tenants or tenants with many rows).
//
// Rows of x are placed in LDS with their 16-byte chunks XOR-swizzled by the
// row index, so fragment reads of 16 consecutive rows hit distinct banks.
// Partial sums of the 8 waves are added in a fixed order: results are bitwise
// deterministic.
#include "device.h"
#include "internal.h"
#include "ldscopy.h"

namespace bitdelta {
namespace {

constexpr int kFeat = 16;
constexpr int kWaves = 8;
constexpr int kTileBlocks = 8;          // k-blocks per tile (one per wave)
constexpr int kRowBytes = kTileBlocks * 64;   // 512 B: one row of a tile
constexpr int kSlots = 16;              // tenant slots per pass
constexpr int kBlocksPerPass = 16;      // tenant blocks per pass
constexpr int kRowsMax = 64;

template <int MB>
struct MultiCfg {
    static constexpr int kWBytes = kFeat * kRowBytes;                 // 8 KB
    static constexpr int kSBytes = kSlots * kFeat * 32;               // 8 KB
    static constexpr int kXBytes = MB * 16 * kRowBytes;               // 8 KB per 16 rows
    static constexpr int kTileBytes = kWBytes + kSBytes + kXBytes;
    static constexpr int kNB = MB == 1 ? 6 : (MB == 2 ? 4 : 3);       // ring depth
    static constexpr int kRingBytes = kNB * kTileBytes;
    static constexpr int kOpsPerTile = 1 + 1 + MB;                    // W + S + x copies per wave
    static constexpr int kRedBytes = 2 * kWaves * kRowsMax * kFeat * 4;
    static constexpr int kLdsBytes = kRingBytes > kRedBytes ? kRingBytes : kRedBytes;
};

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ (row & 15); }

template <int MB>
__global__ __launch_bounds__(kWaves * 64) void multi_kernel(
    const uint16_t* __restrict__ x, int M, int K, const uint16_t* __restrict__ w, int N,
    const uint32_t* __restrict__ packed, const float* __restrict__ alpha,
    const int32_t* __restrict__ tenant_ids, int T, void* __restrict__ y, int y_dtype) {
    using C = MultiCfg<MB>;
    constexpr int NB = C::kNB;
    constexpr int D = NB - 1;                  // tiles in flight ahead of the one computed
    __shared__ __attribute__((aligned(16))) char ring[C::kLdsBytes];
    __shared__ int row_tenant[kRowsMax];       // tenant of row m, -1 = id out of range
    __shared__ int row_block[kRowsMax];        // tenant block of row m, -1 = none
    __shared__ int blk_rows[kRowsMax][16];     // gathered row of each block slot, -1 = empty
    __shared__ int blk_tenant[kRowsMax];
    __shared__ int pass_slot_tenant[kSlots];   // tenant held in each slot of this pass
    __shared__ int blk_slot[kBlocksPerPass];   // slot of each block of this pass
    __shared__ int nblk_sh;
    __shared__ float sign_sum[kRowsMax][kFeat];

    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nl = lane & 15, g = lane >> 4;
    const int n0 = blockIdx.x * kFeat;
    const int KB = K >> 5, KW = K >> 5;
    const int KT = (KB + kTileBlocks - 1) / kTileBlocks;

    // ---- group rows by tenant (wave 0): ballots, one per distinct tenant ----
    if (wv == 0) {
        int t = -2;
        if (lane < M) {
            t = tenant_ids[lane];
            if (t < 0 || t >= T) t = -1;
        }
        row_tenant[lane] = t;
        row_block[lane] = -1;
#pragma unroll
        for (int i = 0; i < 16; ++i) blk_rows[lane][i] = -1;
        unsigned long long remaining = __ballot(t >= 0);
        int nb = 0;
        while (remaining) {
            const int leader = __ffsll((long long)remaining) - 1;
            const int tl = __shfl(t, leader);
            const unsigned long long grp = __ballot(t == tl) & remaining;
            remaining &= ~grp;
            if ((grp >> lane) & 1ull) {
                const int rank = __popcll(grp & ((1ull << lane) - 1ull));
                blk_rows[nb + rank / 16][rank % 16] = lane;
                row_block[lane] = nb + rank / 16;
                if (rank % 16 == 0) blk_tenant[nb + rank / 16] = tl;
            }
            nb += (__popcll(grp) + 15) / 16;
        }
        if (lane == 0) nblk_sh = nb;
    }
    __syncthreads();
    const int nblk = nblk_sh;

    f32x4 accb[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) accb[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // copy sources that do not depend on the tile
    //   W: this wave copies features 2*wv, 2*wv+1; lane -> (feature, chunk slot)
    const int wf = 2 * wv + (lane >> 5), wslot = lane & 31;
    const int wchunk = swz(wf, wslot);
    const uint16_t* wsrc = w + (size_t)min(n0 + wf, N - 1) * K;
    //   x: this wave copies rows 2*(wv*MB + i) + lane/32 for i < MB
    //   signs: slots 2*wv, 2*wv+1; lane -> (slot, feature, half)
    //   (LDS layout [slot][half][feature][16 B]: conflict-free byte reads)
    const int sslot = 2 * wv + (lane >> 5), shalf = (lane >> 4) & 1, sfeat = lane & 15;
    const int sn = min(n0 + sfeat, N - 1);

    for (int p0 = 0; p0 == 0 || p0 < nblk; p0 += kBlocksPerPass) {
        const bool first_pass = (p0 == 0);
        // ---- tenant slots of this pass (one thread) ----
        if (threadIdx.x == 0) {
            int nslot = 0, prev = -1;
            for (int b = 0; b < kBlocksPerPass; ++b) {
                const int blk = p0 + b;
                if (blk < nblk) {
                    const int t = blk_tenant[blk];
                    if (t != prev) { pass_slot_tenant[nslot++] = t; prev = t; }
                    blk_slot[b] = nslot - 1;
                } else {
                    blk_slot[b] = 0;
                }
            }
            if (nslot == 0) pass_slot_tenant[nslot++] = 0;
            for (int s = nslot; s < kSlots; ++s) pass_slot_tenant[s] = pass_slot_tenant[nslot - 1];
        }
        __syncthreads();
        const int nb_pass = min(kBlocksPerPass, max(0, nblk - p0));
        const uint32_t* ssrc = packed + ((size_t)pass_slot_tenant[sslot] * N + sn) * KW;

        // Copies of tile tt into ring buffer tt % NB: W, signs, x (fixed order and count).
        auto issue_tile = [&](int tt) {
            const int tc = min(tt, KT - 1);                      // tail tiles repeat the last one
            char* buf = ring + (tt % NB) * C::kTileBytes;
            const int kb_w = min(tc * kTileBlocks + (wchunk >> 2), KB - 1);
            copy16_to_lds(wsrc + (size_t)kb_w * 32 + 8 * (wchunk & 3),
                          buf + wv * 1024);
            const int kw0 = min(tc * kTileBlocks + 4 * shalf, max(KW - 4, 0));
            copy16_to_lds(ssrc + kw0, buf + C::kWBytes + wv * 1024);
#pragma unroll
            for (int i = 0; i < MB; ++i) {
                const int xr = 2 * (wv * MB + i) + (lane >> 5);
                const int xc = swz(xr, wslot);
                const int kb_x = min(tc * kTileBlocks + (xc >> 2), KB - 1);
                copy16_to_lds(x + (size_t)min(xr, M - 1) * K + (size_t)kb_x * 32 + 8 * (xc & 3),
                              buf + C::kWBytes + C::kSBytes + (wv * MB + i) * 1024);
            }
            // the vmcnt arithmetic assumes each tile's copies are issued as one group
            __builtin_amdgcn_sched_barrier(0);
        };

        // One pass over K for NBP tenant blocks (NBP >= nb_pass; the extra
        // blocks are inert: their x reads are masked off and results dropped).
        auto run_pass = [&](auto nbp_tag) {
            constexpr int NBP = decltype(nbp_tag)::value;
            // Tile-invariant LDS byte offsets of this lane's operands.  Padding
            // slots of a tenant block read row 0: they only feed output rows
            // that are dropped, so no masking is needed.
            const int c = 4 * wv + g;                            // logical chunk of this lane
            int xoff[NBP], soff[NBP];
            f32x4 accs[NBP];
#pragma unroll
            for (int b = 0; b < NBP; ++b) {
                const int r0 = (b < nb_pass) ? blk_rows[p0 + b][nl] : -1;
                const int r = r0 < 0 ? 0 : r0;
                xoff[b] = r * kRowBytes + 16 * swz(r, c);
                soff[b] = __builtin_amdgcn_readfirstlane(blk_slot[b]) * (kFeat * 32) +
                          (wv >> 2) * (kFeat * 16) + nl * 16 + 4 * (wv & 3) + g;
                accs[b] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
            int boff[MB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) boff[mb] = (mb * 16 + nl) * kRowBytes + 16 * swz(mb * 16 + nl, c);
            const int woff = nl * kRowBytes + 16 * swz(nl, c);

            // Each pass starts on an idle ring: all earlier reads are behind a barrier.
            __syncthreads();
#pragma unroll
            for (int i = 0; i < D; ++i) issue_tile(i);
            for (int t = 0; t < KT; ++t) {
                // tile t was issued D tiles ago; D-1 tiles of copies may stay in flight
                wait_vm_lgkm0<(D - 1) * C::kOpsPerTile>();
                raw_barrier();
                issue_tile(t + D);      // into the buffer of tile t-1, free after the barrier
                if (t * kTileBlocks + wv < KB) {
                    const char* buf = ring + (t % NB) * C::kTileBytes;
                    const char* sl = buf + C::kWBytes;
                    const char* xl = buf + C::kWBytes + C::kSBytes;
                    if (first_pass) {
                        const u32x4 bw = *reinterpret_cast<const u32x4*>(buf + woff);
#pragma unroll
                        for (int mb = 0; mb < MB; ++mb)
                            accb[mb] = mfma16(*reinterpret_cast<const u32x4*>(xl + boff[mb]), bw, accb[mb]);
                    }
                    // tenant blocks in chunks of 8: the chunk's LDS reads first,
                    // then its decodes and MFMAs
                    constexpr int CH = NBP < 8 ? NBP : 8;
#pragma unroll
                    for (int b0 = 0; b0 < NBP; b0 += CH) {
                        u32x4 ga[CH];
                        uint32_t sb[CH];
#pragma unroll
                        for (int i = 0; i < CH; ++i) {
                            sb[i] = *reinterpret_cast<const uint8_t*>(sl + soff[b0 + i]);
                            ga[i] = *reinterpret_cast<const u32x4*>(xl + xoff[b0 + i]);
                        }
#pragma unroll
                        for (int i = 0; i < CH; ++i) accs[b0 + i] = mfma16(ga[i], decode_signs8(sb[i]), accs[b0 + i]);
                    }
                }
            }
            // drain the tail copies before the ring is reused
            wait_vm_lgkm0<0>();
            __syncthreads();

            // ---- reduce this pass's sign partials into sign_sum (fixed wave order) ----
            float* red = reinterpret_cast<float*>(ring);          // [wave][row][feat]
#pragma unroll
            for (int b = 0; b < NBP; ++b) {
                if (b < nb_pass) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int row = blk_rows[p0 + b][4 * g + r];
                        if (row >= 0) red[(wv * kRowsMax + row) * kFeat + nl] = accs[b][r];
                    }
                }
            }
        };
        if (nb_pass <= 2)
            run_pass(std::integral_constant<int, 2>{});
        else if (nb_pass <= 4)
            run_pass(std::integral_constant<int, 4>{});
        else if (nb_pass <= 8)
            run_pass(std::integral_constant<int, 8>{});
        else
            run_pass(std::integral_constant<int, 16>{});
        __syncthreads();
        {
            const float* red = reinterpret_cast<const float*>(ring);
            for (int idx = threadIdx.x; idx < kRowsMax * kFeat; idx += kWaves * 64) {
                const int m = idx / kFeat, f = idx % kFeat;
                const int blk = row_block[m];
                if (m < M && blk >= p0 && blk < p0 + kBlocksPerPass) {
                    float s = 0.f;
#pragma unroll
                    for (int v = 0; v < kWaves; ++v) s += red[(v * kRowsMax + m) * kFeat + f];
                    sign_sum[m][f] = s;
                }
            }
        }
        __syncthreads();
    }

    // ---- base partials, then the epilogue ----
    float* red = reinterpret_cast<float*>(ring);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[(wv * kRowsMax + mb * 16 + 4 * g + r) * kFeat + nl] = accb[mb][r];
    __syncthreads();
    for (int idx = threadIdx.x; idx < MB * 16 * kFeat; idx += kWaves * 64) {
        const int m = idx / kFeat, f = idx % kFeat;
        const int nn = n0 + f;
        if (m >= M || nn >= N) continue;
        const int t = row_tenant[m];
        float out;
        if (t < 0) {
            out = __builtin_nanf("");
        } else {
            float b = 0.f;
#pragma unroll
            for (int v = 0; v < kWaves; ++v) b += red[(v * kRowsMax + m) * kFeat + f];
            out = __builtin_fmaf(alpha[t], sign_sum[m][f], b);
        }
        if (y_dtype == kF32)
            reinterpret_cast<float*>(y)[(size_t)m * N + nn] = out;
        else
            reinterpret_cast<uint16_t*>(y)[(size_t)m * N + nn] = to_bf16(out);
    }
}

template <int MB>
hipError_t launch_mb(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                     const uint32_t* packed, const float* alpha, const int32_t* tenant_ids, int T,
                     void* y, int y_dtype, hipStream_t stream) {
    const int grid = (N + kFeat - 1) / kFeat;
    multi_kernel<MB><<<grid, kWaves * 64, 0, stream>>>(x, M, K, w, N, packed, alpha, tenant_ids,
                                                       T, y, y_dtype);
    return hipGetLastError();
}

}  // namespace

bool multi_supported(int K) { return K >= 128 && (K & 127) == 0; }

hipError_t launch_multi(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                        const uint32_t* packed, const float* alpha, const int32_t* tenant_ids,
                        int T, void* y, int y_dtype, hipStream_t stream) {
    switch ((M + 15) / 16) {
        case 1: return launch_mb<1>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
        case 2: return launch_mb<2>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
        case 3: return launch_mb<3>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
        default: return launch_mb<4>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
    }
}

}  // namespace bitdelta
