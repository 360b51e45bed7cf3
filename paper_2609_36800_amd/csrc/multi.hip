// Batched (multi-tenant) binary-delta matmul for at most 64 token rows:
//
//   y[m][n] = sum_k x[m][k] W[n][k] + alpha[t(m)] * sum_k x[m][k] s_t(m)[n][k]
//
// (the batched BitDelta GEMM of Section 4.4).  Row m selects its tenant's
// sign matrix by id; every W byte and the sign bytes of each tenant present
// are read once from HBM.
//
// Work split: a 256-thread workgroup owns 16 output features, and two
// workgroups share a CU (about 70 KB of LDS each), so one can compute while
// the other waits on memory.  The contraction runs in tiles of 4 k-blocks
// (128 k); in each tile wave w owns k-block w.  The operand streams of a tile
//   W      16 features x 128 k  bf16                     4 KB
//   signs  P tenant slots x 16 features x 4 words        P x 256 B
//   x      16*MB rows x 128 k    bf16                    4 KB per 16 rows
// are copied global -> LDS by the DMA path (no register staging) into a ring
// of NB tile buffers, NB-1 tiles ahead of the tile being computed.  Every
// wave issues the same number of copies per tile in a fixed order, so one
// s_waitcnt vmcnt((NB-2)*ops_per_tile) plus a barrier makes a tile visible
// without draining the copies still in flight (the memory counter retires
// loads in issue order).  Only the slots a pass needs are staged (P = 4, 8
// or 16).
//
// Per k-block a wave reads the x fragments of all rows once (A operands, 16
// rows each) and the W fragment (B operand of x*W^T).  Each tenant slot's
// sign bytes are then decoded in registers into bf16 +1/-1 B operands
// (decode_signs8) and multiplied against every row fragment: the x
// fragments are reused from registers for all tenants, and the rows of other
// tenants are discarded at the end, where each row takes the accumulator of
// its own slot.  A pass covers up to 16 slots (8 for more than 32 rows, to
// bound the accumulators); more distinct tenants re-stream x and signs.
//
// Rows of x are placed in LDS with their 16-byte chunks XOR-swizzled by the
// row index, so fragment reads of 16 consecutive rows hit distinct banks.
// Partial sums of the 4 waves are added in a fixed order: results are bitwise
// deterministic.
#include "device.h"
#include "internal.h"
#include "ldscopy.h"

namespace bitdelta {
namespace {

constexpr int kFeat = 16;
constexpr int kWaves = 4;
constexpr int kTileBlocks = 4;                // k-blocks per tile (one per wave)
constexpr int kRowBytes = kTileBlocks * 64;   // 256 B: one row of a tile
constexpr int kSlotBytes = kFeat * 16;        // 256 B: one slot's sign words of a tile
constexpr int kRowsMax = 64;
constexpr int kMaxSlots = 16;
constexpr int kRingBytes = 68 * 1024;         // two workgroups per CU

// MB: 16-row fragments of x; P: tenant slots staged per tile.
template <int MB, int P>
struct MultiCfg {
    static constexpr int kWBytes = kFeat * kRowBytes;                 // 4 KB
    static constexpr int kSBytes = P * kSlotBytes;
    static constexpr int kXBytes = MB * 16 * kRowBytes;               // 4 KB per 16 rows
    static constexpr int kTileBytes = kWBytes + kSBytes + kXBytes;
    static constexpr int kNB = kRingBytes / kTileBytes < 6 ? kRingBytes / kTileBytes : 6;
    static constexpr int kSOps = P == 16 ? 1 : P / 4;                 // sign copies per wave
    static constexpr int kOps = 1 + kSOps + MB;                       // W + signs + x copies per wave
    static_assert(kNB >= 3, "ring too shallow");
};

// slots computed per pass: the accumulators stay at 4 * MB * slots <= 128
template <int MB>
constexpr int pass_slots() { return MB <= 2 ? 16 : 8; }

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ (row & 15); }

template <int ET, int MB>
__global__ __launch_bounds__(kWaves * 64, 2) void multi_kernel(
    const uint16_t* __restrict__ x, int M, int K, const uint16_t* __restrict__ w, int N,
    const uint32_t* __restrict__ packed, const float* __restrict__ alpha,
    const int32_t* __restrict__ tenant_ids, int T, void* __restrict__ y, int y_dtype) {
    constexpr int PS = pass_slots<MB>();
    static_assert(kRingBytes >= 2 * kWaves * kRowsMax * kFeat * 4, "reduction area must fit");
    __shared__ __attribute__((aligned(16))) char ring[kRingBytes];
    __shared__ int row_tenant[kRowsMax];       // tenant of row m, -1 = id out of range
    __shared__ int row_slot[kRowsMax];         // distinct-tenant slot of row m, -1 = none
    __shared__ int slot_tenant[kRowsMax];      // tenant of each slot
    __shared__ int pass_slot_tenant[kMaxSlots];
    __shared__ int nslot_sh;
    __shared__ float sign_sum[kRowsMax][kFeat];

    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nl = lane & 15, g = lane >> 4;
    const int n0 = blockIdx.x * kFeat;
    const int KB = K >> 5, KW = K >> 5;
    const int KT = (KB + kTileBlocks - 1) / kTileBlocks;

    // ---- distinct tenants (wave 0): ballots, one per distinct tenant ----
    if (wv == 0) {
        int t = -2;
        if (lane < M) {
            t = tenant_ids[lane];
            if (t < 0 || t >= T) t = -1;
        }
        row_tenant[lane] = t;
        int my_slot = -1;
        unsigned long long remaining = __ballot(t >= 0);
        int ns = 0;
        while (remaining) {
            const int leader = __ffsll((long long)remaining) - 1;
            const int tl = __shfl(t, leader);
            const unsigned long long grp = __ballot(t == tl) & remaining;
            remaining &= ~grp;
            if ((grp >> lane) & 1ull) my_slot = ns;
            if (lane == 0) slot_tenant[ns] = tl;
            ++ns;
        }
        row_slot[lane] = my_slot;
        if (lane == 0) nslot_sh = ns;
    }
    __syncthreads();
    const int nslot = nslot_sh;

    f32x4 accb[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) accb[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // ---- copy assignment (tile-invariant parts): lane -> (row, chunk slot) ----
    const int cslot = lane & 15, crow = lane >> 4;
    const int wf = 4 * wv + crow;                                // W: features 4wv .. 4wv+3
    const int wchunk = swz(wf, cslot);
    const uint16_t* wsrc = w + (size_t)min(n0 + wf, N - 1) * K + 8 * (wchunk & 3);
    const int wkb = wchunk >> 2;

    // ---- fragment offsets: A row / B column nl, k-slots 8g .. 8g+7 of k-block wv ----
    const int c = 4 * wv + g;
    int xoff[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) xoff[mb] = (mb * 16 + nl) * kRowBytes + 16 * swz(mb * 16 + nl, c);
    const int woff = nl * kRowBytes + 16 * swz(nl, c);
    const int soff = nl * 16 + 4 * wv + g;                       // sign byte in a slot's block

    for (int p0 = 0; p0 == 0 || p0 < nslot; p0 += PS) {
        const bool first_pass = (p0 == 0);
        if (threadIdx.x < kMaxSlots) {
            const int sl = min(p0 + (int)threadIdx.x, nslot - 1);
            pass_slot_tenant[threadIdx.x] = sl >= 0 ? slot_tenant[sl] : 0;
        }
        __syncthreads();
        const int ns_pass = min(PS, max(0, nslot - p0));

        // One pass over K for P staged slots (P >= ns_pass; surplus slots hold
        // copies of a real tenant and their results are never selected).
        auto run_pass = [&](auto p_tag) {
            constexpr int P = decltype(p_tag)::value;
            using C = MultiCfg<MB, P>;
            constexpr int NB = C::kNB;
            constexpr int D = NB - 1;                  // tiles in flight ahead of the one computed

            // sign-copy sources: P = 16 -> 16 B per lane (slots 4wv .. 4wv+3,
            // 4 words = the tile's 4 k-blocks); P = 8, 4 -> 4 B per lane
            const uint32_t* ssrc[C::kSOps];
            int sdst[C::kSOps];
#pragma unroll
            for (int j = 0; j < C::kSOps; ++j) {
                if constexpr (P == 16) {
                    const int sl = 4 * wv + (lane >> 4), ft = lane & 15;
                    ssrc[j] = packed + ((size_t)pass_slot_tenant[sl] * N + min(n0 + ft, N - 1)) * KW;
                    sdst[j] = wv * 1024;
                } else {
                    const int sl = wv * C::kSOps + j, ft = lane >> 2;
                    ssrc[j] = packed + ((size_t)pass_slot_tenant[sl] * N + min(n0 + ft, N - 1)) * KW + (lane & 3);
                    sdst[j] = sl * kSlotBytes;
                }
            }

            auto issue_tile = [&](int tt) {
                const int tc = min(tt, KT - 1);                      // tail tiles repeat the last one
                char* buf = ring + (tt % NB) * C::kTileBytes;
                // later passes re-read a fixed W tile (cached) to keep the copy count
                const int kb_w = first_pass ? min(tc * kTileBlocks + wkb, KB - 1) : 0;
                if (first_pass) copy16_to_lds_nt(wsrc + (size_t)kb_w * 32, buf + wv * 1024);
                else copy16_to_lds(wsrc + (size_t)kb_w * 32, buf + wv * 1024);
                const int kw0 = min(tc * kTileBlocks, KW - 4);       // K is a multiple of 128
#pragma unroll
                for (int j = 0; j < C::kSOps; ++j) {
                    if constexpr (P == 16)
                        copy16_to_lds(ssrc[j] + kw0, buf + C::kWBytes + sdst[j]);
                    else
                        copy4_to_lds(ssrc[j] + kw0, buf + C::kWBytes + sdst[j]);
                }
#pragma unroll
                for (int i = 0; i < MB; ++i) {
                    const int xr = 4 * (wv * MB + i) + crow;
                    const int xc = swz(xr, cslot);
                    const int kb_x = min(tc * kTileBlocks + (xc >> 2), KB - 1);
                    copy16_to_lds(x + (size_t)min(xr, M - 1) * K + (size_t)kb_x * 32 + 8 * (xc & 3),
                                  buf + C::kWBytes + C::kSBytes + (wv * MB + i) * 1024);
                }
                // the vmcnt arithmetic assumes each tile's copies are issued as one group
                __builtin_amdgcn_sched_barrier(0);
            };

            f32x4 accs[P][MB];
#pragma unroll
            for (int s0 = 0; s0 < P; ++s0)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) accs[s0][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

            // Each pass starts on an idle ring: all earlier reads are behind a barrier.
            __syncthreads();
#pragma unroll
            for (int i = 0; i < D; ++i) issue_tile(i);
            for (int t = 0; t < KT; ++t) {
                // tile t was issued D tiles ago; D-1 tiles of copies may stay in flight
                wait_vm_lgkm0<(D - 1) * C::kOps>();
                raw_barrier();
                issue_tile(t + D);      // into the buffer of tile t-1, free after the barrier
                if (t * kTileBlocks + wv < KB) {
                    const char* buf = ring + (t % NB) * C::kTileBytes;
                    const char* sl = buf + C::kWBytes;
                    const char* xl = buf + C::kWBytes + C::kSBytes;
                    u32x4 xa[MB];
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) xa[mb] = *reinterpret_cast<const u32x4*>(xl + xoff[mb]);
                    if (first_pass) {
                        const u32x4 bw = *reinterpret_cast<const u32x4*>(buf + woff);
#pragma unroll
                        for (int mb = 0; mb < MB; ++mb) accb[mb] = mfma16<ET>(xa[mb], bw, accb[mb]);
                    }
                    // slots in chunks: the chunk's sign-byte reads first, then
                    // its decodes and MFMAs
                    constexpr int CH = (P < 8 || MB >= 3) ? 4 : 8;
#pragma unroll
                    for (int s0 = 0; s0 < P; s0 += CH) {
                        uint32_t sb[CH];
#pragma unroll
                        for (int i = 0; i < CH; ++i)
                            sb[i] = *reinterpret_cast<const uint8_t*>(sl + (s0 + i) * kSlotBytes + soff);
#pragma unroll
                        for (int i = 0; i < CH; ++i) {
                            const u32x4 bs = decode_signs8<ET>(sb[i]);
#pragma unroll
                            for (int mb = 0; mb < MB; ++mb) accs[s0 + i][mb] = mfma16<ET>(xa[mb], bs, accs[s0 + i][mb]);
                        }
                    }
                }
            }
            // drain the tail copies before the ring is reused
            wait_vm_lgkm0<0>();
            __syncthreads();

            // ---- each row keeps its own slot's sums: red[wave][row][feature] ----
            float* red = reinterpret_cast<float*>(ring);
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = mb * 16 + 4 * g + r;
                    const int rs = row_slot[row] - p0;
                    float v = 0.f;
#pragma unroll
                    for (int s0 = 0; s0 < P; ++s0) v = (rs == s0) ? accs[s0][mb][r] : v;
                    if (rs >= 0 && rs < ns_pass) red[(wv * kRowsMax + row) * kFeat + nl] = v;
                }
        };
        if (ns_pass <= 4)
            run_pass(std::integral_constant<int, 4>{});
        else if (PS == 8 || ns_pass <= 8)
            run_pass(std::integral_constant<int, 8>{});
        else
            run_pass(std::integral_constant<int, (PS > 8 ? 16 : 8)>{});
        __syncthreads();
        {
            const float* red = reinterpret_cast<const float*>(ring);
            for (int idx = threadIdx.x; idx < MB * 16 * kFeat; idx += kWaves * 64) {
                const int m = idx / kFeat, f = idx % kFeat;
                const int rs = row_slot[m] - p0;
                if (m < M && rs >= 0 && rs < ns_pass) {
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
        store_y<ET>(y, (size_t)m * N + nn, out, y_dtype);
    }
}

template <int ET, int MB>
hipError_t launch_mb(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                     const uint32_t* packed, const float* alpha, const int32_t* tenant_ids, int T,
                     void* y, int y_dtype, hipStream_t stream) {
    const int grid = (N + kFeat - 1) / kFeat;
    multi_kernel<ET, MB><<<grid, kWaves * 64, 0, stream>>>(x, M, K, w, N, packed, alpha, tenant_ids,
                                                       T, y, y_dtype);
    return hipGetLastError();
}

template <int ET>
hipError_t launch_multi_et(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                           const uint32_t* packed, const float* alpha, const int32_t* tenant_ids,
                           int T, void* y, int y_dtype, hipStream_t stream) {
    switch ((M + 15) / 16) {
        case 1: return launch_mb<ET, 1>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
        case 2: return launch_mb<ET, 2>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
        case 3: return launch_mb<ET, 3>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
        default: return launch_mb<ET, 4>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
    }
}

}  // namespace

bool multi_supported(int K) { return K >= 128 && (K & 127) == 0; }

hipError_t launch_multi(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                        const uint32_t* packed, const float* alpha, const int32_t* tenant_ids,
                        int T, void* y, int y_dtype, int et, hipStream_t stream) {
    if (et == kF16)
        return launch_multi_et<kF16>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
    return launch_multi_et<kBF16>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
}

}  // namespace bitdelta
