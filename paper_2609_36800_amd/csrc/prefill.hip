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
// Two kernels share that contraction and the output tiling:
//
// prefill_stream_kernel (K a multiple of 64; the common case).  A 256-thread
// workgroup (4 waves, 2x2) owns a 256x256 output tile, each wave 128x128 =
// 4x4 v_mfma_f32_32x32x16_bf16 tiles (256 fp32 accumulators per lane).  Per
// 64-wide k-tile:
//   * the x tile goes global -> LDS by direct copies (no registers), into
//     one of two LDS buffers as soon as the barrier frees it, a tile ahead
//     of its use; one explicit vmcnt wait before the next barrier covers
//     them (measured 4% faster in bf16 than staging x through registers);
//   * the raw W tile and its sign words are loaded into registers two tiles
//     ahead (buffer loads: 32-bit per-lane offsets, the k offset in a scalar
//     register; two register sets), and the effective weights of the next
//     tile are formed and written to the other of two LDS buffers while the
//     matrix cores work on the current one: the 64 MFMAs of a k-tile are
//     issued one per scheduling slot, and each slot carries a share of the
//     decode (one bf16 pair), the LDS writes and the next loads;
//   * one barrier per k-tile publishes both buffers.
// The two LDS buffers of each operand are separate objects so the compiler
// can tell a write into one from a read of the other and count the writes
// exactly when it places its waits.
// Every W element is decoded once per workgroup; with alpha's sign moved onto
// W (s*W + alpha, rounded, then the sign restored -- round-to-nearest-even is
// symmetric) all eight weights of a chunk add the same alpha.
//
// prefill_general_kernel (any K that is a multiple of 32): the same tiling
// with both operands staged through registers and zero-filled past K.
//
// LDS rows are 128 bytes (64 bf16).  Chunk c of row r is stored at slot
// c ^ f(r), f(r) = (r & 7) ^ ((r >> 3) & 1): the 16-byte fragment reads of 16
// consecutive rows then fall in distinct bank groups whether LDS serves 8 or
// 16 lanes of a 128-bit read per cycle.
//
// Workgroups are renumbered so that the 32 resident on one XCD (the hardware
// deals workgroups round-robin over the 8 XCDs) cover a 4 x 8 block of tiles
// and share their x and W panels in that XCD's L2.
#include <type_traits>

#include "device.h"
#include "internal.h"
#include "ldscopy.h"

namespace bitdelta {
namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kCUs = 256;            // MI355X compute units (one output tile each per round)
constexpr int kThreads = 256;
constexpr int kChunks = BM * BK / 8 / kThreads;  // 16-byte chunks per thread per operand = 8
constexpr int kGroupM = 4;

struct PrefillLds {
    uint16_t a[2][BM * BK];
    uint16_t b[2][BN * BK];
};

__device__ __forceinline__ int lds_off(int row, int chunk) {
    return row * BK + ((chunk ^ (row & 7) ^ ((row >> 3) & 1)) << 3);
}

template <int ET>
__global__ __launch_bounds__(kThreads, 1) void prefill_general_kernel(
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
    // bf16: fp32 bits of -alpha; fp16: the pair (fp16(-alpha), fp16(-alpha))
    uint32_t neg_alpha;
    if constexpr (ET == kF16) {
        const uint32_t h = to_f16(-alpha[0]);
        neg_alpha = h | (h << 16);
    } else {
        neg_alpha = __builtin_bit_cast(uint32_t, -alpha[0]);
    }

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
            const uint32_t byte = (rs[i] >> (8 * (q & 3))) & 0xFFu;
            u32x4 fused;
            if constexpr (ET == kF16) fused = fuse_weights8_f16(rb[i], byte, neg_alpha);
            else fused = fuse_weights8(rb[i], byte, neg_alpha);
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
                for (int j = 0; j < 4; ++j) acc[i][j] = mfma32<ET>(af[i], bf[j], acc[i][j]);
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
                if (row < M && col < N) store_y<ET>(y, (size_t)row * N + col, acc[i][j][r], y_dtype);
            }
        }
}

// ------------------------------------------------------------ streaming kernel

// Output-tile assignment (XCD-aware, groups of kGroupM tile rows) of block
// `bid` < tiles_m * tiles_n.
__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int& tile_m, int& tile_n) {
    const int nwg = tiles_m * tiles_n;
    if ((nwg & 7) == 0) bid = (bid & 7) * (nwg >> 3) + (bid >> 3);
    const int group = bid / (kGroupM * tiles_n);
    const int first_m = group * kGroupM;
    const int gm = min(tiles_m - first_m, kGroupM);
    const int local = bid - group * kGroupM * tiles_n;
    tile_m = first_m + local % gm;
    tile_n = local / gm;
}

// ---------------------------------------------------- batched (grouped) form
//
// With a tenant id per row the fused GEMM runs once per tenant over that
// tenant's rows (the batched BitDelta GEMM of Section 4.4): the rows of tenant
// t, in increasing row order, form ceil(c_t / 256) row tiles, numbered tenant
// by tenant, and each output tile decodes its own tenant's effective weights.
// Every workgroup routes the rows itself, so no scratch memory and no extra
// launch are needed: it histograms the ids (one histogram per wave over a
// quarter of the rows, in LDS that the operand buffers reuse afterwards),
// scans the per-tenant tile counts, picks its tile from its block index (the
// number of tiles is known only on the device, so the grid covers the upper
// bound and surplus workgroups leave), and collects its tile's row indices.
constexpr int kMaxGroupedTenants = BM * BK * 2 / (4 * 4);  // 4 histograms of T ints in 32 KB
constexpr size_t kSplitChunkBytes = (size_t)BM * BN * 4;   // fp32 partial sums of one tile
constexpr int kSplitVecs = 4 * 4 * 4;                       // f32x4 partials per thread
constexpr int kSplitMetaInts = BM + 4;                      // row map, column origin, counts

// Work items.  With at most kCUs output tiles (or no room for partial sums)
// block b takes tile b.  With more tiles, blocks 0 .. kCUs-1 take tiles 0 ..
// kCUs-1 whole (one round), and the L leftover tiles are split along K into
// S chunks, S = min(8, k-tiles, room / L, kCUs / L): blocks kCUs + l*S + c
// take chunk c of leftover tile l, so the second round runs on every CU for
// 1/S of a tile's time.  A chunk's fp32 partial sums go to `part`, and the
// reduction launch that follows adds the S partials of a tile in chunk order
// and writes its rows, so the result does not depend on timing.
struct WorkItem {
    int chunk, nchunks, leftover;   // chunk c of nchunks (1: whole tile); leftover tile index
    int nleft;                      // leftover tiles (split ones)
};

__device__ __forceinline__ int split_chunks(int ntiles, int room, int KT) {
    if (ntiles <= kCUs || room <= 0) return 1;
    const int L = ntiles - kCUs;
    const int cap = room < kCUs ? room : kCUs;
    int S = cap / L;
    S = S < 8 ? S : 8;
    S = S < KT ? S : KT;
    return S > 1 ? S : 1;
}

// Returns false (for the whole workgroup) when block `bid` owns no work;
// else `tenant`, `tile_n`, the work item and rows[0..255] (row index, -1 past
// the tenant's last row).  hist: 4*T ints of LDS; info: 8 ints of LDS.
// room: leftover chunks the partial-sum buffer holds (0: none).
__device__ bool route_rows(const int32_t* __restrict__ ids, int M, int T, int tiles_n, int bid,
                           int room, int KT, int* split_hdr, int* hist, int* rows, int* info, int& tenant,
                           int& tile_n, WorkItem& item) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int seg = ((M + 255) >> 8) << 6;  // rows per wave, a multiple of 64
    const int r_beg = min(M, seg * wv), r_end = min(M, seg * (wv + 1));

    int* h = hist + wv * T;
    for (int i = lane; i < T; i += 64) h[i] = 0;
    // the ids of 1024 rows per step, all loads issued together; the first
    // step's stay in registers for the row collection below
    constexpr int kIdRegs = 16;
    auto load_ids = [&](int base, int (&v)[kIdRegs]) {
#pragma unroll
        for (int u = 0; u < kIdRegs; ++u) {
            const int m = base + 64 * u + lane;
            v[u] = m < r_end ? ids[m] : -1;
        }
    };
    // a 64-row run of one id (prompts are runs of rows) is one LDS add, not
    // 64 adds to one address
    auto add_hist = [&](const int (&v)[kIdRegs]) {
#pragma unroll
        for (int u = 0; u < kIdRegs; ++u) {
            const int f = __builtin_amdgcn_readfirstlane(v[u]);
            if (__ballot(v[u] != f) == 0) {
                if (lane == 0 && (unsigned)f < (unsigned)T) atomicAdd(&h[f], 64);
            } else if ((unsigned)v[u] < (unsigned)T) {
                atomicAdd(&h[v[u]], 1);
            }
        }
    };
    int idr[kIdRegs];
    load_ids(r_beg, idr);
    __syncthreads();
    add_hist(idr);
    for (int base = r_beg + 64 * kIdRegs; base < r_end; base += 64 * kIdRegs) {
        int v[kIdRegs];
        load_ids(base, v);
        add_hist(v);
    }
    __syncthreads();

    // Row tiles, in this order: every tenant's full (256-row) tiles, tenant by
    // tenant; then the tenants' last, partly filled tiles, in eight classes of
    // decreasing row count (224-255 rows, 192-223, ..., 1-31), tenant by tenant
    // within a class.  So the row tiles at the end -- the ones split when there
    // are more tiles than CUs -- hold the fewest rows, and their partial sums
    // (stored only for rows that exist) the fewest bytes.  Class 0 counts full
    // tiles, class 1 + j partial tiles of row class j; one exclusive scan per
    // class over the tenants (thread i takes a run of tenants).
    constexpr int kClasses = 9;
    const int per = (T + kThreads - 1) / kThreads;
    const int t_beg = min(T, tid * per), t_end = min(T, t_beg + per);
    auto count = [&](int t) { return hist[t] + hist[T + t] + hist[2 * T + t] + hist[3 * T + t]; };
    auto class_of_last = [](int c) { return 1 + (BM - 1 - c % BM) / 32; };   // c % BM != 0
    // this thread's tenants' row counts, all read at once (at most 8 tenants)
    constexpr int kPer = kMaxGroupedTenants / kThreads;
    static_assert(kPer * kThreads == kMaxGroupedTenants && kPer <= 8, "tenants per thread");
    int cnt[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) cnt[i] = t_beg + i < t_end ? count(t_beg + i) : 0;
    int sc[kClasses], ex[kClasses];
#pragma unroll
    for (int k = 0; k < kClasses; ++k) sc[k] = 0;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int c = cnt[i];
        sc[0] += c / BM;
        if (c % BM != 0) {
            const int k = class_of_last(c);
#pragma unroll
            for (int kk = 1; kk < kClasses; ++kk) sc[kk] += kk == k;
        }
    }
    // Inclusive wave scans of the nine counts in four words, interleaved: the
    // full-tile count alone, the partial-tile class counts three to a word in
    // 10-bit fields (at most 8 tenants per thread, so at most 512 per wave).
    static_assert(kMaxGroupedTenants <= 8 * kThreads, "class count fields");
    int pk[4] = {sc[0], sc[1] | sc[2] << 10 | sc[3] << 20, sc[4] | sc[5] << 10 | sc[6] << 20,
                 sc[7] | sc[8] << 10};
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        int o[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] = __shfl_up(pk[j], d);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (lane >= d) pk[j] += o[j];
    }
    const int inc[kClasses] = {pk[0],
                               pk[1] & 1023, (pk[1] >> 10) & 1023, pk[1] >> 20,
                               pk[2] & 1023, (pk[2] >> 10) & 1023, pk[2] >> 20,
                               pk[3] & 1023, pk[3] >> 10};
#pragma unroll
    for (int k = 0; k < kClasses; ++k) {
        if (lane == 63) rows[4 * k + wv] = inc[k];
        ex[k] = inc[k] - sc[k];
    }
    __syncthreads();
    // the four waves' class totals, all read at once, then combined without
    // branches: class starts, and this wave's offset within each class
    static_assert(kThreads == 4 * 64, "four waves");
    int wtot[kClasses][4];
#pragma unroll
    for (int k = 0; k < kClasses; ++k)
#pragma unroll
        for (int w2 = 0; w2 < 4; ++w2) wtot[k][w2] = rows[4 * k + w2];
    int cls_first[kClasses + 1];                 // first row tile of each class
    cls_first[0] = 0;
#pragma unroll
    for (int k = 0; k < kClasses; ++k) {
        cls_first[k + 1] = cls_first[k] + wtot[k][0] + wtot[k][1] + wtot[k][2] + wtot[k][3];
        ex[k] += (wv > 0 ? wtot[k][0] : 0) + (wv > 1 ? wtot[k][1] : 0) + (wv > 2 ? wtot[k][2] : 0);
    }
    const int total = cls_first[kClasses];
    __syncthreads();            // the totals are read before info[4..5] and rows[] are reused
    const int ntiles = total * tiles_n;
    const int S = split_chunks(ntiles, room, KT);
    // block 0 records this call's split for the reduction launch that follows
    if (bid == 0 && tid == 0 && split_hdr != nullptr) {
        split_hdr[0] = S > 1 ? ntiles - kCUs : 0;
        split_hdr[1] = S;
    }
    int tile_idx = bid;
    item = WorkItem{0, 1, -1, 0};
    if (S > 1 && bid >= kCUs) {
        item.nleft = ntiles - kCUs;
        const int u = bid - kCUs;
        if (u >= (ntiles - kCUs) * S) return false;
        item.leftover = u / S;
        item.chunk = u - item.leftover * S;
        item.nchunks = S;
        tile_idx = kCUs + item.leftover;
    }
    if (tile_idx >= ntiles) return false;
    int tile_v;
    if (S > 1 && kCUs % tiles_n == 0) {
        // the whole tiles are the first kCUs / tiles_n row tiles (grouped for
        // L2 as in the one-round case); the leftover ones follow row by row
        if (tile_idx < kCUs) {
            tile_of(tile_idx, kCUs / tiles_n, tiles_n, tile_v, tile_n);
        } else {
            const int l = tile_idx - kCUs;
            tile_v = kCUs / tiles_n + l / tiles_n;
            tile_n = l % tiles_n;
        }
    } else {
        tile_of(tile_idx, total, tiles_n, tile_v, tile_n);
    }
    int k = 0;
#pragma unroll
    for (int kk = 1; kk < kClasses; ++kk) k += tile_v >= cls_first[kk];
    const int pv = tile_v - cls_first[k];        // index within its class
    int exk = 0, sck = 0;
#pragma unroll
    for (int kk = 0; kk < kClasses; ++kk)
        if (kk == k) {
            exk = ex[kk];
            sck = sc[kk];
        }
    if (pv >= exk && pv < exk + sck) {
        int first = exk;
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int t = t_beg + i;
            if (t >= t_end) break;
            const int c = cnt[i];
            if (k == 0) {
                const int nf = c / BM;
                if (pv < first + nf) {
                    info[4] = t;
                    info[5] = pv - first;
                    break;
                }
                first += nf;
            } else if (c % BM != 0 && class_of_last(c) == k) {
                if (pv == first) {
                    info[4] = t;
                    info[5] = c / BM;
                    break;
                }
                ++first;
            }
        }
    }
    rows[tid] = -1;
    __syncthreads();

    // rank of each row among its tenant's rows: this wave's base from the
    // earlier waves' histograms, then ballots over 64-row chunks in order
    const int t = info[4], lo = info[5] * BM;
    int rank = 0;
    for (int w2 = 0; w2 < wv; ++w2) rank += hist[w2 * T + t];
    auto collect = [&](int base, const int (&v)[kIdRegs]) {
#pragma unroll
        for (int u = 0; u < kIdRegs; ++u) {
            const uint64_t mask = __ballot(v[u] == t);
            if (v[u] == t) {
                const int below = (int)__builtin_amdgcn_mbcnt_hi(
                    (uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
                const int r = rank + below - lo;
                if (r >= 0 && r < BM) rows[r] = base + 64 * u + lane;
            }
            rank += __popcll(mask);
        }
    };
    if (rank < lo + BM) collect(r_beg, idr);
    for (int base = r_beg + 64 * kIdRegs; base < r_end && rank < lo + BM; base += 64 * kIdRegs) {
        int v[kIdRegs];
        load_ids(base, v);
        collect(base, v);
    }
    __syncthreads();
    tenant = t;
    return true;
}

// Rows whose tenant id lies outside [0, T) are written as quiet NaN, columns
// [n0, n0 + 256) (one workgroup per column tile).
template <int ET, int YDT>
__device__ void write_invalid_rows(const int32_t* __restrict__ ids, int M, int T, int N, int n0,
                                   void* __restrict__ y) {
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    for (int base = 64 * wv; base < M; base += 4 * 64 * 4) {
        int v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int m = base + 256 * u + lane;
            v[u] = m < M ? ids[m] : 0;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int m = base + 256 * u + lane;
            uint64_t mask = __ballot(m < M && (unsigned)v[u] >= (unsigned)T);
            while (mask) {
                const int r = base + 256 * u + __builtin_ctzll(mask);
                mask &= mask - 1;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int col = n0 + 4 * lane + e;
                    if (col >= N) continue;
                    if constexpr (YDT == kF32)
                        reinterpret_cast<float*>(y)[(size_t)r * N + col] = __builtin_nanf("");
                    else
                        reinterpret_cast<uint16_t*>(y)[(size_t)r * N + col] = to_half<ET>(__builtin_nanf(""));
                }
            }
        }
    }
}

template <int P, class T>
__device__ __forceinline__ T& pick(T& a, T& b) {
    if constexpr (P == 0) return a; else return b;
}

// Hides a value from the optimiser so that a shift-and-mask sequence built on
// it is emitted as written.
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
    asm("" : "+v"(v));
    return v;
}

typedef __attribute__((ext_vector_type(2))) float f32x2v;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2v;

// One bf16 pair of effective weights, in two halves of four VALU operations
// so that the work can be spread over two MFMA issue slots.  `s` carries the
// chunk's eight sign bits twice (bit i and bit i+15); shifting by 15-2p
// brings the bits of pair p to positions 15 and 31.  Where the bit is set
// (sign +1) the weight's sign is flipped, -alpha is added in fp32, the sum is
// rounded to bf16 (v_cvt_pk_bf16_f32, nearest even) and the flip is undone:
// -bf16(-w - alpha) = bf16(w + alpha); where it is clear, w - alpha is rounded
// directly.  The mask is hidden from the optimiser between its two uses so
// each use folds into a single three-input bit operation.
struct PairWork {
    uint32_t xm;
    float lo, hi;
};

__device__ __forceinline__ PairWork fuse_pair_a(uint32_t w, uint32_t s, int p) {
    PairWork r;
    const uint32_t xm = s << (15 - 2 * p);
    const uint32_t v = opaque(w ^ (xm & kSignBits));
    r.lo = __builtin_bit_cast(float, v << 16);
    r.hi = __builtin_bit_cast(float, v & 0xFFFF0000u);
    r.xm = opaque(xm);
    return r;
}

__device__ __forceinline__ uint32_t fuse_pair_b(const PairWork& q, float neg_alpha) {
    const f32x2v f = {q.lo + neg_alpha, q.hi + neg_alpha};
    const uint32_t r = __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2v));
    return r ^ (q.xm & kSignBits);
}

__device__ __forceinline__ uint32_t fuse_pair(uint32_t w, uint32_t s, int p, float neg_alpha) {
    return fuse_pair_b(fuse_pair_a(w, s, p), neg_alpha);
}

// fp16 pair: fp16 has a packed add, so the whole pair is three operations: the
// shift, one bit operation that moves the signs onto the (-a, -a) pair, and
// v_pk_add_f16 (nearest even): fp16(w + fp16(+-alpha)).
__device__ __forceinline__ uint32_t fuse_pair_f16(uint32_t w, uint32_t s, int p,
                                                  uint32_t neg_alpha_pair) {
    return add_f16x2(w, neg_alpha_pair ^ ((s << (15 - 2 * p)) & kSignBits));
}

// Two fp32 values -> one dword of two 16-bit outputs (nearest even).
template <int ET>
__device__ __forceinline__ uint32_t cvt_pair(f32x2v f) {
    if constexpr (ET == kF16) return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, f16x2));
    else return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2v));
}

// ET: 16-bit type of x and W; YDT: output dtype (kF32 or ET); ALIGNED: output
// rows start on 16-byte boundaries (N a multiple of 8 for 16-bit outputs, of 4
// for fp32), which allows 16-byte stores.
// GROUPED: the batched form (tenant id per row, at most kMaxGroupedTenants
// tenants); blocks below g_tiles take the work items of route_rows, and
// tiles_n more blocks past g_tiles write the rows of invalid ids.  part /
// counters / room: partial-sum buffer (room chunks of 256 KB) and the split
// record (header of 4 ints, then per leftover tile its row map and column
// origin) that prefill_reduce_kernel reads; room 0 disables the split.
template <int ET, int YDT, bool ALIGNED, bool GROUPED>
__global__ __launch_bounds__(kThreads, 1) void prefill_stream_kernel(
    const uint16_t* __restrict__ x, int M, int K, const uint16_t* __restrict__ w, int N,
    const uint32_t* __restrict__ packed, const float* __restrict__ alpha_p,
    const int32_t* __restrict__ ids, int T, void* __restrict__ y, int tiles_m, int tiles_n,
    float* __restrict__ part, int* __restrict__ counters, int room, int g_tiles) {
    // Two buffers per operand, each [256 rows][64 k] bf16 = 32 KB.
    __shared__ __attribute__((aligned(1024))) uint16_t sA0[BM * BK];
    __shared__ __attribute__((aligned(1024))) uint16_t sA1[BM * BK];
    __shared__ __attribute__((aligned(1024))) uint16_t sB0[BN * BK];
    __shared__ __attribute__((aligned(1024))) uint16_t sB1[BN * BK];
    __shared__ int sRows[GROUPED ? BM : 1];   // global row of each tile row, -1 = none
    __shared__ int sInfo[GROUPED ? 8 : 1];

    int tile_m = 0, tile_n, tenant = 0;
    WorkItem item{0, 1, -1, 0};
    if constexpr (GROUPED) {
        if ((int)blockIdx.x >= g_tiles) {
            write_invalid_rows<ET, YDT>(ids, M, T, N, ((int)blockIdx.x - g_tiles) * BN, y);
            return;
        }
        if (!route_rows(ids, M, T, tiles_n, blockIdx.x, room, K / BK, counters, reinterpret_cast<int*>(sA0),
                        sRows, sInfo, tenant, tile_n, item))
            return;
        // the chunk is needed again only after the k-loop: keep it in LDS, not
        // in registers across the loop (sInfo[6], [7] are free after routing)
        if (threadIdx.x == 0) {
            sInfo[6] = item.leftover * item.nchunks + item.chunk;
            sInfo[7] = item.nchunks;
        }
    } else {
        tile_of(blockIdx.x, tiles_m, tiles_n, tile_m, tile_n);
    }
    const int m0 = tile_m * BM, n0 = tile_n * BN;
    // global row g of tile row lr; false when the tile row holds no row
    auto out_row = [&](int lr, int& g) -> bool {
        if constexpr (GROUPED) {
            g = sRows[lr];
            return g >= 0;
        } else {
            g = m0 + lr;
            return g < M;
        }
    };

    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wv >> 1, wn = wv & 1;
    // k-tiles of this work item: all of K, or chunk c of a split leftover tile
    const int kb0 = item.chunk * (K / BK) / item.nchunks;
    const int KT = (item.chunk + 1) * (K / BK) / item.nchunks - kb0;
    const int KW = K >> 5;
    const float neg_alpha = -alpha_p[tenant];
    const uint32_t neg_alpha_h = to_f16(neg_alpha) | ((uint32_t)to_f16(neg_alpha) << 16);
    packed += (size_t)tenant * N * KW;
    // one pair of effective weights in one go (prologue)
    auto fuse_full = [&](uint32_t wd, uint32_t sw_, int p) -> uint32_t {
        if constexpr (ET == kF16) return fuse_pair_f16(wd, sw_, p, neg_alpha_h);
        else return fuse_pair(wd, sw_, p, neg_alpha);
    };

    // ---- staging assignment: per instruction i a wave moves rows
    //      32i + 8wv + (lane >> 3), lane l landing at LDS slot l & 7 ----
    const int fst = (lane >> 3) ^ (wv & 1);          // f(row) of the staged rows
    const int ch = (lane & 7) ^ fst;                 // global 16-byte chunk moved
    uint32_t xoff[8], woff[8], soff[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int r = 32 * i + 8 * wv + (lane >> 3);
        // rows past the end (or past the tenant's last row) re-read a valid row
        uint32_t xr;
        if constexpr (GROUPED) xr = (uint32_t)(sRows[r] >= 0 ? sRows[r] : sRows[0]);
        else xr = (uint32_t)min(m0 + r, M - 1);
        const uint32_t wr = (uint32_t)min(n0 + r, N - 1);
        xoff[i] = (xr * (uint32_t)K + 8u * ch) * 2u + (uint32_t)kb0 * (BK * 2);
        woff[i] = (wr * (uint32_t)K + 8u * ch) * 2u + (uint32_t)kb0 * (BK * 2);
        soff[i] = (wr * (uint32_t)KW + (uint32_t)(ch >> 2)) * 4u + (uint32_t)kb0 * 8u;
    }
    const int sbit = (ch & 3) * 8;
    const int st_lane = 8 * wv * BK + 8 * lane;      // bf16 offset of the lane's slot, row block 0

    // ---- fragment reads: row (lane & 31) of a 32-row block, chunk 2kk + (lane >> 5) ----
    const int frd = (lane & 7) ^ ((lane >> 3) & 1);
    int rdo[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) rdo[kk] = (lane & 31) * BK + 8 * ((2 * kk + (lane >> 5)) ^ frd);
    const int a_row0 = wm * 128 * BK, b_row0 = wn * 128 * BK;

    // Buffer resources: per-lane 32-bit byte offsets (row and chunk) plus a
    // wave-uniform k-tile offset in an SGPR, so no address arithmetic is
    // spent per load.  Row indices are clamped, so every access is in range.
    constexpr int kRawBufferFlags = 0x00020000;  // untyped 32-bit data format
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(w), (short)0, (int)((uint32_t)N * (uint32_t)K * 2u), kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t sres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint32_t*>(packed), (short)0, (int)((uint32_t)N * (uint32_t)KW * 4u), kRawBufferFlags);

    auto load_w = [&](u32x4& dst, int i, int kt) {
        dst = __builtin_amdgcn_raw_buffer_load_b128(wres, (int)woff[i], kt * (BK * 2), 0);
    };
    auto load_s = [&](uint32_t& dst, int i, int kt) {
        dst = __builtin_amdgcn_raw_buffer_load_b32(sres, (int)soff[i], kt * 8, 0);
    };
    auto sign_word = [&](uint32_t d) {
        const uint32_t byte = (d >> sbit) & 0xFFu;
        return opaque(byte | (byte << 15));
    };
    // x chunk i of k-tile kt straight into LDS by a global->LDS copy: lane l
    // lands at slot l of the wave's 1 KB, the layout st_lane describes
    auto copy_x = [&](uint16_t* buf, int i, int kt) {
        copy16_to_lds(reinterpret_cast<const char*>(x) + xoff[i] + (size_t)kt * (BK * 2),
                      buf + i * 32 * BK + 8 * wv * BK);
    };
    auto frag = [&](const uint16_t* buf, int row0, int blk, int kk) {
        return *reinterpret_cast<const u32x4*>(buf + row0 + blk * 32 * BK + rdo[kk]);
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // Raw W / sign-word register sets.  Chunk c of the tile decoded in the
    // second half of the decode stream... concretely: body t decodes chunks
    // 2..7 of tile t+1 (set (t+1)&1) and chunks 0..1 of tile t+2 (set t&1),
    // and refills every chunk it consumed with the tile two further on.
    u32x4 w0[8], w1[8];
    uint32_t s0[8], s1[8];

    // ---- prologue: tile 0 and chunks 0..1 of tile 1 staged, registers primed ----
    const int k1 = min(1, KT - 1), k2 = min(2, KT - 1), k3 = min(3, KT - 1);
#pragma unroll
    for (int i = 0; i < 8; ++i) copy_x(sA0, i, 0);
#pragma unroll
    for (int i = 0; i < 8; ++i) copy_x(sA1, i, k1);
#pragma unroll
    for (int i = 0; i < 8; ++i) { load_w(w0[i], i, 0); load_s(s0[i], i, 0); }
#pragma unroll
    for (int i = 0; i < 8; ++i) { load_w(w1[i], i, k1); load_s(s1[i], i, k1); }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const uint32_t sw0 = sign_word(s0[i]);
        u32x4 o;
#pragma unroll
        for (int p = 0; p < 4; ++p) o[p] = fuse_full(w0[i][p], sw0, p);
        *reinterpret_cast<u32x4*>(sB0 + i * 32 * BK + st_lane) = o;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) { load_w(w0[i], i, k2); load_s(s0[i], i, k2); }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const uint32_t sw1 = sign_word(s1[i]);
        u32x4 o;
#pragma unroll
        for (int p = 0; p < 4; ++p) o[p] = fuse_full(w1[i][p], sw1, p);
        *reinterpret_cast<u32x4*>(sB1 + i * 32 * BK + st_lane) = o;
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) { load_w(w1[i], i, k3); load_s(s1[i], i, k3); }
    uint32_t sw = sign_word(s1[2]);
    wait_vm_lgkm0<0>();                              // x of tiles 0 and 1 in LDS
    raw_barrier();
    u32x4 fa[4], fb[4], na[4], nb[4];
    fa[0] = frag(sA0, a_row0, 0, 0);
#pragma unroll
    for (int j = 0; j < 4; ++j) fb[j] = frag(sB0, b_row0, j, 0);
#pragma unroll
    for (int i = 1; i < 4; ++i) fa[i] = frag(sA0, a_row0, i, 0);

    // Loads per slot: each run of eight slots issues one sign-word load (its
    // seventh slot) and one W load (its eighth).  The x copies of tile t+2 go
    // out in slots 48..55 of body t, the last before slot 55's W load; up to
    // the barrier of body t+1 (slot 48) come that W load, the two loads of
    // slots 56..63 and the twelve of body t+1's slots 0..47.
    constexpr int kXWait = 1 + 2 + 12;

    // Body t: the 64 MFMAs of tile t.  Fragments are always read one k-step
    // ahead, so the barrier that publishes tile t+1 sits between k-steps 2
    // and 3: by then every read of tile t has been issued and waited for, the
    // buffers of tile t are free for tile t+2, and k-step 3 overlaps the reads
    // of tile t+1's first fragments.  Slot g (0..63) also carries position
    // p of the decode stream: g < 48 -> chunks 2..7 of tile t+1 (p = g+16),
    // g >= 48 -> chunks 0..1 of tile t+2 (p = g-48); chunk p/8, step p%8:
    // even steps form half a pair, odd steps finish it; step 6 refills the
    // sign word, step 7 writes the chunk to LDS and refills its raw weights.
    auto body = [&](auto par, int t) {
        constexpr int P = decltype(par)::value;
        uint16_t* const Ac = P ? sA1 : sA0;
        uint16_t* const An = P ? sA0 : sA1;
        uint16_t* const Bc = P ? sB1 : sB0;
        uint16_t* const Bn = P ? sB0 : sB1;
        u32x4(&wn1)[8] = pick<P ^ 1>(w0, w1);      // tile t+1
        uint32_t(&sn1)[8] = pick<P ^ 1>(s0, s1);
        u32x4(&wn2)[8] = pick<P>(w0, w1);          // tile t+2
        uint32_t(&sn2)[8] = pick<P>(s0, s1);
        const int kr1 = min(t + 3, KT - 1), kr2 = min(t + 4, KT - 1);

        PairWork pw;
        u32x4 o;
        uint32_t sw_next = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            if (b == 3) {
                // this wave's LDS writes of tile t+1 are complete, and so are its
                // x copies of tile t+1 (the previous body's slots 48..55): after
                // them came kXWait loads (wait_vm_lgkm0 below); publish them
                wait_vm_lgkm0<kXWait>();
                raw_barrier();
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int m = 0; m < 16; ++m) {
                const int i = m >> 2, j = m & 3;
                // tile t's buffers are free after the barrier: x of tile t+2
                if (b == 3 && m < 8) copy_x(Ac, m, min(t + 2, KT - 1));
                acc[i][j] = mfma32<ET>(fb[j], fa[i], acc[i][j]);
                if (m < 8) {
                    const uint16_t* abuf = b < 3 ? Ac : An;
                    const uint16_t* bbuf = b < 3 ? Bc : Bn;
                    const int kk = b < 3 ? b + 1 : 0;
                    if (m == 0) na[0] = frag(abuf, a_row0, 0, kk);
                    else if (m < 5) nb[m - 1] = frag(bbuf, b_row0, m - 1, kk);
                    else na[m - 4] = frag(abuf, a_row0, m - 4, kk);
                }
                const int g = b * 16 + m;
                const bool first = g < 48;
                const int pos = first ? g + 16 : g - 48;
                const int c = pos >> 3, u = pos & 7;
                u32x4(&ws)[8] = first ? wn1 : wn2;
                uint32_t(&ss)[8] = first ? sn1 : sn2;
                uint16_t* const dst = first ? Bn : Bc;
                const int kr = first ? kr1 : kr2;
                if constexpr (ET == kF16) {
                    if ((u & 1) == 0) o[u >> 1] = fuse_pair_f16(ws[c][u >> 1], sw, u >> 1, neg_alpha_h);
                } else {
                    if ((u & 1) == 0) pw = fuse_pair_a(ws[c][u >> 1], sw, u >> 1);
                    else o[u >> 1] = fuse_pair_b(pw, neg_alpha);
                }
                if (u == 6) {
                    // sign word of the next chunk in stream order
                    sw_next = c < 7 ? sign_word(ss[c + 1]) : sign_word(sn2[0]);
                    load_s(ss[c], c, kr);
                }
                if (u == 7) {
                    *reinterpret_cast<u32x4*>(dst + c * 32 * BK + st_lane) = o;
                    load_w(ws[c], c, kr);
                    sw = sw_next;
                }
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) { fa[r] = na[r]; fb[r] = nb[r]; }
        }
    };

    int t = 0;
    for (; t + 1 < KT; t += 2) {
        body(std::integral_constant<int, 0>{}, t);
        body(std::integral_constant<int, 1>{}, t + 1);
    }
    if (t < KT) body(std::integral_constant<int, 0>{}, t);
    wait_vm_lgkm0<0>();                              // the last x copies are in before LDS is reused

    // ---- a chunk of a split tile: store the partial sums (and, chunk 0, the
    //      tile's row map and column origin); prefill_reduce_kernel, launched
    //      next on the stream, adds the chunks in chunk order and writes y ----
    if constexpr (GROUPED) {
        const int nchunks = sInfo[7];
        if (nchunks > 1) {
            const int tid = threadIdx.x;
            const int unit = sInfo[6];                   // leftover * nchunks + chunk
            f32x4* mine = reinterpret_cast<f32x4*>(part) + (size_t)unit * kSplitVecs * kThreads;
            // partials of tile rows that hold no output row are neither stored
            // nor read by the reduction
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (sRows[wm * 128 + 32 * i + (lane & 31)] < 0) continue;
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        mine[((i * 4 + j) * 4 + q) * kThreads + tid] =
                            f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
            }
            if (unit % nchunks == 0) {
                int* meta = counters + 4 + kSplitMetaInts * (unit / nchunks);  // [rows 256][n0]
                meta[tid] = sRows[tid];
                if (tid == 0) meta[BM] = n0;
            }
            return;
        }
    }

    // ---- epilogue.  The W fragment is the MFMA's first operand, so acc[i][j][r]
    //      holds y[mrow + 32i][ncol + 32j + 8(r >> 2) + (r & 3)]: four
    //      consecutive columns per register quad ----
    const int lrow = wm * 128 + (lane & 31);
    const int ncol = n0 + wn * 128 + 4 * (lane >> 5);
    if constexpr (YDT != kF32 && ALIGNED) {
        // Rows go through LDS, 64 at a time, so that each lane stores 16
        // contiguous bytes and a store instruction covers whole 256-byte rows.
        raw_barrier();  // every wave is done with the operand buffers
        uint16_t* const stage = wv == 0 ? sA0 : wv == 1 ? sA1 : wv == 2 ? sB0 : sB1;
        constexpr int kStageRow = 136;  // bf16 per staged row: 128 + 8 padding
#pragma unroll
        for (int half = 0; half < 2; ++half) {
#pragma unroll
            for (int ii = 0; ii < 2; ++ii)
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int i = 2 * half + ii;
                        const f32x2v lo = {acc[i][j][4 * q], acc[i][j][4 * q + 1]};
                        const f32x2v hi = {acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
                        uint2 v;
                        v.x = cvt_pair<ET>(lo);
                        v.y = cvt_pair<ET>(hi);
                        *reinterpret_cast<uint2*>(stage + (32 * ii + (lane & 31)) * kStageRow + 32 * j +
                                                  8 * q + 4 * (lane >> 5)) = v;
                    }
            // each wave reads back only rows it wrote itself
#pragma unroll
            for (int t = 0; t < 16; ++t) {
                const int qd = lane + 64 * t, row = qd >> 4, c8 = qd & 15;
                const u32x4 v = *reinterpret_cast<const u32x4*>(stage + row * kStageRow + c8 * 8);
                int gm;
                const bool ok = out_row(wm * 128 + 64 * half + row, gm);
                const int gn = n0 + wn * 128 + c8 * 8;
                if (ok && gn < N)
                    *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(y) + (size_t)gm * N + gn) = v;
            }
        }
    } else if constexpr (YDT == kF32) {
        constexpr bool vec = ALIGNED;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    int row;
                    if (!out_row(lrow + 32 * i, row)) continue;
                    const int col = ncol + 32 * j + 8 * q;
                    float* dst = reinterpret_cast<float*>(y) + (size_t)row * N + col;
                    if constexpr (vec) {
                        if (col >= N) continue;
                        const f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                         acc[i][j][4 * q + 3]};
                        *reinterpret_cast<f32x4*>(dst) = v;
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (col + e < N) dst[e] = acc[i][j][4 * q + e];
                    }
                }
    } else {
        // 16-bit rows not 16-byte aligned: element stores
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    int row;
                    const bool ok = out_row(lrow + 32 * i, row);
                    const int col = ncol + 32 * j + 8 * (r >> 2) + (r & 3);
                    if (ok && col < N)
                        reinterpret_cast<uint16_t*>(y)[(size_t)row * N + col] = to_half<ET>(acc[i][j][r]);
                }
    }
}

// The chunks of the split leftover tiles: sum them in chunk order and write
// the tiles' rows.  Sixteen blocks per leftover tile, each taking four of the
// 64 partial vectors of every thread of the chunk blocks (the same thread
// layout, so row and column follow as in the main epilogue).  Partials of
// tile rows that hold no output row are not read.
template <int ET>
__global__ __launch_bounds__(kThreads) void prefill_reduce_kernel(const float* __restrict__ part,
                                                                  const int* __restrict__ split, void* __restrict__ y,
                                                                  int N, int y_dtype) {
    constexpr int kPerBlock = 4, kBlocks = kSplitVecs / kPerBlock;
    const int nleft = split[0], S = split[1];
    const int l = blockIdx.x / kBlocks, vb = blockIdx.x % kBlocks;
    if (l >= nleft || S < 2) return;
    const int* meta = split + 4 + kSplitMetaInts * l;
    const int n0 = meta[BM];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int wm = wv >> 1, wn = wv & 1;
    const f32x4* all = reinterpret_cast<const f32x4*>(part) + (size_t)l * S * kSplitVecs * kThreads;
    // every load of the block's vectors (all chunks) is issued before the
    // first add, so their latencies overlap
    int rows[kPerBlock];
#pragma unroll
    for (int vv = 0; vv < kPerBlock; ++vv) {
        const int v = vb * kPerBlock + vv;
        rows[vv] = meta[wm * 128 + 32 * (v >> 4) + (lane & 31)];
    }
    f32x4 pc[kPerBlock][8];
#pragma unroll
    for (int vv = 0; vv < kPerBlock; ++vv) {
        const int v = vb * kPerBlock + vv;
#pragma unroll
        for (int c = 0; c < 8; ++c)
            if (rows[vv] >= 0 && c < S) pc[vv][c] = all[((size_t)c * kSplitVecs + v) * kThreads + tid];
    }
#pragma unroll
    for (int vv = 0; vv < kPerBlock; ++vv) {
        const int v = vb * kPerBlock + vv;              // (i * 4 + j) * 4 + q
        const int j = (v >> 2) & 3, q = v & 3;
        const int row = rows[vv];
        if (row < 0) continue;
        f32x4 sum = pc[vv][0];
#pragma unroll
        for (int c = 1; c < 8; ++c)
            if (c < S) {
                sum[0] += pc[vv][c][0];
                sum[1] += pc[vv][c][1];
                sum[2] += pc[vv][c][2];
                sum[3] += pc[vv][c][3];
            }
        const int col = n0 + wn * 128 + 32 * j + 8 * q + 4 * (lane >> 5);
        const size_t at = (size_t)row * N + col;
        if ((N & 3) == 0 && col + 3 < N) {
            // four consecutive outputs in one store (col and N multiples of 4)
            if (y_dtype == kF32) {
                *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(y) + at) = sum;
            } else {
                uint2 v;
                v.x = cvt_pair<ET>(f32x2v{sum[0], sum[1]});
                v.y = cvt_pair<ET>(f32x2v{sum[2], sum[3]});
                *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(y) + at) = v;
            }
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (col + e < N) store_y<ET>(y, at + e, sum[e], y_dtype);
        }
    }
}

}  // namespace

// The streaming kernel addresses x and W through buffer resources whose byte
// extents must fit in 31 bits, and steps K in tiles of 64.
bool prefill_stream_supported(int M, int N, int K) {
    return K >= BK && K % BK == 0 && (int64_t)M * K < ((int64_t)1 << 30) &&
           (int64_t)N * K < ((int64_t)1 << 30);
}

namespace {

template <int ET, bool GROUPED>
void launch_stream_et(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                      const uint32_t* packed, const float* alpha, const int32_t* ids, int T,
                      void* y, int y_dtype, int tiles_m, int grid, int tiles_n,
                      hipStream_t stream, float* part = nullptr, int* counters = nullptr, int room = 0,
                      int g_tiles = 0) {
    const dim3 g(grid), block(kThreads);
    if (y_dtype != kF32 && N % 8 == 0)
        prefill_stream_kernel<ET, ET, true, GROUPED><<<g, block, 0, stream>>>(
            x, M, K, w, N, packed, alpha, ids, T, y, tiles_m, tiles_n, part, counters, room, g_tiles);
    else if (y_dtype != kF32)
        prefill_stream_kernel<ET, ET, false, GROUPED><<<g, block, 0, stream>>>(
            x, M, K, w, N, packed, alpha, ids, T, y, tiles_m, tiles_n, part, counters, room, g_tiles);
    else if (N % 4 == 0)
        prefill_stream_kernel<ET, kF32, true, GROUPED><<<g, block, 0, stream>>>(
            x, M, K, w, N, packed, alpha, ids, T, y, tiles_m, tiles_n, part, counters, room, g_tiles);
    else
        prefill_stream_kernel<ET, kF32, false, GROUPED><<<g, block, 0, stream>>>(
            x, M, K, w, N, packed, alpha, ids, T, y, tiles_m, tiles_n, part, counters, room, g_tiles);
}

}  // namespace

hipError_t launch_prefill(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                          const uint32_t* packed, const float* alpha, void* y, int y_dtype,
                          int et, hipStream_t stream) {
    const int tiles_m = (M + BM - 1) / BM;
    const int tiles_n = (N + BN - 1) / BN;
    const int grid = tiles_m * tiles_n;
    if (prefill_stream_supported(M, N, K)) {
        if (et == kF16)
            launch_stream_et<kF16, false>(x, M, K, w, N, packed, alpha, nullptr, 1, y, y_dtype,
                                          tiles_m, grid, tiles_n, stream);
        else
            launch_stream_et<kBF16, false>(x, M, K, w, N, packed, alpha, nullptr, 1, y, y_dtype,
                                           tiles_m, grid, tiles_n, stream);
    } else if (et == kF16) {
        prefill_general_kernel<kF16><<<grid, kThreads, 0, stream>>>(x, M, K, w, N, packed, alpha, y,
                                                                   y_dtype, tiles_m, tiles_n);
    } else {
        prefill_general_kernel<kBF16><<<grid, kThreads, 0, stream>>>(x, M, K, w, N, packed, alpha, y,
                                                                    y_dtype, tiles_m, tiles_n);
    }
    return hipGetLastError();
}

bool prefill_grouped_supported(int M, int N, int K, int T) {
    return prefill_stream_supported(M, N, K) && T >= 1 && T <= kMaxGroupedTenants;
}

constexpr size_t kSplitMetaBytes = (4 + (size_t)kCUs * kSplitMetaInts) * sizeof(int);
static_assert((size_t)kCUs * kSplitChunkBytes + kSplitMetaBytes == kPrefillSplitBytes, "split buffer size");
size_t prefill_split_bytes() { return kPrefillSplitBytes; }

hipError_t launch_prefill_grouped(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                                  const uint32_t* packed, const float* alpha,
                                  const int32_t* tenant_ids, int T, void* y, int y_dtype,
                                  int et, hipStream_t stream, void* scratch, size_t scratch_bytes) {
    // sum_t ceil(c_t / BM) over the U <= min(T, M) tenants present, with
    // sum_t c_t <= M, is at most (M + (BM - 1) * U) / BM
    const int64_t U = T < M ? T : M;
    const int tiles_m = (int)(((int64_t)M + (BM - 1) * U) / BM);
    const int tiles_n = (N + BN - 1) / BN;
    // partial-sum room: the split record sits at the start of the buffer,
    // the chunks after it
    int room = 0;
    float* part = nullptr;
    int* split = nullptr;
    if (scratch != nullptr && scratch_bytes >= kSplitMetaBytes + 2 * kSplitChunkBytes) {
        const size_t chunks = (scratch_bytes - kSplitMetaBytes) / kSplitChunkBytes;
        room = (int)(chunks < (size_t)kCUs ? chunks : (size_t)kCUs);
        split = static_cast<int*>(scratch);
        part = reinterpret_cast<float*>(static_cast<char*>(scratch) + kSplitMetaBytes);
    }
    // blocks: every whole tile, and kCUs + room for the split chunks
    int g_tiles = tiles_m * tiles_n;
    if (g_tiles <= kCUs) room = 0;                     // one round at most: nothing to split
    if (room > 0 && g_tiles < kCUs + room) g_tiles = kCUs + room;
    const int grid = g_tiles + tiles_n;
    if (et == kF16)
        launch_stream_et<kF16, true>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype,
                                     tiles_m, grid, tiles_n, stream, part, split, room, g_tiles);
    else
        launch_stream_et<kBF16, true>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype,
                                      tiles_m, grid, tiles_n, stream, part, split, room, g_tiles);
    if (room > 0) {
        // at most room / 2 leftover tiles are split (two chunks or more each)
        const int rgrid = (kSplitVecs / 4) * (room / 2);
        if (et == kF16)
            prefill_reduce_kernel<kF16><<<rgrid, kThreads, 0, stream>>>(part, split, y, N, y_dtype);
        else
            prefill_reduce_kernel<kBF16><<<rgrid, kThreads, 0, stream>>>(part, split, y, N, y_dtype);
    }
    return hipGetLastError();
}

}  // namespace bitdelta
