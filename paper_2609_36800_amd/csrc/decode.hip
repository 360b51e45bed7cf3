// Single-tenant decode GEMV/skinny kernel for M <= 16 token rows:
//
//   y[m][n] = sum_k x[m][k] W[n][k] + alpha * sum_k x[m][k] s[n][k]
//
// (the standard BitDelta GEMM of Section 4.4 at decode shapes).  Bound by HBM:
// every byte of W and of the packed signs is read once.
//
// Work split: a 512-thread workgroup owns 16 output features; its 8 waves split
// the contraction into contiguous runs of 32-wide k-blocks, processed in rounds
// of D blocks.  Per round a wave
//   * streams W straight into registers as MFMA B operands: one 16-byte load
//     per lane per block (8 consecutive k of one feature), D loads in flight;
//   * loads the packed signs of its 16 features x D blocks (D*4 bytes per row)
//     with one coalesced 16-byte load per lane into a private LDS area;
//   * loads its slice of x (up to 16 rows x D*64 bytes) with one coalesced
//     1-KB load per row into the same area.
// Scattered per-block loads of sign bytes and of x rows cost more request
// slots than the W stream itself, so they go through LDS once per round and the
// MFMA fragments are read back from there.  Signs become bf16 +1/-1 operands in
// registers (decode_signs8, two values per two ops), and x*W^T and x*S^T are
// accumulated apart in fp32 on v_mfma_f32_16x16x32_bf16; the epilogue forms
// acc_base + alpha*acc_sign, so W + alpha*s is never rounded.
//
// Partial sums of the 8 waves are added in a fixed order through LDS: results
// are bitwise deterministic.
#include "device.h"
#include "internal.h"
#include "ldscopy.h"

namespace bitdelta {
namespace {

constexpr int kFeat = 16;        // output features per workgroup
constexpr int kWaves = 8;
constexpr int kRound = 16;       // k-blocks per wave per round (D)
constexpr int kSignStride = 80;  // bytes per feature row of staged signs (64 + pad)

template <int XR>
struct DecodeLayout {
    static constexpr int kXStride = kRound * 64 + 16;            // bytes per staged x row
    static constexpr int kXBytes = XR * kXStride;
    static constexpr int kWaveBytes = kXBytes + kFeat * kSignStride;
    static constexpr int kTotal = kWaves * kWaveBytes;
    static_assert(kTotal >= 2 * kWaves * 16 * kFeat * 4, "reduction area must fit");
};

__device__ __forceinline__ u32x4 lds_read16(const char* p) {
    return *reinterpret_cast<const u32x4*>(p);
}

template <int ET, int XR>
__global__ __launch_bounds__(kWaves * 64) void decode_kernel(
    const uint16_t* __restrict__ x, int M, int K, const uint16_t* __restrict__ w, int N,
    const uint32_t* __restrict__ packed, const float* __restrict__ alpha,
    void* __restrict__ y, int y_dtype) {
    using L = DecodeLayout<XR>;
    __shared__ __attribute__((aligned(16))) char smem[L::kTotal];

    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nl = lane & 15, g = lane >> 4;
    const int n0 = blockIdx.x * kFeat;
    const int KB = K >> 5, KW = K >> 5;

    char* xs = smem + wv * L::kWaveBytes;        // staged x rows of this wave
    char* ss = xs + L::kXBytes;                  // staged sign words of this wave

    // W: this lane's feature (clamped; rows past N feed unstored outputs only)
    const int n = min(n0 + nl, N - 1);
    const uint16_t* wp = w + (size_t)n * K + 8 * g;
    // signs: lane l stages row l/4, words 4*(l%4) .. +3 of the round
    const int srow = lane >> 2, squad = lane & 3;
    const uint32_t* sp = packed + (size_t)min(n0 + srow, N - 1) * KW;
    // x: MFMA row nl reads staged row min(nl, XR-1); source rows clamped to M-1
    const int xrow_lds = min(nl, XR - 1);

    f32x4 accb = {0.f, 0.f, 0.f, 0.f}, accs = {0.f, 0.f, 0.f, 0.f};
    const int per = (KB + kWaves - 1) / kWaves;
    const int kb0 = min(KB, wv * per);
    const int kb1 = min(KB, kb0 + per);
    const bool aligned_signs = (KW & 3) == 0;

    for (int base = kb0; base < kb1; base += kRound) {
        const int c = min(kRound, kb1 - base);   // blocks in this round (uniform)

        // ---- issue: signs, x slice, then the W stream (oldest first) ----
        uint32_t sw[4];
        if (aligned_signs && c == kRound && (base & 3) == 0) {
            const u32x4 v = *reinterpret_cast<const u32x4*>(sp + base + 4 * squad);
            sw[0] = v[0]; sw[1] = v[1]; sw[2] = v[2]; sw[3] = v[3];
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) sw[i] = sp[base + min(4 * squad + i, c - 1)];
        }
        u32x4 xv[XR];
        const int xchunk = min(lane, 4 * c - 1);   // 16-byte chunk of the row slice
#pragma unroll
        for (int r = 0; r < XR; ++r)
            xv[r] = load16(x + (size_t)min(r, M - 1) * K + (size_t)base * 32 + 8 * xchunk);
        __builtin_amdgcn_sched_barrier(0);
        u32x4 wf[kRound];
#pragma unroll
        for (int j = 0; j < kRound; ++j) {
            wf[j] = load16(wp + (size_t)(base + min(j, c - 1)) * 32);
            __builtin_amdgcn_sched_barrier(0);
        }

        // ---- stage signs and x in this wave's LDS area ----
#pragma unroll
        for (int i = 0; i < 4; ++i)
            *reinterpret_cast<uint32_t*>(ss + srow * kSignStride + 16 * squad + 4 * i) = sw[i];
#pragma unroll
        for (int r = 0; r < XR; ++r)
            *reinterpret_cast<u32x4*>(xs + r * L::kXStride + 16 * lane) = xv[r];

        // ---- consume, oldest block first ----
        auto consume = [&](int j) {
            const u32x4 xa = lds_read16(xs + xrow_lds * L::kXStride + j * 64 + 16 * g);
            const uint32_t sb = *reinterpret_cast<const uint8_t*>(ss + nl * kSignStride + 4 * j + g);
            accb = mfma16<ET>(xa, wf[j], accb);
            accs = mfma16<ET>(xa, decode_signs8<ET>(sb), accs);
        };
        if (c == kRound) {
#pragma unroll
            for (int j = 0; j < kRound; ++j) consume(j);
        } else {
#pragma unroll
            for (int j = 0; j < kRound; ++j)
                if (j < c) consume(j);
        }
    }

    // ---- combine the waves' partial sums (fixed order) ----
    __syncthreads();
    float* red_b = reinterpret_cast<float*>(smem);                 // [wave][16 rows][16 feat]
    float* red_s = red_b + kWaves * 16 * kFeat;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        red_b[(wv * 16 + 4 * g + r) * kFeat + nl] = accb[r];
        red_s[(wv * 16 + 4 * g + r) * kFeat + nl] = accs[r];
    }
    __syncthreads();
    if (threadIdx.x < 16 * kFeat) {
        const int m = threadIdx.x / kFeat, f = threadIdx.x % kFeat;
        const int nn = n0 + f;
        if (m < M && nn < N) {
            float b = 0.f, s = 0.f;
#pragma unroll
            for (int v = 0; v < kWaves; ++v) {
                b += red_b[(v * 16 + m) * kFeat + f];
                s += red_s[(v * 16 + m) * kFeat + f];
            }
            const float out = __builtin_fmaf(alpha[0], s, b);
            store_y<ET>(y, (size_t)m * N + nn, out, y_dtype);
        }
    }
}


// ---------------------------------------------------------------------------
// Streaming variant (K a multiple of 128): W and x reach LDS by global->LDS
// copies in 256-k tiles, NB-1 tiles ahead of the one being computed, and the
// workgroup's sign words for the whole K are staged once up front.  Each copy
// instruction moves whole 512-byte row segments, so every request is a full
// cache line (the register path above issues 64-byte half lines), and the
// streaming does not depend on how many waves are resident.  In step t wave w
// computes k-block 8d + w of the step's tile d from LDS; one vmcnt wait plus
// one barrier per step.
// W and the sign rows are read once per launch and copied with the
// non-temporal hint; x, shared by every workgroup through L2, is not.  The
// ring stops at the last tile of K (no repeat copies to drain at the end).
// Workgroups start K at different tiles: the 32 workgroups resident on one XCD
// (the hardware deals workgroups round-robin over the 8 XCDs) take up to 16
// different starting tiles (K/256 of them), so that at any moment their W rows are read at
// spread-out offsets (measured 2% faster at 16x4096x4096 and 5% at 1x11008x4096
// than all workgroups walking K in step).
// ---------------------------------------------------------------------------
constexpr int kTileBlocks = 8;                  // k-blocks per tile (one per wave)
constexpr int kTileRow = kTileBlocks * 64;      // bytes of one row segment of a tile

// XUP: x (XR rows x K <= 4096) is staged once up front instead of per tile.
template <int XR, bool XUP>
struct StreamCfg {
    static constexpr int kWBytes = kFeat * kTileRow;          // W: 16 rows x 512 B
    static constexpr int kXBytes = XUP ? 0 : XR * kTileRow;   // x: XR rows x 512 B per tile
    static constexpr int kTileBytes = kWBytes + kXBytes;
    // ring depth (tiles): with x copied per tile 5 (16 rows at 4096x4096, medians
    // of five rounds in one process: 8.42 us against 8.59 for 6, 8.49 for 4 and
    // 8.75 for 7 or 8); with x up front 6, level with 8 (4, 5 and 10 slower)
    static constexpr int kNB = XUP ? 6 : 5;
    static constexpr int kRing = kNB * kTileBytes;
    static constexpr int kOpsPerTile = XUP ? 1 : 2;           // copies per wave per tile
    static constexpr int kXLanes = XR * 4;                    // lanes of a wave copying x
    static constexpr int kXRowUp = 4096 * 2 + 64;             // up-front x row stride (padded)
    static constexpr int kXUpBytes = XUP ? XR * kXRowUp : 0;
};

__device__ __forceinline__ int tswz(int row, int chunk) { return chunk ^ (row & 15); }

// SB: bytes reserved for the staged signs (16 features x K/8 bytes).
template <int ET, int XR, int SB, bool XUP>
__global__ __launch_bounds__(kWaves * 64) void stream_decode_kernel(
    const uint16_t* __restrict__ x, int M, int K, const uint16_t* __restrict__ w, int N,
    const uint32_t* __restrict__ packed, const float* __restrict__ alpha,
    void* __restrict__ y, int y_dtype) {
    using C = StreamCfg<XR, XUP>;
    constexpr int NB = C::kNB;
    constexpr int D = NB - 1;
    static_assert(C::kRing >= 2 * kWaves * 16 * kFeat * 4, "reduction area must fit");
    __shared__ __attribute__((aligned(16))) char lds[C::kRing + SB + C::kXUpBytes];
    char* ring = lds;
    char* sg = lds + C::kRing;      // signs: [chunk of 4 words][feature][16 B]
    char* xu = sg + SB;             // up-front x rows (XUP)

    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nl = lane & 15, g = lane >> 4;
    const int n0 = blockIdx.x * kFeat;
    const int KB = K >> 5, KW = K >> 5;
    const int KT = (KB + kTileBlocks - 1) / kTileBlocks;
    // step t works on tile (t + rot) mod KT
    const int rot = ((int)blockIdx.x >> 3) % KT;
    auto tile_of = [&](int t) { const int d = t + rot; return d >= KT ? d - KT : d; };

    // ---- stage all sign words of the 16 features (same count on every wave) ----
    {
        const int nq = (KW + 15) >> 4;                        // copies of 4 chunks x 16 features
        const int per_wave = (nq + kWaves - 1) / kWaves;
        const uint32_t* srow = packed + (size_t)min(n0 + (lane & 15), N - 1) * KW;
        for (int i = 0; i < per_wave; ++i) {
            const int q = min(wv + i * kWaves, nq - 1);       // surplus copies repeat the last one
            const int chunk = min(4 * q + (lane >> 4), KW / 4 - 1);
            copy16_to_lds_nt(srow + 4 * chunk, sg + q * 1024);
        }
    }

    // ---- up-front x (XUP): XR rows x K, 1 KB per copy, same count on every wave ----
    if constexpr (XUP) {
        // a row of 2K bytes takes ceil(2K / 1 KB) copies; lanes past the row's end
        // re-read its last 16 bytes into the unused tail of the padded row stride
        const int per_row = (K + 511) >> 9;
        const int nx = XR * per_row;
        const int per_wave = (nx + kWaves - 1) / kWaves;
        for (int i = 0; i < per_wave; ++i) {
            const int q = min(wv + i * kWaves, nx - 1);
            const int r = q / per_row, part = q - r * per_row;
            const int e = min(part * 512 + 8 * lane, K - 8);
            copy16_to_lds(x + (size_t)min(r, M - 1) * K + e, xu + r * C::kXRowUp + part * 1024);
        }
    }

    // ---- ring of W and x tiles ----
    const int wf = 2 * wv + (lane >> 5), wslot = lane & 31;
    const int wchunk = tswz(wf, wslot);
    const uint16_t* wsrc = w + (size_t)min(n0 + wf, N - 1) * K;
    const int xidx = wv * C::kXLanes + lane;                  // chunk index inside the x tile
    const int xr = xidx >> 5, xchunk = tswz(xr, xidx & 31);
    const uint16_t* xsrc = x + (size_t)min(xr, M - 1) * K;
    // Tiles past the end are never issued: the last D tiles run in an unrolled
    // tail whose waits leave only the real tiles after them in flight.
    auto issue_tile = [&](int tt) {
        char* buf = ring + (tt % NB) * C::kTileBytes;
        const int d = tile_of(tt);
        const int kbw = min(d * kTileBlocks + (wchunk >> 2), KB - 1);
        copy16_to_lds_nt(wsrc + (size_t)kbw * 32 + 8 * (wchunk & 3), buf + wv * 1024);
        if (!XUP && lane < C::kXLanes) {
            const int kbx = min(d * kTileBlocks + (xchunk >> 2), KB - 1);
            copy16_to_lds(xsrc + (size_t)kbx * 32 + 8 * (xchunk & 3),
                          buf + C::kWBytes + wv * (C::kXLanes * 16));
        }
        __builtin_amdgcn_sched_barrier(0);
    };

    const int c = 4 * wv + g;                                 // this lane's chunk of a tile row
    const int woff = nl * kTileRow + 16 * tswz(nl, c);
    const int xrow = min(nl, XR - 1);
    const int xoff = C::kWBytes + xrow * kTileRow + 16 * tswz(xrow, c);
    f32x4 accb = {0.f, 0.f, 0.f, 0.f}, accs = {0.f, 0.f, 0.f, 0.f};
    auto compute = [&](int t) {
        const int kb = tile_of(t) * kTileBlocks + wv;
        if (kb < KB) {
            const char* buf = ring + (t % NB) * C::kTileBytes;
            const u32x4 bw = *reinterpret_cast<const u32x4*>(buf + woff);
            const u32x4 xa = XUP ? *reinterpret_cast<const u32x4*>(xu + xrow * C::kXRowUp + kb * 64 + 16 * g)
                                 : *reinterpret_cast<const u32x4*>(buf + xoff);
            const uint32_t sb = *reinterpret_cast<const uint8_t*>(
                sg + (kb >> 2) * 256 + nl * 16 + 4 * (kb & 3) + g);
            accb = mfma16<ET>(xa, bw, accb);
            accs = mfma16<ET>(xa, decode_signs8<ET>(sb), accs);
        }
    };

#pragma unroll
    for (int i = 0; i < D; ++i)
        if (i < KT) issue_tile(i);
    // tile t's copies are waited for with the D-1 later tiles left in flight
    for (int t = 0; t < KT - D; ++t) {
        wait_vm_lgkm0<(D - 1) * C::kOpsPerTile>();
        raw_barrier();
        issue_tile(t + D);              // into the buffer of tile t-1, free after the barrier
        compute(t);
    }
    // the last D tiles: tile KT-D+i has D-1-i real tiles after it in flight
    static_for<D>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        const int t = KT - D + i;
        if (t >= 0) {
            wait_vm_lgkm0<(D - 1 - i) * C::kOpsPerTile>();
            raw_barrier();
            compute(t);
        }
    });
    wait_vm_lgkm0<0>();
    __syncthreads();

    // ---- combine the waves' partial sums (fixed order) ----
    float* red_b = reinterpret_cast<float*>(lds);             // [wave][16 rows][16 feat]
    float* red_s = red_b + kWaves * 16 * kFeat;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        red_b[(wv * 16 + 4 * g + r) * kFeat + nl] = accb[r];
        red_s[(wv * 16 + 4 * g + r) * kFeat + nl] = accs[r];
    }
    __syncthreads();
    if (threadIdx.x < 16 * kFeat) {
        const int m = threadIdx.x / kFeat, f = threadIdx.x % kFeat;
        const int nn = n0 + f;
        if (m < M && nn < N) {
            float b = 0.f, s = 0.f;
#pragma unroll
            for (int v = 0; v < kWaves; ++v) {
                b += red_b[(v * 16 + m) * kFeat + f];
                s += red_s[(v * 16 + m) * kFeat + f];
            }
            const float out = __builtin_fmaf(alpha[0], s, b);
            store_y<ET>(y, (size_t)m * N + nn, out, y_dtype);
        }
    }
}

template <int ET, int XR>
hipError_t launch_stream(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                         const uint32_t* packed, const float* alpha, void* y, int y_dtype,
                         hipStream_t stream) {
    const int grid = (N + kFeat - 1) / kFeat;
    if constexpr (XR <= 4) {
        if (K <= 4096) {
            stream_decode_kernel<ET, XR, 8192, true><<<grid, kWaves * 64, 0, stream>>>(x, M, K, w, N, packed, alpha, y, y_dtype);
            return hipGetLastError();
        }
    }
    if (K <= 4096)
        stream_decode_kernel<ET, XR, 8192, false><<<grid, kWaves * 64, 0, stream>>>(x, M, K, w, N, packed, alpha, y, y_dtype);
    else
        stream_decode_kernel<ET, XR, 32768, false><<<grid, kWaves * 64, 0, stream>>>(x, M, K, w, N, packed, alpha, y, y_dtype);
    return hipGetLastError();
}

template <int ET>
hipError_t launch_decode_et(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                            const uint32_t* packed, const float* alpha, void* y, int y_dtype,
                            hipStream_t stream) {
    if (K >= 128 && (K & 127) == 0 && K <= 16384) {
        // signs of 16 features x K fit the staging area; rows of W split into whole chunks
        if (M == 1) return launch_stream<ET, 1>(x, M, K, w, N, packed, alpha, y, y_dtype, stream);
        if (M <= 4) return launch_stream<ET, 4>(x, M, K, w, N, packed, alpha, y, y_dtype, stream);
        return launch_stream<ET, 16>(x, M, K, w, N, packed, alpha, y, y_dtype, stream);
    }
    const int grid = (N + kFeat - 1) / kFeat;
    if (M == 1)
        decode_kernel<ET, 1><<<grid, kWaves * 64, 0, stream>>>(x, M, K, w, N, packed, alpha, y, y_dtype);
    else if (M <= 4)
        decode_kernel<ET, 4><<<grid, kWaves * 64, 0, stream>>>(x, M, K, w, N, packed, alpha, y, y_dtype);
    else
        decode_kernel<ET, 16><<<grid, kWaves * 64, 0, stream>>>(x, M, K, w, N, packed, alpha, y, y_dtype);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                         const uint32_t* packed, const float* alpha, void* y, int y_dtype,
                         int et, hipStream_t stream) {
    if (et == kF16) return launch_decode_et<kF16>(x, M, K, w, N, packed, alpha, y, y_dtype, stream);
    return launch_decode_et<kBF16>(x, M, K, w, N, packed, alpha, y, y_dtype, stream);
}

}  // namespace bitdelta
