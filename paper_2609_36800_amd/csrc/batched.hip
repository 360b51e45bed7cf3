// Batched (multi-tenant) binary-delta matmul for up to 64 token rows with at
// most 16 distinct tenants per call, K a multiple of 128 or 256 by
// configuration (batched_supported says which requests take it):
//
//   y[m][n] = sum_k x[m][k] W[n][k] + alpha[t(m)] * sum_k x[m][k] s_t(m)[n][k]
//
// (the batched BitDelta GEMM of Section 4.4 at decode shapes).
//
// Cost model.  Every byte of W and the sign bits of each tenant present are
// read once from HBM; x (a few hundred KB) is re-read from L2 by every
// workgroup.  Turning one byte of sign bits into the eight bf16 +-1 values of
// an MFMA operand takes nine VALU instructions, against 16 cycles for the
// v_mfma_f32_16x16x32 that consumes them, so each tenant's signs are decoded
// once per (16 features, 32-k block) and drive one product over all of that
// tenant's rows.
//
// Routing.  The rows of each tenant are gathered into fragments of up to 16
// rows (F fragments in all, a tenant with more rows gets more).  Per 32-k
// block a fragment costs one x fragment read, one sign decode and two MFMAs
// (x*W^T and x*S_t^T on the gathered rows).  F is known only on the device:
// every workgroup computes the routing (wave 0, ballots) and enters the loop
// specialised for its F.  Sign slot u holds tenant u when there are at most
// as many tenants as slots, so the first tiles' copies go out before the
// routing is known (after it, the slots of tenants without rows are filled
// from a present tenant's rows, which L2 already holds); with more tenants the
// slots are compacted to the tenants present and the copies wait for the
// routing.
//
// Memory path.  A workgroup of WV waves (8 or 4) owns 16 output features; K
// runs in 32*WV-k tiles and wave w computes k-block w of every tile.  All
// operands reach LDS by global->LDS copies of long row segments (a full cache
// line or more per row), in three rings:
//   W      16 rows x 64*WV B per tile, NWR slots, issued NWR-1 tiles ahead;
//   x      XR rows x 64*WV B per tile, NXR slots, issued NXR-1 tiles ahead;
//   signs  UMAX tenant slots x 16 rows x 16*WV B per super-tile (four
//          tiles), 2 slots.  The next super-tile is copied in two halves
//          during the first two tiles of the current one (its slot was last
//          read by the previous super-tile), and the last two tiles repeat
//          the second half, so every tile issues the same copies.
// Each tile's issue group is [sign part, x, W]: loads retire in issue order,
// so one s_waitcnt vmcnt for the x of the tile about to be computed also
// covers every earlier sign part while the deeper W ring stays in flight, and
// one barrier per tile publishes the tile.
//
// Occupancy.  The 8-wave configurations take 133 to 157 KB of LDS, one
// workgroup per CU: with at most 256 workgroups (N <= 4096) the whole grid is
// resident at once and each workgroup's eight waves split K finely.  Larger
// grids run in rounds; there the 4-wave configurations (49 to 69 KB) hold two
// or three workgroups per CU, so one workgroup's waits and barriers overlap
// another's copies and products, and the last round is shorter.
//
// The waves' partial sums are added in a fixed order through LDS, so the
// result is bitwise deterministic.
#include <utility>

#include "device.h"
#include "internal.h"
#include "ldscopy.h"

namespace bitdelta {
namespace {

constexpr int kFeat = 16;
constexpr int kRowsMax = 64;
constexpr int kSuperTiles = 4;                 // tiles per sign super-tile
constexpr int kCUs = 256;                      // MI355X compute units

// Tile geometry of a WV-wave workgroup: one 32-k block per wave and tile.
template <int WV>
struct Geo {
    static constexpr int kWaves = WV;
    static constexpr int kTileK = 32 * WV;                        // k per tile
    static constexpr int kRowBytes = 2 * kTileK;                  // one row of a W or x tile
    static constexpr int kLanesPerRow = kRowBytes / 16;           // 16-byte chunks per row
    static constexpr int kRowsPerCopy = 64 / kLanesPerRow;        // rows per 1 KB copy
    static constexpr int kSignRowBytes = kSuperTiles * kTileK / 8;   // sign bits of a row per super-tile
    static constexpr int kSLanes = kSignRowBytes / 16;            // chunks per sign row
    static constexpr int kSRowsPerCopy = 64 / kSLanes;
    // Sign rows are read one byte per feature row li; rows kSignRowBytes apart
    // repeat the bank pattern every 256 / kSignRowBytes rows, and XOR-ing the
    // chunk with the bits above that period puts those rows in distinct banks.
    static __device__ __forceinline__ int sswz(int row) {
        return kSLanes == 8 ? (row & 7) : ((row >> 2) & 3);
    }
    static_assert(kSLanes == 8 || kSLanes == 4, "sign row layout");
};

__device__ __forceinline__ int swz16(int row, int chunk) { return chunk ^ (row & 15); }

struct Routing {
    int tenant_of_row[kRowsMax];          // -1: id out of range
    int frag_of_row[kRowsMax];            // fragment holding row m, -1: none
    int frag_row[kRowsMax][16];           // row in slot i of fragment f, -1: empty
    int frag_slot[kRowsMax];              // sign slot (distinct-tenant index) of fragment f
    int slot_tenant[16];                  // tenant of sign slot u
    uint32_t key_sorted[kRowsMax];
    int sorted_row[kRowsMax];
    int nfrag, nslot;
};

template <int XR, int UMAX, int NWR, int NXR, int WV>
struct BatchedLayout {
    using G = Geo<WV>;
    static constexpr int kW = kFeat * G::kRowBytes;               // per W slot (one copy per wave)
    static constexpr int kX = XR * G::kRowBytes;                  // per x slot
    static constexpr int kS = UMAX * kFeat * G::kSignRowBytes;    // per sign slot
    static constexpr int kWOff = 0;
    static constexpr int kXOff = NWR * kW;
    static constexpr int kSOff = kXOff + NXR * kX;
    static constexpr int kRouteOff = kSOff + 2 * kS;
    static constexpr int kTotal = kRouteOff + (int)sizeof(Routing);
    // per-wave partials [wave][row][feature], base then sign, reuse the W and x rings
    static constexpr int kRed = WV * XR * kFeat * 4;             // rows m < M <= XR
    static_assert(2 * kRed <= kSOff, "reduction area must fit in the W and x rings");
    static_assert(kTotal <= 160 * 1024, "LDS budget");
    // copies per wave per tile: sign part, x, W
    static constexpr int kXOps = XR * G::kRowBytes / 1024 / WV;
    static constexpr int kSOps = UMAX * 8 / G::kSRowsPerCopy / WV;   // half a super-tile
    static_assert(kW == 1024 * WV, "one W copy per wave and tile");
    static_assert(kXOps >= 1 && kXOps * 1024 * WV == kX, "x copies");
    static_assert(kSOps >= 1 && kSOps * G::kSRowsPerCopy * WV == UMAX * 8, "sign copies");
    static_assert(UMAX == 8 || UMAX == 16, "sign slots");
    static_assert(NXR >= 2 && NWR >= NXR, "ring depths");
};

// The global->LDS copies of one wave's share of the rings: W rows, x rows and
// sign rows of copy-wave index cw (normally the wave's own index; another wave
// can issue a share on its behalf).  All sources are clamped in range; surplus
// rows feed unstored outputs.  tenant_of_slot(u) gives the tenant whose sign
// rows fill slot u.
template <int XR, int UMAX, int NWR, int NXR, int WV>
struct Copier {
    using L = BatchedLayout<XR, UMAX, NWR, NXR, WV>;
    using G = Geo<WV>;
    static constexpr int DX = NXR - 1, DW = NWR - 1;
    char* lds;
    int cw, KT, KW, NS, schunk;
    const uint16_t* wsrc;
    const uint16_t* xsrc[L::kXOps];
    int srow[2][L::kSOps];
    const uint32_t* ssrc[2][L::kSOps];

    template <class SlotFn>
    __device__ __forceinline__ Copier(char* lds_, int cw_, int lane, const uint16_t* __restrict__ x, int M, int K,
                                      const uint16_t* __restrict__ w, int N, const uint32_t* __restrict__ packed,
                                      int n0, SlotFn tenant_of_slot)
        : lds(lds_), cw(cw_) {
        KT = K / G::kTileK;
        KW = K >> 5;
        NS = (KT + kSuperTiles - 1) / kSuperTiles;
        // W: copy-wave c copies rows c*RPC .. (RPC rows per copy), lane l its row's
        // 16-byte chunk l % LPR, swizzled
        const int lrow = lane / G::kLanesPerRow, lch = lane % G::kLanesPerRow;
        const int wrow = G::kRowsPerCopy * cw + lrow;
        wsrc = w + (size_t)min(n0 + wrow, N - 1) * K + 8 * swz16(wrow, lch);
        // x: copy i of copy-wave c holds rows RPC*(c*XOPS + i) ..
#pragma unroll
        for (int i = 0; i < L::kXOps; ++i) {
            const int r = G::kRowsPerCopy * (cw * L::kXOps + i) + lrow;
            xsrc[i] = x + (size_t)min(r, M - 1) * K + 8 * swz16(r, lch);
        }
        // signs: the UMAX*16 (slot, feature) rows of a super-tile, SRPC per copy
        // with SL lanes per row; half h holds rows [h*UMAX*8, (h+1)*UMAX*8), copy j
        // of copy-wave c its rows SRPC*(c*kSOps + j) ..
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int j = 0; j < L::kSOps; ++j) {
                srow[h][j] = h * UMAX * 8 + G::kSRowsPerCopy * (cw * L::kSOps + j) + lane / G::kSLanes;
                const int u = srow[h][j] >> 4, f = srow[h][j] & 15;
                ssrc[h][j] = packed + ((size_t)tenant_of_slot(u) * N + min(n0 + f, N - 1)) * KW;
            }
        schunk = lane % G::kSLanes;
    }
    __device__ __forceinline__ void issue_x(int tt) const {
        const int tc = min(tt, KT - 1);
        char* buf = lds + L::kXOff + (tt % NXR) * L::kX;
#pragma unroll
        for (int i = 0; i < L::kXOps; ++i)
            copy16_to_lds(xsrc[i] + (size_t)tc * G::kTileK, buf + (cw * L::kXOps + i) * 1024);
    }
    __device__ __forceinline__ void issue_w(int tt) const {
        const int tc = min(tt, KT - 1);
        copy16_to_lds_nt(wsrc + (size_t)tc * G::kTileK, lds + L::kWOff + (tt % NWR) * L::kW + cw * 1024);
    }
    // half h of super-tile s
    __device__ __forceinline__ void issue_s(int s, int h) const {
        const int sc = min(s, NS - 1);
#pragma unroll
        for (int j = 0; j < L::kSOps; ++j) {
            const int c = schunk ^ G::sswz(srow[h][j]);            // source chunk at this position
            const int word = min(G::kSignRowBytes / 4 * sc + 4 * c, KW - 4);
            const int drow = h * UMAX * 8 + G::kSRowsPerCopy * (cw * L::kSOps + j);   // first row of this copy
            copy16_to_lds(ssrc[h][j] + word, lds + L::kSOff + (s & 1) * L::kS + drow * G::kSignRowBytes);
        }
    }
    // prologue: super-tile 0, then x(0 .. DX-1) and W(0 .. DW-1)
    __device__ __forceinline__ void prologue_s() const {
        issue_s(0, 0);
        issue_s(0, 1);
    }
    __device__ __forceinline__ void prologue_xw(bool do_x, bool do_w) const {
#pragma unroll
        for (int i = 0; i < DW; ++i) {
            if (do_x && i < DX) issue_x(i);
            if (do_w) issue_w(i);
        }
    }
};

// One pass over K for fragments f0 .. f0+F-1.  With `issued` the prologue
// copies (super-tile 0, x(0 .. DX-1), W(0 .. DW-1)) are already in flight.
template <int ET, int XR, int UMAX, int NWR, int NXR, int WV, int F>
__device__ __forceinline__ void batched_loop(char* lds, const Routing& rt, const uint16_t* __restrict__ x,
                                             int M, int K, const uint16_t* __restrict__ w, int N,
                                             const uint32_t* __restrict__ packed, int n0, int lane, int wv,
                                             int f0, bool issued) {
    using L = BatchedLayout<XR, UMAX, NWR, NXR, WV>;
    using G = Geo<WV>;
    const int li = lane & 15, g = lane >> 4;
    const int KT = K / G::kTileK;
    const Copier<XR, UMAX, NWR, NXR, WV> cp(lds, wv, lane, x, M, K, w, N, packed, n0,
                                            [&](int u) { return rt.slot_tenant[min(u, rt.nslot - 1)]; });

    // ---- fragment read offsets ----
    const int wchunk = 4 * wv + g;                                  // this lane's chunk of a tile row
    const int woff = li * G::kRowBytes + 16 * swz16(li, wchunk);
    // sign rows are (slot * 16 + feature): the swizzle key sswz(row) is sswz(li)
    // for every slot, and a fragment's slot only moves the row base (wave-uniform)
    int xoff[F];
    uint32_t sslot[F];
#pragma unroll
    for (int f = 0; f < F; ++f) {
        int r = rt.frag_row[f0 + f][li];
        if (r < 0) r = rt.frag_row[f0 + f][0];
        xoff[f] = r * G::kRowBytes + 16 * swz16(r, wchunk);
        sslot[f] = __builtin_amdgcn_readfirstlane((uint32_t)rt.frag_slot[f0 + f] * (kFeat * G::kSignRowBytes));
    }
    const int slane = li * G::kSignRowBytes + g + 4 * (wv & 3);    // + chunk per tile
    const int sswz = G::sswz(li);
    f32x4 accb[F], accs[F];
#pragma unroll
    for (int f = 0; f < F; ++f) {
        accb[f] = f32x4{0.f, 0.f, 0.f, 0.f};
        accs[f] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // ---- prologue: super-tile 0, then the issue groups of tiles 0 .. NXR-2 / NWR-2 ----
    constexpr int DX = NXR - 1, DW = NWR - 1;
    if (!issued) {
        cp.prologue_s();
        cp.prologue_xw(true, true);
    }
    __builtin_amdgcn_sched_barrier(0);

    // vmcnt after which the x of tile t (and so every sign part before it) and
    // the W of tile t have landed: the copies issued later are the W of the
    // group that issued x(t) (unless that group issued W(t) itself) and the DX-1
    // whole groups after it
    constexpr int kGroup = L::kSOps + L::kXOps + 1;
    constexpr int kWait = (DW > DX ? 1 : 0) + (DX - 1) * kGroup;
    for (int t = 0; t < KT; ++t) {
        if (t == 0) wait_vm_lgkm0<0>();
        else wait_vm_lgkm0<kWait>();
        raw_barrier();
        // issue group: sign half (t&3 < 2 ? t&3 : 1) of super-tile t/4+1, x(t+DX), W(t+DW)
        cp.issue_s((t >> 2) + 1, min(t & 3, 1));
        cp.issue_x(t + DX);
        cp.issue_w(t + DW);
        __builtin_amdgcn_sched_barrier(0);

        const int kb = t * WV + wv;
        if (kb < (K >> 5)) {
            const char* wbuf = lds + L::kWOff + (t % NWR) * L::kW;
            const char* xbuf = lds + L::kXOff + (t % NXR) * L::kX;
            const char* sbuf = lds + L::kSOff + ((t >> 2) & 1) * L::kS;
            // this wave's word of the tile is word WV*(t&3) + wv of the super-tile
            // row: chunk (WV*(t&3) + wv) / 4, stored at chunk ^ sswz(row)
            const char* srd = sbuf + slane + 16 * (((WV * (t & 3) + wv) >> 2) ^ sswz);
            const u32x4 bw = *reinterpret_cast<const u32x4*>(wbuf + woff);
            // all of the tile's LDS reads first, so their latencies overlap
            uint32_t sb[F];
            u32x4 xa[F];
#pragma unroll
            for (int f = 0; f < F; ++f) {
                sb[f] = *reinterpret_cast<const uint8_t*>(srd + sslot[f]);
                xa[f] = *reinterpret_cast<const u32x4*>(xbuf + xoff[f]);
            }
#pragma unroll
            for (int f = 0; f < F; ++f) {
                accb[f] = mfma16<ET>(xa[f], bw, accb[f]);
                accs[f] = mfma16<ET>(xa[f], decode_signs8<ET>(sb[f]), accs[f]);
            }
        }
    }
    // drain the copies of the tail tiles, then the rings become the reduction area
    wait_vm_lgkm0<0>();
    __syncthreads();
    float* red_b = reinterpret_cast<float*>(lds);                  // [wave][row][feature]
    float* red_s = red_b + WV * XR * kFeat;
#pragma unroll
    for (int f = 0; f < F; ++f)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = rt.frag_row[f0 + f][4 * g + r];
            if (row >= 0) {
                red_b[(wv * XR + row) * kFeat + li] = accb[f][r];
                red_s[(wv * XR + row) * kFeat + li] = accs[f][r];
            }
        }
}

// Waves per SIMD the register budget must allow: three 4-wave workgroups per
// CU where three fit in LDS, else two workgroups (4 waves) or one (8 waves).
template <int XR, int UMAX, int NWR, int NXR, int WV>
constexpr int waves_per_simd() {
    return (WV == 4 && 3 * BatchedLayout<XR, UMAX, NWR, NXR, WV>::kTotal <= 160 * 1024) ? 3 : 2;
}

template <int ET, int XR, int UMAX, int NWR, int NXR, int WV>
__global__ __launch_bounds__(WV * 64, (waves_per_simd<XR, UMAX, NWR, NXR, WV>())) void batched_decode_kernel(
    const uint16_t* __restrict__ x, int M, int K, const uint16_t* __restrict__ w, int N,
    const uint32_t* __restrict__ packed, const float* __restrict__ alpha,
    const int32_t* __restrict__ tenant_ids, int T, void* __restrict__ y, int y_dtype) {
    using L = BatchedLayout<XR, UMAX, NWR, NXR, WV>;
    constexpr int kThreads = WV * 64;
    __shared__ __attribute__((aligned(16))) char lds[L::kTotal];
    Routing& rt = *reinterpret_cast<Routing*>(lds + L::kRouteOff);
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n0 = blockIdx.x * kFeat;
    constexpr uint32_t kKeyInvalid = 0x80000000u, kKeyPad = 0x80000001u;

    // ---- with at most UMAX tenants, sign slot u holds tenant u (absent tenants'
    //      slots are copied and not read), so the first tiles' copies do not
    //      depend on the routing and go out now, while wave 0 routes.  Wave 0's
    //      share is issued by the last three waves: its id load must not queue
    //      behind copies of its own. ----
    const bool ident = T <= UMAX;
    if (ident && wv != 0) {
        auto ident_slot = [&](int u) { return min(u, T - 1); };
        const Copier<XR, UMAX, NWR, NXR, WV> own(lds, wv, lane, x, M, K, w, N, packed, n0, ident_slot);
        own.prologue_s();
        own.prologue_xw(true, true);
        if (wv >= WV - 3) {
            const Copier<XR, UMAX, NWR, NXR, WV> w0(lds, 0, lane, x, M, K, w, N, packed, n0, ident_slot);
            if (wv == WV - 3) w0.prologue_s();
            w0.prologue_xw(wv == WV - 2, wv == WV - 1);
        }
    }

    for (int i = threadIdx.x; i < kRowsMax * 16; i += kThreads) (&rt.frag_row[0][0])[i] = -1;
    // ---- routing (wave 0): stable sort of the rows by tenant ----
    if (wv == 0) {
        uint32_t key = kKeyPad;
        if (lane < M) {
            const int t = tenant_ids[lane];
            key = (t >= 0 && t < T) ? (uint32_t)t : kKeyInvalid;
        }
        int rank = 0;
        for (int j = 0; j < kRowsMax; ++j) {
            const uint32_t kj = __builtin_amdgcn_readlane(key, j);
            rank += (kj < key || (kj == key && j < lane)) ? 1 : 0;
        }
        rt.sorted_row[rank] = lane < M ? lane : 0;
        rt.key_sorted[rank] = key;
        rt.tenant_of_row[lane] = key < kKeyInvalid ? (int)key : -1;
        rt.frag_of_row[lane] = -1;
    }
    __syncthreads();
    // ---- fragments (runs of up to 16 rows of one tenant) and sign slots ----
    if (wv == 0) {
        const int p = lane;
        const uint32_t kp = rt.key_sorted[p];
        const uint32_t kprev = p > 0 ? rt.key_sorted[p - 1] : 0xFFFFFFFFu;
        const bool valid = kp < kKeyInvalid;
        const unsigned long long upto = p == 63 ? ~0ull : ((2ull << p) - 1ull);
        const unsigned long long tstart = __ballot(valid && kp != kprev);
        const int first = 63 - __builtin_clzll((tstart & upto) | 1ull);
        const int rank = p - first;
        const int slot = ident ? (int)kp : __popcll(tstart & upto) - 1;
        const unsigned long long fstart = __ballot(valid && (rank & 15) == 0);
        const int fidx = __popcll(fstart & upto) - 1;
        if (valid) {
            rt.frag_row[fidx][rank & 15] = rt.sorted_row[p];
            rt.frag_of_row[rt.sorted_row[p]] = fidx;
            if ((rank & 15) == 0) rt.frag_slot[fidx] = slot;
            if (!ident && rank == 0 && slot < 16) rt.slot_tenant[slot] = (int)kp;
        }
        if (ident) {
            // slot u holds tenant u; the slots of tenants without rows (never
            // read) copy the first present tenant's rows instead, from L2
            const uint32_t k0 = __builtin_amdgcn_readfirstlane(kp);
            if (lane < T) rt.slot_tenant[lane] = k0 < kKeyInvalid ? (int)k0 : 0;
            if (valid && kp != kprev) rt.slot_tenant[kp] = (int)kp;
        }
        if (lane == 0) {
            rt.nfrag = __popcll(fstart);
            rt.nslot = ident ? T : __popcll(tstart);
        }
    }
    __syncthreads();
    const int F = rt.nfrag;

    // ---- main loop, specialised for the fragment count; passes of FMAX fragments ----
    // fragments per pass: all of them up to 16 (12 for 64 rows x 16 tenants, to fit registers)
    constexpr int FMAX = (XR == 64 && UMAX == 16) ? 12 : ((XR / 16 + UMAX) < 16 ? (XR / 16 + UMAX) : 16);
    const float* red_b = reinterpret_cast<const float*>(lds);
    const float* red_s = red_b + WV * XR * kFeat;
    for (int f0 = 0; f0 < F; f0 += FMAX) {
        const int fc = min(FMAX, F - f0);
        static_for<FMAX>([&](auto ic) {
            constexpr int FC = decltype(ic)::value + 1;
            if (fc == FC)
                batched_loop<ET, XR, UMAX, NWR, NXR, WV, FC>(lds, rt, x, M, K, w, N, packed, n0, lane, wv, f0,
                                                         ident && f0 == 0);
        });
        __syncthreads();
        for (int idx = threadIdx.x; idx < M * kFeat; idx += kThreads) {
            const int m = idx >> 4, ff = idx & 15;
            const int nn = n0 + ff;
            const int fr = rt.frag_of_row[m];
            if (nn >= N || fr < f0 || fr >= f0 + fc) continue;
            float bsum = 0.f, ssum = 0.f;
#pragma unroll
            for (int v = 0; v < WV; ++v) {
                bsum += red_b[(v * XR + m) * kFeat + ff];
                ssum += red_s[(v * XR + m) * kFeat + ff];
            }
            store_y<ET>(y, (size_t)m * N + nn, __builtin_fmaf(alpha[rt.tenant_of_row[m]], ssum, bsum), y_dtype);
        }
        __syncthreads();        // the next pass reuses the rings
    }
    // rows whose tenant id is out of range
    for (int idx = threadIdx.x; idx < M * kFeat; idx += kThreads) {
        const int m = idx >> 4, nn = n0 + (idx & 15);
        if (nn < N && rt.tenant_of_row[m] < 0) store_y<ET>(y, (size_t)m * N + nn, __builtin_nanf(""), y_dtype);
    }
}

template <int ET, int XR, int UMAX, int NWR, int NXR, int WV = 8>
hipError_t launch_cfg(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                      const uint32_t* packed, const float* alpha, const int32_t* tenant_ids, int T,
                      void* y, int y_dtype, hipStream_t stream) {
    if (M > XR || K % Geo<WV>::kTileK != 0) return hipErrorInvalidValue;   // x rows staged, whole tiles
    const int grid = (N + kFeat - 1) / kFeat;
    batched_decode_kernel<ET, XR, UMAX, NWR, NXR, WV><<<grid, WV * 64, 0, stream>>>(
        x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype);
    return hipGetLastError();
}

// More workgroups than CUs: the grid runs in rounds.
bool several_rounds(int N) { return (N + kFeat - 1) / kFeat > kCUs; }

template <int ET>
hipError_t launch_et(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                     const uint32_t* packed, const float* alpha, const int32_t* tenant_ids, int T,
                     void* y, int y_dtype, hipStream_t stream) {
    // Measured on MI355X (us, 4096 deep, 8 / 16 tenants):
    //   64 x 4096:  8 waves 24.6, 4 waves 29  (one round: 8 waves)
    //   64 x 11008: 8 waves 65.8, 4 waves x 2/CU 61.4; at 16 slots 137 / 147
    //   32 x 11008: tenant-slot kernel 52.3 / 76.8, 4 waves 41.3 (3/CU) / 68.4
    //   16 x 11008: tenant-slot kernel 43.5, 4 waves x 3/CU 38.3
    // Ring depths between 2 and 7 tiles move the 8-wave times by under 5%
    // (32 rows x 4096^2, 8 tenants: 20.1-20.5 us at 3 x 3, 19.3-19.5 at 4 x 4).
    const bool few = min(T, M) <= 8;
    const bool rounds = several_rounds(N);
#define BD_CFG(XR, U, NW, NX, WV) \
    return launch_cfg<ET, XR, U, NW, NX, WV>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream)
    if (M <= 32) {
        if (rounds) {
            if (few) BD_CFG(32, 8, 3, 2, 4);        // 49 KB LDS, 163 VGPRs: three per CU
            BD_CFG(32, 16, 4, 2, 4);                // 69 KB: two per CU
        }
        if (few) BD_CFG(32, 8, 4, 4, 8);            // 133 KB: 4% faster than 3-deep rings
        BD_CFG(32, 16, 3, 3, 8);
    }
    if (few) {
        if (rounds) BD_CFG(64, 8, 4, 2, 4);         // 69 KB: two per CU
        BD_CFG(64, 8, 3, 3, 8);
    }
    BD_CFG(64, 16, 3, 2, 8);
#undef BD_CFG
}

}  // namespace

bool batched_supported(int M, int N, int K, int T) {
    // Asked only for requests the wide form (wide.hip: 48 or 64 features per
    // workgroup where those groups fill the CUs) does not take.
    // One round (N <= 4096): the 8-wave kernel for 17 to 64 rows; the
    // tenant-slot kernel (multi.hip, two workgroups per CU) is as fast or
    // faster at 16 rows and below.  Several rounds: every row count from 17,
    // and 8 to 16 rows with at most 8 tenant slots (three 4-wave workgroups per
    // CU); at fewer rows, or more slots, a fragment carries too few rows to
    // gain over the tenant-slot kernel.  Tiles are 256 deep for 8 waves, 128
    // for 4; 33 to 64 rows over more than 8 slots keep 8 waves.
    const int u = min(T, M);
    if (M < 1 || M > kRowsMax || u > 16 || K < 128 || K % 128 != 0) return false;
    if (!several_rounds(N)) return M > 16 && K % 256 == 0;
    if (M > 32) return u <= 8 || K % 256 == 0;
    return M > 16 || (M >= 8 && u <= 8);
}

hipError_t launch_batched(const uint16_t* x, int M, int K, const uint16_t* w, int N,
                          const uint32_t* packed, const float* alpha, const int32_t* tenant_ids,
                          int T, void* y, int y_dtype, int et, hipStream_t stream) {
    if (et == kF16)
        return launch_et<kF16>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
    return launch_et<kBF16>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
}

}  // namespace bitdelta
