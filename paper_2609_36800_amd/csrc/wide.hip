// Batched (multi-tenant) binary-delta matmul at decode shapes, wide form: 17
// to 64 token rows, at most 8 or 16 distinct tenants present, K a multiple of
// 128, and N such that groups of 48 or 64 features fill the CUs:
//
//   y[m][n] = sum_k x[m][k] W[n][k] + alpha[t(m)] * sum_k x[m][k] s_t(m)[n][k]
//
// (the batched BitDelta GEMM of Section 4.4 at decode shapes).
//
// Cost model.  W and the sign rows of the tenants present are read once from
// HBM; x is re-read from L2 by every workgroup.  What limits a copy stream on
// this part is less its bytes than the number of distinct cache lines each
// CU has in flight, so every copy here moves whole lines (128-byte row
// segments of W and x, 64-byte segments of sign rows) and a workgroup owns 48
// or 64 output features: x lines per W line fall to rows/48 or rows/64
// (rows/16 with 16 features).
//
// Routing.  Wave 0 sorts the rows by tenant (ballots) into fragments of up to
// 16 rows of one tenant; past the first 512-k super-tile, sign slot u holds the
// u-th tenant present, so only present tenants' signs are copied (the first
// super-tile holds tenant u in slot u and is copied while wave 0 routes).
// Wave w computes the sign products of
// fragments w, w+8, w+16 against all 16*FB features (per 32-k block one x
// read, FB sign decodes and FB MFMAs) and x*W^T on the rows in their own order
// for its share of the (16-row block, 16-feature block) pairs (one MFMA per 16
// rows rather than per fragment); the two sums meet in LDS at the end as
// acc_base + alpha*acc_sign.
//
// Memory path (8 waves, one workgroup per CU).  K runs in 64-k tiles.  A ring
// of NB slots holds W (16*FB rows x 128 B) and x (XR rows x 128 B) per tile,
// issued NB tiles ahead with up to 8 sign slots (a slot is refilled as soon as
// its tile's operands are in registers), NB - 1 with 16; signs come in 512-k
// super-tiles (64 B per row), double-buffered, super-tile j+1 issued in pieces
// during the first steps of super-tile j, early enough that the in-order wait
// for a tile also covers the signs it reads.  Every wave issues the same
// number of copies per step (past the end of K, or with no real work, a copy
// of one hot line instead), so one s_waitcnt vmcnt count and one barrier per
// step hand a tile over.  Operands
// are read from LDS one step ahead of the arithmetic that uses them.  The loop
// runs sixteen steps per pass, so ring slots, super-tile phases and sign words
// are compile-time offsets of the LDS reads.
#include "device.h"
#include "internal.h"
#include "ldscopy.h"

namespace bitdelta {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kTK = 64;                  // k per tile: two 32-k blocks
constexpr int kRowB = kTK * 2;           // bytes of one W or x row per tile (one cache line)
constexpr int kSK = 512;                 // k per sign super-tile
constexpr int kSRowB = kSK / 8;          // bytes of one sign row per super-tile
constexpr int kR = kSK / kTK;            // tiles per super-tile
constexpr int kMaxRows = 64;
constexpr int kMaxFrags = 24;            // 3 per wave
constexpr int kCUs = 256;
static_assert(kR == 8, "tile -> super-tile arithmetic uses shifts by 3");

struct WideRouting {
    int tenant_of_row[kMaxRows];         // -1: id out of range or no row
    int frag_row[kMaxFrags][16];         // row in slot i of fragment f, -1: empty
    int frag_slot[kMaxFrags];            // sign slot of fragment f
    int slot_tenant[16];                 // tenant of sign slot u
    int sorted_row[kMaxRows];
    uint32_t key_sorted[kMaxRows];
    int nfrag, nslot;
};

// FB: 16-feature blocks per workgroup; XR: x rows staged (>= M); U: sign slots;
// NB: ring slots (a power of two dividing 8).
template <int FB, int XR, int U, int NB>
struct WideCfg {
    static constexpr int NF = 16 * FB;
    // Tiles issued ahead.  With up to 8 sign slots a slot is refilled as soon
    // as its tile's operands are in registers (D = NB, 1-3% faster); with 16
    // the larger sign pieces make the shallower order faster (D = NB - 1, 2%).
    static constexpr bool kEarly = U <= 8;
    static constexpr int D = kEarly ? NB : NB - 1;
    static constexpr int kW = NF * kRowB;
    static constexpr int kX = XR * kRowB;
    static constexpr int kSlot = kW + kX;
    static constexpr int kWRows = NF / kWaves, kXRows = XR / kWaves;   // rows each wave copies per tile
    static constexpr int kSBuf = U * NF * kSRowB;          // one sign super-tile
    static constexpr int nSup = kSBuf / 1024;              // its 1-KB copies
    static constexpr int kPieces = kR - D + 1;             // steps of a super-tile that issue the next one
    static constexpr int cS = (nSup + kWaves * kPieces - 1) / (kWaves * kPieces);
    static constexpr int ops = 2 + cS;                     // copies per wave per step
    static constexpr int FW = U == 8 ? 2 : 3;              // fragments per wave
    static constexpr int RB = XR / 16;                     // natural row blocks
    static constexpr int NBJ = (RB * FB + kWaves - 1) / kWaves;   // base pairs per wave
    // LDS: signs first, then the ring (the uniform parts of the read addresses
    // then fit the 16-bit offset field), the padding target, the routing
    static constexpr int kRingOff = 2 * kSBuf;
    static constexpr int kDummyOff = kRingOff + NB * kSlot;
    static constexpr int kRouteOff = kDummyOff + 1024;
    static constexpr int kTotal = kRouteOff + (int)sizeof(WideRouting);
    static_assert(kTotal <= 160 * 1024, "LDS budget");
    static_assert(NB == 2 || NB == 4 || NB == 8, "ring slots: a power of two dividing 8");
    static_assert(kPieces >= 1 && D >= 2, "ring depth");
    static_assert((kMaxRows + 15 * U) / 16 <= kWaves * FW, "fragments per wave");
    static_assert(NF % kWaves == 0 && XR % kWaves == 0 && kWaves % RB == 0, "copy and base split");
    static_assert((NB - 1) * kSlot + (FB - 1) * 16 * kRowB < 65536, "ring read offsets");
    static_assert(kSBuf + (FB - 1) * 16 * kSRowB + 12 < 65536, "sign read offsets");
};

// Row r of a 128-byte-row tile stores its 16-byte chunk c at 16*(c ^ key128(r)),
// and row r of a 64-byte sign row block its chunk c at 16*(c ^ key64(r)):
// sixteen consecutive rows then cover all banks once.
__device__ __forceinline__ int key128(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ int key64(int r) { return (r >> 2) & 3; }

// The sign bytes of both 32-k blocks of a tile -> their two MFMA operands
// (eight +1/-1 each, as decode_signs8).  Each byte, duplicated 15 bits up,
// sits in one half of a 64-bit value, so one 64-bit shift serves both blocks;
// bits shifted across the halves land below bit 6 and are masked off.
// (Measured 9-10% faster than two decode_signs8 at 32 and 64 rows.)
template <int ET>
__device__ __forceinline__ void decode_signs8x2(uint32_t w0, uint32_t w1, int bit0, u32x4& r0, u32x4& r1) {
    const uint32_t b0 = __builtin_amdgcn_ubfe(w0, bit0, 8), b1 = __builtin_amdgcn_ubfe(w1, bit0, 8);
    const uint64_t s = (uint64_t)opaque_u32(b0 | (b0 << 15)) | ((uint64_t)opaque_u32(b1 | (b1 << 15)) << 32);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        uint64_t t;
        asm("v_lshlrev_b64 %0, %1, %2" : "=v"(t) : "n"(15 - 2 * j), "v"(s));
        r0[j] = kMinusOnePair<ET> ^ ((uint32_t)t & kSignBits);
        r1[j] = kMinusOnePair<ET> ^ ((uint32_t)(t >> 32) & kSignBits);
    }
}

template <int ET, int FB, int XR, int U, int NB>
__global__ __launch_bounds__(kThreads) void wide_batched_kernel(
    const uint16_t* __restrict__ x, int M, int K, const uint16_t* __restrict__ w, int N,
    const uint32_t* __restrict__ packed, const float* __restrict__ alpha,
    const int32_t* __restrict__ tenant_ids, int T, void* __restrict__ y, int y_dtype) {
    using C = WideCfg<FB, XR, U, NB>;
    constexpr int NF = C::NF, D = C::D, FW = C::FW, RB = C::RB, NBJ = C::NBJ;
    __shared__ __attribute__((aligned(16))) char lds[C::kTotal];
    WideRouting& rt = *reinterpret_cast<WideRouting*>(lds + C::kRouteOff);
    char* const ring = lds + C::kRingOff;
    char* const dummy = lds + C::kDummyOff;
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nl = lane & 15, g = lane >> 4;
    const int n0 = blockIdx.x * NF;
    const int KT = K / kTK;                                // 2 or more; steps past KT issue only padding copies
    const int KW = K >> 5;
    const char* const hot = reinterpret_cast<const char*>(packed);

    // ---- W and x copies: wave wv copies W rows [wv*kWRows, +kWRows) and x rows
    //      [wv*kXRows, +kXRows) of each tile, 8 lanes per 128-byte row ----
    const int crow = lane >> 3, cch = lane & 7;
    const bool w_on = crow < C::kWRows, x_on = crow < C::kXRows;
    const char* wsrc;
    const char* xsrc;
    {
        const int r = wv * C::kWRows + crow;
        wsrc = reinterpret_cast<const char*>(w + (size_t)min(n0 + min(r, NF - 1), N - 1) * K + 8 * (cch ^ key128(r)));
        const int q = wv * C::kXRows + crow;
        xsrc = reinterpret_cast<const char*>(x + (size_t)min(q, M - 1) * K + 8 * (cch ^ key128(q)));
    }
    const int wdst = wv * C::kWRows * kRowB, xdst = C::kW + wv * C::kXRows * kRowB;
    // copies of tile tt into ring slot SL, or two copies of one hot line past
    // the end of K: every step issues the same count
    auto issue_tile = [&](int tt, auto slc) {
        constexpr int SL = decltype(slc)::value;
        if (tt < KT) {
            const size_t off = (size_t)tt * kRowB;
            if (w_on) copy16_to_lds_nt(wsrc + off, ring + SL * C::kSlot + wdst);
            if (x_on) copy16_to_lds(xsrc + off, ring + SL * C::kSlot + xdst);
        } else {
            copy16_to_lds(hot, dummy);
            copy16_to_lds(hot, dummy);
        }
    };
    auto pads = [&](int n) {
        for (int i = 0; i < n; ++i) copy16_to_lds(hot, dummy);
    };

    // ---- signs: rows are slot-major (row = u*NF + f); copy q of a super-tile
    //      holds rows 16q .. 16q+15, 4 lanes of 16 B each, and lane l's chunk is
    //      (l & 3) ^ key64(row) = (l & 3) ^ (l >> 4) ----
    const int sc4 = 4 * ((lane & 3) ^ (lane >> 4));       // word of the lane's chunk in a super-tile
    // There are never more tenants than sign slots (T <= U, which the launch
    // checks), so super-tile 0 holds tenant u in slot u (absent tenants' rows
    // are copied and never read) and need not wait for the routing; later
    // super-tiles hold only the tenants present, in the compacted slots the
    // routing assigns.

    // ---- routing (wave 0) while the other waves start super-tile 0 (tenant u
    //      in slot u) and tile 0 ----
    if (wv != 0) {
        for (int q = wv - 1; q < C::nSup; q += kWaves - 1) {
            const int row = 16 * q + (lane >> 2), u = row / NF, f = row - u * NF;
            if ((16 * q) / NF < T)
                copy16_to_lds(packed + ((size_t)u * N + min(n0 + f, N - 1)) * KW + min(sc4, KW - 4), lds + q * 1024);
        }
        issue_tile(0, std::integral_constant<int, 0>{});
        pads(C::cS);
    } else {
        for (int i = lane; i < kMaxFrags * 16; i += 64) (&rt.frag_row[0][0])[i] = -1;
        constexpr uint32_t kInvalid = 0x80000000u, kPad = 0x80000001u;
        uint32_t key = kPad;
        if (lane < M) {
            const int t = tenant_ids[lane];
            key = (t >= 0 && t < T) ? (uint32_t)t : kInvalid;
        }
        int rank = 0;
        for (int j = 0; j < kMaxRows; ++j) {
            const uint32_t kj = __builtin_amdgcn_readlane(key, j);
            rank += (kj < key || (kj == key && j < lane)) ? 1 : 0;
        }
        rt.sorted_row[rank] = lane;
        rt.key_sorted[rank] = key;
        rt.tenant_of_row[lane] = key < kInvalid ? (int)key : -1;
        __builtin_amdgcn_s_waitcnt(0xC07F);                // lgkmcnt(0): sorted arrays written
        const uint32_t kp = rt.key_sorted[lane];
        const uint32_t kprev = lane > 0 ? rt.key_sorted[lane - 1] : 0xFFFFFFFFu;
        const bool valid = kp < kInvalid;
        const unsigned long long upto = lane == 63 ? ~0ull : ((2ull << lane) - 1ull);
        const unsigned long long tstart = __ballot(valid && kp != kprev);
        const int first = 63 - __builtin_clzll((tstart & upto) | 1ull);
        const int r = lane - first;                        // rank inside the tenant's rows
        const int slot = __popcll(tstart & upto) - 1;
        const unsigned long long fstart = __ballot(valid && (r & 15) == 0);
        const int fidx = __popcll(fstart & upto) - 1;
        if (valid) {
            rt.frag_row[fidx][r & 15] = rt.sorted_row[lane];
            if ((r & 15) == 0) rt.frag_slot[fidx] = slot;
            if (r == 0) rt.slot_tenant[slot] = (int)kp;
        }
        if (lane == 0) {
            rt.nfrag = __popcll(fstart);
            rt.nslot = __popcll(tstart);
        }
    }
    raw_barrier();
    const int nslot = __builtin_amdgcn_readfirstlane(rt.nslot);
    const int F = __builtin_amdgcn_readfirstlane(rt.nfrag);
    // this wave's fragments' alpha, loaded now rather than after the loop (the
    // loads are older than every tile copy still to come, so the in-order
    // copy counts below are unaffected)
    float afr[FW];
#pragma unroll
    for (int i = 0; i < FW; ++i) {
        const int f = wv + kWaves * i;
        afr[i] = f < F ? alpha[rt.slot_tenant[rt.frag_slot[f]]] : 0.f;
    }
    if (wv == 0) {
        issue_tile(0, std::integral_constant<int, 0>{});
        pads(C::cS);
    }

    auto sign_row = [&](int row) {
        const int u = row / NF, f = row - u * NF;
        return packed + ((size_t)rt.slot_tenant[u] * N + min(n0 + f, N - 1)) * KW;
    };
    const uint32_t* ssrc[C::kPieces * C::cS];
    uint32_t pmask = 0;                                    // piece copies of a present slot
#pragma unroll
    for (int p = 0; p < C::kPieces * C::cS; ++p) {
        const int q = p * kWaves + wv;
        const bool real = q < C::nSup && (16 * q) / NF < nslot;
        ssrc[p] = real ? sign_row(16 * q + (lane >> 2)) : packed;
        if (real) pmask |= 1u << p;
    }
    static_for<D>([&](auto sc) {
        if constexpr (decltype(sc)::value > 0) {
            issue_tile(decltype(sc)::value, sc);
            pads(C::cS);
        }
    });
    __builtin_amdgcn_sched_barrier(0);
    const int nsuper = (KT + kR - 1) / kR;
    // step t of super-tile j (phase PH = t & 7) issues piece PH of super-tile j+1
    auto issue_piece = [&](int t, auto phc) {
        constexpr int PH = decltype(phc)::value;
        const int j1 = (t >> 3) + 1;
        char* dst = lds + (j1 & 1) * C::kSBuf;
        const bool live = j1 < nsuper;
        const bool ragged = 16 * j1 + 16 > KW;             // the last super-tile ends inside
#pragma unroll
        for (int i = 0; i < C::cS; ++i) {
            if (PH < C::kPieces) {
                const int p = PH * C::cS + i;
                if (live && ((pmask >> p) & 1u)) {
                    const int word = ragged ? min(16 * j1 + sc4, KW - 4) : 16 * j1 + sc4;
                    copy16_to_lds(ssrc[p] + word, dst + (p * kWaves + wv) * 1024);
                    continue;
                }
            }
            copy16_to_lds(hot, dummy);
        }
    };

    // ---- this wave's share: the sign products of fragments wv + 8i (i < na),
    //      and x*W^T for (row block, feature block) pairs p = fb*RB + rb with
    //      p % 8 == wv, that is row block wv % RB and feature blocks
    //      wv/RB + j*8/RB ----
    const int na = F > wv ? min(FW, (F - wv + kWaves - 1) / kWaves) : 0;
    const int rbw = wv % RB;
    int bj[NBJ];
#pragma unroll
    for (int j = 0; j < NBJ; ++j) {
        const int b = wv / RB + j * (kWaves / RB);
        bj[j] = (b < FB && 16 * rbw < M) ? b : -1;
    }
    const int wkey = key128(nl);                           // rows fb*16 + nl and 16*rb + nl share it
    int woff[2], xnoff[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const int ch = 16 * ((4 * kb + g) ^ wkey);
        woff[kb] = C::kRingOff + nl * kRowB + ch;
        xnoff[kb] = C::kRingOff + C::kW + (16 * rbw + nl) * kRowB + ch;
    }

    auto run = [&](auto nac) {
        constexpr int NA = decltype(nac)::value;
        constexpr int NA1 = NA > 0 ? NA : 1;
        // soff: sign row of the fragment's slot; during super-tile 0 shifted by
        // sdelta to the row of the tenant itself
        int xoff[NA1][2], soff[NA1][4], sdelta[NA1];
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int f = wv + kWaves * i;
            int r = rt.frag_row[f][nl];
            if (r < 0) r = rt.frag_row[f][0];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
                xoff[i][kb] = C::kRingOff + C::kW + r * kRowB + 16 * ((4 * kb + g) ^ key128(r));
            const int slot = rt.frag_slot[f];
            sdelta[i] = __builtin_amdgcn_readfirstlane((rt.slot_tenant[slot] - slot) * NF * kSRowB);
            const int sbase = (slot * NF + nl) * kSRowB + sdelta[i];
#pragma unroll
            for (int q = 0; q < 4; ++q) soff[i][q] = sbase + 16 * (q ^ key64(nl));
        }
        f32x4 accs[NA1][FB], accn[NBJ];
#pragma unroll
        for (int j = 0; j < NBJ; ++j) accn[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < NA1; ++i)
#pragma unroll
            for (int b = 0; b < FB; ++b) accs[i][b] = f32x4{0.f, 0.f, 0.f, 0.f};

        // the LDS operands of one tile: sign words, x fragments, and the natural
        // x rows and W fragments of the base pairs
        struct Ops {
            uint2 s2[NA1][FB];
            u32x4 xa[NA1][2], xn[2], bw[NBJ][2];
        };
        // tile of phase I = t mod 16: ring slot I mod NB, sign buffer (I >> 3) & 1,
        // sign words 2*(I & 7) and 2*(I & 7) + 1 of the super-tile row
        auto load = [&](auto ic, Ops& o) {
            constexpr int I = decltype(ic)::value & 15;
            constexpr int SLOT = (I % NB) * C::kSlot;
            constexpr int WI = 2 * (I & 7);
            constexpr int SBUF = ((I >> 3) & 1) * C::kSBuf;
#pragma unroll
            for (int i = 0; i < NA; ++i)
#pragma unroll
                for (int b = 0; b < FB; ++b)
                    o.s2[i][b] = *reinterpret_cast<const uint2*>(lds + soff[i][WI >> 2] + SBUF + 16 * b * kSRowB + 4 * (WI & 3));
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
                for (int i = 0; i < NA; ++i) o.xa[i][kb] = *reinterpret_cast<const u32x4*>(lds + xoff[i][kb] + SLOT);
                if (bj[0] >= 0) {
                    o.xn[kb] = *reinterpret_cast<const u32x4*>(lds + xnoff[kb] + SLOT);
#pragma unroll
                    for (int j = 0; j < NBJ; ++j)
                        if (bj[j] >= 0)
                            o.bw[j][kb] = *reinterpret_cast<const u32x4*>(lds + woff[kb] + SLOT + bj[j] * 16 * kRowB);
                }
            }
        };
        auto compute = [&](const Ops& o) {
#pragma unroll
            for (int b = 0; b < FB; ++b) {
                u32x4 sb[NA1][2];
#pragma unroll
                for (int i = 0; i < NA; ++i) decode_signs8x2<ET>(o.s2[i][b].x, o.s2[i][b].y, 8 * g, sb[i][0], sb[i][1]);
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < NA; ++i) accs[i][b] = mfma16<ET>(o.xa[i][kb], sb[i][kb], accs[i][b]);
            }
            if (bj[0] >= 0)
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int j = 0; j < NBJ; ++j)
                        if (bj[j] >= 0) accn[j] = mfma16<ET>(o.xn[kb], o.bw[j][kb], accn[j]);
        };

        // ---- main loop, sixteen steps per pass.  D = NB: step t waits until
        //      tile t + 1 and its signs have landed (only the copies of tiles
        //      t + 2 .. t + D - 1 in flight), then, past the barrier, issues the
        //      copies of tile t + D into the slot of tile t (whose operands were
        //      read into registers in the previous step; those reads completed
        //      before the barrier).  D = NB - 1: step t first issues tile t + D
        //      into the slot of tile t - 1 (its reads completed at the previous
        //      barrier), then waits for tile t + 1 the same way.  Either way the
        //      step then reads tile t + 1's operands and computes tile t from
        //      the operands read one step earlier, so their LDS latency overlaps
        //      the previous step's arithmetic ----
        Ops oa, ob;
        wait_vm_lgkm0<(D - 1) * C::ops>();
        raw_barrier();
        load(std::integral_constant<int, 0>{}, oa);
        for (int t0 = 0; t0 < KT; t0 += 16) {
            static_for<16>([&](auto ic) {
                constexpr int I = decltype(ic)::value;
                const int t = t0 + I;
                if (t < KT) {
                    if constexpr (C::kEarly) {
                        wait_vm_lgkm0<(D - 2) * C::ops>();
                        raw_barrier();
                    }
                    issue_tile(t + D, std::integral_constant<int, (I + D) % NB>{});
                    issue_piece(t, std::integral_constant<int, I & 7>{});
                    __builtin_amdgcn_sched_barrier(0);
                    if constexpr (!C::kEarly) {
                        wait_vm_lgkm0<(D - 1) * C::ops>();
                        raw_barrier();
                    }
                    Ops& cur = (I & 1) ? ob : oa;
                    Ops& nxt = (I & 1) ? oa : ob;
                    if constexpr (I == 7) {
                        // tile 8 starts super-tile 1: compacted slots from here on
                        if (t0 == 0)
#pragma unroll
                            for (int i = 0; i < NA; ++i)
#pragma unroll
                                for (int q = 0; q < 4; ++q) soff[i][q] -= sdelta[i];
                    }
                    if (t + 1 < KT) load(std::integral_constant<int, I + 1>{}, nxt);
                    compute(cur);
                }
            });
        }
        wait_vm_lgkm0<0>();

        // ---- epilogue: base sums through LDS (the ring is free once every wave
        //      is past its last tile), then y = base + alpha * sign ----
        float* red = reinterpret_cast<float*>(ring);       // [XR rows][NF features]
        __syncthreads();
#pragma unroll
        for (int j = 0; j < NBJ; ++j)
            if (bj[j] >= 0)
#pragma unroll
                for (int r = 0; r < 4; ++r) red[(16 * rbw + 4 * g + r) * NF + 16 * bj[j] + nl] = accn[j][r];
        __syncthreads();
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int f = wv + kWaves * i;
            const float a = afr[i];
#pragma unroll
            for (int b = 0; b < FB; ++b) {
                const int n = n0 + 16 * b + nl;
                if (n >= N) continue;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = rt.frag_row[f][4 * g + r];
                    if (row >= 0)
                        store_y<ET>(y, (size_t)row * N + n, __builtin_fmaf(a, accs[i][b][r], red[row * NF + 16 * b + nl]),
                                    y_dtype);
                }
            }
        }
    };
    static_for<FW + 1>([&](auto ic) {
        if (na == decltype(ic)::value) run(ic);
    });

    // rows whose tenant id is out of range
    for (int idx = threadIdx.x; idx < M * NF; idx += kThreads) {
        const int m = idx / NF, n = n0 + idx % NF;
        if (n < N && rt.tenant_of_row[m] < 0) store_y<ET>(y, (size_t)m * N + n, __builtin_nanf(""), y_dtype);
    }
}

constexpr int kNB = 4;

// LDS of a configuration (same layout as WideCfg, for the host-side choice).
constexpr int wide_lds(int fb, int xr, int u) {
    return 2 * u * 16 * fb * kSRowB + kNB * (16 * fb * kRowB + xr * kRowB) + 1024 + (int)sizeof(WideRouting);
}

struct WidePlan {
    int fb, xr, u;
};

// Shape -> form.  One workgroup per CU: the feature groups must fill most of
// the 256 CUs (48 features per group from 161 groups, else 64 from 193), with
// at most 16 distinct tenants, and the signs and rings must fit the LDS.
// Other shapes take the 16-feature kernels.
bool plan_wide(int M, int N, int K, int T, WidePlan* p) {
    const int u = T < M ? T : M;
    if (M < 17 || M > kMaxRows || u > 16 || K < 128 || K % 128 != 0) return false;
    p->u = u <= 8 ? 8 : 16;
    if (T > p->u) return false;                            // super-tile 0 holds tenant u in slot u
    p->xr = M <= 32 ? 32 : 64;
    const int fg3 = (N + 47) / 48, fg4 = (N + 63) / 64;
    if (fg3 > 5 * kCUs / 8 && fg3 <= kCUs) p->fb = 3;
    else if (fg4 > 3 * kCUs / 4 && fg4 <= kCUs) p->fb = 4;
    else return false;
    return K / kTK >= kNB - 1 && wide_lds(p->fb, p->xr, p->u) <= 160 * 1024;
}

template <int ET, int FB, int XR, int U>
hipError_t launch_cfg(const uint16_t* x, int M, int K, const uint16_t* w, int N, const uint32_t* packed,
                      const float* alpha, const int32_t* tenant_ids, int T, void* y, int y_dtype,
                      hipStream_t stream) {
    if constexpr (wide_lds(FB, XR, U) > 160 * 1024) {
        return hipErrorInvalidValue;
    } else {
        const int grid = (N + 16 * FB - 1) / (16 * FB);
        wide_batched_kernel<ET, FB, XR, U, kNB><<<grid, kThreads, 0, stream>>>(x, M, K, w, N, packed, alpha,
                                                                              tenant_ids, T, y, y_dtype);
        return hipGetLastError();
    }
}

template <int ET, int XR, int U>
hipError_t launch_xu(const WidePlan& p, const uint16_t* x, int M, int K, const uint16_t* w, int N,
                     const uint32_t* packed, const float* alpha, const int32_t* tenant_ids, int T, void* y,
                     int y_dtype, hipStream_t stream) {
    if (p.fb == 3)
        return launch_cfg<ET, 3, XR, U>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
    return launch_cfg<ET, 4, XR, U>(x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
}

template <int ET>
hipError_t launch_et(const WidePlan& p, const uint16_t* x, int M, int K, const uint16_t* w, int N,
                     const uint32_t* packed, const float* alpha, const int32_t* tenant_ids, int T, void* y,
                     int y_dtype, hipStream_t stream) {
    if (p.xr == 32 && p.u == 8)
        return launch_xu<ET, 32, 8>(p, x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
    if (p.xr == 32)
        return launch_xu<ET, 32, 16>(p, x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
    if (p.u == 8)
        return launch_xu<ET, 64, 8>(p, x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
    return launch_xu<ET, 64, 16>(p, x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
}

}  // namespace

bool wide_supported(int M, int N, int K, int T) {
    WidePlan p;
    return plan_wide(M, N, K, T, &p);
}

hipError_t launch_wide(const uint16_t* x, int M, int K, const uint16_t* w, int N, const uint32_t* packed,
                       const float* alpha, const int32_t* tenant_ids, int T, void* y, int y_dtype, int et,
                       hipStream_t stream) {
    WidePlan p;
    if (!plan_wide(M, N, K, T, &p)) return hipErrorInvalidValue;
    if (et == kF16) return launch_et<kF16>(p, x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
    return launch_et<kBF16>(p, x, M, K, w, N, packed, alpha, tenant_ids, T, y, y_dtype, stream);
}

}  // namespace bitdelta
