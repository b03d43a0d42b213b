// The per-item body of the gathered fine attention (steps 3-5 at the finer levels; Sec. 3.2,
// Fig. 1; QuadTree-A scores Eq. 4, QuadTree-B softmax Eq. 6; the finest level's combination,
// Eqs. 2 and 5), included by the fine kernels of every finer level.
//
// Work item = one parent query P at level l+1 and one head. Its four children at level l are
// sibling queries with one shared candidate set: the 2x2 children of the K keys P kept (4K <= 256
// candidates). One wave owns one item; candidate slot s = 4r + c is child c, in the order (0,0),
// (0,1),(1,0),(1,1), of kept key r; lane l owns slots l, l + 64, ... (up to four), and the slots
// are taken in tiles of 16:
//   1. the candidates' key and value rows of this head are gathered once for the four queries with
//      16-byte loads: lane 16g + n loads chunks g, g+4, ... of the row of slot n of each tile, so
//      one instruction reads 16 whole rows. The value rows go to wave-private LDS (transposed for
//      bf16); the key rows stay in registers;
//   2. logits on the 16x16 MFMA straight from those registers: the key chunks are the B operand,
//      the four queries the A operand, query g on rows 4g .. 4g+3 (the d channels are contracted in
//      the order the chunks arrive, the same for both operands). Lane 16g + n then holds query g's
//      logit of slot 16t + n from tile t: a lane keeps one query's logits over the tiles;
//   3. B: a softmax per query over its 16-lane row (DPP butterflies) and the lane's tiles;
//      A: a softmax over each lane quad (the children of one kept key) times the parent's score;
//   4. levels above 0: the ranking keys move to one slot per lane (lane l: slots l, l + 64, ...) by
//      a 4x4 transpose across the wave's 16-lane rows per four tiles (row swaps, no LDS), then the
//      K best candidates of each query by a bitwise radix select on wave ballots (ties at the cut to
//      the lower flat index); A drops their weight from its message;
//   5. messages m = P V on the 4x4 MFMA, blocks split over 4-channel groups (and slot halves);
//   6. levels above 0 store m; level 0 adds the ancestors' messages (times w for B) and stores the
//      output in the storage type. With a fused position encoding (PE, maps of more than one row)
//      every level first adds to m the 3x3 depth-wise cross-correlation of its own value map around
//      each query (zero outside the map) plus the bias: the 4x4 tokens around the sibling block are
//      read once per wave and passed through the wave's LDS.
#ifndef QTA_FINE_ITEM_H
#define QTA_FINE_ITEM_H

#include "qta_device.h"
#include "qta_internal.h"

namespace qta {
namespace fine {

typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

constexpr int kMaxSlots = 256;         // candidate slots of one item: 4 K_l for K_l <= 64, up to four per lane
constexpr int kMaxSlotsPe = 64;        // with a fused position encoding: one slot per lane
constexpr int kSplitSlots = 64;        // bf16 value rows staged at a time when a group has 65 .. 128 slots
constexpr int kPrefetchLevels = 4;    // the finest level prefetches up to this many ancestors
// LDS pitch (elements) of one channel's 16 tokens in the fused position encoding: 20 puts the four lane
// groups' writes and neighbouring channels' row reads in different banks (16 would stack them)
constexpr int kPeTokenPitch = 20;

// Byte layout of one wave's LDS region for nsp padded slots (a multiple of 16): the value rows
// and the weights P.
struct WaveLds {
    int v, p, total;
    int vpitch;    // bf16: elements per transposed value row; fp32: floats per value row
};

template <typename T, int D>
__host__ __device__ inline WaveLds wave_lds(int nsp)
{
    constexpr int TB = sizeof(T);
    WaveLds L;
    L.v = 0;
    int vbytes;
    if (TB == 2) {
        // Vt[channel][slot]; with 65 .. 128 slots the rows are staged in two halves of at most 64
        // slots (half the LDS per wave, so that registers rather than LDS bound the occupancy)
        L.vpitch = (nsp > kSplitSlots && nsp <= 2 * kSplitSlots ? kSplitSlots : nsp) + 8;
        vbytes = D * L.vpitch * 2;
    } else {
        L.vpitch = D + 4;                   // Vs[slot][channel]
        vbytes = nsp * L.vpitch * 4;
    }
    // (the fused position encoding stages 16 tokens of one head here, kPeTokenPitch elements per channel)
    if (vbytes < D * kPeTokenPitch * TB) vbytes = D * kPeTokenPitch * TB;
    L.p = L.v + vbytes;
    L.total = (L.p + 4 * nsp * TB + 15) / 16 * 16;
    return L;
}

__device__ __forceinline__ float pick4(const float4_t& v, int i)
{
    return i == 0 ? v[0] : i == 1 ? v[1] : i == 2 ? v[2] : v[3];
}

__device__ __forceinline__ float pick4(const float (&v)[4], int i)
{
    return i == 0 ? v[0] : i == 1 ? v[1] : i == 2 ? v[2] : v[3];
}

// The loads of a work item that need no other load, with the item's coordinates: its parents' kept
// keys (each lane's gather key of every slot tile), their scores (QuadTree-A) and the query rows
// (MFMA A operand: row n16 holds query n16 >> 2). Vector memory counters drain in order, and a load
// inside a divergent branch makes the compiler wait for it at the join, so every load here is
// unconditional, at a clamped address that is always in bounds, with validity applied when the
// value is used.
template <typename T, int D, int NSP, bool VA, bool ROW>
struct ItemHead {
    int b, h, P, Py, Px;
    bool pair2;                 // ROW: the second parent exists
    bool q_ok;                  // this lane's query (n16 >> 2) lies on the map
    int J_g[NSP / 16];
    float pkey[VA ? NSP / 16 : 1];   // QuadTree-A: the parent's score of the lane's slot in each tile
    uint4 qa[D * sizeof(T) / 64];
};

// FINEST: the finest level, whose queries are always stored NHWC (the layout flag is not read).
template <typename T, int D, int NSP, bool VA, bool ROW, bool FINEST>
__device__ __forceinline__ void item_head(const FineArgs& a, const int item, ItemHead<T, D, NSP, VA, ROW>& hd)
{
    constexpr int TB = sizeof(T);
    constexpr int RB = D * TB;
    constexpr int NJ = RB / 64;
    constexpr int NT = NSP / 16;
    const int lane = threadIdx.x & 63;
    const int n16 = lane & 15, g = lane >> 4;
    const int Np = a.Hp * a.Wp;
    const int bp = fast_div(item, a.div_heads);
    const int h = item - bp * a.heads;
    const int NI = ROW ? (Np + 1) / 2 : Np;               // items per (batch, head)
    const int b = fast_div(bp, a.div_items);
    const int P = ROW ? 2 * (bp - b * NI) : bp - b * NI;  // ROW: the pair's first parent
    const int Py = ROW ? 0 : fast_div(P, a.div_Wp), Px = ROW ? P : P - Py * a.Wp;
    const bool pair2 = ROW && P + 1 < Np;
    const int H = a.H, W = a.W, C = a.C, K = a.Kp;
    hd.b = b;
    hd.h = h;
    hd.P = P;
    hd.Py = Py;
    hd.Px = Px;
    hd.pair2 = pair2;
    // per batch element a 64-bit base, within it 32-bit offsets (one element's map is below 2^31 bytes,
    // so its kept-key table and its coarser messages are too)
    const int32_t* prow = a.parent_idx + static_cast<size_t>(b) * static_cast<uint32_t>(a.heads * Np * K) +
                          static_cast<uint32_t>((h * Np + P) * K);
    // the kept-key entry of slot s: s >> 2 (ROW: s >> 1, the pair's two rows being contiguous)
    constexpr int kSlotShift = ROW ? 1 : 2;
    const int last_sel = (ROW && pair2 ? 2 * K : K) - 1;
#pragma unroll
    for (int t = 0; t < NT; ++t)
        hd.J_g[t] = load_at<int32_t>(prow, static_cast<uint32_t>(min(((16 * t) >> kSlotShift) + (n16 >> kSlotShift), last_sel)) * 4u);
    if constexpr (VA) {
        const float* pk = a.parent_key + ((static_cast<size_t>(b) * a.heads + h) * Np + P) * K;
#pragma unroll
        for (int t = 0; t < NT; ++t)
            hd.pkey[t] = load_at<float>(pk, static_cast<uint32_t>(min(((16 * t) >> kSlotShift) + (n16 >> kSlotShift), last_sel)) * 4u);
    } else {
        hd.pkey[0] = 0.f;
    }
    const int qi = n16 >> 2;
    const int qy = ROW ? 0 : 2 * Py + (qi >> 1), qx = ROW ? 2 * P + qi : 2 * Px + (qi & 1);
    hd.q_ok = qy < H && qx < W;
    const int qyc = qy < H ? qy : H - 1, qxc = qx < W ? qx : W - 1;
    // uniform base of this (batch, head) plus a 32-bit per-lane offset. ROW, blocked: query 4p + qi
    // is child qi & 1 of parent 2p + (qi >> 1)
    const bool qb = !FINEST && a.q_blocked;
    const unsigned char* qbase = static_cast<const unsigned char*>(a.q) +
        (qb ? ((static_cast<size_t>(b) * a.heads + h) * Np + P) * 4 * RB
                     : (static_cast<size_t>(b) * H * W * C + h * D) * TB);
    // (a query off the map may belong to a parent past the last one: read the first block instead)
    const int qblk = ROW ? (hd.q_ok ? (qi >> 1) * 4 + (qi & 1) : 0) : qi;
    const uint32_t qoff = qb ? static_cast<uint32_t>(qblk * RB)
                                      : __umul24(static_cast<uint32_t>(__mul24(qyc, W) + qxc), static_cast<uint32_t>(C * TB));
#pragma unroll
    for (int j = 0; j < NJ; ++j)
        hd.qa[j] = *reinterpret_cast<const uint4*>(qbase + (qoff + static_cast<uint32_t>((g + 4 * j) * 16)));
}

// One work item (parent query P at level l+1, head h; item = (b*Np + P)*heads + h), whose
// independent loads item_head has issued, on the calling wave, whose private LDS region of wave_lds<T, D>(nsp).total bytes starts at `base`. The whole
// wave must call it with the same item.
// ROW: maps of one row (attention along epipolar lines). A parent there has only two children and
// its kept keys two children each, so one item takes two neighbouring parents P0 = 2p, P1 = 2p + 1
// (item = (b*ceil(Np/2) + p)*heads + h): its four queries are tokens 4p .. 4p+3, candidate slot
// s = 2*(half*K + r) + c is child c of kept key r of parent `half`, and query q uses the slots of
// half q >> 1 only.
template <typename T, int D, int NSP, bool VA, bool FINEST, bool ROW = false, bool PE = false>
__device__ __forceinline__ void fine_item(const FineArgs& a, const ItemHead<T, D, NSP, VA, ROW>& hd, unsigned char* const base)
{
    using S = Storage<T>;
    constexpr bool kBf16 = sizeof(T) == 2;
    constexpr int TB = sizeof(T);
    constexpr int RB = D * TB;             // bytes of one head's row
    constexpr int E = S::kPer16B;          // elements per 16-byte chunk
    constexpr int NJ = RB / 64;            // 16-byte chunks per lane and row (lane group g: g, g+4, ...)
    constexpr int NT = NSP / 16;           // slot tiles (upper bound)
    // tiles whose rows are in registers at once (at most four: eight would cost occupancy with 128 slots)
    constexpr int kTB = (8 / NJ) < 4 ? ((8 / NJ) < NT ? (8 / NJ) : NT) : (4 < NT ? 4 : NT);
    constexpr int NCG = D / 4;             // PV: 4-channel groups
    constexpr int NH = 16 / NCG;           // PV: slot halves (2 for d = 32, 1 for d = 64)
    constexpr int QPL = 4 / NH;            // output queries per lane
    constexpr int SPL = NSP > 64 ? NSP / 64 : 1;   // candidate slots per lane: lane + 64u
    // bf16 with 65 .. 128 slots: slots 0 .. 63 are staged as their tiles are consumed, the value rows
    // of slots 64 .. are held in registers and staged after the first half of the messages
    constexpr bool kSplitV = kBf16 && NSP == 2 * kSplitSlots;
    constexpr int kTS = kSplitSlots / 16;           // tiles of the first half
    static_assert(!PE || !ROW, "the fused position encoding is for maps of more than one row");
    static_assert(NSP <= kMaxSlotsPe || !PE, "a fused position encoding takes at most 64 slots");

    const int lane = threadIdx.x & 63;
    const int Np = a.Hp * a.Wp;
    const int b = hd.b, h = hd.h, P = hd.P, Py = hd.Py, Px = hd.Px;
    const bool pair2 = hd.pair2;
    const int H = a.H, W = a.W, C = a.C, K = a.Kp, Ks = a.Ks;
    const int N = H * W;
    const int nslot = 4 * K;
    const int nsp = (nslot + 15) & ~15;                // <= NSP

    const WaveLds lay = wave_lds<T, D>(nsp);
    unsigned char* Vb = base + lay.v;
    unsigned char* Pb = base + lay.p;

    // flat index at level l of child (s & 3) of kept key J (a level l+1 index), or -1. Map sizes are
    // below 2^24 tokens, so coordinate products fit the 24-bit multiplier. ROW: child s & 1 of J.
    // Computed without branches: the early returns of a plain form became divergent branches per
    // tile, with their exec-mask bookkeeping on the scalar unit.
    auto child_of_slot_J = [&](int J, int s) -> int {
        const int Jc = J < 0 ? 0 : J;
        if constexpr (ROW) {
            const int cx = 2 * Jc + (s & 1);
            const bool ok = s < nslot && J >= 0 && (pair2 || s < 2 * K) && cx < W;
            return ok ? cx : -1;
        }
        const int Jy = fast_div(Jc, a.div_Wp), Jx = Jc - __mul24(Jy, a.Wp);
        const int cy = 2 * Jy + ((s >> 1) & 1), cx = 2 * Jx + (s & 1);
        const bool ok = s < nslot && J >= 0 && cy < H && cx < W;
        return ok ? __mul24(cy, W) + cx : -1;
    };
    // query r of the item: its map coordinates
    auto query_yx = [&](int r, int& qy, int& qx) {
        if constexpr (ROW) {
            qy = 0;
            qx = 2 * P + r;
        } else {
            qy = 2 * Py + (r >> 1);
            qx = 2 * Px + (r & 1);
        }
    };

    // ---- 1. loads: item_head issued the phase A loads (kept keys, scores, query rows); phase B,
    //      the gathers, needs the kept keys ----
    // With more tiles than one batch of registers holds, a compiler barrier: the kept keys of the
    // later batches (gathered behind a uniform bound) would otherwise be sunk to those batches,
    // leaving each a dependent load chain of its own (detection's 128-slot finest level +1.6 us).
    // With a single batch the barrier only constrains the schedule (backbone's finest +2 us).
    if constexpr (NT > kTB) asm volatile("" ::: "memory");
    const int n16 = lane & 15, g = lane >> 4;
    const int ntile = nsp / 16;
    const int (&J_g)[NT] = hd.J_g;
    // lane 16g + n16 owns slots 64u + 16g + n16: the gather keys of tiles g + 4u
    int J_own[SPL];
#pragma unroll
    for (int u = 0; u < SPL; ++u) J_own[u] = -1;
#pragma unroll
    for (int t = 0; t < NT; ++t) J_own[t >> 2] = g == (t & 3) ? J_g[t] : J_own[t >> 2];
    const float (&pkey)[VA ? NT : 1] = hd.pkey;
    const uint4 (&qa)[NJ] = hd.qa;
    // phase B: the gathers. NHWC: child f of this head at kg + f*C*TB. Blocked: the four children
    // of kept key J are the 4*RB bytes at kg + J*4*RB (this (batch, head)'s blocks start at kg).
    // The finest level's keys and values are always NHWC.
    const bool kvb = !FINEST && a.kv_blocked;
    const size_t kv_base = kvb ? (static_cast<size_t>(b) * a.heads + h) * Np * 4 * RB
                               : (static_cast<size_t>(b) * N * C + h * D) * TB;
    const unsigned char* kg = static_cast<const unsigned char*>(a.k) + kv_base;
    const unsigned char* vg = static_cast<const unsigned char*>(a.v) + kv_base;
    // at most 4 MiB (heads*d <= 2^20 by the host checks): token index times row bytes fits the
    // 24-bit multiplier
    const uint32_t tok_bytes = static_cast<uint32_t>(C * TB);
    bool gok[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) gok[t] = false;
    uint4 kc[kTB][NJ], vc[kTB][NJ];
    auto load_tiles = [&](int t0) {
#pragma unroll
        for (int i = 0; i < kTB; ++i) {
            const int t = t0 + i, s = 16 * t + n16;
            if (t >= NT || t >= ntile) break;                 // uniform
            const int f = child_of_slot_J(J_g[t], s);
            gok[t] = f >= 0;
            // 32-bit byte offset within this (batch, head)'s map (below 2^31 by the host's checks); a
            // missing candidate reads the map's first row
            uint32_t off = __umul24(static_cast<uint32_t>(gok[t] ? f : 0), tok_bytes);
            if constexpr (!FINEST) {
                // the layout as a mask, not a branch per tile
                const unsigned kvb_m = opaque_mask(kvb);
                const uint32_t boff = static_cast<uint32_t>(gok[t] ? J_g[t] * 4 + (ROW ? (s & 1) : (s & 3)) : 0) * RB;
                off = (boff & kvb_m) | (off & ~kvb_m);
            }
            const uint32_t goff = off + g * 16;
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                kc[i][j] = *reinterpret_cast<const uint4*>(kg + (goff + 64 * j));
                vc[i][j] = *reinterpret_cast<const uint4*>(vg + (goff + 64 * j));
            }
        }
    };
    // Output ownership (step 6): lane 4*blk + t4 with blk = cg*NH + hh owns channel 4*cg + t4 of
    // queries hh*QPL .. hh*QPL + QPL-1.
    const int blk = lane >> 2, t4 = lane & 3;
    const int cg = blk / NH, hh = blk % NH;
    const int ch = 4 * cg + t4;
    constexpr int kPre = FINEST ? kPrefetchLevels : 1;
    float anc[ROW ? QPL : 1][kPre];     // ROW: the two parents of a pair have different ancestors
    float wq[FINEST ? QPL : 1][kPre + 1];
    float peq[FINEST ? QPL : 1] = {};
    const bool prefetch = FINEST && a.levels <= kPre + 1;
    // the finest level's combination inputs: the ancestors' messages and the encoding of level 0,
    // and w. With d = 64 (and no fused encoding) the ancestors and the encoding are requested before
    // the gathers (backbone's layer 75.9 -> 73.2 us); with d = 32, or with the fused encoding's own
    // early loads, that costs more occupancy than it saves (stereo +0.6 us, backbone_pe +3 us), so
    // there they follow the gathers, and their latency overlaps the softmax and the messages. w
    // always follows the gathers: its twenty scattered loads per lane ahead of them held the gathers
    // back (backbone +1.9 us).
    constexpr bool kEarlyCombination = D == 64 && !PE;
    auto request_ancestors = [&]() {
        if constexpr (FINEST) {
            if (prefetch) {                                      // uniform
                const int L = a.levels;
#pragma unroll
                for (int lev = 1; lev <= kPre; ++lev) {
                    if (lev >= L) break;                         // uniform
                    if constexpr (ROW) {
#pragma unroll
                        for (int u = 0; u < QPL; ++u) {
                            const int qi = (NH == 2 ? hh * QPL : 0) + u;
                            // clamped: a query off the map may lie past the last ancestor
                            const uint32_t an = min((2 * P + qi) >> lev, a.lvl_W[lev] - 1);
                            anc[u][lev - 1] = load_at<float>(a.coarser_msg[lev] + static_cast<size_t>(b) * static_cast<uint32_t>(a.lvl_N[lev] * C),
                                                             (an * static_cast<uint32_t>(C) + static_cast<uint32_t>(h * D + ch)) * 4u);
                        }
                    } else {
                        // the ancestor is shared by the four siblings: a uniform address plus the channel
                        const uint32_t an = static_cast<uint32_t>(((2 * Py) >> lev) * a.lvl_W[lev] + ((2 * Px) >> lev));
                        anc[0][lev - 1] = load_at<float>(a.coarser_msg[lev] + static_cast<size_t>(b) * static_cast<uint32_t>(a.lvl_N[lev] * C),
                                                         (an * static_cast<uint32_t>(C) + static_cast<uint32_t>(h * D + ch)) * 4u);
                    }
                }
                if (a.pe0) {                                     // uniform
                    const float* pb = a.pe0 + (static_cast<size_t>(b) * N * a.heads + h) * D + ch;
#pragma unroll
                    for (int u = 0; u < QPL; ++u) {
                        const int qi = (NH == 2 ? hh * QPL : 0) + u;
                        int py, px;
                        query_yx(qi, py, px);
                        py = min(py, H - 1);
                        px = min(px, W - 1);
                        peq[u] = pb[static_cast<uint32_t>(__mul24(py, W) + px) * static_cast<uint32_t>(a.heads * D)];
                    }
                }
            }
        }
    };
    auto request_weights = [&]() {
        if constexpr (FINEST) {
            if (prefetch) {                                      // uniform
                const int L = a.levels;
                if (!VA && a.w) {                                // uniform
                    const float* wb = a.w + (static_cast<size_t>(b) * N * a.heads + h) * L;
#pragma unroll
                    for (int u = 0; u < QPL; ++u) {
                        const int qi = (NH == 2 ? hh * QPL : 0) + u;
                        int wy, wx;
                        query_yx(qi, wy, wx);
                        wy = min(wy, H - 1);
                        wx = min(wx, W - 1);
                        // (a batch element's w is below 2^31 bytes: heads*L*4 <= heads*d*b)
                        const uint32_t wrow = __umul24(static_cast<uint32_t>(__mul24(wy, W) + wx), static_cast<uint32_t>(a.heads * L));
#pragma unroll
                        for (int lev = 0; lev <= kPre; ++lev) {
                            if (lev >= L) break;                 // uniform
                            wq[u][lev] = load_at<float>(wb, (wrow + lev) * 4u);
                        }
                    }
                }
            }
        }
    };
    if constexpr (kEarlyCombination) request_ancestors();
    load_tiles(0);
    int flat[SPL];
    bool ok[SPL];
#pragma unroll
    for (int u = 0; u < SPL; ++u) {
        const int s = 64 * u + lane;
        flat[u] = child_of_slot_J(s < nslot ? J_own[u] : -1, s);
        ok[u] = flat[u] >= 0;
    }

    // ---- 2. logits on MFMA and the value rows into LDS, one batch of tiles at a time ----
    // xs[t]: this lane's query's (g's) logit of slot 16t + n16 (unscaled)
    float xs[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) xs[t] = 0.f;
    uint4 vkeep[kSplitV ? NT - kTS : 1][NJ];
    auto consume_tiles = [&](int t0) {
#pragma unroll
        for (int i = 0; i < kTB; ++i) {
            const int t = t0 + i, s = 16 * t + n16;
            if (t >= NT || t >= ntile) break;                 // uniform
            float4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                // An off-map query's or a missing candidate's row was read at a clamped, valid address
                // (finite by the interface's contract) and its logits are masked below, so with d = 32
                // the operands go in unzeroed; with d = 64 the zeroing stays (without it that kernel
                // measured slower: backbone's finest level 36.0 -> 37.9 us)
                const uint4 qq = (D == 32 || hd.q_ok) ? qa[j] : make_uint4(0, 0, 0, 0);
                const uint4 kk = (D == 32 || gok[t]) ? kc[i][j] : make_uint4(0, 0, 0, 0);
                if constexpr (kBf16) {
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, qq),
                                                                  __builtin_bit_cast(bf16x8_t, kk), acc, 0, 0, 0);
                } else {
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(qq.x), __uint_as_float(kk.x), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(qq.y), __uint_as_float(kk.y), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(qq.z), __uint_as_float(kk.z), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(qq.w), __uint_as_float(kk.w), acc, 0, 0, 0);
                }
            }
            // rows 4g .. 4g+3 of the product are all query g
            xs[t] = acc[0];
            // value rows
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                // (a missing candidate's row gets weight 0 in the messages)
                const uint4 vv = (D == 32 || gok[t]) ? vc[i][j] : make_uint4(0, 0, 0, 0);
                const int c0 = (g + 4 * j) * E;               // first channel of this chunk
                if (kSplitV && t >= kTS) {                    // compile-time after unrolling
                    vkeep[kSplitV ? t - kTS : 0][j] = vv;
                } else if constexpr (kBf16) {
                    uint16_t* vt = reinterpret_cast<uint16_t*>(Vb);
                    const uint32_t w4[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const uint32_t bits = (e & 1) ? (w4[e >> 1] >> 16) : (w4[e >> 1] & 0xFFFFu);
                        vt[(c0 + e) * lay.vpitch + s] = static_cast<uint16_t>(bits);
                    }
                } else {
                    *reinterpret_cast<uint4*>(Vb + (s * lay.vpitch + c0) * 4) = vv;
                }
            }
        }
    };
    consume_tiles(0);
#pragma unroll
    for (int t0 = kTB; t0 < NT; t0 += kTB) {
        if (t0 >= ntile) break;                               // uniform
        load_tiles(t0);
        consume_tiles(t0);
    }
    // fused position encoding: the 4x4 tokens (2Py-1 .. 2Py+2) x (2Px-1 .. 2Px+2) of v around the
    // sibling block, token n16 = (by, bx), chunks g, g+4, ... of its row (as in the gathers; tokens off
    // the map read a clamped row and count as zero), and this lane's channel's 3x3 kernel and bias,
    // requested here so that their latency overlaps the weights and the messages
    uint4 peb[PE ? NJ : 1];
    float pek[PE ? 9 : 1];
    float pebias = 0.f;
    bool pe_ok = false;
    if constexpr (PE) {
        const int by = 2 * Py - 1 + (n16 >> 2), bx = 2 * Px - 1 + (n16 & 3);
        pe_ok = by >= 0 && by < H && bx >= 0 && bx < W;
        const int byc = min(max(by, 0), H - 1), bxc = min(max(bx, 0), W - 1);
        // this (batch, head)'s value map as for the gathers: NHWC rows, or child (by & 1, bx & 1) of
        // parent block (by >> 1, bx >> 1)
        const uint32_t boff = (kvb ? static_cast<uint32_t>(((__mul24(byc >> 1, a.Wp) + (bxc >> 1)) * 4 + (byc & 1) * 2 +
                                                            (bxc & 1)) * RB)
                                   : __umul24(static_cast<uint32_t>(__mul24(byc, W) + bxc), tok_bytes)) + g * 16;
#pragma unroll
        for (int j = 0; j < NJ; ++j) peb[j] = *reinterpret_cast<const uint4*>(vg + (boff + 64 * j));
        const float* wp = a.pe_w + static_cast<uint32_t>(h * D + ch) * 9u;
#pragma unroll
        for (int i = 0; i < 9; ++i) pek[i] = wp[i];
        pebias = a.pe_b ? a.pe_b[h * D + ch] : 0.f;
    }
    if constexpr (!kEarlyCombination) request_ancestors();
    request_weights();
    // this lane's query g and its slots 16t + n16 (ROW: only those of its own parent, half g >> 1)
    bool okt[NT];
    float xt[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int s = 16 * t + n16;
        okt[t] = t < ntile && gok[t] && (!ROW || ((s >> 1) >= K) == ((g >> 1) != 0));
        xt[t] = okt[t] ? xs[t] * a.scale : -INFINITY;
    }

    // ---- 3. weights (unnormalised for B: exp(x - max); the 1/sum is applied to the message) ----
    float wt[NT];
    float inv_g = 1.f;                                       // B: 1/sum of this lane's query
    if constexpr (!VA) {
        float m = xt[0];
#pragma unroll
        for (int t = 1; t < NT; ++t) m = fmaxf(m, xt[t]);
        m = row_allreduce(m, [](float u, float v) { return fmaxf(u, v); });
        float se = 0.f;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            wt[t] = okt[t] ? __expf(xt[t] - m) : 0.f;
            se += wt[t];
        }
        inv_g = fast_rcp(row_allreduce(se, [](float u, float v) { return u + v; }));   // >= 1: the maximum's term
    } else {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            // t: a softmax over the children of one kept key (a lane quad; ROW: a lane pair)
            float m = fmaxf(xt[t], xchg_f32<1>(xt[t]));
            if constexpr (!ROW) m = fmaxf(m, xchg_f32<2>(m));
            const float e = okt[t] ? __expf(xt[t] - m) : 0.f;
            float se = e + xchg_f32<1>(e);
            if constexpr (!ROW) se += xchg_f32<2>(se);
            wt[t] = okt[t] ? pkey[t] * e * fast_rcp(se) : 0.f;   // se >= 1
        }
    }
    // the four queries' normalisers, wave-uniform
    float inv_sum[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) inv_sum[r] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(inv_g), 16 * r));

    // ---- 5a. the weights P into the wave's LDS, [query][slot] ----
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        if (t >= ntile) break;                               // uniform
        const int s = 16 * t + n16;
        if constexpr (kBf16)
            reinterpret_cast<uint16_t*>(Pb)[g * nsp + s] = static_cast<uint16_t>(f32_to_bf16_bits(wt[t]));
        else
            reinterpret_cast<float*>(Pb)[g * nsp + s] = wt[t];
    }

    // ---- 4. this level's selection (levels above the finest) ----
    if constexpr (!FINEST) {
        // the ranking keys (B: the logit, ordered as the probability; A: the score) to one slot per
        // lane: tiles 4u .. 4u+3 of query row g become query r's keys of slots 64u + lane
        float kvs[SPL][4];
#pragma unroll
        for (int u = 0; u < SPL; ++u) {
            float c[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int t = 4 * u + j;
                c[j] = t < NT ? (VA ? wt[t] : xt[t]) : (VA ? 0.f : -INFINITY);
            }
            rows_transpose4(c);
#pragma unroll
            for (int r = 0; r < 4; ++r) kvs[u][r] = c[r];
        }
        // B: query r's maximum logit, for its kept keys' probabilities
        float mx[4] = {0.f, 0.f, 0.f, 0.f};
        if constexpr (!VA) {
            float m = xt[0];
#pragma unroll
            for (int t = 1; t < NT; ++t) m = fmaxf(m, xt[t]);
            m = row_allreduce(m, [](float u, float v) { return fmaxf(u, v); });
#pragma unroll
            for (int r = 0; r < 4; ++r) mx[r] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(m), 16 * r));
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            int qy, qx;
            query_yx(r, qy, qx);
            if (qy >= H || qx >= W) continue;                 // uniform across the wave
            bool okr[SPL];
            float kv[SPL];
            int nvalid = 0;
#pragma unroll
            for (int u = 0; u < SPL; ++u) {
                const int s = 64 * u + lane;
                okr[u] = ROW ? ok[u] && ((s >> 1) >= K) == ((r >> 1) != 0) : ok[u];
                kv[u] = kvs[u][r];
                nvalid += __popcll(__ballot(okr[u]));
            }
            const int keff = Ks < nvalid ? Ks : nvalid;
            uint32_t key[SPL], name[SPL];
#pragma unroll
            for (int u = 0; u < SPL; ++u) {
                key[u] = okr[u] ? ordered_bits(kv[u]) : 0u;
                name[u] = static_cast<uint32_t>(flat[u]);
            }
            bool kept[SPL];
            wave_select_top<SPL>(key, name, keff, kept);
            const size_t orow = ((static_cast<size_t>(b) * a.heads + h) * N + qy * W + qx) * Ks;
            int before = 0;
#pragma unroll
            for (int u = 0; u < SPL; ++u) {
                const uint64_t mask = __ballot(kept[u]);
                if (kept[u]) {
                    const int pos = before + lanes_below(mask);
                    a.sel_idx[orow + pos] = flat[u];
                    a.sel_key[orow + pos] = VA ? kv[u] : __expf(kv[u] - mx[r]) * inv_sum[r];
                    if constexpr (VA) {                       // refined at the next level (Omega)
                        const int s = 64 * u + lane;
                        if constexpr (kBf16) reinterpret_cast<uint16_t*>(Pb)[r * nsp + s] = 0;
                        else reinterpret_cast<float*>(Pb)[r * nsp + s] = 0.f;
                    }
                }
                before += __popcll(mask);
            }
            if (lane >= keff && lane < Ks) {
                a.sel_idx[orow + lane] = -1;
                a.sel_key[orow + lane] = 0.f;
            }
        }
    }
    wave_lds_sync();

    // ---- 5b. messages on MFMA ----
    float4_t o = {0.f, 0.f, 0.f, 0.f};
    if constexpr (kBf16) {
        // slots [s0, s0 + n) staged at Vt columns 0 .. n-1; lane half hh sums its half of them
        auto pv_part = [&](int s0, int n) {
            const int sph = n / NH;
            const uint16_t* prow_l = reinterpret_cast<const uint16_t*>(Pb) + t4 * nsp + s0 + hh * sph;
            const uint16_t* vrow_l = reinterpret_cast<const uint16_t*>(Vb) + (4 * cg + t4) * lay.vpitch + hh * sph;
            for (int st = 0; st < sph; st += 4) {
                const uint2 pa = *reinterpret_cast<const uint2*>(prow_l + st);
                const uint2 vb = *reinterpret_cast<const uint2*>(vrow_l + st);
                short4_t av, bv;
                av[0] = static_cast<short>(pa.x); av[1] = static_cast<short>(pa.x >> 16);
                av[2] = static_cast<short>(pa.y); av[3] = static_cast<short>(pa.y >> 16);
                bv[0] = static_cast<short>(vb.x); bv[1] = static_cast<short>(vb.x >> 16);
                bv[2] = static_cast<short>(vb.y); bv[3] = static_cast<short>(vb.y >> 16);
                o = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(av, bv, o, 0, 0, 0);
            }
        };
        if constexpr (kSplitV) {
            pv_part(0, kSplitSlots);
            // the second half's value rows over the first's (same lane layout as in the tiles)
            wave_lds_sync();
            uint16_t* vt = reinterpret_cast<uint16_t*>(Vb);
#pragma unroll
            for (int t = kTS; t < NT; ++t) {
                if (t >= ntile) break;                        // uniform
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    const uint4 vv = vkeep[t - kTS][j];
                    const int c0 = (g + 4 * j) * E;
                    const uint32_t w4[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const uint32_t bits = (e & 1) ? (w4[e >> 1] >> 16) : (w4[e >> 1] & 0xFFFFu);
                        vt[(c0 + e) * lay.vpitch + 16 * (t - kTS) + n16] = static_cast<uint16_t>(bits);
                    }
                }
            }
            wave_lds_sync();
            pv_part(kSplitSlots, nsp - kSplitSlots);
        } else {
            pv_part(0, nsp);
        }
    } else {
        const int sph = nsp / NH;
        const float* prow_l = reinterpret_cast<const float*>(Pb) + t4 * nsp + hh * sph;
        const float* vcol = reinterpret_cast<const float*>(Vb) + 4 * cg + t4;
        for (int st = 0; st < sph; ++st)
            o = __builtin_amdgcn_mfma_f32_4x4x1f32(prow_l[st], vcol[(hh * sph + st) * lay.vpitch], o, 0, 0, 0);
    }
    if constexpr (NH == 2) {
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r] += xchg_f32<4>(o[r]);
    }

    float pe_f[PE ? QPL : 1] = {};
    if constexpr (PE) {
        // the block into the wave's LDS as [channel][16 tokens, pitch kPeTokenPitch] (the value rows are no
        // longer read)
        wave_lds_sync();
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const uint4 vv = pe_ok ? peb[j] : make_uint4(0, 0, 0, 0);   // zero outside the map
            const int c0 = (g + 4 * j) * E;
            if constexpr (kBf16) {
                uint16_t* pt = reinterpret_cast<uint16_t*>(Vb);
                const uint32_t w4[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    pt[(c0 + e) * kPeTokenPitch + n16] =
                        static_cast<uint16_t>((e & 1) ? (w4[e >> 1] >> 16) : (w4[e >> 1] & 0xFFFFu));
            } else {
                float* pt = reinterpret_cast<float*>(Vb);
                pt[(c0 + 0) * kPeTokenPitch + n16] = __uint_as_float(vv.x);
                pt[(c0 + 1) * kPeTokenPitch + n16] = __uint_as_float(vv.y);
                pt[(c0 + 2) * kPeTokenPitch + n16] = __uint_as_float(vv.z);
                pt[(c0 + 3) * kPeTokenPitch + n16] = __uint_as_float(vv.w);
            }
        }
        wave_lds_sync();
        // this lane's channel over the 4x4 block (row r: four tokens), then each of its queries,
        // which sits at block position (1 + (qi >> 1), 1 + (qi & 1))
        float blkv[4][4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            if constexpr (kBf16) {
                const uint2 u = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(Vb) + ch * kPeTokenPitch + r * 4);
                blkv[r][0] = __uint_as_float(u.x << 16);
                blkv[r][1] = __uint_as_float(u.x & 0xFFFF0000u);
                blkv[r][2] = __uint_as_float(u.y << 16);
                blkv[r][3] = __uint_as_float(u.y & 0xFFFF0000u);
            } else {
                const float4 u = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(Vb) + ch * kPeTokenPitch + r * 4);
                blkv[r][0] = u.x;
                blkv[r][1] = u.y;
                blkv[r][2] = u.z;
                blkv[r][3] = u.w;
            }
        }
        // (with two lanes per channel, NH = 2, the lane's queries are row hh of the sibling block, so the
        // window rows are hh .. hh + 2, chosen by a select between the two possible rows)
#pragma unroll
        for (int u = 0; u < QPL; ++u) {
            const int rx = u & 1;                     // the window's left column in the block
            const int ry = NH == 2 ? 0 : u >> 1;      // its top row (NH = 2: plus hh)
            float acc = pebias;
#pragma unroll
            for (int ky = 0; ky < 3; ++ky)
#pragma unroll
                for (int kx = 0; kx < 3; ++kx) {
                    float val;
                    if constexpr (NH == 2)
                        val = hh ? blkv[ky + 1][rx + kx] : blkv[ky][rx + kx];
                    else
                        val = blkv[ry + ky][rx + kx];
                    acc = fmaf(pek[ky * 3 + kx], val, acc);
                }
            pe_f[u] = acc;
        }
    }

    // ---- 6. outputs ----
#pragma unroll
    for (int u = 0; u < QPL; ++u) {
        const int qi = (NH == 2 ? hh * QPL : 0) + u;
        int qy, qx;
        query_yx(qi, qy, qx);
        if (qy >= H || qx >= W) continue;
        const float m = pick4(o, qi) * pick4(inv_sum, qi);
        const uint32_t qpos = static_cast<uint32_t>(__mul24(qy, W) + qx);      // token within the map
        if constexpr (!FINEST) {
            float* mb = a.msg + (static_cast<size_t>(b) * N * a.heads + h) * D;  // uniform
            // (a batch element's message is below 2^32 bytes: twice a bf16 map at most)
            store_at<float>(mb, (qpos * static_cast<uint32_t>(a.heads * D) + ch) * 4u, PE ? m + pe_f[PE ? u : 0] : m);
        } else {
            const size_t qtok = static_cast<size_t>(b) * N + qpos;
            const int L = a.levels;
            const float wdef = a.inv_levels;
            float out;
            if (prefetch) {
                out = (VA ? 1.0f : (a.w ? wq[u][0] : wdef)) * (m + (PE ? pe_f[PE ? u : 0] : peq[u]));
#pragma unroll
                for (int lev = 1; lev <= kPre; ++lev) {
                    if (lev >= L) break;
                    out += (VA ? 1.0f : (a.w ? wq[u][lev] : wdef)) * anc[ROW ? u : 0][lev - 1];
                }
            } else {
                const float* wrow = a.w ? a.w + (qtok * a.heads + h) * L : nullptr;
                const float pe = PE ? pe_f[PE ? u : 0] : (a.pe0 ? a.pe0[(qtok * a.heads + h) * D + ch] : 0.f);
                out = (VA ? 1.0f : (wrow ? wrow[0] : wdef)) * (m + pe);
                for (int lev = 1; lev < L; ++lev) {
                    const size_t an = static_cast<size_t>(b) * a.lvl_N[lev] +
                                      static_cast<size_t>(qy >> lev) * a.lvl_W[lev] + (qx >> lev);
                    const float wl = VA ? 1.0f : (wrow ? wrow[lev] : wdef);
                    out += wl * a.coarser_msg[lev][(an * a.heads + h) * D + ch];
                }
            }
            void* ob = static_cast<unsigned char*>(a.out) + (static_cast<size_t>(b) * N * C + h * D) * TB;  // uniform
            S::store1_at(ob, qpos * static_cast<uint32_t>(C) + ch, out);
        }
    }
}

}  // namespace fine
}  // namespace qta

#endif
