// Backward pass of QuadTree attention: gradients of q, k, v (and QuadTree-B's w) for an upstream
// gradient of the output, with the kept-key sets of the forward held fixed (top-K is a selection,
// not differentiated). The chain rule runs through the forward's steps in reverse (Sec. 3.2):
//   1. combination (Eqs. 2, 5), inside the finest level's query pass: dm^l of a level-l token sums
//      w_{i,l} dout_i over its finest descendants (each sibling group adds its four queries' share
//      to its ancestors); dw_{i,l} = <dout_i, m^l of the ancestor>
//   2. each finer level, finest first, in two passes:
//      query pass, one wave per sibling group as in the forward: the logits and <dm, v> of every
//      candidate on MFMA, the softmax gradient (B: over the candidates, Eq. 6; A: over each kept
//      key's children with s = sigma t, Eq. 4, sending d sigma back to the parent level), dq on
//      MFMA; it keeps each query's softmax statistics and counts how many parents kept each key
//                                                                        (bwd_level_kernel)
//      key pass: the parents are sorted by the key they kept (a counting sort: the query pass's
//      count atomics also give each pair its place in its key's list; a scan, a fill), and one
//      wave per chunk of up to kKeyChunk parents of one kept key gathers those parents' four
//      children and forms dk and dv of the key's four children from the recomputed
//      probabilities; a key's rows are written once (summed over its chunks when it has several)
//                                                   (bwd_scan_*, bwd_fill, bwd_key, bwd_key_reduce)
//   3. the coarsest level (Eq. 1), in coarse_bwd.hip: a pass over query tiles (dq, softmax
//      statistics) and a pass over key tiles (dk, dv) that recomputes the probabilities, both on
//      MFMA and without atomics
//   4. pyramids: a pooled token hands 1/n of its gradient to each of its n valid children; the
//      level-0 gradients add every ancestor's, scaled along the chain      (bwd_unpool_kernel)
// All gradients are fp32. The message gradients of levels >= 2 are summed with atomics and the
// parents within one kept key's list come in the order the query pass's count atomics hand out, so
// the last bits of the gradients may differ between runs.
#include "qta_device.h"
#include "qta_internal.h"

namespace qta {

namespace {

typedef float float4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

// ---------------------------------------------------------------------------------------------
// zero fill (no hipMemsetAsync: the launch sequence may be captured in a graph)
// ---------------------------------------------------------------------------------------------

struct FillArgs {
    FillRange r[4];
    int n;
};

__global__ __launch_bounds__(256) void fill_zero_kernel(FillArgs a)
{
    const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
    for (int k = 0; k < a.n; ++k) {
        float4* p = reinterpret_cast<float4*>(a.r[k].p);
        const size_t n4 = a.r[k].n / 4;
        for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n4; i += stride)
            p[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
}

// ---------------------------------------------------------------------------------------------
// 2. finer levels
// ---------------------------------------------------------------------------------------------

// Byte layout of one wave's LDS region for nsp padded slots: the gathered key rows in fp32 (B
// operand of dq) and per slot the four queries' logit gradients.
struct BwdLds {
    int ks, dx, total;
    int kpitch;     // elements per key row (bf16 rows stay bf16: exact, and half the LDS per wave)
};

template <typename T, int D>
__host__ __device__ inline BwdLds bwd_lds(int nsp)
{
    constexpr int TB = sizeof(T);
    BwdLds L;
    // rows of 16-byte multiples; bf16 rows with d = 32 unpadded: the dq loop's two slot halves are 32
    // rows apart and meet the same banks with a padded pitch as well, the row writes conflict more,
    // and the 5 KB a wave then takes with 64 slots lets LDS hold 8 waves per SIMD instead of 6, which
    // outweighs that (d = 64 keeps its padding: unpadded it measured slower, with registers, not
    // LDS, bounding its occupancy)
    L.kpitch = TB == 2 ? (D == 32 ? D : D + 8) : D + 4;
    L.ks = 0;
    L.dx = L.ks + nsp * L.kpitch * TB;
    L.total = L.dx + nsp * 16;
    return L;
}

__device__ __forceinline__ float pick4(const float4_t& v, int i)
{
    return i == 0 ? v[0] : i == 1 ? v[1] : i == 2 ? v[2] : v[3];
}

// v[off + i] for i in 0..3 (off a compile-time constant), by selects
template <int N>
__device__ __forceinline__ float pick4_at(const float (&v)[N], int off, int i)
{
    return i == 0 ? v[off] : i == 1 ? v[off + 1] : i == 2 ? v[off + 2] : v[off + 3];
}

// One work item: parent query P at level l+1 and head h (item = (b*Np + P)*heads + h); its four
// children at level l share the candidate slots 4r + c (child c of the parent's kept key r).
template <typename T, int D, int NSP, bool VA, bool FINEST>
__device__ __forceinline__ void bwd_item(const BwdLevelArgs& a, const int item, unsigned char* const base)
{
    using S = Storage<T>;
    constexpr bool kBf16 = sizeof(T) == 2;
    constexpr int TB = sizeof(T);
    constexpr int RB = D * TB;             // bytes of one head's row
    constexpr int E = S::kPer16B;          // elements per 16-byte chunk
    constexpr int NJ = RB / 64;            // chunks per lane and row (lane group g: g, g+4, ...)
    constexpr int NT = NSP / 16;
    constexpr int NCG = D / 4;
    constexpr int NH = 16 / NCG;
    constexpr int QPL = 4 / NH;

    const int lane = threadIdx.x & 63;
    const int Np = a.Hp * a.Wp;
    const int bp = fast_div(item, a.div_heads);
    const int h = item - bp * a.heads;
    const int b = fast_div(bp, a.div_Np);
    const int P = bp - b * Np;
    const int Py = fast_div(P, a.div_Wp), Px = P - Py * a.Wp;
    const int H = a.H, W = a.W, C = a.C, K = a.Kp;
    const int N = H * W;
    const int nslot = 4 * K;
    const int nsp = (nslot + 15) & ~15;
    const BwdLds lay = bwd_lds<T, D>(nsp);
    float* Ks = reinterpret_cast<float*>(base + lay.ks);
    float* dxs = reinterpret_cast<float*>(base + lay.dx);      // [slot][4]

    const size_t prow_off = (static_cast<size_t>(b) * a.heads + h) * Np + P;
    const int32_t* prow = a.parent_idx + prow_off * K;
    auto child_of_slot_J = [&](int J, int s) -> int {
        if (s >= nslot || J < 0) return -1;
        const int Jy = fast_div(J, a.div_Wp), Jx = J - __mul24(Jy, a.Wp);
        const int cy = 2 * Jy + ((s >> 1) & 1), cx = 2 * Jx + (s & 1);
        return (cy < H && cx < W) ? __mul24(cy, W) + cx : -1;
    };
    const int n16 = lane & 15, g = lane >> 4;
    const int ntile = nsp / 16;
    const int last_sel = K - 1;
    int J_g[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) J_g[t] = prow[min(4 * t + (n16 >> 2), last_sel)];
    // QuadTree-A: the parent's score of this lane's slot in each tile
    float pkey[VA ? NT : 1];
    if constexpr (VA) {
#pragma unroll
        for (int t = 0; t < NT; ++t) pkey[t] = a.parent_key[prow_off * K + min(4 * t + (n16 >> 2), last_sel)];
    }

    // queries: A operand rows 4g .. 4g+3 hold query g, so lane 16g + n receives query g's logit (and
    // <dm, v>) of slot 16t + n from every tile t
    const int qi = n16 >> 2;
    const int qy = 2 * Py + (qi >> 1), qx = 2 * Px + (qi & 1);
    const bool q_ok = qy < H && qx < W;
    const uint32_t qtok = static_cast<uint32_t>(__mul24(min(qy, H - 1), W) + min(qx, W - 1));
    uint4 qa[NJ];
    {
        const unsigned char* qbase = static_cast<const unsigned char*>(a.q) +
            (a.blocked ? prow_off * 4 * RB : (static_cast<size_t>(b) * N * C + h * D) * TB);
        const uint32_t qoff = a.blocked ? static_cast<uint32_t>(qi * RB) : qtok * static_cast<uint32_t>(C * TB);
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const uint4 raw = *reinterpret_cast<const uint4*>(qbase + (qoff + static_cast<uint32_t>((g + 4 * j) * 16)));
            qa[j] = q_ok ? raw : make_uint4(0, 0, 0, 0);
        }
    }
    // gradient of the queries' messages, same layout: level 0 the upstream gradient (times w_0 in
    // the weights below), other levels dm^l in fp32
    uint4 da[FINEST ? NJ : 1];
    float dmA[FINEST ? 1 : NJ][E];
    const size_t grow = (static_cast<size_t>(b) * N + qtok) * C + h * D;    // element offset of the row
    if constexpr (FINEST) {
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const uint4 raw = *reinterpret_cast<const uint4*>(static_cast<const unsigned char*>(a.dout) +
                                                              (grow + (g + 4 * j) * E) * TB);
            da[j] = q_ok ? raw : make_uint4(0, 0, 0, 0);
        }
    } else {
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
#pragma unroll
            for (int e4 = 0; e4 < E; e4 += 4) {
                const float4 raw = *reinterpret_cast<const float4*>(a.dm + grow + (g + 4 * j) * E + e4);
                dmA[j][e4 + 0] = q_ok ? raw.x : 0.f;
                dmA[j][e4 + 1] = q_ok ? raw.y : 0.f;
                dmA[j][e4 + 2] = q_ok ? raw.z : 0.f;
                dmA[j][e4 + 3] = q_ok ? raw.w : 0.f;
            }
        }
    }
    // level 0: w_{g,0} (QuadTree-B; 1/L without w; 1 for A), below. Per batch element
    // a 64-bit base, within it 32-bit offsets (one element's map is below 2^31 bytes, and so are its
    // level weights and softmax statistics)
    const size_t wq_off = static_cast<size_t>(b) * static_cast<uint32_t>(N * a.heads * a.levels);
    const float* wq_b = a.w + wq_off;
    float* const st_b = a.stats + static_cast<size_t>(b * a.heads + h) * static_cast<uint32_t>(N * 2 * (VA ? K : 1));
    // the products' lanes hold query g (row g of the wave): its position, and w_{g,0}
    const int ry_q = 2 * Py + (g >> 1), rx_q = 2 * Px + (g & 1);
    const bool qv = ry_q < H && rx_q < W;                     // this lane's query lies on the map
    const uint32_t qpos = static_cast<uint32_t>(__mul24(min(ry_q, H - 1), W) + min(rx_q, W - 1));
    float w0 = 1.f;
    if constexpr (FINEST && !VA) w0 = a.w ? wq_b[(qpos * a.heads + h) * a.levels] : 1.0f / a.levels;
    // how many parents kept each key of level l+1 (for the key pass's counting sort); the count a
    // pair finds is its place in the key's list
    if (lane < K) {
        const int Jr = prow[min(lane, last_sel)];
        if (Jr >= 0) a.slot[prow_off * K + lane] = atomicAdd(a.count + (static_cast<size_t>(b) * a.heads + h) * Np + Jr, 1);
    }

    // ---- gathers, logits and <dm, v> on MFMA, key rows to LDS, one tile of 16 slots at a time ----
    const bool kvb = a.blocked;
    const size_t kv_base = kvb ? (static_cast<size_t>(b) * a.heads + h) * Np * 4 * RB
                               : (static_cast<size_t>(b) * N * C + h * D) * TB;
    const unsigned char* kg = static_cast<const unsigned char*>(a.k) + kv_base;
    const unsigned char* vg = static_cast<const unsigned char*>(a.v) + kv_base;
    const uint32_t tok_bytes = static_cast<uint32_t>(C * TB);
    float acc_x[NT], acc_g[NT];
    bool gok[NT];
    int flat_t[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        acc_x[t] = 0.f;
        acc_g[t] = 0.f;
        gok[t] = false;
        flat_t[t] = -1;
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        if (t >= ntile) break;                                // uniform
        const int s = 16 * t + n16;
        const int f = child_of_slot_J(J_g[t], s);
        gok[t] = f >= 0;
        flat_t[t] = f;
        const uint32_t goff = (!gok[t] ? 0u : (kvb ? static_cast<uint32_t>(J_g[t] * 4 + (s & 3)) * RB
                                                    : static_cast<uint32_t>(f) * tok_bytes)) + g * 16;
        uint4 kc[NJ], vc[NJ];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            kc[j] = *reinterpret_cast<const uint4*>(kg + (goff + 64 * j));
            vc[j] = *reinterpret_cast<const uint4*>(vg + (goff + 64 * j));
        }
        float4_t ax = {0.f, 0.f, 0.f, 0.f}, ag = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const uint4 kk = gok[t] ? kc[j] : make_uint4(0, 0, 0, 0);
            const uint4 vv = gok[t] ? vc[j] : make_uint4(0, 0, 0, 0);
            if constexpr (kBf16) {
                ax = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, qa[j]),
                                                             __builtin_bit_cast(bf16x8_t, kk), ax, 0, 0, 0);
            } else {
                ax = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(qa[j].x), __uint_as_float(kk.x), ax, 0, 0, 0);
                ax = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(qa[j].y), __uint_as_float(kk.y), ax, 0, 0, 0);
                ax = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(qa[j].z), __uint_as_float(kk.z), ax, 0, 0, 0);
                ax = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(qa[j].w), __uint_as_float(kk.w), ax, 0, 0, 0);
            }
            float vf[E];
            S::unpack(vv, vf);
            if constexpr (FINEST && kBf16) {
                ag = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, da[j]),
                                                             __builtin_bit_cast(bf16x8_t, vv), ag, 0, 0, 0);
            } else if constexpr (FINEST) {
                ag = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(da[j].x), vf[0], ag, 0, 0, 0);
                ag = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(da[j].y), vf[1], ag, 0, 0, 0);
                ag = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(da[j].z), vf[2], ag, 0, 0, 0);
                ag = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(da[j].w), vf[3], ag, 0, 0, 0);
            } else {
#pragma unroll
                for (int e = 0; e < E; ++e)
                    ag = __builtin_amdgcn_mfma_f32_16x16x4f32(dmA[j][e], vf[e], ag, 0, 0, 0);
            }
            // the key row in the storage type (zeros for missing candidates)
            if constexpr (kBf16) {
                *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(Ks) + s * lay.kpitch + (g + 4 * j) * E) = kk;
            } else {
                *reinterpret_cast<uint4*>(Ks + s * lay.kpitch + (g + 4 * j) * E) = kk;
            }
        }
        // rows 4g .. 4g+3 of the products are all query g
        acc_x[t] = ax[0];
        acc_g[t] = ag[0];
    }

    // ---- softmax gradients of this lane's query g, slots 16t + n16 ----
    float x[NT], gsl[NT], dxt[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const bool okt = t < ntile && gok[t];
        x[t] = okt ? acc_x[t] * a.scale : -INFINITY;
        gsl[t] = FINEST ? w0 * acc_g[t] : acc_g[t];        // dLoss/d(weight) on Omega
        dxt[t] = 0.f;
    }
    // The sum over the query's slots of one value per tile, in the order of a butterfly over the
    // 64 slots (each tile over its 16-lane row, then tiles (0 + 1) + (2 + 3)), so that the softmax
    // statistics round as a full-wave sum of one slot per lane does
    auto slots_sum = [&](const float (&v)[NT]) -> float {
        float r[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < NT; ++t) r[t] = row_allreduce(v[t], [](float u, float w) { return u + w; });
        return (r[0] + r[1]) + (r[2] + r[3]);
    };
    if constexpr (!VA) {
        static_assert(NT <= 4, "at most 64 candidate slots");
        // a softmax per query over its 16-lane row and the lane's tiles
        float m = x[0];
#pragma unroll
        for (int t = 1; t < NT; ++t) m = fmaxf(m, x[t]);
        m = row_allreduce(m, [](float u, float v) { return fmaxf(u, v); });
        float e[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) e[t] = (t < ntile && gok[t]) ? __expf(x[t] - m) : 0.f;
        const float sum = slots_sum(e);
        const float inv = fast_rcp(sum);                      // sum >= 1 (the maximum's term)
        float pg[NT], pa[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const float p = e[t] * inv;
            e[t] = p;
            pg[t] = p * gsl[t];
            pa[t] = p * acc_g[t];
        }
        const float Dr = slots_sum(pg);
#pragma unroll
        for (int t = 0; t < NT; ++t) dxt[t] = qv ? e[t] * (gsl[t] - Dr) : 0.f;
        // the key pass recomputes p = exp(x - lse) and needs D
        if (n16 == 0 && qv) *reinterpret_cast<float2*>(st_b + qpos * 2) = make_float2(m + fast_ln(sum), Dr);
        if constexpr (FINEST) {
            if (a.w && a.dw) {                                // uniform
                const float dw0 = slots_sum(pa);
                if (n16 == 0 && qv) a.dw[wq_off + static_cast<uint32_t>((qpos * a.heads + h) * a.levels)] = dw0;
            }
        }
    } else {
        // d sigma of each slot's key: a key this lane's query keeps is refined at level l-1, and its
        // score's gradient comes from there
        float dsT[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) dsT[t] = gsl[t];
        if constexpr (!FINEST) {
            const size_t srow = ((static_cast<size_t>(b) * a.heads + h) * N + qpos) * a.Ks;
            for (int mm = 0; mm < a.Ks; ++mm) {
                const int kept = a.sel_idx[srow + mm];
                const float dv = a.dsig_in[srow + mm];
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    if (t < ntile && gok[t] && kept == flat_t[t]) dsT[t] = dv;
            }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            if (t >= ntile) break;                            // uniform
            const bool okt = gok[t];
            // a softmax over the children of one kept key (a lane quad)
            float m = fmaxf(x[t], xchg_f32<1>(x[t]));
            m = fmaxf(m, xchg_f32<2>(m));
            const float e = okt ? __expf(x[t] - m) : 0.f;
            float sum = e + xchg_f32<1>(e);
            sum += xchg_f32<2>(sum);
            const float tt = okt ? e * fast_rcp(sum) : 0.f;   // sum >= 1
            const float sc = pkey[t] * tt;
            const float ds = dsT[t];
            float dsq = tt * ds;                              // this query's d sigma of the kept key
            dsq += xchg_f32<1>(dsq);
            dsq += xchg_f32<2>(dsq);
            dxt[t] = qv ? sc * (ds - dsq) : 0.f;
            // the key pass recomputes t = exp(x - lse) per kept parent key and needs sum t ds
            const int key = 4 * t + (n16 >> 2);
            if ((n16 & 3) == 0 && key < K && qv)
                *reinterpret_cast<float2*>(st_b + static_cast<uint32_t>(qpos * K + key) * 2) =
                    make_float2(m + fast_ln(sum), dsq);
            // the four queries' sum, across the wave's rows
            float dsig = qv ? dsq : 0.f;
            dsig += xchg_f32<16>(dsig);
            dsig += xchg_f32<32>(dsig);
            if (g == 0 && (n16 & 3) == 0 && key < K) a.dsig_out[prow_off * K + key] = dsig;
        }
    }
    // the logit gradients into LDS as [slot][query] (the B operand of dq)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        if (t >= ntile) break;                                // uniform
        dxs[(16 * t + n16) * 4 + g] = dxt[t];
    }
    wave_lds_sync();

    // ---- dq = scale * sum_s dx_s k_s on the 4x4 MFMA (blocks over 4-channel groups, slot halves) ----
    {
        float* const dq_b = a.dq + static_cast<size_t>(b) * N * C + h * D;
        const int blk = lane >> 2, t4 = lane & 3;
        const int cg = blk / NH, hh = blk % NH;
        const int ch = 4 * cg + t4;
        const int sph = nsp / NH;
        float4_t o = {0.f, 0.f, 0.f, 0.f};
        for (int st = 0; st < sph; ++st) {
            const int sl = hh * sph + st;
            float kv;
            if constexpr (kBf16)
                kv = bf16_bits_to_f32(reinterpret_cast<const uint16_t*>(Ks)[sl * lay.kpitch + 4 * cg + t4]);
            else
                kv = Ks[sl * lay.kpitch + 4 * cg + t4];
            o = __builtin_amdgcn_mfma_f32_4x4x1f32(dxs[sl * 4 + t4], kv, o, 0, 0, 0);
        }
        if constexpr (NH == 2) {
#pragma unroll
            for (int r = 0; r < 4; ++r) o[r] += xchg_f32<4>(o[r]);
        }
#pragma unroll
        for (int u = 0; u < QPL; ++u) {
            const int r = (NH == 2 ? hh * QPL : 0) + u;
            const int ry = 2 * Py + (r >> 1), rx = 2 * Px + (r & 1);
            if (ry >= H || rx >= W) continue;
            // (uniform base, 32-bit offset: a batch element's fp32 gradient is below 2^32 bytes)
            store_at<float>(dq_b, (static_cast<uint32_t>(__mul24(ry, W) + rx) * static_cast<uint32_t>(C) + ch) * 4u,
                            a.scale * pick4(o, r));
        }
    }

    // ---- level 0: the combination's backward for the coarser levels. The four queries are the
    //      children of P, so at every level j >= 1 they share one ancestor: dm^j of that ancestor
    //      receives sum_r w_{r,j} dout_r (written at j = 1, where the ancestor is P itself, and
    //      added with atomics above), and dw_{r,j} = <dout_r, m^j of the ancestor>. ----
    if constexpr (FINEST) {
        const int L = a.levels;
        const bool want_dw = !VA && a.w && a.dw;
        // w of query n16 >> 2: a uniform base and a 32-bit offset (a batch element's w is below 2^31 bytes)
        const float* const w_b = a.w ? a.w + static_cast<size_t>(b) * N * a.heads * L : nullptr;
        const uint32_t wrow = (qtok * static_cast<uint32_t>(a.heads) + h) * static_cast<uint32_t>(L);
        float gv[NJ][E];
#pragma unroll
        for (int j = 0; j < NJ; ++j) S::unpack(da[j], gv[j]);                    // zero off the map
        // the coarser levels in blocks: each block's weights and forward messages are all requested
        // before any is used, so their latencies overlap. Blocks of four need about 20 more VGPRs,
        // which costs occupancy unless the LDS already caps it (64 candidate slots)
        constexpr int kBlk = NSP == 64 ? 4 : 1;
        for (int lv0 = 1; lv0 < L; lv0 += kBlk) {
            float wl[kBlk];
            float4 mq[kBlk][NJ * E / 4];
            size_t arow[kBlk];
#pragma unroll
            for (int i = 0; i < kBlk; ++i) {
                const int lv = min(lv0 + i, L - 1);                               // clamped: unused past L-1
                wl[i] = VA ? 1.0f : (a.w ? load_at<float>(w_b, (wrow + lv) * 4u) : 1.0f / L);
                const size_t anc = static_cast<size_t>(b) * a.lvl_N[lv] +
                                   static_cast<size_t>((2 * Py) >> lv) * a.lvl_W[lv] + ((2 * Px) >> lv);
                arow[i] = (anc * a.heads + h) * D;
                if (want_dw) {                                                    // uniform
#pragma unroll
                    for (int j = 0; j < NJ; ++j)
#pragma unroll
                        for (int e4 = 0; e4 < E; e4 += 4)
                            mq[i][(j * E + e4) / 4] =
                                load_at<float4>(a.msg_fwd[lv] + arow[i], ((g + 4 * j) * E + e4) * 4u);
                }
            }
#pragma unroll
            for (int i = 0; i < kBlk; ++i) {
                const int lv = lv0 + i;
                if (lv >= L) break;                                               // uniform
                float part = 0.f;
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    const int c0 = (g + 4 * j) * E;
                    if (want_dw) {
#pragma unroll
                        for (int e4 = 0; e4 < E; e4 += 4) {
                            const float4 m4 = mq[i][(j * E + e4) / 4];
                            part += gv[j][e4] * m4.x + gv[j][e4 + 1] * m4.y + gv[j][e4 + 2] * m4.z + gv[j][e4 + 3] * m4.w;
                        }
                    }
                    // lane 16g + e stores element e of chunk g + 4j (one instruction covers the head's
                    // channels contiguously): the sum over the four queries (query n16 >> 2, on lanes
                    // 4 apart). Lane 4q + i contributes its query's elements i (and, with eight per
                    // chunk, i + 4); after the sums over lanes 4 apart, lanes 0-3 hold elements 0-3
                    // and lanes 4-7 elements 4-7
                    const int ei = n16 & 3;
                    float mine = row_sum_stride4(wl[i] * pick4_at(gv[j], 0, ei));
                    if constexpr (E == 8) {
                        const float hi = row_sum_stride4(wl[i] * pick4_at(gv[j], 4, ei));
                        mine = n16 < 4 ? mine : hi;
                    }
                    if (n16 < E) {
                        float* dst = a.dm_out[lv] + arow[i] + c0 + n16;
                        if (lv == 1)
                            *dst = mine;
                        else
                            atomicAddNoRet(dst, mine);
                    }
                }
                if (want_dw) {
                    part += xchg_f32<16>(part);
                    part += xchg_f32<32>(part);
                    if (g == 0 && (n16 & 3) == 0 && q_ok) store_at<float>(a.dw + static_cast<size_t>(b) * N * a.heads * L, (wrow + lv) * 4u, part);
                }
            }
        }
    }
}

template <typename T, int D, int NSP, bool VA, bool FINEST>
__global__ __launch_bounds__(256) void bwd_level_kernel(BwdLevelArgs a)
{
    const int wave = threadIdx.x >> 6;
    const int wpb = blockDim.x >> 6;
    const long long nitems = static_cast<long long>(a.B) * a.heads * a.Hp * a.Wp;
    const int item = __builtin_amdgcn_readfirstlane(xcd_remap(blockIdx.x, gridDim.x) * wpb + wave);
    if (item >= nitems) return;            // whole wave leaves; only wave-level syncs follow
    extern __shared__ __align__(16) unsigned char smem[];
    const int nsp = (4 * a.Kp + 15) & ~15;
    bwd_item<T, D, NSP, VA, FINEST>(a, item, smem + static_cast<size_t>(wave) * bwd_lds<T, D>(nsp).total);
}

template <typename T, int D, int NSP, bool VA, bool FINEST>
hipError_t launch_level_one(const BwdLevelArgs& a, hipStream_t stream)
{
    const int nsp = (4 * a.Kp + 15) & ~15;
    const size_t wave_bytes = bwd_lds<T, D>(nsp).total;
    int wpb = 4;
    while (wpb > 1 && wpb * wave_bytes > 64 * 1024) --wpb;
    if (wpb * wave_bytes > device_max_lds()) return hipErrorInvalidValue;
    static std::atomic<unsigned long long> configured{0};     // devices whose LDS limit is raised
    if (hipError_t e = set_max_lds_once(reinterpret_cast<const void*>(&bwd_level_kernel<T, D, NSP, VA, FINEST>), configured);
        e != hipSuccess)
        return e;
    const long long items = static_cast<long long>(a.B) * a.heads * a.Hp * a.Wp;
    const long long blocks = (items + wpb - 1) / wpb;
    if (blocks * wpb >= 0x7FFFFFFFLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((bwd_level_kernel<T, D, NSP, VA, FINEST>), dim3(static_cast<unsigned>(blocks)),
                       dim3(wpb * kWave), wpb * wave_bytes, stream, a);
    return hipGetLastError();
}

template <typename T, int D, bool VA, bool FINEST>
hipError_t launch_level_nsp(const BwdLevelArgs& a, hipStream_t stream)
{
    const int nslot = 4 * a.Kp;
    if (nslot <= 16) return launch_level_one<T, D, 16, VA, FINEST>(a, stream);
    if (nslot <= 32) return launch_level_one<T, D, 32, VA, FINEST>(a, stream);
    return launch_level_one<T, D, 64, VA, FINEST>(a, stream);
}

template <typename T, int D>
hipError_t launch_level_td(const BwdLevelArgs& a, bool variant_a, bool finest, hipStream_t stream)
{
    if (variant_a)
        return finest ? launch_level_nsp<T, D, true, true>(a, stream) : launch_level_nsp<T, D, true, false>(a, stream);
    return finest ? launch_level_nsp<T, D, false, true>(a, stream) : launch_level_nsp<T, D, false, false>(a, stream);
}

// ---- counting sort of the parents by the key they kept ----

// Block-wide exclusive scan of two counters per element over 256 threads x 4 elements; returns
// the block total in `total` (all threads).
__device__ __forceinline__ void block_scan_256x4(int2 (&v)[4], int2& total)
{
    __shared__ int2 wsum[4];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int2 run = make_int2(0, 0);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int2 t = v[e];
        v[e] = run;
        run.x += t.x;
        run.y += t.y;
    }
    // inclusive scan of the thread sums over the wave
    int2 inc = run;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int ux = __shfl_up(inc.x, o, kWave), uy = __shfl_up(inc.y, o, kWave);
        if (lane >= o) {
            inc.x += ux;
            inc.y += uy;
        }
    }
    if (lane == 63) wsum[wave] = inc;
    __syncthreads();
    int2 before = make_int2(inc.x - run.x, inc.y - run.y);
    total = make_int2(0, 0);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const int2 t = wsum[w];
        if (w < wave) {
            before.x += t.x;
            before.y += t.y;
        }
        total.x += t.x;
        total.y += t.y;
    }
    __syncthreads();
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        v[e].x += before.x;
        v[e].y += before.y;
    }
}

__device__ __forceinline__ int chunks_of(int n) { return n > 0 ? (n + kKeyChunk - 1) / kKeyChunk : 1; }

// (count, chunk count) of the key slots i0 .. i0+3 (i0 a multiple of 4) from one 16-byte load, and
// (0, 0) past the last slot. The count array is padded to a multiple of four slots, so the load
// (clamped to the last quad) stays inside it; it is unconditional and masked rather than selected,
// so that the compiler keeps every such load of a thread in flight at once.
__device__ __forceinline__ void quad_counts(const int32_t* count, int i0, int n, int2 (&c)[4])
{
    const int4 r = *reinterpret_cast<const int4*>(count + min(i0, (n - 1) & ~3));
    const int v[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int valid = i0 + e < n;
        const int x = v[e] & -valid;
        c[e] = make_int2(x, chunks_of(x) & -valid);
    }
}

// Elements i0 .. i0+3 of p below n: one 16-byte store for a full quad (i0 a multiple of 4).
__device__ __forceinline__ void store_quad(int32_t* p, int i0, int n, int x, int y, int z, int w)
{
    if (i0 + 3 < n) {
        *reinterpret_cast<int4*>(p + i0) = make_int4(x, y, z, w);
    } else {
        if (i0 < n) p[i0] = x;
        if (i0 + 1 < n) p[i0 + 1] = y;
        if (i0 + 2 < n) p[i0 + 2] = z;
    }
}

// Per block of 1024 kept-key slots: the sums of the counts and of the chunk counts.
__global__ __launch_bounds__(256) void bwd_scan_reduce_kernel(BwdScanArgs a)
{
    int2 v[4];
    quad_counts(a.count, blockIdx.x * 1024 + threadIdx.x * 4, a.n, v);
    int2 total;
    block_scan_256x4(v, total);
    if (threadIdx.x == 0) {
        a.block_sums[2 * blockIdx.x] = total.x;
        a.block_sums[2 * blockIdx.x + 1] = total.y;
    }
}

// One block: exclusive scan of the block sums, in place.
__global__ __launch_bounds__(256) void bwd_scan_blocks_kernel(BwdScanArgs a)
{
    int2 carry = make_int2(0, 0);
    for (int t0 = 0; t0 < a.nblocks; t0 += 1024) {
        int2 v[4];
        const int base = t0 + threadIdx.x * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int i = base + e;
            const int j = 2 * min(i, a.nblocks - 1);
            const int2 b = make_int2(a.block_sums[j], a.block_sums[j + 1]);
            v[e] = i < a.nblocks ? b : make_int2(0, 0);
        }
        int2 total;
        block_scan_256x4(v, total);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int i = base + e;
            if (i < a.nblocks) {
                a.block_sums[2 * i] = v[e].x + carry.x;
                a.block_sums[2 * i + 1] = v[e].y + carry.y;
            }
        }
        carry.x += total.x;
        carry.y += total.y;
    }
    if (threadIdx.x == 0) {
        a.off[a.n] = carry.x;
        a.coff[a.n] = carry.y;
    }
}

// Per block: the exclusive scans of the counts (list offsets) and of the chunk counts, and the
// kept key of every chunk.
__global__ __launch_bounds__(256) void bwd_scan_write_kernel(BwdScanArgs a)
{
    int2 v[4], c[4];
    const int base = blockIdx.x * 1024 + threadIdx.x * 4;
    quad_counts(a.count, base, a.n, c);
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = c[e];
    int2 total;
    block_scan_256x4(v, total);
    const int2 bo = make_int2(a.block_sums[2 * blockIdx.x], a.block_sums[2 * blockIdx.x + 1]);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        v[e].x += bo.x;
        v[e].y += bo.y;
    }
    store_quad(a.off, base, a.n, v[0].x, v[1].x, v[2].x, v[3].x);
    store_quad(a.coff, base, a.n, v[0].y, v[1].y, v[2].y, v[3].y);
    store_quad(a.count, base, a.n, 0, 0, 0, 0);               // the last reader: zero for the next level
#pragma unroll
    for (int e = 0; e < 4; ++e)
        if (base + e < a.n)
            for (int t = 0; t < c[e].y; ++t) a.chunk_key[v[e].y + t] = base + e;
}

// Up to kSingleScanMax key slots: the whole scan in one workgroup of 1024 threads (four tiles of
// 4096 slots), in place of the three-kernel scan. Every load comes first and every store last: a
// store issued between two waits for loads would be waited for too.
constexpr int kSingleScanMax = 16384;

__global__ __launch_bounds__(1024) void bwd_scan_single_kernel(BwdScanArgs a)
{
    __shared__ int2 wsum[4][16];                              // one row per tile: a single barrier each
    constexpr int kTile = 4096;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int2 c[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t) quad_counts(a.count, t * kTile + tid * 4, a.n, c[t]);
    int2 x[4][4];                                             // exclusive scans (list offset, first chunk)
    int2 carry = make_int2(0, 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        if (t * kTile < a.n) {                                // uniform; no early exit, so c stays in registers
            int2 run = make_int2(0, 0);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                x[t][e] = run;
                run.x += c[t][e].x;
                run.y += c[t][e].y;
            }
            int2 inc = run;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int ux = __shfl_up(inc.x, o, kWave), uy = __shfl_up(inc.y, o, kWave);
                if (lane >= o) {
                    inc.x += ux;
                    inc.y += uy;
                }
            }
            if (lane == 63) wsum[t][wave] = inc;
            __syncthreads();
            int2 before = make_int2(carry.x + inc.x - run.x, carry.y + inc.y - run.y), total = make_int2(0, 0);
#pragma unroll
            for (int w = 0; w < 16; ++w) {
                const int2 ws = wsum[t][w];
                if (w < wave) {
                    before.x += ws.x;
                    before.y += ws.y;
                }
                total.x += ws.x;
                total.y += ws.y;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                x[t][e].x += before.x;
                x[t][e].y += before.y;
            }
            carry.x += total.x;
            carry.y += total.y;
        }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int i0 = t * kTile + tid * 4;
        store_quad(a.off, i0, a.n, x[t][0].x, x[t][1].x, x[t][2].x, x[t][3].x);
        store_quad(a.coff, i0, a.n, x[t][0].y, x[t][1].y, x[t][2].y, x[t][3].y);
        store_quad(a.count, i0, a.n, 0, 0, 0, 0);             // read above by this thread only
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (i0 + e < a.n)
                for (int u = 0; u < c[t][e].y; ++u) a.chunk_key[x[t][e].y + u] = i0 + e;
    }
    if (tid == 0) {
        a.off[a.n] = carry.x;
        a.coff[a.n] = carry.y;
    }
}

// Every kept (parent, rank) pair into the list of the key it kept, at the place its count atomic
// handed out in the query pass.
__global__ __launch_bounds__(256) void bwd_fill_kernel(BwdFillArgs a)
{
    const long long tid = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (tid >= a.nentries) return;
    const int J = a.parent_idx[tid];
    if (J < 0) return;
    const int row = static_cast<int>(tid / a.Kp);          // bh * Np + P
    const int r = static_cast<int>(tid - static_cast<long long>(row) * a.Kp);
    const int bh = row / a.Np, P = row - bh * a.Np;
    a.entries[a.off[bh * a.Np + J] + a.slot[tid]] = P * a.Kp + r;
}

// Key pass: one wave per chunk of one kept key J's parent list (up to kKeyChunk = 16 parents, so
// 64 query slots s = 4e + child). It mirrors the forward's fine kernel with the roles of queries and
// keys exchanged: the four children of J (keys) are the MFMA operand repeated over the rows, the
// slots' query rows are gathered 16 at a time (lane 16g + n takes chunks g, g+4, ... of slot n of a
// tile), lane s keeps tile s/16 of the products and so ends with slot s's logits and <dm, v> for
// the four keys. The weights dx and vw go to LDS, and dk = scale * dx^T Q, then dv = vw^T dM, run on
// the 4x4 MFMA from the slots' q rows, then their dm rows, in one LDS buffer (layout in key_lds).
// Only the tiles that hold parents are gathered. A key whose list spans several chunks has each
// chunk store its partial rows, and bwd_key_reduce_kernel adds them up. (Letting the last chunk add
// them, with a counter and device-scope fences, was ten times slower: every such fence writes back
// the L2.)
struct KeyLds {
    int rows, dx, vw, total;
    int qpitch;     // elements per query row
    int mpitch;     // elements per dm row
    int mslots;     // dm rows the buffer holds at once (all 64, or 32 per pass)
};

// With bf16 inputs the query rows are bf16 values and stay bf16 (exact, half the LDS). So do the
// finest level's dm rows, which are dout (its w_0 moves into the weights vw). The coarser levels'
// dm rows are fp32 and go through the buffer 32 slots at a time, so that it stays at the size of
// the bf16 query rows.
template <typename T, int D, bool FINEST>
__host__ __device__ inline KeyLds key_lds()
{
    constexpr bool bf = sizeof(T) == 2;
    KeyLds L;
    L.qpitch = bf ? D + 8 : D + 4;                         // rows of 16-byte multiples
    L.mpitch = bf && FINEST ? D + 8 : D + 4;
    L.mslots = bf && !FINEST ? 2 * kKeyChunk : 4 * kKeyChunk;
    const int qbytes = 4 * kKeyChunk * L.qpitch * (bf ? 2 : 4);
    const int mbytes = L.mslots * L.mpitch * (bf && FINEST ? 2 : 4);
    L.rows = 0;
    L.dx = L.rows + (qbytes > mbytes ? qbytes : mbytes);
    L.vw = L.dx;                                           // the weights replace dx once dk is done
    L.total = L.dx + 4 * kKeyChunk * 16;
    return L;
}

template <typename T, int D, bool VA, bool FINEST>
__global__ __launch_bounds__(64) void bwd_key_kernel(BwdLevelArgs a)
{
    using S = Storage<T>;
    constexpr bool kBf16 = sizeof(T) == 2;
    constexpr int TB = sizeof(T);
    constexpr int RB = D * TB;               // bytes of one head's row (storage)
    constexpr int E = S::kPer16B;            // storage elements per 16-byte chunk
    constexpr int NJ = RB / 64;              // storage chunks per lane and row
    constexpr int NJF = D / 16;              // fp32 4-channel chunks per lane and row
    constexpr int NT = 4 * kKeyChunk / 16;   // tiles of 16 slots
    constexpr int NCG = D / 4;
    constexpr int NH = 16 / NCG;
    constexpr int QPL = 4 / NH;
    static_assert(kKeyChunk == 16, "one wave holds the 64 query slots of a chunk");

    const int lane = threadIdx.x & 63;
    const int Np = a.Hp * a.Wp;
    const int n = a.B * a.heads * Np;
    // chunks of neighbouring keys (whose parents overlap) run on one XCD and share its L2: the
    // workgroups that have a chunk (the grid is an upper bound) are remapped onto contiguous ranges
    const int nchunks = a.coff[n];
    if (static_cast<int>(blockIdx.x) >= nchunks) return;    // whole wave
    const int chunk = __builtin_amdgcn_readfirstlane(xcd_remap(static_cast<int>(blockIdx.x), nchunks));
    extern __shared__ __align__(16) unsigned char smem[];
    const KeyLds lay = key_lds<T, D, FINEST>();
    constexpr bool kRows16 = kBf16 && FINEST;                // query and dm rows kept as bf16
    constexpr bool kSplit = kBf16 && !FINEST;                // bf16 query rows, fp32 dm rows in two passes
    uint16_t* const Rs16 = reinterpret_cast<uint16_t*>(smem + lay.rows);
    auto q_elem = [&](int sl, int c) -> float {
        if constexpr (kBf16) return bf16_bits_to_f32(Rs16[sl * lay.qpitch + c]);
        else return reinterpret_cast<const float*>(smem + lay.rows)[sl * lay.qpitch + c];
    };
    auto m_elem = [&](int sl, int c) -> float {
        if constexpr (kRows16) return bf16_bits_to_f32(Rs16[sl * lay.mpitch + c]);
        else return reinterpret_cast<const float*>(smem + lay.rows)[sl * lay.mpitch + c];
    };
    float* Rs = reinterpret_cast<float*>(smem + lay.rows);    // q rows, then dm rows
    float* dxs = reinterpret_cast<float*>(smem + lay.dx);     // [slot][4 keys]
    float* vws = reinterpret_cast<float*>(smem + lay.vw);

    const int key = a.chunk_key[chunk];      // bh * Np + J
    const int bh = fast_div(key, a.div_Np), J = key - bh * Np;
    const int b = fast_div(bh, a.div_heads), h = bh - b * a.heads;
    const int H = a.H, W = a.W, C = a.C, N = H * W, K = a.Kp;
    const int first = a.coff[key], nch = a.coff[key + 1] - first;
    const int beg = a.off[key] + (chunk - first) * kKeyChunk;
    const int nent = min(a.off[key + 1] - beg, kKeyChunk);
    const int Jy = fast_div(J, a.div_Wp), Jx = J - Jy * a.Wp;
    const int n16 = lane & 15, g = lane >> 4;
    const bool kvb = a.blocked;
    const unsigned char* qbase = static_cast<const unsigned char*>(a.q);

    // the four keys (children of J); rows n16 of the A operand hold key n16 & 3
    bool jv[4];
    int jtok[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const int y = 2 * Jy + (c >> 1), x = 2 * Jx + (c & 1);
        jv[c] = y < H && x < W;
        jtok[c] = jv[c] ? y * W + x : 0;
    }
    const int kc = n16 & 3;
    const bool kc_ok = kc == 0 ? jv[0] : kc == 1 ? jv[1] : kc == 2 ? jv[2] : jv[3];
    const int kc_tok = kc == 0 ? jtok[0] : kc == 1 ? jtok[1] : kc == 2 ? jtok[2] : jtok[3];
    const size_t krow = kvb ? (static_cast<size_t>(key) * 4 + kc) * RB
                            : ((static_cast<size_t>(b) * N + kc_tok) * C + h * D) * TB;
    uint4 kA[NJ], vA[NJ];
    float vAf[NJF][4];
    const unsigned km = opaque_mask(kc_ok);                   // (a key off the map reads a clamped row)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        kA[j] = masked4(*reinterpret_cast<const uint4*>(static_cast<const unsigned char*>(a.k) + krow + (g + 4 * j) * 16), km);
        vA[j] = masked4(*reinterpret_cast<const uint4*>(static_cast<const unsigned char*>(a.v) + krow + (g + 4 * j) * 16), km);
    }
    if constexpr (!FINEST) {
        // V in 4-channel chunks g, g+4, ... to meet the fp32 dm rows channel for channel
#pragma unroll
        for (int j = 0; j < NJF; ++j) {
            const int c0 = (g + 4 * j) * 4;
            if constexpr (kBf16) {
                const uint2 vr = *reinterpret_cast<const uint2*>(static_cast<const unsigned char*>(a.v) + krow + c0 * 2);
                vAf[j][0] = bf16_bits_to_f32(vr.x & 0xFFFFu);
                vAf[j][1] = bf16_bits_to_f32(vr.x >> 16);
                vAf[j][2] = bf16_bits_to_f32(vr.y & 0xFFFFu);
                vAf[j][3] = bf16_bits_to_f32(vr.y >> 16);
            } else {
                const float4 vr = *reinterpret_cast<const float4*>(static_cast<const unsigned char*>(a.v) + krow + c0 * 4);
                vAf[j][0] = vr.x;
                vAf[j][1] = vr.y;
                vAf[j][2] = vr.z;
                vAf[j][3] = vr.w;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) vAf[j][e] = masked(vAf[j][e], km);
        }
    }

    // the chunk's parents: lane e < nent holds entry e
    const int ent_lane = nent > 0 ? a.entries[beg + min(lane, nent - 1)] : 0;   // an empty list reads nothing
    // where slot s's query lives: entry s >> 2, child s & 3
    auto slot_query = [&](int s, int ent, int& P, int& r, int& qtok, bool& qv) {
        P = fast_div(ent, a.div_Kp);
        r = ent - P * K;
        const int Py = fast_div(P, a.div_Wp), Px = P - Py * a.Wp;
        const int qi = s & 3;
        const int qy = 2 * Py + (qi >> 1), qx = 2 * Px + (qi & 1);
        qv = (s >> 2) < nent && qy < H && qx < W;
        qtok = min(qy, H - 1) * W + min(qx, W - 1);
    };

    const int ntile = (nent + 3) / 4;                         // tiles that hold parents
    const int nsp = 16 * ntile;
    // uniform bases of this (batch, head): query rows (blocked: this (batch, head)'s parent blocks),
    // dout or dm rows, w (a batch element's map, its messages and w are below 2^32 bytes)
    const unsigned char* const qb_base = kvb ? qbase + static_cast<size_t>(bh) * Np * 4 * RB
                                             : qbase + (static_cast<size_t>(b) * N * C + h * D) * TB;
    const unsigned char* const d_base = FINEST ? static_cast<const unsigned char*>(a.dout) +
                                                     (static_cast<size_t>(b) * N * C + h * D) * TB
                                               : nullptr;
    const float* const m_base = FINEST ? nullptr : a.dm + static_cast<size_t>(b) * N * C + h * D;
    const float* const w_base = a.w ? a.w + static_cast<size_t>(b) * N * a.heads * a.levels : nullptr;
    float acc_x[4] = {0.f, 0.f, 0.f, 0.f}, acc_g[4] = {0.f, 0.f, 0.f, 0.f};
    // each tile's dm chunks (level 0: w_0 dout; bf16: dout as stored), kept for dv
    float mreg[NT][kRows16 ? 1 : (FINEST ? NJ * E : NJF * 4)];
    uint4 dreg[kRows16 ? NT : 1][kRows16 ? NJ : 1];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        if (t >= ntile) break;                                // uniform
        const int s = 16 * t + n16;
        const int ent = __shfl(ent_lane, s >> 2, kWave);
        int P, r, qtok;
        bool qv;
        slot_query(s, ent, P, r, qtok, qv);
        // every load unconditional at a clamped, valid address and zeroed for a slot without a
        // query by an opaque mask (a visible select on a loaded value became a branch around the
        // load that waited for it at the join); uniform bases with 32-bit per-lane offsets
        const unsigned qm = opaque_mask(qv);
        const uint32_t qoff = kvb ? static_cast<uint32_t>((P * 4 + (s & 3)) * RB)
                                  : static_cast<uint32_t>(qtok) * static_cast<uint32_t>(C * TB);
        uint4 qB[NJ];
#pragma unroll
        for (int j = 0; j < NJ; ++j) qB[j] = masked4(load_at<uint4>(qb_base, qoff + (g + 4 * j) * 16), qm);
        float w0 = 1.0f;
        if constexpr (FINEST && !VA)
            w0 = a.w ? load_at<float>(w_base, (static_cast<uint32_t>(qtok) * a.heads + h) * a.levels * 4u) : 1.0f / a.levels;
        float4_t ax = {0.f, 0.f, 0.f, 0.f}, ag = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            if constexpr (kBf16) {
                ax = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kA[j]),
                                                             __builtin_bit_cast(bf16x8_t, qB[j]), ax, 0, 0, 0);
            } else {
                ax = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kA[j].x), __uint_as_float(qB[j].x), ax, 0, 0, 0);
                ax = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kA[j].y), __uint_as_float(qB[j].y), ax, 0, 0, 0);
                ax = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kA[j].z), __uint_as_float(qB[j].z), ax, 0, 0, 0);
                ax = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kA[j].w), __uint_as_float(qB[j].w), ax, 0, 0, 0);
            }
            // the query row for dk (fp32, or bf16 as stored)
            if constexpr (kBf16) {
                *reinterpret_cast<uint4*>(Rs16 + s * lay.qpitch + (g + 4 * j) * E) = qB[j];
            } else {
                float qf[E];
                S::unpack(qB[j], qf);
                float* qd = Rs + s * lay.qpitch + (g + 4 * j) * E;
#pragma unroll
                for (int e4 = 0; e4 < E; e4 += 4)
                    *reinterpret_cast<float4*>(qd + e4) = make_float4(qf[e4], qf[e4 + 1], qf[e4 + 2], qf[e4 + 3]);
            }
        }
        if constexpr (FINEST) {
            // <dout, v> on the storage type (times w_0 below), and w_0 dout in fp32 for dv
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                const uint4 dd = masked4(load_at<uint4>(d_base, static_cast<uint32_t>(qtok) * static_cast<uint32_t>(C * TB) +
                                                                    (g + 4 * j) * 16), qm);
                if constexpr (kBf16) {
                    ag = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, vA[j]),
                                                                 __builtin_bit_cast(bf16x8_t, dd), ag, 0, 0, 0);
                } else {
                    ag = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(vA[j].x), __uint_as_float(dd.x), ag, 0, 0, 0);
                    ag = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(vA[j].y), __uint_as_float(dd.y), ag, 0, 0, 0);
                    ag = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(vA[j].z), __uint_as_float(dd.z), ag, 0, 0, 0);
                    ag = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(vA[j].w), __uint_as_float(dd.w), ag, 0, 0, 0);
                }
                if constexpr (kRows16) {
                    dreg[t][j] = dd;
                } else {
                    float gf[E];
                    S::unpack(dd, gf);
#pragma unroll
                    for (int e = 0; e < E; ++e) mreg[t][j * E + e] = w0 * gf[e];
                }
            }
        } else {
            // <dm, v> with dm in fp32, 4-channel chunks g, g+4, ...
#pragma unroll
            for (int j = 0; j < NJF; ++j) {
                const uint4 dr = masked4(load_at<uint4>(m_base, (static_cast<uint32_t>(qtok) * static_cast<uint32_t>(C) +
                                                                 (g + 4 * j) * 4) * 4u), qm);
                const float4 dm4 = make_float4(__uint_as_float(dr.x), __uint_as_float(dr.y), __uint_as_float(dr.z),
                                               __uint_as_float(dr.w));
                ag = __builtin_amdgcn_mfma_f32_16x16x4f32(vAf[j][0], dm4.x, ag, 0, 0, 0);
                ag = __builtin_amdgcn_mfma_f32_16x16x4f32(vAf[j][1], dm4.y, ag, 0, 0, 0);
                ag = __builtin_amdgcn_mfma_f32_16x16x4f32(vAf[j][2], dm4.z, ag, 0, 0, 0);
                ag = __builtin_amdgcn_mfma_f32_16x16x4f32(vAf[j][3], dm4.w, ag, 0, 0, 0);
                mreg[t][4 * j] = dm4.x;
                mreg[t][4 * j + 1] = dm4.y;
                mreg[t][4 * j + 2] = dm4.z;
                mreg[t][4 * j + 3] = dm4.w;
            }
        }
        // rows 4g + c of the products are key c for every g: lane 16g + n keeps tile g
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            acc_x[c] = g == t ? ax[c] : acc_x[c];
            acc_g[c] = g == t ? ag[c] : acc_g[c];
        }
    }

    // ---- slot `lane`: its query's statistics and the weights of the four keys ----
    float4 vw_lane;                       // staged over dx once dk has read it
    {
        const int s = lane;
        int P, r, qtok;
        bool qv;
        slot_query(s, __shfl(ent_lane, s >> 2, kWave), P, r, qtok, qv);
        const size_t qrow = static_cast<size_t>(bh) * N + qtok;
        const float2 st = VA ? *reinterpret_cast<const float2*>(a.stats + (qrow * K + r) * 2)
                             : *reinterpret_cast<const float2*>(a.stats + qrow * 2);
        const float sigma = VA ? a.parent_key[(static_cast<size_t>(bh) * Np + P) * K + r] : 1.0f;
        float w0 = 1.0f;
        if constexpr (FINEST && !VA)
            w0 = a.w ? a.w[((static_cast<size_t>(b) * N + qtok) * a.heads + h) * a.levels] : 1.0f / a.levels;
        float dx[4], vw[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const bool valid = qv && jv[c];
            const float pr = valid ? __expf(acc_x[c] * a.scale - st.x) : 0.f;   // B: p; A: t
            const float gsv = FINEST ? w0 * acc_g[c] : acc_g[c];
            if constexpr (!VA) {
                dx[c] = pr * (gsv - st.y);
                vw[c] = pr;
            } else {
                const float sc = sigma * pr;
                float ds = gsv;
                bool kept = false;
                if constexpr (!FINEST) {
                    const size_t srow = qrow * a.Ks;
                    for (int mm = 0; mm < a.Ks; ++mm)
                        if (valid && a.sel_idx[srow + mm] == jtok[c]) {
                            kept = true;
                            ds = a.dsig_in[srow + mm];
                        }
                }
                dx[c] = sc * (ds - st.y);
                vw[c] = kept ? 0.f : sc;
            }
        }
        if constexpr (kRows16) {
#pragma unroll
            for (int c = 0; c < 4; ++c) vw[c] *= w0;         // the dout rows are stored without w_0
        }
        *reinterpret_cast<float4*>(dxs + s * 4) = make_float4(dx[0], dx[1], dx[2], dx[3]);
        vw_lane = make_float4(vw[0], vw[1], vw[2], vw[3]);
    }
    wave_lds_sync();

    // ---- dk = dx^T Q, then dv = vw^T dM, on the 4x4 MFMA (blocks over 4-channel groups, slot halves) ----
    const int blk = lane >> 2, t4 = lane & 3;
    const int cg = blk / NH, hh = blk % NH;
    const int ch = 4 * cg + t4;
    const int sph = nsp / NH;
    float4_t ok_ = {0.f, 0.f, 0.f, 0.f}, ov = {0.f, 0.f, 0.f, 0.f};
    for (int st = 0; st < sph; ++st) {
        const int sl = hh * sph + st;
        ok_ = __builtin_amdgcn_mfma_f32_4x4x1f32(dxs[sl * 4 + t4], q_elem(sl, ch), ok_, 0, 0, 0);
    }
    // the dm rows into the same buffer (lane 16g + n holds slot 16t + n's chunks g, g+4, ...), all
    // slots at once or (kSplit) 32 at a time; slot sl of a pass is row sl - first
    constexpr int kPasses = kSplit ? 2 : 1;
#pragma unroll
    for (int pass = 0; pass < kPasses; ++pass) {
        const int first = pass * lay.mslots;
        if (first >= nsp) break;                              // uniform
        wave_lds_sync();
        if (pass == 0) *reinterpret_cast<float4*>(vws + lane * 4) = vw_lane;   // (vws aliases dxs)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            if (t >= ntile) break;                            // uniform
            if (16 * t < first || 16 * t >= first + lay.mslots) continue;   // uniform
            const int s = 16 * t + n16 - first;
            if constexpr (kRows16) {
#pragma unroll
                for (int j = 0; j < NJ; ++j) *reinterpret_cast<uint4*>(Rs16 + s * lay.mpitch + (g + 4 * j) * E) = dreg[t][j];
            } else if constexpr (FINEST) {
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    float* md = Rs + s * lay.mpitch + (g + 4 * j) * E;
#pragma unroll
                    for (int e4 = 0; e4 < E; e4 += 4)
                        *reinterpret_cast<float4*>(md + e4) = make_float4(mreg[t][j * E + e4], mreg[t][j * E + e4 + 1],
                                                                          mreg[t][j * E + e4 + 2], mreg[t][j * E + e4 + 3]);
                }
            } else {
#pragma unroll
                for (int j = 0; j < NJF; ++j)
                    *reinterpret_cast<float4*>(Rs + s * lay.mpitch + (g + 4 * j) * 4) =
                        make_float4(mreg[t][4 * j], mreg[t][4 * j + 1], mreg[t][4 * j + 2], mreg[t][4 * j + 3]);
            }
        }
        wave_lds_sync();
        const int cnt = min(nsp - first, lay.mslots);         // a multiple of 16
        const int sphp = cnt / NH;
        for (int st = 0; st < sphp; ++st) {
            const int sl = hh * sphp + st;
            ov = __builtin_amdgcn_mfma_f32_4x4x1f32(vws[(first + sl) * 4 + t4], m_elem(sl, ch), ov, 0, 0, 0);
        }
    }
    if constexpr (NH == 2) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            ok_[c] += xchg_f32<4>(ok_[c]);
            ov[c] += xchg_f32<4>(ov[c]);
        }
    }
    if (nch > 1) {
        // this chunk's rows; bwd_key_reduce_kernel adds up the key's chunks
#pragma unroll
        for (int u = 0; u < QPL; ++u) {
            const int c = (NH == 2 ? hh * QPL : 0) + u;
            float* pk = a.partial + ((static_cast<size_t>(chunk) * 4 + c) * 2) * D + ch;
            pk[0] = pick4(ok_, c);
            pk[D] = pick4(ov, c);
        }
        return;
    }
#pragma unroll
    for (int u = 0; u < QPL; ++u) {
        const int c = (NH == 2 ? hh * QPL : 0) + u;
        const bool cv = c == 0 ? jv[0] : c == 1 ? jv[1] : c == 2 ? jv[2] : jv[3];
        const int ct = c == 0 ? jtok[0] : c == 1 ? jtok[1] : c == 2 ? jtok[2] : jtok[3];
        if (!cv) continue;
        const size_t row = (static_cast<size_t>(b) * N + ct) * C + h * D + ch;
        a.dk[row] = a.scale * pick4(ok_, c);
        a.dv[row] = pick4(ov, c);
    }
}

// Keys whose list spans several chunks: the sum of the chunks' partial rows. One thread per
// (kept-key slot, child, 4 channels).
__global__ __launch_bounds__(256) void bwd_key_reduce_kernel(BwdLevelArgs a, int d)
{
    const int Np = a.Hp * a.Wp;
    const long long n = static_cast<long long>(a.B) * a.heads * Np;
    const int q4n = d / 4;
    const long long tid = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (tid >= n * 4 * q4n) return;
    const int qd = static_cast<int>(tid % q4n);
    const int c = static_cast<int>((tid / q4n) % 4);
    const int key = static_cast<int>(tid / (4LL * q4n));
    const int first = a.coff[key], nch = a.coff[key + 1] - first;
    if (nch <= 1) return;
    const int bh = fast_div(key, a.div_Np), J = key - bh * Np;
    const int b = fast_div(bh, a.div_heads), h = bh - b * a.heads;
    const int Jy = fast_div(J, a.div_Wp), Jx = J - Jy * a.Wp;
    const int y = 2 * Jy + (c >> 1), x = 2 * Jx + (c & 1);
    if (y >= a.H || x >= a.W) return;
    float4 sk = make_float4(0.f, 0.f, 0.f, 0.f), sv = sk;
    for (int t = 0; t < nch; ++t) {
        const float* pk = a.partial + ((static_cast<size_t>(first + t) * 4 + c) * 2) * d + 4 * qd;
        const float4 k4 = *reinterpret_cast<const float4*>(pk);
        const float4 v4 = *reinterpret_cast<const float4*>(pk + d);
        sk.x += k4.x; sk.y += k4.y; sk.z += k4.z; sk.w += k4.w;
        sv.x += v4.x; sv.y += v4.y; sv.z += v4.z; sv.w += v4.w;
    }
    const size_t row = (static_cast<size_t>(b) * a.H * a.W + y * a.W + x) * a.C + h * d + 4 * qd;
    *reinterpret_cast<float4*>(a.dk + row) = make_float4(a.scale * sk.x, a.scale * sk.y, a.scale * sk.z, a.scale * sk.w);
    *reinterpret_cast<float4*>(a.dv + row) = sv;
}

template <typename T, int D, bool VA, bool FINEST>
hipError_t launch_key_tdv(const BwdLevelArgs& a, long long max_chunks, hipStream_t stream)
{
    if (max_chunks >= 0x7FFFFFFFLL) return hipErrorInvalidValue;
    const size_t lds = key_lds<T, D, FINEST>().total;
    if (lds > device_max_lds()) return hipErrorInvalidValue;
    hipLaunchKernelGGL((bwd_key_kernel<T, D, VA, FINEST>), dim3(static_cast<unsigned>(max_chunks)), dim3(kWave), lds,
                       stream, a);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_key_td(const BwdLevelArgs& a, bool variant_a, bool finest, long long max_chunks, hipStream_t stream)
{
    if (variant_a)
        return finest ? launch_key_tdv<T, D, true, true>(a, max_chunks, stream)
                      : launch_key_tdv<T, D, true, false>(a, max_chunks, stream);
    return finest ? launch_key_tdv<T, D, false, true>(a, max_chunks, stream)
                  : launch_key_tdv<T, D, false, false>(a, max_chunks, stream);
}

// 3. the coarsest level: coarse_bwd.hip

// ---------------------------------------------------------------------------------------------
// 4. pyramids
// ---------------------------------------------------------------------------------------------

template <int LMAX>
__global__ __launch_bounds__(256) void bwd_unpool_kernel(BwdUnpoolArgs a)
{
    // one thread per tensor (q, k or v: blockIdx.y) and 4 channels of the (up to) 2x2 level-0 tokens
    // under one level-1 token, which share every ancestor: the ancestors' rows are loaded once for four
    // tokens. A batch element takes a.bpb consecutive blocks (its maps are below 2^31 bytes, so chunk
    // indices fit 32 bits)
    const int m = blockIdx.y;
    // given V levels are not pooled from v: their gradients are returned as they are, and v's level-0
    // gradient receives nothing from them
    if (m == 2 && !a.v_pooled) return;                        // whole block
    const int cpt = a.C / 4;
    const int n1 = a.H[1] * a.W[1] * cpt;
    const int b = static_cast<int>(blockIdx.x) / a.bpb;
    const int t = (static_cast<int>(blockIdx.x) - b * a.bpb) * blockDim.x + threadIdx.x;
    if (t >= n1) return;
    const int i = fast_div(t, a.div_cpt);
    const int ch = t - i * cpt;
    const int y1 = fast_div(i, a.div_W1), x1 = i - y1 * a.W[1];
    float* const dst = m == 0 ? a.dq : m == 1 ? a.dk : a.dv;
    // the four tokens' rows first (they are used last), then the ancestors' rows, then the sums
    const int H0 = a.H[0], W0 = a.W[0];
    const size_t base = static_cast<size_t>(b) * static_cast<uint32_t>(H0 * W0 * a.C) + 4 * ch;
    uint32_t tok[4];
    bool ok[4];
    float4 r[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const int y = 2 * y1 + (c >> 1), x = 2 * x1 + (c & 1);
        ok[c] = y < H0 && x < W0;
        tok[c] = static_cast<uint32_t>((min(y, H0 - 1) * W0 + min(x, W0 - 1)) * a.C);   // clamped onto the map
        r[c] = *reinterpret_cast<const float4*>(dst + base + tok[c]);
    }
    // (eight levels at a time: all of a group's loads before its sums)
    constexpr int kGroup = 8;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    float fl = 1.0f;
#pragma unroll
    for (int l0 = 1; l0 < LMAX; l0 += kGroup) {
        if (l0 >= a.L) break;                                 // uniform
        float4 g[kGroup];
        float f[kGroup];
#pragma unroll
        for (int j = 0; j < kGroup; ++j) {
            const int l = l0 + j;
            if (l >= LMAX || l >= a.L) break;                 // uniform
            const int yl = y1 >> (l - 1), xl = x1 >> (l - 1);
            const int ny = (2 * yl + 1 < a.H[l - 1]) ? 2 : 1, nx = (2 * xl + 1 < a.W[l - 1]) ? 2 : 1;
            fl *= 1.0f / static_cast<float>(ny * nx);
            f[j] = fl;
            const size_t off = static_cast<size_t>(b) * static_cast<uint32_t>(a.H[l] * a.W[l] * a.C) +
                               static_cast<uint32_t>((yl * a.W[l] + xl) * a.C + 4 * ch);
            const float* const gl = m == 0 ? a.gq[l] : m == 1 ? a.gk[l] : a.gv[l];
            g[j] = *reinterpret_cast<const float4*>(gl + off);
        }
#pragma unroll
        for (int j = 0; j < kGroup; ++j) {
            if (l0 + j >= LMAX || l0 + j >= a.L) break;       // uniform
            s.x += f[j] * g[j].x;
            s.y += f[j] * g[j].y;
            s.z += f[j] * g[j].z;
            s.w += f[j] * g[j].w;
        }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c)
        if (ok[c])
            *reinterpret_cast<float4*>(dst + base + tok[c]) = make_float4(r[c].x + s.x, r[c].y + s.y, r[c].z + s.z, r[c].w + s.w);
}

}  // namespace

hipError_t launch_fill_zero(const FillRange* r, int n, hipStream_t stream)
{
    if (n <= 0) return hipSuccess;
    if (n > 4) return hipErrorInvalidValue;
    FillArgs a{};
    size_t most = 0;
    for (int k = 0; k < n; ++k) {
        a.r[k] = r[k];
        if (r[k].n > most) most = r[k].n;
    }
    a.n = n;
    const size_t blocks = (most / 4 + 255) / 256;
    const unsigned grid = static_cast<unsigned>(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096);
    hipLaunchKernelGGL(fill_zero_kernel, dim3(grid), dim3(256), 0, stream, a);
    return hipGetLastError();
}

// The multiply-high constants of the divisions the level kernels make by the map sizes.
BwdLevelArgs with_divisors(const BwdLevelArgs& a)
{
    BwdLevelArgs b = a;
    b.div_Wp = make_fastdiv(a.Wp);
    b.div_Np = make_fastdiv(a.Hp * a.Wp);
    b.div_heads = make_fastdiv(a.heads);
    b.div_Kp = make_fastdiv(a.Kp);
    return b;
}

hipError_t launch_bwd_level(const BwdLevelArgs& a, int d, bool variant_a, bool use_bf16, bool finest,
                            hipStream_t stream)
{
    if (4 * a.Kp > 64) return hipErrorInvalidValue;
    const BwdLevelArgs b = with_divisors(a);
    if (use_bf16) {
        if (d == 32) return launch_level_td<bf16, 32>(b, variant_a, finest, stream);
        if (d == 64) return launch_level_td<bf16, 64>(b, variant_a, finest, stream);
    } else {
        if (d == 32) return launch_level_td<float, 32>(b, variant_a, finest, stream);
        if (d == 64) return launch_level_td<float, 64>(b, variant_a, finest, stream);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_bwd_keys(const BwdLevelArgs& a, const BwdScanArgs& sc, int d, bool variant_a, bool use_bf16,
                           bool finest, hipStream_t stream)
{
    if (sc.n <= 0) return hipErrorInvalidValue;
    hipError_t e;
    if (sc.n <= kSingleScanMax) {
        hipLaunchKernelGGL(bwd_scan_single_kernel, dim3(1), dim3(1024), 0, stream, sc);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    } else {
        const unsigned nb = static_cast<unsigned>(sc.nblocks);
        hipLaunchKernelGGL(bwd_scan_reduce_kernel, dim3(nb), dim3(256), 0, stream, sc);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(bwd_scan_blocks_kernel, dim3(1), dim3(256), 0, stream, sc);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(bwd_scan_write_kernel, dim3(nb), dim3(256), 0, stream, sc);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    BwdFillArgs f{a.parent_idx, a.slot, static_cast<long long>(sc.n) * a.Kp, a.Kp, a.Hp * a.Wp, sc.off, a.entries};
    const long long fb = (f.nentries + 255) / 256;
    if (fb >= 0x7FFFFFFFLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL(bwd_fill_kernel, dim3(static_cast<unsigned>(fb)), dim3(256), 0, stream, f);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const long long max_chunks = static_cast<long long>(sc.n) + (static_cast<long long>(sc.n) * a.Kp + kKeyChunk - 1) / kKeyChunk;
    const BwdLevelArgs k = with_divisors(a);
    if (use_bf16) {
        if (d == 32) e = launch_key_td<bf16, 32>(k, variant_a, finest, max_chunks, stream);
        else if (d == 64) e = launch_key_td<bf16, 64>(k, variant_a, finest, max_chunks, stream);
        else return hipErrorInvalidValue;
    } else {
        if (d == 32) e = launch_key_td<float, 32>(k, variant_a, finest, max_chunks, stream);
        else if (d == 64) e = launch_key_td<float, 64>(k, variant_a, finest, max_chunks, stream);
        else return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    const long long rb = (static_cast<long long>(sc.n) * 4 * (d / 4) + 255) / 256;
    if (rb >= 0x7FFFFFFFLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL(bwd_key_reduce_kernel, dim3(static_cast<unsigned>(rb)), dim3(256), 0, stream, k, d);
    return hipGetLastError();
}

hipError_t launch_bwd_unpool(const BwdUnpoolArgs& a, hipStream_t stream)
{
    if (a.L < 2) return hipErrorInvalidValue;
    const long long n0 = static_cast<long long>(a.H[0]) * a.W[0] * a.C;          // floats of a level-0 map
    const long long n1 = static_cast<long long>(a.H[1]) * a.W[1] * (a.C / 4);    // threads per batch element
    const long long bpb = (n1 + 255) / 256;
    if (n0 >= 0x7FFFFFFFLL || bpb * a.B >= 0x7FFFFFFFLL) return hipErrorInvalidValue;
    BwdUnpoolArgs u = a;
    u.div_cpt = make_fastdiv(a.C / 4);
    u.div_W1 = make_fastdiv(a.W[1]);
    u.bpb = static_cast<int>(bpb);
    const dim3 grid(static_cast<unsigned>(bpb * a.B), 3);     // y: q, k, v
    if (a.L <= 4) hipLaunchKernelGGL(bwd_unpool_kernel<4>, grid, dim3(256), 0, stream, u);
    else if (a.L <= 8) hipLaunchKernelGGL(bwd_unpool_kernel<8>, grid, dim3(256), 0, stream, u);
    else hipLaunchKernelGGL(bwd_unpool_kernel<QTA_MAX_LEVELS>, grid, dim3(256), 0, stream, u);
    return hipGetLastError();
}

}  // namespace qta
