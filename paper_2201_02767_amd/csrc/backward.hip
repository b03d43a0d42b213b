// Backward pass of QuadTree attention: gradients of q, k, v (and QuadTree-B's w) for an upstream
// gradient of the output, with the kept-key sets of the forward held fixed (top-K is a selection,
// not differentiated). The chain rule runs through the forward's steps in reverse (Sec. 3.2):
//   1. combination (Eqs. 2, 5): dm^l of a level-l token sums w_{i,l} dout_i over its finest
//      descendants; dw_{i,l} = <dout_i, m^l of the ancestor>            (bwd_combine_kernel)
//   2. each finer level, finest first, one wave per sibling group as in the forward: the logits
//      and <dm, v> of every candidate on MFMA, then the softmax gradient (B: over the candidates,
//      Eq. 6; A: over each kept key's children with s = sigma t, Eq. 4, sending d sigma back to the
//      parent level), dq on MFMA, and dk, dv scattered to the gathered keys with fp32 atomics
//                                                                        (bwd_level_kernel)
//   3. the coarsest level (Eq. 1): a pass per query (dq, softmax statistics) and a pass per key
//      (dk, dv) that recomputes the probabilities, so neither needs atomics (bwd_coarse_*)
//   4. pyramids: a pooled token hands 1/n of its gradient to each of its n valid children; the
//      level-0 gradients add every ancestor's, scaled along the chain      (bwd_unpool_kernel)
// All gradients are fp32. The order in which the atomics land varies from run to run, so dk and
// dv (and dm at levels >= 2) may differ in the last bits between runs.
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
// 1. combination backward
// ---------------------------------------------------------------------------------------------

// Sum over the d lanes of one head (d = 32 or 64 consecutive lanes, aligned).
__device__ __forceinline__ float head_sum(float x, int d)
{
    x += xchg_f32<1>(x);
    x += xchg_f32<2>(x);
    x += xchg_f32<4>(x);
    x += xchg_f32<8>(x);
    x += xchg_f32<16>(x);
    if (d == 64) x += xchg_f32<32>(x);
    return x;
}

template <typename T>
__global__ __launch_bounds__(256) void bwd_combine_kernel(BwdCombineArgs a)
{
    using S = Storage<T>;
    const int C = a.C, L = a.L;
    const int H1 = a.H[1], W1 = a.W[1], H0 = a.H[0], W0 = a.W[0];
    const long long total = static_cast<long long>(a.B) * H1 * W1 * C;
    const long long tid = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
    // threads past the end run on clamped indices (the head sums need every lane) and store nothing
    const bool active = tid < total;
    const long long t = active ? tid : total - 1;
    const int c = static_cast<int>(t % C);
    const long long pt = t / C;
    const int P = static_cast<int>(pt % (static_cast<long long>(H1) * W1));
    const int b = static_cast<int>(pt / (static_cast<long long>(H1) * W1));
    const int h = c / a.d;
    const int Py = P / W1, Px = P - Py * W1;
    const bool want_dw = a.variant_b && a.w && a.dw;
    // the ancestors' messages at this channel (shared by the 2x2 children of P)
    float manc[QTA_MAX_LEVELS];
#pragma unroll
    for (int l = 1; l < QTA_MAX_LEVELS; ++l) {
        manc[l] = 0.f;
        if (l < L && want_dw) {
            const size_t anc = static_cast<size_t>(b) * a.H[l] * a.W[l] +
                               static_cast<size_t>((2 * Py) >> l) * a.W[l] + ((2 * Px) >> l);
            manc[l] = a.msg[l][anc * C + c];
        }
    }
    float acc[QTA_MAX_LEVELS];
#pragma unroll
    for (int l = 0; l < QTA_MAX_LEVELS; ++l) acc[l] = 0.f;
    const float wdef = a.variant_b ? 1.0f / L : 1.0f;
#pragma unroll
    for (int ci = 0; ci < 4; ++ci) {
        const int y = 2 * Py + (ci >> 1), x = 2 * Px + (ci & 1);
        const bool valid = y < H0 && x < W0;           // the same for every lane of a head
        const size_t tok = static_cast<size_t>(b) * H0 * W0 + static_cast<size_t>(valid ? y : 2 * Py) * W0 +
                           (valid ? x : 2 * Px);
        const float g = valid ? S::load1(a.dout, tok * C + c) : 0.f;
        const float* wrow = a.w ? a.w + (tok * a.heads + h) * L : nullptr;
#pragma unroll
        for (int l = 1; l < QTA_MAX_LEVELS; ++l) {
            if (l >= L) break;
            const float wl = (a.variant_b && wrow) ? wrow[l] : wdef;
            acc[l] += wl * g;
            if (want_dw) {
                const float dot = head_sum(g * manc[l], a.d);
                if (active && valid && (c % a.d) == 0) a.dw[(tok * a.heads + h) * L + l] = dot;
            }
        }
    }
    if (!active) return;
    a.dm[1][(static_cast<size_t>(b) * H1 * W1 + P) * C + c] = acc[1];
#pragma unroll
    for (int l = 2; l < QTA_MAX_LEVELS; ++l) {
        if (l >= L) break;
        const size_t anc = static_cast<size_t>(b) * a.H[l] * a.W[l] + static_cast<size_t>(Py >> (l - 1)) * a.W[l] +
                           (Px >> (l - 1));
        atomicAddNoRet(a.dm[l] + anc * C + c, acc[l]);
    }
}

// ---------------------------------------------------------------------------------------------
// 2. finer levels
// ---------------------------------------------------------------------------------------------

// Byte layout of one wave's LDS region for nsp padded slots: the gathered key rows in fp32 (B
// operand of dq), per slot the four queries' logit gradients and value weights, per channel the
// four queries' q and dm, and the slots' flat key indices.
struct BwdLds {
    int ks, dx, vw, q, dm, flat, total;
    int kpitch;     // floats per key row
};

template <int D>
__host__ __device__ inline BwdLds bwd_lds(int nsp)
{
    BwdLds L;
    L.kpitch = D + 4;
    L.ks = 0;
    L.dx = L.ks + nsp * L.kpitch * 4;
    L.vw = L.dx + nsp * 16;
    L.q = L.vw + nsp * 16;
    L.dm = L.q + D * 16;
    L.flat = L.dm + D * 16;
    L.total = (L.flat + nsp * 4 + 15) / 16 * 16;
    return L;
}

__device__ __forceinline__ float pick4(const float4_t& v, int i)
{
    return i == 0 ? v[0] : i == 1 ? v[1] : i == 2 ? v[2] : v[3];
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
    const int h = item % a.heads;
    const int bp = item / a.heads;
    const int P = bp % Np;
    const int b = bp / Np;
    const int Py = P / a.Wp, Px = P - Py * a.Wp;
    const int H = a.H, W = a.W, C = a.C, K = a.Kp;
    const int N = H * W;
    const int nslot = 4 * K;
    const int nsp = (nslot + 15) & ~15;
    const BwdLds lay = bwd_lds<D>(nsp);
    float* Ks = reinterpret_cast<float*>(base + lay.ks);
    float* dxs = reinterpret_cast<float*>(base + lay.dx);      // [slot][4]
    float* vws = reinterpret_cast<float*>(base + lay.vw);      // [slot][4]
    float* q4 = reinterpret_cast<float*>(base + lay.q);        // [channel][4]
    float* dm4 = reinterpret_cast<float*>(base + lay.dm);      // [channel][4]
    int* flat_l = reinterpret_cast<int*>(base + lay.flat);

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
    int J_own = -1;
#pragma unroll
    for (int t = 0; t < NT; ++t) J_own = g == t ? J_g[t] : J_own;
    const int flat = child_of_slot_J(lane < nslot ? J_own : -1, lane);
    const bool ok = flat >= 0;
    float pkey = 0.f;
    if constexpr (VA) pkey = a.parent_key[prow_off * K + min(lane >> 2, last_sel)];

    // queries: A operand row n16 holds query n16 & 3
    const int qi = n16 & 3;
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
    // level 0: w_{r,0} of the four queries (QuadTree-B; 1/L without w; 1 for A)
    float w0[4] = {1.f, 1.f, 1.f, 1.f};
    bool qv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int ry = 2 * Py + (r >> 1), rx = 2 * Px + (r & 1);
        qv[r] = ry < H && rx < W;
        if constexpr (FINEST && !VA) {
            const uint32_t rt = static_cast<uint32_t>(__mul24(min(ry, H - 1), W) + min(rx, W - 1));
            w0[r] = a.w ? a.w[((static_cast<size_t>(b) * N + rt) * a.heads + h) * a.levels] : 1.0f / a.levels;
        }
    }
    // q and dm of the four queries per channel, fp32, for dk and dv (lanes n16 < 4 hold query n16)
    if (n16 < 4) {
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            float qf[E];
            S::unpack(qa[j], qf);
            float gf[E];
            if constexpr (FINEST) {
                S::unpack(da[j], gf);
#pragma unroll
                for (int e = 0; e < E; ++e) gf[e] *= pick4(float4_t{w0[0], w0[1], w0[2], w0[3]}, n16);
            } else {
#pragma unroll
                for (int e = 0; e < E; ++e) gf[e] = dmA[j][e];
            }
            const int c0 = (g + 4 * j) * E;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                q4[(c0 + e) * 4 + n16] = qf[e];
                dm4[(c0 + e) * 4 + n16] = gf[e];
            }
        }
    }

    // ---- gathers, logits and <dm, v> on MFMA, key rows to LDS, one tile of 16 slots at a time ----
    const bool kvb = a.blocked;
    const size_t kv_base = kvb ? (static_cast<size_t>(b) * a.heads + h) * Np * 4 * RB
                               : (static_cast<size_t>(b) * N * C + h * D) * TB;
    const unsigned char* kg = static_cast<const unsigned char*>(a.k) + kv_base;
    const unsigned char* vg = static_cast<const unsigned char*>(a.v) + kv_base;
    const uint32_t tok_bytes = static_cast<uint32_t>(C * TB);
    float acc_x[4] = {0.f, 0.f, 0.f, 0.f}, acc_g[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        if (t >= ntile) break;                                // uniform
        const int s = 16 * t + n16;
        const int f = child_of_slot_J(J_g[t], s);
        const bool gok = f >= 0;
        const uint32_t goff = (!gok ? 0u : (kvb ? static_cast<uint32_t>(J_g[t] * 4 + (s & 3)) * RB
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
            const uint4 kk = gok ? kc[j] : make_uint4(0, 0, 0, 0);
            const uint4 vv = gok ? vc[j] : make_uint4(0, 0, 0, 0);
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
            // the key row in fp32 (zeros for missing candidates)
            float kf[E];
            S::unpack(kk, kf);
            float* krow = Ks + s * lay.kpitch + (g + 4 * j) * E;
#pragma unroll
            for (int e4 = 0; e4 < E; e4 += 4)
                *reinterpret_cast<float4*>(krow + e4) = make_float4(kf[e4], kf[e4 + 1], kf[e4 + 2], kf[e4 + 3]);
        }
        // rows 4g + r of the products are query r for every g: lane 16g + n keeps tile g
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            acc_x[r] = g == t ? ax[r] : acc_x[r];
            acc_g[r] = g == t ? ag[r] : acc_g[r];
        }
    }
    if (lane < nsp) flat_l[lane] = flat;

    // ---- softmax gradients of slot `lane` for the four queries ----
    float x[4], gsl[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        x[r] = ok ? acc_x[r] * a.scale : -INFINITY;
        gsl[r] = FINEST ? w0[r] * acc_g[r] : acc_g[r];      // dLoss/d(weight) on Omega
    }
    float dxr[4], vwr[4];
    if constexpr (!VA) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float m = wave_max_fast(x[r]);
            const float e = ok ? __expf(x[r] - m) : 0.f;
            const float p = e / wave_sum_fast(e);
            const float Dr = wave_sum_fast(p * gsl[r]);
            dxr[r] = qv[r] ? p * (gsl[r] - Dr) : 0.f;
            vwr[r] = qv[r] ? p : 0.f;
            if constexpr (FINEST) {
                if (a.w && a.dw) {                            // uniform
                    const float dw0 = wave_sum_fast(p * acc_g[r]);
                    if (lane == 0 && qv[r]) {
                        const int ry = 2 * Py + (r >> 1), rx = 2 * Px + (r & 1);
                        a.dw[((static_cast<size_t>(b) * N + ry * W + rx) * a.heads + h) * a.levels] = dw0;
                    }
                }
            }
        }
    } else {
        float dsig_acc = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float m = fmaxf(x[r], xchg_f32<1>(x[r]));
            m = fmaxf(m, xchg_f32<2>(m));
            const float e = ok ? __expf(x[r] - m) : 0.f;
            float sum = e + xchg_f32<1>(e);
            sum += xchg_f32<2>(sum);
            const float tt = ok ? e / sum : 0.f;
            const float sc = pkey * tt;
            float ds = gsl[r];
            bool kept = false;
            if constexpr (!FINEST) {
                // a key this query keeps is refined at level l-1: its score's gradient comes from there
                const int ry = 2 * Py + (r >> 1), rx = 2 * Px + (r & 1);
                const size_t srow = ((static_cast<size_t>(b) * a.heads + h) * N + __mul24(min(ry, H - 1), W) +
                                     min(rx, W - 1)) * a.Ks;
                for (int mm = 0; mm < a.Ks; ++mm) {
                    const int32_t j = a.sel_idx[srow + mm];
                    if (ok && j == flat) {
                        kept = true;
                        ds = a.dsig_in[srow + mm];
                    }
                }
            }
            float dsq = tt * ds;                              // this query's d sigma of the kept key
            dsq += xchg_f32<1>(dsq);
            dsq += xchg_f32<2>(dsq);
            dxr[r] = qv[r] ? sc * (ds - dsq) : 0.f;
            vwr[r] = (qv[r] && !kept) ? sc : 0.f;
            dsig_acc += qv[r] ? dsq : 0.f;
        }
        if ((lane & 3) == 0 && (lane >> 2) < K) a.dsig_out[prow_off * K + (lane >> 2)] = dsig_acc;
    }
    if (lane < nsp) {
        *reinterpret_cast<float4*>(dxs + lane * 4) = make_float4(dxr[0], dxr[1], dxr[2], dxr[3]);
        *reinterpret_cast<float4*>(vws + lane * 4) = make_float4(vwr[0], vwr[1], vwr[2], vwr[3]);
    }
    wave_lds_sync();

    // ---- dq = scale * sum_s dx_s k_s on the 4x4 MFMA (blocks over 4-channel groups, slot halves) ----
    {
        const int blk = lane >> 2, t4 = lane & 3;
        const int cg = blk / NH, hh = blk % NH;
        const int ch = 4 * cg + t4;
        const int sph = nsp / NH;
        float4_t o = {0.f, 0.f, 0.f, 0.f};
        const float* kcol = Ks + 4 * cg + t4;
        for (int st = 0; st < sph; ++st) {
            const int sl = hh * sph + st;
            o = __builtin_amdgcn_mfma_f32_4x4x1f32(dxs[sl * 4 + t4], kcol[sl * lay.kpitch], o, 0, 0, 0);
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
            a.dq[(static_cast<size_t>(b) * N + __mul24(ry, W) + rx) * C + h * D + ch] = a.scale * pick4(o, r);
        }
    }

    // ---- dk and dv of the gathered keys: lanes over (slot, channel), coalesced atomics ----
    for (int idx = lane; idx < nslot * D; idx += kWave) {
        const int s = idx / D, c = idx - s * D;
        const int f = flat_l[s];
        if (f < 0) continue;
        const float4 dx4 = *reinterpret_cast<const float4*>(dxs + s * 4);
        const float4 vw4 = *reinterpret_cast<const float4*>(vws + s * 4);
        const float4 qc = *reinterpret_cast<const float4*>(q4 + c * 4);
        const float4 gc = *reinterpret_cast<const float4*>(dm4 + c * 4);
        const float dkv = a.scale * (dx4.x * qc.x + dx4.y * qc.y + dx4.z * qc.z + dx4.w * qc.w);
        const float dvv = vw4.x * gc.x + vw4.y * gc.y + vw4.z * gc.z + vw4.w * gc.w;
        const size_t row = (static_cast<size_t>(b) * N + f) * C + h * D + c;
        atomicAddNoRet(a.dk + row, dkv);
        atomicAddNoRet(a.dv + row, dvv);
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
    bwd_item<T, D, NSP, VA, FINEST>(a, item, smem + static_cast<size_t>(wave) * bwd_lds<D>(nsp).total);
}

template <typename T, int D, int NSP, bool VA, bool FINEST>
hipError_t launch_level_one(const BwdLevelArgs& a, hipStream_t stream)
{
    const int nsp = (4 * a.Kp + 15) & ~15;
    const size_t wave_bytes = bwd_lds<D>(nsp).total;
    int wpb = 4;
    while (wpb > 1 && wpb * wave_bytes > 64 * 1024) --wpb;
    if (wpb * wave_bytes > device_max_lds()) return hipErrorInvalidValue;
    static bool configured = false;
    if (!configured) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&bwd_level_kernel<T, D, NSP, VA, FINEST>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           static_cast<int>(device_max_lds()));
        if (e != hipSuccess) return e;
        configured = true;
    }
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

// ---------------------------------------------------------------------------------------------
// 3. coarsest level
// ---------------------------------------------------------------------------------------------

constexpr int kCoarseChunks = QTA_MAX_COARSE / kWave;   // keys (or queries) per lane, at most

// <x, row> over one head's D channels: x fp32 in LDS (broadcast reads), row in the storage type
// (or fp32) in HBM, streamed 16 bytes at a time.
template <typename T, int D>
__device__ __forceinline__ float dot_row(const float* x, const void* base, size_t elem)
{
    using S = Storage<T>;
    constexpr int E = S::kPer16B;
    const uint4* p = reinterpret_cast<const uint4*>(static_cast<const unsigned char*>(base) + elem * sizeof(T));
    float acc = 0.f;
#pragma unroll
    for (int cc = 0; cc < D / E; ++cc) {
        float f[E];
        S::unpack(p[cc], f);
#pragma unroll
        for (int e = 0; e < E; ++e) acc += x[cc * E + e] * f[e];
    }
    return acc;
}

// acc[c] += s * row[c] over one head's D channels.
template <typename T, int D>
__device__ __forceinline__ void axpy_row(float s, const void* base, size_t elem, float* acc)
{
    using S = Storage<T>;
    constexpr int E = S::kPer16B;
    const uint4* p = reinterpret_cast<const uint4*>(static_cast<const unsigned char*>(base) + elem * sizeof(T));
#pragma unroll
    for (int cc = 0; cc < D / E; ++cc) {
        float f[E];
        S::unpack(p[cc], f);
#pragma unroll
        for (int e = 0; e < E; ++e) acc[cc * E + e] += s * f[e];
    }
}

// Sum over the wave of each acc[c]; lane c < D receives the total of channel c.
template <int D>
__device__ __forceinline__ float wave_sum_to_lane(const float* acc)
{
    const int lane = threadIdx.x & 63;
    float mine = 0.f;
#pragma unroll
    for (int c = 0; c < D; ++c) {
        const float s = wave_sum_fast(acc[c]);
        if (lane == c) mine = s;
    }
    return mine;
}

// The gradient of coarse message row `tok` at channel c: dm^c when there are finer levels,
// otherwise w_0 dout (QuadTree-B) or dout (A).
template <typename T>
__device__ __forceinline__ float dm_elem(const BwdCoarseArgs& a, size_t tok, int h, int D, int c)
{
    if (a.dm) return a.dm[tok * a.C + h * D + c];
    const float w0 = (a.variant_b && a.w) ? a.w[tok * a.heads + h] : 1.0f;
    return w0 * Storage<T>::load1(a.dout, tok * a.C + h * D + c);
}

// Per query (one wave per (b, h, i), lanes over keys): softmax statistics, dq and, for a single
// QuadTree-B level with w, dw. The query's q, dm (and dout) rows sit in the wave's LDS.
template <typename T, int D, bool VA>
__global__ __launch_bounds__(256) void bwd_coarse_query_kernel(BwdCoarseArgs a)
{
    const int lane = threadIdx.x & 63;
    const long long nitems = static_cast<long long>(a.B) * a.heads * a.N;
    const long long item = static_cast<long long>(blockIdx.x) * (blockDim.x >> 6) + (threadIdx.x >> 6);
    if (item >= nitems) return;                              // whole wave
    __shared__ __align__(16) float rows[4][3][D];
    float* qs = rows[threadIdx.x >> 6][0];
    float* gs_row = rows[threadIdx.x >> 6][1];
    float* go = rows[threadIdx.x >> 6][2];
    const int N = a.N;
    const int i = static_cast<int>(item % N);
    const int bh = static_cast<int>(item / N);
    const int h = bh % a.heads, b = bh / a.heads;
    const size_t qtok = static_cast<size_t>(b) * N + i;
    const bool want_dw = !a.dm && a.variant_b && a.w && a.dw;
    if (lane < D) {
        qs[lane] = Storage<T>::load1(a.q, qtok * a.C + h * D + lane);
        gs_row[lane] = dm_elem<T>(a, qtok, h, D, lane);
        go[lane] = want_dw ? Storage<T>::load1(a.dout, qtok * a.C + h * D + lane) : 0.f;
    }
    wave_lds_sync();
    float x[kCoarseChunks], gg[kCoarseChunks], g0[kCoarseChunks];
    float mx = -INFINITY;
#pragma unroll
    for (int ch = 0; ch < kCoarseChunks; ++ch) {
        x[ch] = -INFINITY;
        gg[ch] = 0.f;
        g0[ch] = 0.f;
        if (ch * kWave >= N) continue;                        // uniform
        const int j = ch * kWave + lane;
        const size_t krow = (static_cast<size_t>(b) * N + min(j, N - 1)) * a.C + h * D;
        const float xs = dot_row<T, D>(qs, a.k, krow);
        gg[ch] = dot_row<T, D>(gs_row, a.v, krow);
        if (want_dw) g0[ch] = dot_row<T, D>(go, a.v, krow);
        x[ch] = j < N ? xs * a.scale : -INFINITY;
        mx = fmaxf(mx, x[ch]);
    }
    mx = wave_max_fast(mx);
    float sum = 0.f;
#pragma unroll
    for (int ch = 0; ch < kCoarseChunks; ++ch) {
        x[ch] = __expf(x[ch] - mx);                           // 0 for missing keys
        sum += x[ch];
    }
    sum = wave_sum_fast(sum);
    const float inv = 1.0f / sum;
    // QuadTree-A's kept keys: their score's gradient comes from the level below
    if (VA && a.K > 0) {
        const size_t srow = (static_cast<size_t>(bh) * N + i) * a.K;
        for (int mm = 0; mm < a.K; ++mm) {
            const int32_t j = a.sel_idx[srow + mm];
            if (j < 0) continue;
            const float dsv = a.dsig[srow + mm];
#pragma unroll
            for (int ch = 0; ch < kCoarseChunks; ++ch)
                if (j == ch * kWave + lane) gg[ch] = dsv;
        }
    }
    float Dsum = 0.f, dwsum = 0.f;
#pragma unroll
    for (int ch = 0; ch < kCoarseChunks; ++ch) {
        x[ch] *= inv;                                         // p
        Dsum += x[ch] * gg[ch];
        dwsum += x[ch] * g0[ch];
    }
    Dsum = wave_sum_fast(Dsum);
    float dq[D];
#pragma unroll
    for (int c = 0; c < D; ++c) dq[c] = 0.f;
#pragma unroll
    for (int ch = 0; ch < kCoarseChunks; ++ch) {
        if (ch * kWave >= N) continue;                        // uniform
        const int j = ch * kWave + lane;
        const float dx = x[ch] * (gg[ch] - Dsum);             // 0 for missing keys (p = 0)
        axpy_row<T, D>(dx, a.k, (static_cast<size_t>(b) * N + min(j, N - 1)) * a.C + h * D, dq);
    }
    const float mine = wave_sum_to_lane<D>(dq);
    if (lane < D) a.dq[qtok * a.C + h * D + lane] = a.scale * mine;
    if (lane == 0)
        *reinterpret_cast<float4*>(a.stats + (static_cast<size_t>(bh) * N + i) * 4) = make_float4(mx, sum, Dsum, 0.f);
    if (want_dw) {
        dwsum = wave_sum_fast(dwsum);
        if (lane == 0) a.dw[qtok * a.heads + h] = dwsum;
    }
}

// Per key (one wave per (b, h, j), lanes over queries): dk and dv from the recomputed probabilities.
template <typename T, int D, bool VA>
__global__ __launch_bounds__(256) void bwd_coarse_key_kernel(BwdCoarseArgs a)
{
    const int lane = threadIdx.x & 63;
    const long long nitems = static_cast<long long>(a.B) * a.heads * a.N;
    const long long item = static_cast<long long>(blockIdx.x) * (blockDim.x >> 6) + (threadIdx.x >> 6);
    if (item >= nitems) return;                              // whole wave
    __shared__ __align__(16) float rows[4][2][D];
    float* ks = rows[threadIdx.x >> 6][0];
    float* vs = rows[threadIdx.x >> 6][1];
    const int N = a.N;
    const int j = static_cast<int>(item % N);
    const int bh = static_cast<int>(item / N);
    const int h = bh % a.heads, b = bh / a.heads;
    const size_t ktok = static_cast<size_t>(b) * N + j;
    if (lane < D) {
        ks[lane] = Storage<T>::load1(a.k, ktok * a.C + h * D + lane);
        vs[lane] = Storage<T>::load1(a.v, ktok * a.C + h * D + lane);
    }
    wave_lds_sync();
    float dk[D], dv[D];
#pragma unroll
    for (int c = 0; c < D; ++c) {
        dk[c] = 0.f;
        dv[c] = 0.f;
    }
    for (int ch = 0; ch < kCoarseChunks; ++ch) {
        if (ch * kWave >= N) break;                           // uniform
        const int i = ch * kWave + lane;
        const int ic = min(i, N - 1);
        const size_t qtok = static_cast<size_t>(b) * N + ic;
        const size_t qrow = qtok * a.C + h * D;
        const float4 st = *reinterpret_cast<const float4*>(a.stats + (static_cast<size_t>(bh) * N + ic) * 4);
        const float xs = dot_row<T, D>(ks, a.q, qrow);
        // <dm_i, v_j>: dm^c rows are fp32; for a single level, w_0 dout in the storage type
        float w0 = 1.0f, gsv;
        if (a.dm) {
            gsv = dot_row<float, D>(vs, a.dm, qrow);
        } else {
            if (a.variant_b && a.w) w0 = a.w[qtok * a.heads + h];
            gsv = w0 * dot_row<T, D>(vs, a.dout, qrow);
        }
        const float p = i < N ? __expf(xs * a.scale - st.x) / st.y : 0.f;
        float ds = gsv;
        bool kept = false;
        if (VA && a.K > 0) {
            const size_t srow = (static_cast<size_t>(bh) * N + ic) * a.K;
            for (int mm = 0; mm < a.K; ++mm)
                if (a.sel_idx[srow + mm] == j) {
                    kept = true;
                    ds = a.dsig[srow + mm];
                }
        }
        const float dx = p * (ds - st.z);
        const float vw = kept ? 0.f : p;
        axpy_row<T, D>(dx, a.q, qrow, dk);
        if (a.dm)
            axpy_row<float, D>(vw, a.dm, qrow, dv);
        else
            axpy_row<T, D>(vw * w0, a.dout, qrow, dv);
    }
    const float mk = wave_sum_to_lane<D>(dk);
    const float mv = wave_sum_to_lane<D>(dv);
    if (lane < D) {
        a.dk[ktok * a.C + h * D + lane] = a.scale * mk;
        a.dv[ktok * a.C + h * D + lane] = mv;
    }
}

template <typename T, int D, bool VA>
hipError_t launch_coarse_tdv(const BwdCoarseArgs& a, hipStream_t stream)
{
    const long long items = static_cast<long long>(a.B) * a.heads * a.N;
    const int wpb = 4;
    const long long blocks = (items + wpb - 1) / wpb;
    if (blocks >= 0x7FFFFFFFLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((bwd_coarse_query_kernel<T, D, VA>), dim3(static_cast<unsigned>(blocks)), dim3(wpb * kWave), 0,
                       stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((bwd_coarse_key_kernel<T, D, VA>), dim3(static_cast<unsigned>(blocks)), dim3(wpb * kWave), 0,
                       stream, a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------------------------
// 4. pyramids
// ---------------------------------------------------------------------------------------------

__global__ __launch_bounds__(256) void bwd_unpool_kernel(BwdUnpoolArgs a)
{
    const int cpt = a.C / 4;
    const long long N0 = static_cast<long long>(a.H[0]) * a.W[0];
    const long long total = a.B * N0 * cpt;
    const long long tid = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (tid >= total) return;
    const int ch = static_cast<int>(tid % cpt);
    const long long tok = tid / cpt;
    const int i = static_cast<int>(tok % N0);
    const int b = static_cast<int>(tok / N0);
    const int y = i / a.W[0], x = i - y * a.W[0];
    float4 aq = make_float4(0.f, 0.f, 0.f, 0.f), ak = aq, av = aq;
    float f = 1.0f;
    for (int l = 1; l < a.L; ++l) {
        const int yl = y >> l, xl = x >> l;
        const int ny = (2 * yl + 1 < a.H[l - 1]) ? 2 : 1, nx = (2 * xl + 1 < a.W[l - 1]) ? 2 : 1;
        f *= 1.0f / static_cast<float>(ny * nx);
        const size_t off = ((static_cast<size_t>(b) * a.H[l] + yl) * a.W[l] + xl) * a.C + 4 * ch;
        const float4 gq = *reinterpret_cast<const float4*>(a.gq[l] + off);
        const float4 gk = *reinterpret_cast<const float4*>(a.gk[l] + off);
        const float4 gv = *reinterpret_cast<const float4*>(a.gv[l] + off);
        aq.x += f * gq.x; aq.y += f * gq.y; aq.z += f * gq.z; aq.w += f * gq.w;
        ak.x += f * gk.x; ak.y += f * gk.y; ak.z += f * gk.z; ak.w += f * gk.w;
        av.x += f * gv.x; av.y += f * gv.y; av.z += f * gv.z; av.w += f * gv.w;
    }
    const size_t o = static_cast<size_t>(tok) * a.C + 4 * ch;
    float4* pq = reinterpret_cast<float4*>(a.dq + o);
    float4* pk = reinterpret_cast<float4*>(a.dk + o);
    float4* pv = reinterpret_cast<float4*>(a.dv + o);
    float4 q = *pq, k = *pk, v = *pv;
    q.x += aq.x; q.y += aq.y; q.z += aq.z; q.w += aq.w;
    k.x += ak.x; k.y += ak.y; k.z += ak.z; k.w += ak.w;
    v.x += av.x; v.y += av.y; v.z += av.z; v.w += av.w;
    *pq = q;
    *pk = k;
    *pv = v;
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

hipError_t launch_bwd_combine(const BwdCombineArgs& a, bool use_bf16, hipStream_t stream)
{
    const long long total = static_cast<long long>(a.B) * a.H[1] * a.W[1] * a.C;
    const long long blocks = (total + 255) / 256;
    if (blocks >= 0x7FFFFFFFLL) return hipErrorInvalidValue;
    if (use_bf16)
        hipLaunchKernelGGL(bwd_combine_kernel<bf16>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(bwd_combine_kernel<float>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_bwd_level(const BwdLevelArgs& a, int d, bool variant_a, bool use_bf16, bool finest,
                            hipStream_t stream)
{
    if (4 * a.Kp > 64) return hipErrorInvalidValue;
    BwdLevelArgs b = a;
    b.div_Wp = make_fastdiv(a.Wp);
    if (use_bf16) {
        if (d == 32) return launch_level_td<bf16, 32>(b, variant_a, finest, stream);
        if (d == 64) return launch_level_td<bf16, 64>(b, variant_a, finest, stream);
    } else {
        if (d == 32) return launch_level_td<float, 32>(b, variant_a, finest, stream);
        if (d == 64) return launch_level_td<float, 64>(b, variant_a, finest, stream);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_bwd_coarse(const BwdCoarseArgs& a, int d, bool variant_a, bool use_bf16, hipStream_t stream)
{
    if (a.N > QTA_MAX_COARSE) return hipErrorInvalidValue;
    if (use_bf16) {
        if (d == 32) return variant_a ? launch_coarse_tdv<bf16, 32, true>(a, stream) : launch_coarse_tdv<bf16, 32, false>(a, stream);
        if (d == 64) return variant_a ? launch_coarse_tdv<bf16, 64, true>(a, stream) : launch_coarse_tdv<bf16, 64, false>(a, stream);
    } else {
        if (d == 32) return variant_a ? launch_coarse_tdv<float, 32, true>(a, stream) : launch_coarse_tdv<float, 32, false>(a, stream);
        if (d == 64) return variant_a ? launch_coarse_tdv<float, 64, true>(a, stream) : launch_coarse_tdv<float, 64, false>(a, stream);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_bwd_unpool(const BwdUnpoolArgs& a, hipStream_t stream)
{
    const long long total = static_cast<long long>(a.B) * a.H[0] * a.W[0] * (a.C / 4);
    const long long blocks = (total + 255) / 256;
    if (blocks >= 0x7FFFFFFFLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL(bwd_unpool_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace qta
