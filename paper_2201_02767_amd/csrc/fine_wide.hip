// Steps 3-5 at the finer levels for large K (4K > 64 candidates per sibling group): gathered
// attention over the children of the parent's kept keys (Sec. 3.2, Fig. 1), QuadTree-A scores
// (Eq. 4) or QuadTree-B softmax (Eq. 6), the next level's top-K, and at level 0 the combination of
// all levels' messages (Eqs. 2 and 5). The common case K <= 16 runs the MFMA kernel of fine.hip.
//
// Work item = one parent query P at level l+1 and one head. Its four children at level l are
// sibling queries with the same candidate set: the 2x2 children of the K keys P kept. One wave
// owns one item:
//   1. slot 4r+c names child c ((0,0),(0,1),(1,0),(1,1)) of kept key r; lane = slot;
//   2. the candidates' key and value rows of this head (d elements each) are gathered once with
//      16-byte loads, several lanes per row, into wave-private LDS, together with the four
//      queries (scaled by the temperature);
//   3. each lane computes its candidate's logits against the four queries;
//   4. B: a wave-wide softmax per query; A: a softmax over each quad of lanes (the children of
//      one kept key) times the parent's score;
//   5. levels above 0: a wave-wide bitonic sort per query of (score, flat index) words yields
//      this level's kept keys; A drops their weight from the message (refined one level down);
//   6. the message m = sum w v: lane = (query, d/16 channels), reading weights and values from LDS;
//   7. levels above 0 store m; level 0 adds the ancestors' messages (times w for B) and stores
//      the output in the storage type.
// A workgroup holds up to four independent waves; nothing synchronises across waves.
#include "qta_device.h"
#include "qta_internal.h"

namespace qta {

namespace {

__host__ __device__ inline size_t fine_wave_bytes(int nslot, int d, int tbytes)
{
    const size_t rb = static_cast<size_t>(d) * tbytes;
    return static_cast<size_t>(nslot) * (rb + 16) + static_cast<size_t>(nslot) * rb + 4 * d * sizeof(float) +
           4 * static_cast<size_t>(nslot) * sizeof(float);
}

template <typename T, int CPL>
__device__ __forceinline__ void load_vals(const unsigned char* p, float (&o)[CPL])
{
    if constexpr (sizeof(T) == 4) {
        if constexpr (CPL == 2) {
            const float2 v = *reinterpret_cast<const float2*>(p);
            o[0] = v.x;
            o[1] = v.y;
        } else {
            const float4 v = *reinterpret_cast<const float4*>(p);
            o[0] = v.x;
            o[1] = v.y;
            o[2] = v.z;
            o[3] = v.w;
        }
    } else {
        if constexpr (CPL == 2) {
            const uint32_t v = *reinterpret_cast<const uint32_t*>(p);
            o[0] = __uint_as_float(v << 16);
            o[1] = __uint_as_float(v & 0xFFFF0000u);
        } else {
            const uint2 v = *reinterpret_cast<const uint2*>(p);
            o[0] = __uint_as_float(v.x << 16);
            o[1] = __uint_as_float(v.x & 0xFFFF0000u);
            o[2] = __uint_as_float(v.y << 16);
            o[3] = __uint_as_float(v.y & 0xFFFF0000u);
        }
    }
}

template <typename T, int CPL>
__device__ __forceinline__ void store_vals(void* base, size_t elem, const float (&o)[CPL])
{
    if constexpr (sizeof(T) == 4) {
        float* p = static_cast<float*>(base) + elem;
        if constexpr (CPL == 2) *reinterpret_cast<float2*>(p) = make_float2(o[0], o[1]);
        else *reinterpret_cast<float4*>(p) = make_float4(o[0], o[1], o[2], o[3]);
    } else {
        uint16_t* p = static_cast<uint16_t*>(base) + elem;
        if constexpr (CPL == 2) {
            *reinterpret_cast<uint32_t*>(p) = f32_to_bf16_bits(o[0]) | (f32_to_bf16_bits(o[1]) << 16);
        } else {
            *reinterpret_cast<uint2*>(p) = make_uint2(f32_to_bf16_bits(o[0]) | (f32_to_bf16_bits(o[1]) << 16),
                                                      f32_to_bf16_bits(o[2]) | (f32_to_bf16_bits(o[3]) << 16));
        }
    }
}

template <typename T, int D, bool VA, bool FINEST, int NT>
__global__ __launch_bounds__(256) void fine_attn_kernel(FineArgs a)
{
    using S = Storage<T>;
    constexpr int TB = sizeof(T);
    constexpr int RB = D * TB;            // bytes of one head's row
    constexpr int KP = RB + 16;           // LDS pitch of key rows (padding spreads the banks)
    constexpr int E = S::kPer16B;
    constexpr int LPR = RB / 16;          // lanes per row when gathering
    constexpr int RPP = kWave / LPR;      // rows per gather instruction
    constexpr int CPL = D / 16;           // message channels per lane

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wpb = blockDim.x >> 6;
    const int Np = a.Hp * a.Wp;
    const long long nitems = static_cast<long long>(a.B) * a.heads * Np;
    const long long item = static_cast<long long>(xcd_remap(blockIdx.x, gridDim.x)) * wpb + wave;
    if (item >= nitems) return;           // whole wave leaves; only wave-level syncs follow

    const int h = static_cast<int>(item % a.heads);
    const long long bp = item / a.heads;
    const int P = static_cast<int>(bp % Np);
    const int b = static_cast<int>(bp / Np);
    const int Py = P / a.Wp, Px = P - Py * a.Wp;
    const int H = a.H, W = a.W, C = a.C, K = a.Kp, Ksel = a.Ks;
    const int N = H * W;
    const int nslot = 4 * K;

    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* Ks = smem + static_cast<size_t>(wave) * fine_wave_bytes(nslot, D, TB);
    unsigned char* Vs = Ks + static_cast<size_t>(nslot) * KP;
    float* Qs = reinterpret_cast<float*>(Vs + static_cast<size_t>(nslot) * RB);
    float* Ps = Qs + 4 * D;

    // ---- 1. candidate slots ----
    const size_t prow = ((static_cast<size_t>(b) * a.heads + h) * Np + P) * K;
    int flat[NT];
    float pkey[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int s = lane + kWave * t;
        flat[t] = -1;
        pkey[t] = 0.f;
        if (s < nslot) {
            const int r = s >> 2, c = s & 3;
            const int J = a.parent_idx[prow + r];
            if (J >= 0) {
                const int Jy = J / a.Wp, Jx = J - Jy * a.Wp;
                const int cy = 2 * Jy + (c >> 1), cx = 2 * Jx + (c & 1);
                if (cy < H && cx < W) flat[t] = cy * W + cx;
            }
            if constexpr (VA) pkey[t] = a.parent_key[prow + r];
        }
    }

    // ---- 2. gather key/value rows and the four queries into LDS ----
    {
        const unsigned char* kg = static_cast<const unsigned char*>(a.k) + (static_cast<size_t>(b) * N * C + h * D) * TB;
        const unsigned char* vg = static_cast<const unsigned char*>(a.v) + (static_cast<size_t>(b) * N * C + h * D) * TB;
        const int sub = lane / LPR, chunk = lane % LPR;
        const size_t tok_bytes = static_cast<size_t>(C) * TB;
        constexpr int kBatch = 4;
        for (int s0 = 0; s0 < nslot; s0 += RPP * kBatch) {
            uint4 kc[kBatch], vc[kBatch];
            int ss[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int s = s0 + u * RPP + sub;
                ss[u] = s;
                int f = -1;
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const int ft = __shfl(flat[t], s & 63, kWave);
                    if ((s >> 6) == t) f = ft;
                }
                kc[u] = make_uint4(0, 0, 0, 0);
                vc[u] = make_uint4(0, 0, 0, 0);
                if (s < nslot && f >= 0) {
                    kc[u] = *reinterpret_cast<const uint4*>(kg + f * tok_bytes + chunk * 16);
                    vc[u] = *reinterpret_cast<const uint4*>(vg + f * tok_bytes + chunk * 16);
                }
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                if (ss[u] < nslot) {
                    *reinterpret_cast<uint4*>(Ks + static_cast<size_t>(ss[u]) * KP + chunk * 16) = kc[u];
                    *reinterpret_cast<uint4*>(Vs + static_cast<size_t>(ss[u]) * RB + chunk * 16) = vc[u];
                }
            }
        }
        for (int e = lane; e < 4 * D; e += kWave) {
            const int qi = e / D, c = e - qi * D;
            const int qy = 2 * Py + (qi >> 1), qx = 2 * Px + (qi & 1);
            float val = 0.f;
            if (qy < H && qx < W)
                val = S::load1(a.q, (static_cast<size_t>(b) * N + qy * W + qx) * C + h * D + c) * a.scale;
            Qs[e] = val;
        }
    }
    wave_lds_sync();

    // ---- 3. logits: lane = candidate slot ----
    bool ok[NT];
    float x[NT][4];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int s = lane + kWave * t;
        ok[t] = s < nslot && flat[t] >= 0;
        const int sr = s < nslot ? s : nslot - 1;
        float kf[D];
#pragma unroll
        for (int cc = 0; cc < RB / 16; ++cc) {
            const uint4 c = *reinterpret_cast<const uint4*>(Ks + static_cast<size_t>(sr) * KP + cc * 16);
            float tmp[E];
            S::unpack(c, tmp);
#pragma unroll
            for (int e = 0; e < E; ++e) kf[cc * E + e] = tmp[e];
        }
#pragma unroll
        for (int qi = 0; qi < 4; ++qi) {
            float acc = 0.f;
#pragma unroll
            for (int c = 0; c < D; c += 4) {
                const float4 q4 = *reinterpret_cast<const float4*>(Qs + qi * D + c);
                acc += q4.x * kf[c] + q4.y * kf[c + 1] + q4.z * kf[c + 2] + q4.w * kf[c + 3];
            }
            x[t][qi] = ok[t] ? acc : -INFINITY;
        }
    }

    // ---- 4. weights ----
    float wgt[NT][4];
    float mx[4], inv_sum[4];
    if constexpr (!VA) {
#pragma unroll
        for (int qi = 0; qi < 4; ++qi) {
            float m = -INFINITY;
#pragma unroll
            for (int t = 0; t < NT; ++t) m = fmaxf(m, x[t][qi]);
            m = wave_max(m);
            float sum = 0.f;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                wgt[t][qi] = ok[t] ? __expf(x[t][qi] - m) : 0.f;
                sum += wgt[t][qi];
            }
            sum = wave_sum(sum);
            mx[qi] = m;
            inv_sum[qi] = 1.0f / sum;
        }
    } else {
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int qi = 0; qi < 4; ++qi) {
                float m = x[t][qi];
                m = fmaxf(m, __shfl_xor(m, 1, kWave));
                m = fmaxf(m, __shfl_xor(m, 2, kWave));
                const float e = ok[t] ? __expf(x[t][qi] - m) : 0.f;
                float s = e;
                s += __shfl_xor(s, 1, kWave);
                s += __shfl_xor(s, 2, kWave);
                wgt[t][qi] = ok[t] ? pkey[t] * (e / s) : 0.f;
            }
#pragma unroll
        for (int qi = 0; qi < 4; ++qi) {
            mx[qi] = 0.f;
            inv_sum[qi] = 1.f;
        }
    }

    // ---- 5. this level's selection (levels above the finest) ----
    if constexpr (!FINEST) {
        int nvalid = 0;
#pragma unroll
        for (int t = 0; t < NT; ++t) nvalid += __popcll(__ballot(ok[t]));
        const int keff = Ksel < nvalid ? Ksel : nvalid;
#pragma unroll
        for (int qi = 0; qi < 4; ++qi) {
            const int qy = 2 * Py + (qi >> 1), qx = 2 * Px + (qi & 1);
            if (qy >= H || qx >= W) continue;                  // uniform across the wave
            uint64_t word[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) word[t] = ok[t] ? rank_word(VA ? wgt[t][qi] : x[t][qi], flat[t]) : 0ull;
            wave_bitonic_sort_desc<NT>(word);
            const size_t orow = ((static_cast<size_t>(b) * a.heads + h) * N + qy * W + qx) * Ksel;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int r = kWave * t + lane;
                if (r < Ksel) {
                    const uint64_t wd = word[t];
                    int32_t idx = -1;
                    float key = 0.f;
                    if (wd != 0ull) {
                        idx = rank_word_index(wd);
                        const float sc = rank_word_score(wd);
                        key = VA ? sc : __expf(sc - mx[qi]) * inv_sum[qi];
                    }
                    a.sel_idx[orow + r] = idx;
                    a.sel_key[orow + r] = key;
                }
            }
            if constexpr (VA) {
                // the kept keys are exactly the candidates whose word is >= the keff-th largest
                if (keff > 0) {
                    const int last = keff - 1;
                    uint64_t thr = 0ull;
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        const uint32_t lo = __shfl(static_cast<uint32_t>(word[t]), last & 63, kWave);
                        const uint32_t hi = __shfl(static_cast<uint32_t>(word[t] >> 32), last & 63, kWave);
                        if ((last >> 6) == t) thr = (static_cast<uint64_t>(hi) << 32) | lo;
                    }
#pragma unroll
                    for (int t = 0; t < NT; ++t)
                        if (ok[t] && rank_word(wgt[t][qi], flat[t]) >= thr) wgt[t][qi] = 0.f;
                }
            }
        }
    }

    // ---- 6. message m = sum_slot w * v ----
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int s = lane + kWave * t;
        if (s < nslot)
#pragma unroll
            for (int qi = 0; qi < 4; ++qi) Ps[qi * nslot + s] = wgt[t][qi];
    }
    wave_lds_sync();

    const int pq = lane >> 4, cg = lane & 15;
    float acc[CPL];
#pragma unroll
    for (int e = 0; e < CPL; ++e) acc[e] = 0.f;
    for (int s = 0; s < nslot; s += 4) {
        const float4 p4 = *reinterpret_cast<const float4*>(Ps + pq * nslot + s);
        const float pw[4] = {p4.x, p4.y, p4.z, p4.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            float vv[CPL];
            load_vals<T, CPL>(Vs + static_cast<size_t>(s + u) * RB + cg * CPL * TB, vv);
#pragma unroll
            for (int e = 0; e < CPL; ++e) acc[e] += pw[u] * vv[e];
        }
    }
    const float my_inv = pq == 0 ? inv_sum[0] : pq == 1 ? inv_sum[1] : pq == 2 ? inv_sum[2] : inv_sum[3];
#pragma unroll
    for (int e = 0; e < CPL; ++e) acc[e] *= my_inv;

    // ---- 7. outputs ----
    const int qy = 2 * Py + (pq >> 1), qx = 2 * Px + (pq & 1);
    if (qy >= H || qx >= W) return;
    const size_t qtok = static_cast<size_t>(b) * N + qy * W + qx;
    if constexpr (!FINEST) {
        float* m = a.msg + (qtok * a.heads + h) * D + cg * CPL;
        if constexpr (CPL == 2) *reinterpret_cast<float2*>(m) = make_float2(acc[0], acc[1]);
        else *reinterpret_cast<float4*>(m) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    } else {
        const int L = a.levels;
        const float* wrow = a.w ? a.w + (qtok * a.heads + h) * L : nullptr;
        const float wdef = 1.0f / L;
        float o[CPL];
        const float w0 = VA ? 1.0f : (wrow ? wrow[0] : wdef);
        const float* pe = a.pe0 ? a.pe0 + (qtok * a.heads + h) * D + cg * CPL : nullptr;
#pragma unroll
        for (int e = 0; e < CPL; ++e) o[e] = w0 * (acc[e] + (pe ? pe[e] : 0.f));
        for (int lev = 1; lev < L; ++lev) {
            const size_t anc = static_cast<size_t>(b) * a.lvl_N[lev] + static_cast<size_t>(qy >> lev) * a.lvl_W[lev] +
                               (qx >> lev);
            const float* m = a.coarser_msg[lev] + (anc * a.heads + h) * D + cg * CPL;
            const float wl = VA ? 1.0f : (wrow ? wrow[lev] : wdef);
            float mv[CPL];
            if constexpr (CPL == 2) {
                const float2 t2 = *reinterpret_cast<const float2*>(m);
                mv[0] = t2.x;
                mv[1] = t2.y;
            } else {
                const float4 t4 = *reinterpret_cast<const float4*>(m);
                mv[0] = t4.x;
                mv[1] = t4.y;
                mv[2] = t4.z;
                mv[3] = t4.w;
            }
#pragma unroll
            for (int e = 0; e < CPL; ++e) o[e] += wl * mv[e];
        }
        store_vals<T, CPL>(a.out, qtok * C + h * D + cg * CPL, o);
    }
}

template <typename T, int D, bool VA, bool FINEST, int NT>
hipError_t launch_one(const FineArgs& a, hipStream_t stream)
{
    const int nslot = 4 * a.Kp;
    const size_t wave_bytes = fine_wave_bytes(nslot, D, sizeof(T));
    const size_t kLdsMax = device_max_lds();
    int wpb = 4;
    while (wpb > 1 && wpb * wave_bytes > kLdsMax) --wpb;
    if (wave_bytes > kLdsMax) return hipErrorInvalidValue;
    static std::atomic<unsigned long long> configured{0};     // devices whose LDS limit is raised
    if (hipError_t e = set_max_lds_once(reinterpret_cast<const void*>(&fine_attn_kernel<T, D, VA, FINEST, NT>),
                                        configured);
        e != hipSuccess)
        return e;
    const long long items = static_cast<long long>(a.B) * a.heads * a.Hp * a.Wp;
    const long long blocks = (items + wpb - 1) / wpb;
    if (blocks > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((fine_attn_kernel<T, D, VA, FINEST, NT>), dim3(static_cast<unsigned>(blocks)),
                       dim3(wpb * kWave), wpb * wave_bytes, stream, a);
    return hipGetLastError();
}

template <typename T, int D, bool VA, bool FINEST>
hipError_t launch_nt(const FineArgs& a, hipStream_t stream)
{
    const int nslot = 4 * a.Kp;
    if (nslot <= 64) return launch_one<T, D, VA, FINEST, 1>(a, stream);
    if (nslot <= 128) return launch_one<T, D, VA, FINEST, 2>(a, stream);
    if (nslot <= 256) return launch_one<T, D, VA, FINEST, 4>(a, stream);
    return hipErrorInvalidValue;
}

template <typename T, int D>
hipError_t launch_td(const FineArgs& a, bool variant_a, bool finest, hipStream_t stream)
{
    if (variant_a) return finest ? launch_nt<T, D, true, true>(a, stream) : launch_nt<T, D, true, false>(a, stream);
    return finest ? launch_nt<T, D, false, true>(a, stream) : launch_nt<T, D, false, false>(a, stream);
}

}  // namespace

hipError_t launch_fine_attn_wide(const FineArgs& a, int d, bool variant_a, bool bf16_in, bool finest, hipStream_t stream)
{
    if (bf16_in) {
        if (d == 32) return launch_td<bf16, 32>(a, variant_a, finest, stream);
        if (d == 64) return launch_td<bf16, 64>(a, variant_a, finest, stream);
    } else {
        if (d == 32) return launch_td<float, 32>(a, variant_a, finest, stream);
        if (d == 64) return launch_td<float, 64>(a, variant_a, finest, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace qta
