// Steps 2-3 at the coarsest level: full softmax attention, Eq. (1), plus each query's top-K keys.
//
// One workgroup of 16 waves owns a 16-query tile of one (batch, head):
//   phase 1  logits S = tau * Q_tile K^T on MFMA (16x16 output tiles, waves take key tiles in
//            turn), kept in LDS as fp32 [16][N];
//   phase 2  wave r owns query row r: max, exp and sum over the row, then the K best keys by
//            repeated wave-wide maximum of a (logit, index) word, so ties go to the lower index;
//            QuadTree-A zeroes the kept keys' weights (their mass is refined at the next level);
//   phase 3  m = P V on MFMA: waves split the d columns into 16-wide tiles and the keys into
//            chunks; partial tiles are summed through LDS and written as fp32 messages (or, for a
//            single-level problem, straight to the output in the storage type).
// The coarsest map holds at most QTA_MAX_COARSE tokens, so a row fits in 16 registers per lane.
#include "qta_device.h"
#include "qta_internal.h"

namespace qta {

namespace {

typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kRows = 16;                         // queries per workgroup
constexpr int kWaves = 16;
constexpr int kPerLane = QTA_MAX_COARSE / kWave;  // row elements per lane

__host__ __device__ inline int coarse_pitch(int N) { return (N + 63) / 64 * 64; }

template <typename T, int D, bool VA>
__global__ __launch_bounds__(1024) void coarse_attn_kernel(CoarseArgs a)
{
    using S = Storage<T>;
    constexpr bool kBf16 = sizeof(T) == 2;
    extern __shared__ __align__(16) float smem[];
    const int N = a.N, C = a.C, pitch = coarse_pitch(N);
    float* Sm = smem;                              // [16][pitch]
    float* red = smem + kRows * pitch;             // [16 waves][16][16]
    const int tiles = (N + kRows - 1) / kRows;
    int blk = blockIdx.x;
    const int tile = blk % tiles;
    blk /= tiles;
    const int h = blk % a.heads;
    const int b = blk / a.heads;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const size_t tok0 = static_cast<size_t>(b) * N;           // first token of this batch element
    const size_t hoff = static_cast<size_t>(h) * D;

    // ---- phase 1: logits on MFMA ----
    {
        const int arow = lane & 15, kgrp = lane >> 4;
        const int qi = tile * kRows + arow;
        const bool qok = qi < N;
        for (int kt = wave; kt < tiles; kt += kWaves) {
            const int n = kt * 16 + (lane & 15);
            const bool nok = n < N;
            float4_t acc = {0.f, 0.f, 0.f, 0.f};
            if constexpr (kBf16) {
                const uint16_t* qb = static_cast<const uint16_t*>(a.q) + (tok0 + qi) * C + hoff;
                const uint16_t* kb = static_cast<const uint16_t*>(a.k) + (tok0 + n) * C + hoff;
#pragma unroll
                for (int ks = 0; ks < D / 16; ++ks) {
                    short4_t av = {0, 0, 0, 0}, bv = {0, 0, 0, 0};
                    if (qok) av = *reinterpret_cast<const short4_t*>(qb + ks * 16 + 4 * kgrp);
                    if (nok) bv = *reinterpret_cast<const short4_t*>(kb + ks * 16 + 4 * kgrp);
                    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, bv, acc, 0, 0, 0);
                }
            } else {
                const float* qf = static_cast<const float*>(a.q) + (tok0 + qi) * C + hoff;
                const float* kf = static_cast<const float*>(a.k) + (tok0 + n) * C + hoff;
#pragma unroll
                for (int ks = 0; ks < D / 4; ++ks) {
                    const float av = qok ? qf[ks * 4 + kgrp] : 0.f;
                    const float bv = nok ? kf[ks * 4 + kgrp] : 0.f;
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc, 0, 0, 0);
                }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j)
                Sm[(4 * kgrp + j) * pitch + n] = nok ? acc[j] * a.scale : -INFINITY;
        }
    }
    __syncthreads();

    // ---- phase 2: softmax and selection, one wave per query row ----
    {
        const int r = wave;
        const int qi = tile * kRows + r;
        float* row = Sm + r * pitch;
        float x[kPerLane];
        float mx = -INFINITY;
#pragma unroll
        for (int e = 0; e < kPerLane; ++e) {
            const int j = lane + kWave * e;
            x[e] = j < N ? row[j] : -INFINITY;
            mx = fmaxf(mx, x[e]);
        }
        mx = wave_max(mx);
        float p[kPerLane];
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < kPerLane; ++e) {
            const int j = lane + kWave * e;
            p[e] = j < N ? __expf(x[e] - mx) : 0.f;
            sum += p[e];
        }
        sum = wave_sum(sum);
        const float inv = 1.0f / sum;
#pragma unroll
        for (int e = 0; e < kPerLane; ++e) p[e] *= inv;

        if (a.K > 0 && qi < N) {
            uint64_t word[kPerLane];
#pragma unroll
            for (int e = 0; e < kPerLane; ++e) {
                const int j = lane + kWave * e;
                word[e] = j < N ? rank_word(x[e], j) : 0ull;
            }
            const int keff = a.K < N ? a.K : N;
            const size_t orow = ((static_cast<size_t>(b) * a.heads + h) * N + qi) * a.K;
            for (int rr = 0; rr < a.K; ++rr) {
                if (rr >= keff) {
                    if (lane == 0) {
                        a.sel_idx[orow + rr] = -1;
                        a.sel_key[orow + rr] = 0.f;
                    }
                    continue;
                }
                uint64_t best = 0;
                float bestp = 0.f;
#pragma unroll
                for (int e = 0; e < kPerLane; ++e)
                    if (word[e] > best) {
                        best = word[e];
                        bestp = p[e];
                    }
                const uint64_t g = wave_max_u64(best);
                const int j = rank_word_index(g);
                const float pj = __shfl(bestp, j & 63, kWave);
                if (lane == (j & 63)) {
#pragma unroll
                    for (int e = 0; e < kPerLane; ++e)
                        if (e == (j >> 6)) {
                            word[e] = 0ull;
                            if constexpr (VA) p[e] = 0.f;
                        }
                }
                if (lane == 0) {
                    a.sel_idx[orow + rr] = j;
                    a.sel_key[orow + rr] = pj;
                }
            }
        }
#pragma unroll
        for (int e = 0; e < kPerLane; ++e) {
            const int j = lane + kWave * e;
            if (j < pitch) row[j] = (j < N && qi < N) ? p[e] : 0.f;
        }
    }
    __syncthreads();

    // ---- phase 3: messages m = P V on MFMA ----
    constexpr int NCT = D / 16;          // 16-wide column tiles
    constexpr int NKS = kWaves / NCT;    // key chunks
    {
        const int ct = wave % NCT, ks = wave / NCT;
        const int arow = lane & 15, kgrp = lane >> 4;
        const int ch = ct * 16 + (lane & 15);
        float4_t acc = {0.f, 0.f, 0.f, 0.f};
        if constexpr (kBf16) {
            const uint16_t* vb = static_cast<const uint16_t*>(a.v) + tok0 * C + hoff + ch;
            const int steps = (N + 15) / 16;
            for (int st = ks; st < steps; st += NKS) {
                const float4 pv = *reinterpret_cast<const float4*>(Sm + arow * pitch + st * 16 + 4 * kgrp);
                short4_t av;
                av[0] = static_cast<short>(f32_to_bf16_bits(pv.x));
                av[1] = static_cast<short>(f32_to_bf16_bits(pv.y));
                av[2] = static_cast<short>(f32_to_bf16_bits(pv.z));
                av[3] = static_cast<short>(f32_to_bf16_bits(pv.w));
                short4_t bv;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int cand = st * 16 + 4 * kgrp + e;
                    bv[e] = cand < N ? static_cast<short>(vb[static_cast<size_t>(cand) * C]) : short(0);
                }
                acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, bv, acc, 0, 0, 0);
            }
        } else {
            const float* vf = static_cast<const float*>(a.v) + tok0 * C + hoff + ch;
            const int steps = (N + 3) / 4;
            for (int st = ks; st < steps; st += NKS) {
                const float av = Sm[arow * pitch + st * 4 + kgrp];
                const int cand = st * 4 + kgrp;
                const float bv = cand < N ? vf[static_cast<size_t>(cand) * C] : 0.f;
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc, 0, 0, 0);
            }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) red[(wave * 16 + 4 * kgrp + j) * 16 + (lane & 15)] = acc[j];
    }
    __syncthreads();
    for (int t = threadIdx.x; t < kRows * D; t += blockDim.x) {
        const int r = t / D, ch = t % D;
        const int ct = ch / 16, col = ch % 16;
        float s = 0.f;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) s += red[((ks * NCT + ct) * 16 + r) * 16 + col];
        const int qi = tile * kRows + r;
        if (qi >= N) continue;
        if (a.out) {
            float wl = 1.0f;
            if (!VA) wl = a.w ? a.w[((tok0 + qi) * a.heads + h) * a.levels] : 1.0f / a.levels;
            S::store1(a.out, (tok0 + qi) * C + hoff + ch, wl * s);
        } else {
            a.msg[((tok0 + qi) * a.heads + h) * D + ch] = s;
        }
    }
}

template <typename T, int D, bool VA>
hipError_t launch_one(const CoarseArgs& a, hipStream_t stream)
{
    const size_t lds = (static_cast<size_t>(kRows) * coarse_pitch(a.N) + kWaves * 16 * 16) * sizeof(float);
    if (lds > device_max_lds()) return hipErrorInvalidValue;
    static bool configured = false;
    if (!configured) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&coarse_attn_kernel<T, D, VA>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           static_cast<int>(device_max_lds()));
        if (e != hipSuccess) return e;
        configured = true;
    }
    const int tiles = (a.N + kRows - 1) / kRows;
    const long long blocks = static_cast<long long>(a.B) * a.heads * tiles;
    if (blocks > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((coarse_attn_kernel<T, D, VA>), dim3(static_cast<unsigned>(blocks)), dim3(kWaves * kWave),
                       lds, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_coarse_attn(const CoarseArgs& a, int d, bool variant_a, bool bf16_in, hipStream_t stream)
{
#define QTA_COARSE_CASE(T, D)                                                        \
    if (d == D) return variant_a ? launch_one<T, D, true>(a, stream) : launch_one<T, D, false>(a, stream);
    if (bf16_in) {
        QTA_COARSE_CASE(bf16, 32)
        QTA_COARSE_CASE(bf16, 64)
    } else {
        QTA_COARSE_CASE(float, 32)
        QTA_COARSE_CASE(float, 64)
    }
#undef QTA_COARSE_CASE
    return hipErrorInvalidValue;
}

}  // namespace qta
