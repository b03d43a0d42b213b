// Steps 2-3 at the coarsest level: full softmax attention, Eq. (1), plus each query's top-K keys.
//
// One workgroup of 16 waves owns a 16-query tile of one (batch, head):
//   phase 1  logits S = tau * Q_tile K^T on MFMA (16x16 output tiles, waves take key tiles in
//            turn), kept in LDS as fp32 [16][N];
//   phase 2  wave r owns query row r: max, exp and sum over the row (register butterflies), then
//            the K best keys by a bitwise radix select on wave ballots (ties at the cut go to the
//            lower index), listed in index order; QuadTree-A zeroes the kept keys' weights (their
//            mass is refined at the next level);
//   phase 3  m = P V on fp32 MFMA (values widened to fp32 as they are loaded): waves split the d
//            columns into 16-wide tiles and the keys into chunks; partial tiles are summed through
//            LDS and written as fp32 messages (or, for a single-level problem, straight to the
//            output in the storage type).
// The coarsest map holds at most QTA_MAX_COARSE tokens, so a row fits in 16 registers per lane.
#include "qta_device.h"
#include "qta_internal.h"

namespace qta {

namespace {

typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kRows = 16;                         // queries per workgroup
constexpr int kWaves = 16;

// LDS pitch of a logit row: whole 64-element groups plus 4 floats, so the 16 rows that one MFMA
// operand read touches fall in different banks.
__host__ __device__ inline int coarse_pitch(int N) { return (N + 63) / 64 * 64 + 4; }

// Row elements per lane, rounded up to a power of two (a template parameter, so the selection
// loops carry no bounds checks).
inline int coarse_per_lane(int N)
{
    const int need = (N + kWave - 1) / kWave;
    int p = 1;
    while (p < need) p <<= 1;
    return p;
}

template <typename T, int D, bool VA, int kPerLane>
__global__ __launch_bounds__(1024) void coarse_attn_kernel(CoarseArgs a)
{
    using S = Storage<T>;
    constexpr bool kBf16 = sizeof(T) == 2;
    constexpr int kMaxTilesPerWave = QTA_MAX_COARSE / 16 / kWaves;
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

    // ---- phase 1: logits on MFMA; a wave takes key tiles wave, wave+16, ... (at most 4) ----
    {
        const int arow = lane & 15, kgrp = lane >> 4;
        const int qi = tile * kRows + arow;
        const bool qok = qi < N;
        if constexpr (kBf16) {
            constexpr int KS = D / 16;
            short4_t av[KS], bv[kMaxTilesPerWave][KS];
            const uint16_t* qb = static_cast<const uint16_t*>(a.q) + (tok0 + (qok ? qi : 0)) * C + hoff;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                av[ks] = short4_t{0, 0, 0, 0};
                if (qok) av[ks] = *reinterpret_cast<const short4_t*>(qb + ks * 16 + 4 * kgrp);
            }
#pragma unroll
            for (int it = 0; it < kMaxTilesPerWave; ++it) {
                const int n = (wave + kWaves * it) * 16 + (lane & 15);
                const uint16_t* kb = static_cast<const uint16_t*>(a.k) + (tok0 + (n < N ? n : 0)) * C + hoff;
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    bv[it][ks] = short4_t{0, 0, 0, 0};
                    if (n < N) bv[it][ks] = *reinterpret_cast<const short4_t*>(kb + ks * 16 + 4 * kgrp);
                }
            }
#pragma unroll
            for (int it = 0; it < kMaxTilesPerWave; ++it) {
                const int kt = wave + kWaves * it;
                if (kt >= tiles) break;
                float4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av[ks], bv[it][ks], acc, 0, 0, 0);
                const int n = kt * 16 + (lane & 15);
#pragma unroll
                for (int j = 0; j < 4; ++j) Sm[(4 * kgrp + j) * pitch + n] = n < N ? acc[j] * a.scale : -INFINITY;
            }
        } else {
            constexpr int KS = D / 4;
            float av[KS], bv[kMaxTilesPerWave][KS];
            const float* qf = static_cast<const float*>(a.q) + (tok0 + (qok ? qi : 0)) * C + hoff;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) av[ks] = qok ? qf[ks * 4 + kgrp] : 0.f;
#pragma unroll
            for (int it = 0; it < kMaxTilesPerWave; ++it) {
                const int n = (wave + kWaves * it) * 16 + (lane & 15);
                const float* kf = static_cast<const float*>(a.k) + (tok0 + (n < N ? n : 0)) * C + hoff;
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) bv[it][ks] = n < N ? kf[ks * 4 + kgrp] : 0.f;
            }
#pragma unroll
            for (int it = 0; it < kMaxTilesPerWave; ++it) {
                const int kt = wave + kWaves * it;
                if (kt >= tiles) break;
                float4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[ks], bv[it][ks], acc, 0, 0, 0);
                const int n = kt * 16 + (lane & 15);
#pragma unroll
                for (int j = 0; j < 4; ++j) Sm[(4 * kgrp + j) * pitch + n] = n < N ? acc[j] * a.scale : -INFINITY;
            }
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
        mx = wave_max_fast(mx);
        float p[kPerLane];
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < kPerLane; ++e) {
            const int j = lane + kWave * e;
            p[e] = j < N ? __expf(x[e] - mx) : 0.f;
            sum += p[e];
        }
        const float inv = 1.0f / wave_sum_fast(sum);
#pragma unroll
        for (int e = 0; e < kPerLane; ++e) p[e] *= inv;

        if (a.K > 0 && qi < N) {
            // the K best keys by logit (ties to the lower index), listed in index order
            uint32_t key[kPerLane], name[kPerLane];
            bool kept[kPerLane];
#pragma unroll
            for (int e = 0; e < kPerLane; ++e) {
                const int j = lane + kWave * e;
                key[e] = j < N ? ordered_bits(x[e]) : 0u;
                name[e] = static_cast<uint32_t>(j);
            }
            const int keff = a.K < N ? a.K : N;
            wave_select_top<kPerLane>(key, name, keff, kept);
            const size_t orow = ((static_cast<size_t>(b) * a.heads + h) * N + qi) * a.K;
            int before = 0;
#pragma unroll
            for (int e = 0; e < kPerLane; ++e) {
                const uint64_t mask = __ballot(kept[e]);
                if (kept[e]) {
                    const int pos = before + lanes_below(mask);
                    a.sel_idx[orow + pos] = lane + kWave * e;
                    a.sel_key[orow + pos] = p[e];
                    if constexpr (VA) p[e] = 0.f;           // refined at the next level (Omega)
                }
                before += __popcll(mask);
            }
            if (lane >= keff && lane < a.K) {
                a.sel_idx[orow + lane] = -1;
                a.sel_key[orow + lane] = 0.f;
            }
        }
#pragma unroll
        for (int e = 0; e < kPerLane; ++e) {
            const int j = lane + kWave * e;
            if (j < pitch) row[j] = (j < N && qi < N) ? p[e] : 0.f;
        }
    }
    __syncthreads();

    // ---- phase 3: messages m = P V on fp32 MFMA (values widened on load, so no transpose) ----
    constexpr int NCT = D / 16;          // 16-wide column tiles
    constexpr int NKS = kWaves / NCT;    // key chunks
    {
        const int ct = wave % NCT, ks = wave / NCT;
        const int arow = lane & 15, kgrp = lane >> 4;
        const int ch = ct * 16 + (lane & 15);
        const int steps = (N + 3) / 4;
        float4_t acc = {0.f, 0.f, 0.f, 0.f};
        constexpr int kBatch = 8;
        for (int st0 = ks; st0 < steps; st0 += NKS * kBatch) {
            float bv[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int cand = (st0 + u * NKS) * 4 + kgrp;
                bv[u] = cand < N ? S::load1(a.v, (tok0 + cand) * C + hoff + ch) : 0.f;
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int st = st0 + u * NKS;
                if (st >= steps) break;
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(Sm[arow * pitch + st * 4 + kgrp], bv[u], acc, 0, 0, 0);
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

template <typename T, int D, bool VA, int kPerLane>
hipError_t launch_one(const CoarseArgs& a, hipStream_t stream)
{
    const size_t lds = (static_cast<size_t>(kRows) * coarse_pitch(a.N) + kWaves * 16 * 16) * sizeof(float);
    if (lds > device_max_lds()) return hipErrorInvalidValue;
    static bool configured = false;
    if (!configured) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&coarse_attn_kernel<T, D, VA, kPerLane>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           static_cast<int>(device_max_lds()));
        if (e != hipSuccess) return e;
        configured = true;
    }
    const int tiles = (a.N + kRows - 1) / kRows;
    const long long blocks = static_cast<long long>(a.B) * a.heads * tiles;
    if (blocks > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((coarse_attn_kernel<T, D, VA, kPerLane>), dim3(static_cast<unsigned>(blocks)), dim3(kWaves * kWave),
                       lds, stream, a);
    return hipGetLastError();
}

template <typename T, int D, bool VA>
hipError_t launch_per_lane(const CoarseArgs& a, hipStream_t stream)
{
    switch (coarse_per_lane(a.N)) {
    case 1: return launch_one<T, D, VA, 1>(a, stream);
    case 2: return launch_one<T, D, VA, 2>(a, stream);
    case 4: return launch_one<T, D, VA, 4>(a, stream);
    case 8: return launch_one<T, D, VA, 8>(a, stream);
    case 16: return launch_one<T, D, VA, 16>(a, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_coarse_attn(const CoarseArgs& a, int d, bool variant_a, bool bf16_in, hipStream_t stream)
{
#define QTA_COARSE_CASE(T, D)                                                                     \
    if (d == D) return variant_a ? launch_per_lane<T, D, true>(a, stream) : launch_per_lane<T, D, false>(a, stream);
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
