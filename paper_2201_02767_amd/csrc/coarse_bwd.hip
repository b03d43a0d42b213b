// Backward of the coarsest level (Eq. 1 over the whole map) on MFMA tiles, laid out like the
// forward's coarse kernel: a workgroup of 16 waves owns 16 rows of one (batch, head) against all N
// columns, in two passes.
//   query pass (rows = queries, columns = keys): S = tau Q K^T and G = dM V^T on MFMA into LDS;
//     wave r owns row r: p = softmax(S_r); ds = G_r (QuadTree-A: a key this query kept takes the
//     gradient of its score from the level below); D = sum p ds; dS = p (ds - D); the row's
//     statistics (max, sum, D) go to HBM; dQ = tau dS K on MFMA.
//   key pass (rows = keys, columns = queries): S^T = tau K Q^T and G^T = V dM^T; wave r owns key
//     row r: p from the queries' statistics, dS^T, and the value weights (p, or 0 where QuadTree-A's
//     query kept the key: its mass is refined below); dK = tau dS^T Q and dV = W^T dM on MFMA.
// With a single level dM is w_0 dout (B) or dout (A), and dw_0 = sum_j p_j <dout, v_j>.
// Every element is computed in fp32 from operands widened on load (exact for bf16 inputs). No
// atomics: every output row has one writer.
#include "qta_device.h"
#include "qta_internal.h"

namespace qta {

namespace {

typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kRows = 16;
constexpr int kWaves = 16;

__host__ __device__ inline int bwd_coarse_pitch(int N) { return (N + 63) / 64 * 64 + 4; }

inline int bwd_coarse_per_lane(int N)
{
    const int need = (N + kWave - 1) / kWave;
    static const int counts[] = {1, 2, 3, 4, 5, 6, 8, 12, 16};
    for (int c : counts)
        if (need <= c) return c;
    return 0;
}

// Four consecutive channels [c0, c0+4) of row `tok` (head offset hoff) of a token tensor, widened
// to fp32: the storage type T, or fp32 when `f32` (the message gradients).
template <typename T>
__device__ __forceinline__ float4 load4(const void* base, bool f32, size_t elem)
{
    if (f32) return *reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
    if constexpr (sizeof(T) == 2) {
        const uint2 r = *reinterpret_cast<const uint2*>(static_cast<const unsigned char*>(base) + elem * 2);
        return make_float4(bf16_bits_to_f32(r.x & 0xFFFFu), bf16_bits_to_f32(r.x >> 16), bf16_bits_to_f32(r.y & 0xFFFFu),
                           bf16_bits_to_f32(r.y >> 16));
    } else {
        return *reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
    }
}

template <typename T>
__device__ __forceinline__ float load1(const void* base, bool f32, size_t elem)
{
    if (f32) return static_cast<const float*>(base)[elem];
    return Storage<T>::load1(base, elem);
}

template <typename T, int D, bool VA, int kPerLane, bool KEYS>
__global__ __launch_bounds__(1024) void bwd_coarse_tile_kernel(BwdCoarseArgs a)
{
    constexpr int NJ = D / 16;                     // 4-channel chunks per lane and row
    constexpr int kMaxTilesPerWave = QTA_MAX_COARSE / 16 / kWaves;
    extern __shared__ __align__(16) float smem[];
    const int N = a.N, C = a.C, pitch = bwd_coarse_pitch(N);
    float* Sm = smem;                              // [16][pitch]: logits, then dS
    float* Gm = Sm + kRows * pitch;                // [16][pitch]: <dm, v>, then the value weights
    float* red = Gm + kRows * pitch;               // [16 waves][16][16]
    const int tiles = (N + kRows - 1) / kRows;
    int blk = blockIdx.x;
    const int tile = blk % tiles;
    blk /= tiles;
    const int h = blk % a.heads;
    const int b = blk / a.heads;
    const int bh = b * a.heads + h;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const size_t tok0 = static_cast<size_t>(b) * N;
    const size_t hoff = static_cast<size_t>(h) * D;
    const bool single = a.dm == nullptr;           // one level: dm = w_0 dout (B) or dout
    const void* dmsrc = single ? a.dout : static_cast<const void*>(a.dm);
    const bool dm32 = !single;
    // row operands (A) and column operands (B) of the two products
    const void* rowS = KEYS ? a.k : a.q;
    const void* colS = KEYS ? a.q : a.k;
    const void* rowG = KEYS ? a.v : dmsrc;
    const void* colG = KEYS ? dmsrc : a.v;
    const bool rowG32 = KEYS ? false : dm32, colG32 = KEYS ? dm32 : false;

    // ---- phase 1: S and G on MFMA; a wave takes column tiles wave, wave+16, ... ----
    {
        const int arow = lane & 15, kgrp = lane >> 4;
        const int ri = min(tile * kRows + arow, N - 1);         // rows past N are computed and ignored
        float4 aS[NJ], aG[NJ];
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
            const size_t e = (tok0 + ri) * C + hoff + 4 * (kgrp + 4 * jj);
            aS[jj] = load4<T>(rowS, false, e);
            aG[jj] = load4<T>(rowG, rowG32, e);
        }
#pragma unroll
        for (int it = 0; it < kMaxTilesPerWave; ++it) {
            const int ct = wave + kWaves * it;
            if (ct >= tiles) break;                                   // uniform
            const int n = min(ct * 16 + arow, N - 1);
            float4_t accS = {0.f, 0.f, 0.f, 0.f}, accG = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int jj = 0; jj < NJ; ++jj) {
                const size_t e = (tok0 + n) * C + hoff + 4 * (kgrp + 4 * jj);
                const float4 bS = load4<T>(colS, false, e);
                const float4 bG = load4<T>(colG, colG32, e);
                accS = __builtin_amdgcn_mfma_f32_16x16x4f32(aS[jj].x, bS.x, accS, 0, 0, 0);
                accS = __builtin_amdgcn_mfma_f32_16x16x4f32(aS[jj].y, bS.y, accS, 0, 0, 0);
                accS = __builtin_amdgcn_mfma_f32_16x16x4f32(aS[jj].z, bS.z, accS, 0, 0, 0);
                accS = __builtin_amdgcn_mfma_f32_16x16x4f32(aS[jj].w, bS.w, accS, 0, 0, 0);
                accG = __builtin_amdgcn_mfma_f32_16x16x4f32(aG[jj].x, bG.x, accG, 0, 0, 0);
                accG = __builtin_amdgcn_mfma_f32_16x16x4f32(aG[jj].y, bG.y, accG, 0, 0, 0);
                accG = __builtin_amdgcn_mfma_f32_16x16x4f32(aG[jj].z, bG.z, accG, 0, 0, 0);
                accG = __builtin_amdgcn_mfma_f32_16x16x4f32(aG[jj].w, bG.w, accG, 0, 0, 0);
            }
            const int col = ct * 16 + (lane & 15);
#pragma unroll
            for (int jr = 0; jr < 4; ++jr) {
                Sm[(4 * kgrp + jr) * pitch + col] = col < N ? accS[jr] * a.scale : -INFINITY;
                Gm[(4 * kgrp + jr) * pitch + col] = col < N ? accG[jr] : 0.f;
            }
        }
    }
    __syncthreads();

    // ---- phase 2: one wave per row ----
    {
        const int r = wave;
        const int ri = tile * kRows + r;
        float* srow = Sm + r * pitch;
        float* grow = Gm + r * pitch;
        const bool rv = ri < N;
        if constexpr (!KEYS) {
            float x[kPerLane], g[kPerLane];
            float mx = -INFINITY;
#pragma unroll
            for (int e = 0; e < kPerLane; ++e) {
                const int j = lane + kWave * e;
                x[e] = j < N ? srow[j] : -INFINITY;
                g[e] = j < N ? grow[j] : 0.f;
                mx = fmaxf(mx, x[e]);
            }
            mx = wave_max_fast(mx);
            float sum = 0.f;
#pragma unroll
            for (int e = 0; e < kPerLane; ++e) {
                x[e] = __expf(x[e] - mx);                             // 0 past N
                sum += x[e];
            }
            sum = wave_sum_fast(sum);
            const float inv = 1.0f / sum;
            const size_t qtok = tok0 + min(ri, N - 1);
            const float w0 = (single && a.variant_b && a.w) ? a.w[qtok * a.heads + h] : 1.0f;
            float ds[kPerLane], dw = 0.f;
#pragma unroll
            for (int e = 0; e < kPerLane; ++e) {
                x[e] *= inv;
                ds[e] = w0 * g[e];
                dw += x[e] * g[e];                                    // single level: sum p <dout, v>
            }
            if (VA && a.K > 0 && rv) {
                const size_t sr = (static_cast<size_t>(bh) * N + ri) * a.K;
                for (int mm = 0; mm < a.K; ++mm) {
                    const int32_t j = a.sel_idx[sr + mm];
                    if (j < 0) continue;
                    const float dsv = a.dsig[sr + mm];
#pragma unroll
                    for (int e = 0; e < kPerLane; ++e)
                        if (j == lane + kWave * e) ds[e] = dsv;
                }
            }
            float Dsum = 0.f;
#pragma unroll
            for (int e = 0; e < kPerLane; ++e) Dsum += x[e] * ds[e];
            Dsum = wave_sum_fast(Dsum);
#pragma unroll
            for (int e = 0; e < kPerLane; ++e) {
                const int j = lane + kWave * e;
                if (j < pitch) srow[j] = (j < N && rv) ? x[e] * (ds[e] - Dsum) : 0.f;
            }
            if (rv && lane == 0)
                *reinterpret_cast<float4*>(a.stats + (static_cast<size_t>(bh) * N + ri) * 4) = make_float4(mx, sum, Dsum, 0.f);
            if (single && a.variant_b && a.w && a.dw) {               // uniform
                dw = wave_sum_fast(dw);
                if (rv && lane == 0) a.dw[qtok * a.heads + h] = dw;
            }
        } else {
            // key row ri; column i is a query with statistics (max, sum, D)
#pragma unroll
            for (int e = 0; e < kPerLane; ++e) {
                const int i = lane + kWave * e;
                if (i >= pitch) continue;
                float dsv = 0.f, wv = 0.f;
                if (i < N && rv) {
                    const float4 st = *reinterpret_cast<const float4*>(a.stats + (static_cast<size_t>(bh) * N + i) * 4);
                    const float p = __expf(srow[i] - st.x) / st.y;
                    const float w0 = (single && a.variant_b && a.w) ? a.w[(tok0 + i) * a.heads + h] : 1.0f;
                    float ds = w0 * grow[i];
                    bool kept = false;
                    if (VA && a.K > 0) {
                        const size_t sr = (static_cast<size_t>(bh) * N + i) * a.K;
                        for (int mm = 0; mm < a.K; ++mm)
                            if (a.sel_idx[sr + mm] == ri) {
                                kept = true;
                                ds = a.dsig[sr + mm];
                            }
                    }
                    dsv = p * (ds - st.z);
                    wv = kept ? 0.f : p * w0;                         // w_0 folds the single level's dm
                }
                srow[i] = dsv;
                grow[i] = wv;
            }
        }
    }
    __syncthreads();

    // ---- phase 3: (weights [16 x N]) x (operand rows [N x D]) on fp32 MFMA: lane (kgrp, col)
    //      supplies operand row 4*st + kgrp, column 16*ct + col; waves split the columns into
    //      16-wide tiles and the N rows into chunks; partial tiles are summed through LDS ----
    constexpr int NCT = D / 16;
    constexpr int NKS = kWaves / NCT;
    const int p3_ct = wave % NCT, p3_ks = wave / NCT;
    const int arow = lane & 15, kgrp = lane >> 4;
    const int p3_ch = p3_ct * 16 + arow;
    const int steps = (N + 3) / 4;
    auto product = [&](const float* Wm, const void* src, bool src32, float scale, float* out) {
        float4_t acc = {0.f, 0.f, 0.f, 0.f};
        for (int st = p3_ks; st < steps; st += NKS) {
            const int cand = min(st * 4 + kgrp, N - 1);                // weight 0 past N
            const float bv = load1<T>(src, src32, (tok0 + cand) * C + hoff + p3_ch);
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(Wm[arow * pitch + st * 4 + kgrp], bv, acc, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) red[(wave * 16 + 4 * kgrp + j) * 16 + arow] = acc[j];
        __syncthreads();
        for (int t = threadIdx.x; t < kRows * D; t += blockDim.x) {
            const int rr = t / D, ch = t % D;
            const int ct = ch / 16, col = ch % 16;
            float s = 0.f;
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) s += red[((ks * NCT + ct) * 16 + rr) * 16 + col];
            const int ri = tile * kRows + rr;
            if (ri < N) out[(tok0 + ri) * C + hoff + ch] = scale * s;
        }
        __syncthreads();
    };
    if constexpr (!KEYS) {
        product(Sm, a.k, false, a.scale, a.dq);
    } else {
        product(Sm, a.q, false, a.scale, a.dk);
        product(Gm, dmsrc, dm32, 1.0f, a.dv);
    }
}

template <typename T, int D, bool VA, int kPerLane, bool KEYS>
hipError_t launch_tile(const BwdCoarseArgs& a, hipStream_t stream)
{
    const size_t lds = (2 * static_cast<size_t>(kRows) * bwd_coarse_pitch(a.N) + kWaves * 16 * 16) * sizeof(float);
    if (lds > device_max_lds()) return hipErrorInvalidValue;
    static std::atomic<unsigned long long> configured{0};     // devices whose LDS limit is raised
    if (hipError_t e = set_max_lds_once(reinterpret_cast<const void*>(&bwd_coarse_tile_kernel<T, D, VA, kPerLane, KEYS>), configured);
        e != hipSuccess)
        return e;
    const int tiles = (a.N + kRows - 1) / kRows;
    const long long blocks = static_cast<long long>(a.B) * a.heads * tiles;
    if (blocks > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((bwd_coarse_tile_kernel<T, D, VA, kPerLane, KEYS>), dim3(static_cast<unsigned>(blocks)),
                       dim3(kWaves * kWave), lds, stream, a);
    return hipGetLastError();
}

template <typename T, int D, bool VA, int kPerLane>
hipError_t launch_both(const BwdCoarseArgs& a, hipStream_t stream)
{
    hipError_t e = launch_tile<T, D, VA, kPerLane, false>(a, stream);
    if (e != hipSuccess) return e;
    return launch_tile<T, D, VA, kPerLane, true>(a, stream);
}

template <typename T, int D, bool VA>
hipError_t launch_per_lane(const BwdCoarseArgs& a, hipStream_t stream)
{
    switch (bwd_coarse_per_lane(a.N)) {
    case 1: return launch_both<T, D, VA, 1>(a, stream);
    case 2: return launch_both<T, D, VA, 2>(a, stream);
    case 3: return launch_both<T, D, VA, 3>(a, stream);
    case 4: return launch_both<T, D, VA, 4>(a, stream);
    case 5: return launch_both<T, D, VA, 5>(a, stream);
    case 6: return launch_both<T, D, VA, 6>(a, stream);
    case 8: return launch_both<T, D, VA, 8>(a, stream);
    case 12: return launch_both<T, D, VA, 12>(a, stream);
    case 16: return launch_both<T, D, VA, 16>(a, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_bwd_coarse(const BwdCoarseArgs& a, int d, bool variant_a, bool use_bf16, hipStream_t stream)
{
    if (a.N > QTA_MAX_COARSE) return hipErrorInvalidValue;
#define QTA_BWD_COARSE_CASE(T, DD)                                                                      \
    if (d == DD) return variant_a ? launch_per_lane<T, DD, true>(a, stream) : launch_per_lane<T, DD, false>(a, stream);
    if (use_bf16) {
        QTA_BWD_COARSE_CASE(bf16, 32)
        QTA_BWD_COARSE_CASE(bf16, 64)
    } else {
        QTA_BWD_COARSE_CASE(float, 32)
        QTA_BWD_COARSE_CASE(float, 64)
    }
#undef QTA_BWD_COARSE_CASE
    return hipErrorInvalidValue;
}

}  // namespace qta
