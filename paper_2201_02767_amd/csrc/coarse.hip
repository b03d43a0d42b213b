// Steps 2-3 at the coarsest level: full softmax attention, Eq. (1), plus each query's top-K keys.
//
// One workgroup of Q waves (Q = 8 or 16) owns a tile of Q queries of one (batch, head):
//   phase 1  logits S = tau * Q_tile K^T on MFMA (16x16 output tiles whose rows repeat the Q
//            queries when Q < 16; waves take key tiles in turn, a batch of loads at a time), kept
//            in LDS as fp32 [Q][N];
//   phase 2  wave r owns query row r: max, exp and sum over the row (register butterflies), then
//            the K best keys by a bitwise radix select on wave ballots (ties at the cut go to the
//            lower index), listed in index order; QuadTree-A zeroes the kept keys' weights (their
//            mass is refined at the next level);
//   phase 3  m = P V on fp32 MFMA (values widened to fp32 as they are loaded, two batches of
//            loads in flight): waves split the d columns into 16-wide tiles and the keys into
//            chunks; partial tiles are summed through
//            LDS and written as fp32 messages (or, for a single-level problem, straight to the
//            output in the storage type).
// The coarsest map holds at most QTA_MAX_COARSE tokens, so a row fits in 16 registers per lane.
// Maps of at most 64 tokens take coarse_small_kernel instead (one wave per query row).
#include <type_traits>

#include "qta_device.h"
#include "qta_internal.h"

namespace qta {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));


// LDS pitch of a logit row: whole 64-element groups plus 4 floats, so the 16 rows that one MFMA
// operand read touches fall in different banks.
__host__ __device__ inline int coarse_pitch(int N) { return (N + 63) / 64 * 64 + 4; }

// Row elements per lane: ceil(N / 64) rounded up to the next instantiated count (a template
// parameter, so the selection loops carry no bounds checks and no empty slots for common sizes).
inline int coarse_per_lane(int N)
{
    const int need = (N + kWave - 1) / kWave;
    static const int counts[] = {1, 2, 3, 4, 5, 6, 8, 12, 16};
    for (int c : counts)
        if (need <= c) return c;
    return 0;
}

template <typename T, int D, bool VA, int kPerLane, int Q>
__global__ __launch_bounds__(Q * kWave) void coarse_attn_kernel(CoarseArgs a)
{
    using S = Storage<T>;
    constexpr bool kBf16 = sizeof(T) == 2;
    constexpr int kWaves = Q;                      // one wave per query row in phase 2
    static_assert(Q == 8 || Q == 16, "8 or 16 query rows per workgroup");
    extern __shared__ __align__(16) float smem[];
    const int N = a.N, C = a.C, pitch = coarse_pitch(N);
    float* Sm = smem;                              // [Q][pitch]
    float* red = smem + Q * pitch;                 // [waves][16][16]
    const int tiles = (N + Q - 1) / Q;             // query tiles of this map
    const int ktiles = (N + 15) / 16;              // 16-key tiles
    int blk = blockIdx.x;
    const int tile = blk % tiles;
    blk /= tiles;
    const int h = blk % a.heads;
    const int b = blk / a.heads;
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6)), lane = threadIdx.x & 63;
    const size_t tok0 = static_cast<size_t>(b) * N;           // first token of this batch element
    const size_t hoff = static_cast<size_t>(h) * D;
    // this map's rows as wave-uniform bases; a row's offset from them, below N * C elements
    // (N <= 1024 and C <= 2^20, so under 2^32 bytes), is a 32-bit lane offset
    const size_t map0 = tok0 * C + hoff;
    const unsigned char* qmap = static_cast<const unsigned char*>(a.q) + map0 * sizeof(T);
    const unsigned char* kmap = static_cast<const unsigned char*>(a.k) + map0 * sizeof(T);
    const unsigned char* vmap = static_cast<const unsigned char*>(a.v) + map0 * sizeof(T);
    const uint32_t row_bytes = static_cast<uint32_t>(C) * sizeof(T);   // <= 2^22

    // V operands of phase 3's first two key batches, requested after the logits' operands so that
    // their latency overlaps the logits and the selection (phase 3 layout: lane (kgrp, col) holds
    // V[4*step + kgrp][16*ct + col])
    constexpr int NCT = D / 16;          // 16-wide column tiles of the messages
    constexpr int NKS = kWaves / NCT;    // key chunks
    static_assert(NKS >= 1, "at least one wave per column tile");
    constexpr int kVBatch = 8;           // key steps per V batch
    const int p3_ct = wave % NCT, p3_ks = wave / NCT;
    const int p3_ch = p3_ct * 16 + (lane & 15);
    const int steps = (N + 3) / 4;
    float vb[kVBatch], vb2[kVBatch];
    auto load_v = [&](int st0, float (&dst)[kVBatch]) {
#pragma unroll
        for (int u = 0; u < kVBatch; ++u) {
            const int cand = min((st0 + u * NKS) * 4 + (lane >> 4), N - 1);    // clamped; weight 0 beyond N
            dst[u] = S::load1_at(vmap, __umul24(static_cast<uint32_t>(cand), static_cast<uint32_t>(C)) + p3_ch);
        }
    };

    // ---- phase 1: logits on MFMA; a wave takes key tiles wave, wave + waves, ..., a batch at a time ----
    // The 16 rows of an MFMA tile hold the workgroup's Q query rows (repeated when Q < 16; only the
    // first Q are kept). The contraction over the d channels is taken in a permuted order so that each
    // lane loads whole 16-byte chunks of its query or key row: lane (kgrp, r) loads chunks kgrp,
    // kgrp+4, ... of row r and feeds their elements to consecutive k-steps; Q and K use the same
    // permutation.
    {
        const int arow = lane & 15, kgrp = lane >> 4;
        const int qi = min(tile * Q + (arow & (Q - 1)), N - 1);   // rows past N are computed and ignored
        constexpr int NJ = D * static_cast<int>(sizeof(T)) / 64;   // 16-byte chunks per lane and row
        // key tiles a wave takes (N <= 64 * kPerLane, so at most 4 * kPerLane tiles over Q waves),
        // loaded as one batch where that is at most four: no registers held for tiles no wave has
        constexpr int kTileBatch = (4 * kPerLane + Q - 1) / Q < 4 ? (4 * kPerLane + Q - 1) / Q : 4;
        uint4 qa[NJ];
        const uint32_t qoff = __umul24(static_cast<uint32_t>(qi), row_bytes) + kgrp * 16;
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) qa[jj] = load_at<uint4>(qmap, qoff + 64 * jj);
        bool first = true;
        for (int t0 = wave; t0 < ktiles; t0 += kWaves * kTileBatch) {             // uniform
            uint4 kb[kTileBatch][NJ];
#pragma unroll
            for (int it = 0; it < kTileBatch; ++it) {
                if (t0 + kWaves * it >= ktiles) break;                            // uniform
                const int n = min((t0 + kWaves * it) * 16 + arow, N - 1);         // columns past N set to -inf
                const uint32_t koff = __umul24(static_cast<uint32_t>(n), row_bytes) + kgrp * 16;
#pragma unroll
                for (int jj = 0; jj < NJ; ++jj) kb[it][jj] = load_at<uint4>(kmap, koff + 64 * jj);
            }
            if (first) {
                load_v(p3_ks, vb);
                load_v(p3_ks + NKS * kVBatch, vb2);
                first = false;
            }
#pragma unroll
            for (int it = 0; it < kTileBatch; ++it) {
                const int kt = t0 + kWaves * it;
                if (kt >= ktiles) break;
                float4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int jj = 0; jj < NJ; ++jj) {
                    if constexpr (kBf16) {
                        // 8 bf16 per chunk: one k-step of 32 (eight channels per lane)
                        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, qa[jj]),
                                                                      __builtin_bit_cast(bf16x8_t, kb[it][jj]), acc, 0, 0, 0);
                    } else {
                        // 4 floats per chunk: four k-steps
                        const uint4 qq = qa[jj], kk = kb[it][jj];
                        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(qq.x), __uint_as_float(kk.x), acc, 0, 0, 0);
                        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(qq.y), __uint_as_float(kk.y), acc, 0, 0, 0);
                        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(qq.z), __uint_as_float(kk.z), acc, 0, 0, 0);
                        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(qq.w), __uint_as_float(kk.w), acc, 0, 0, 0);
                    }
                }
                const int n = kt * 16 + (lane & 15);
#pragma unroll
                for (int jr = 0; jr < 4; ++jr)
                    if (4 * kgrp + jr < Q) Sm[(4 * kgrp + jr) * pitch + n] = n < N ? acc[jr] * a.scale : -INFINITY;
            }
        }
        if (first) {                     // a wave with no key tile (more waves than tiles)
            load_v(p3_ks, vb);
            load_v(p3_ks + NKS * kVBatch, vb2);
        }
    }
    // The output element of this thread in the epilogue (Q*D <= the Q*64 threads: one each, or none),
    // and for the fused position encoding its operands, requested now so that they arrive during
    // the softmax: the 3x3 window of v around the query token (clamped addresses, zero outside the
    // map through opaque masks), this channel's kernel and its bias.
    static_assert(D <= kWave, "one output element per thread");
    const int er = static_cast<int>(threadIdx.x) / D, ech = static_cast<int>(threadIdx.x) - er * D;
    const int eqi = tile * Q + er;
    float pev[9], pew[9], peb = 0.f;
    if (a.pe_w) {                                    // uniform
        const int Wc = a.Wc, Hc = N / Wc;
        const int qc = min(eqi, N - 1);
        const int qy = qc / Wc, qx = qc - qy * Wc;
        const float* wk = a.pe_w + (static_cast<size_t>(h) * D + ech) * 9;
#pragma unroll
        for (int ky = 0; ky < 3; ++ky)
#pragma unroll
            for (int kx = 0; kx < 3; ++kx) {
                const int yy = qy + ky - 1, xx = qx + kx - 1;
                const int yc = min(max(yy, 0), Hc - 1), xc = min(max(xx, 0), Wc - 1);
                const unsigned ok = opaque_mask(yy >= 0 && yy < Hc && xx >= 0 && xx < Wc);
                pev[ky * 3 + kx] = masked(S::load1_at(vmap, __umul24(static_cast<uint32_t>(yc * Wc + xc), static_cast<uint32_t>(C)) + ech), ok);
                pew[ky * 3 + kx] = wk[ky * 3 + kx];
            }
        peb = a.pe_b ? a.pe_b[h * D + ech] : 0.f;
    }
    __syncthreads();

    // ---- phase 2: softmax and selection, one wave per query row ----
    {
        const int r = wave;
        const int qi = tile * Q + r;
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
    // A wave takes key steps p3_ks, p3_ks + NKS, ... in batches of kVBatch, two batches in flight.
    {
        const int prow = (lane & 15) & (Q - 1), kgrp = lane >> 4;   // P rows past Q repeat (ignored)
        const float* prw = Sm + prow * pitch + kgrp;
        float4_t acc = {0.f, 0.f, 0.f, 0.f};
        auto mma_batch = [&](int st0, const float (&vv)[kVBatch]) {
#pragma unroll
            for (int u = 0; u < kVBatch; ++u) {
                const int st = st0 + u * NKS;
                if (st >= steps) break;
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(prw[st * 4], vv[u], acc, 0, 0, 0);
            }
        };
        constexpr int kStride = NKS * kVBatch;
        for (int st0 = p3_ks; st0 < steps; st0 += 2 * kStride) {
            mma_batch(st0, vb);
            if (st0 + 2 * kStride < steps) load_v(st0 + 2 * kStride, vb);
            if (st0 + kStride >= steps) break;
            mma_batch(st0 + kStride, vb2);
            if (st0 + 3 * kStride < steps) load_v(st0 + 3 * kStride, vb2);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) red[(wave * 16 + 4 * kgrp + j) * 16 + (lane & 15)] = acc[j];
    }
    __syncthreads();
    if (er < Q && eqi < N) {
        const int r = er, ch = ech;
        const int ct = ch / 16, col = ch % 16;
        float s = 0.f;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) s += red[((ks * NCT + ct) * 16 + r) * 16 + col];
        const int qi = eqi;
        if (a.pe_w) {                                    // uniform: the fused position encoding
            // 3x3 depth-wise cross-correlation of v around token qi, zero outside the map, plus the bias
            float pe = peb;
#pragma unroll
            for (int k = 0; k < 9; ++k) pe = fmaf(pew[k], pev[k], pe);
            s += pe;
        }
        if (a.out) {
            float wl = 1.0f;
            if (!VA) wl = a.w ? a.w[((tok0 + qi) * a.heads + h) * a.levels] : 1.0f / a.levels;
            const float pe = a.pe0 ? a.pe0[((tok0 + qi) * a.heads + h) * D + ch] : 0.f;
            S::store1_at(static_cast<unsigned char*>(a.out) + map0 * sizeof(T), __umul24(static_cast<uint32_t>(qi), static_cast<uint32_t>(C)) + ch, wl * (s + pe));
        } else {
            store_at<float>(a.msg + map0, (__umul24(static_cast<uint32_t>(qi), static_cast<uint32_t>(C)) + ch) * 4u, s);
        }
    }
}

// Sum over each aligned group of G consecutive lanes (G = 4, 8 or 16), the same bits in every lane of
// a group (each step adds two partial sums that the two lanes hold in swapped roles).
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v)
{
    return __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(v), CTRL, 0xF, 0xF, false));
}

template <int G>
__device__ __forceinline__ float group_sum(float x)
{
    static_assert(G == 4 || G == 8 || G == 16, "group of 4, 8 or 16 lanes");
    x += dpp_f32<kDppXor1>(x);
    x += dpp_f32<kDppXor2>(x);
    if constexpr (G >= 8) x += dpp_f32<kDppRowHalfMirror>(x);
    if constexpr (G >= 16) x += dpp_f32<kDppRowMirror>(x);
    return x;
}

// a.lo * b.lo + a.hi * b.hi + c for two packed bf16 pairs, fp32 accumulation
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c)
{
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c, false);
}

// Small coarsest maps (N <= 64, e.g. the many short maps of attention along epipolar lines): a wave
// takes `qpw` consecutive query rows of one (batch, head) map, lane j holding key j. Key row j and
// the value chunks a lane needs are loaded once per wave; per query row the logits are per-lane dot
// products, the softmax and the selection are wave reductions and a ballot radix select, and the
// message is formed from the weights in LDS: lane (c, g) sums chunk c of value rows g, g + G, ...
// and DPP sums over the G lanes of a chunk add the groups.
template <typename T, int D, bool VA>
__global__ __launch_bounds__(256) void coarse_small_kernel(CoarseArgs a, int qpw)
{
    using S = Storage<T>;
    constexpr int E = S::kPer16B;
    constexpr int CH = D / E;                                 // chunks of a head row
    constexpr int G = kWave / CH;                             // key groups of the message, >= E (D <= 64)
    constexpr int NV = kWave / G;                             // value rows a lane covers (N <= 64)
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    const int N = a.N, C = a.C;
    const int wpm = (N + qpw - 1) / qpw;                      // waves per map
    const int gw = static_cast<int>(blockIdx.x) * 4 + wave;   // < 2^31, checked by the launcher
    if (gw >= a.B * a.heads * wpm) return;                    // whole wave
    const int bh = gw / wpm;
    const int q0 = (gw - bh * wpm) * qpw, qend = min(q0 + qpw, N);
    const int h = bh % a.heads, b = bh / a.heads;
    const size_t tok0 = static_cast<size_t>(b) * N;
    const size_t hoff = static_cast<size_t>(h) * D;
    const bool valid = lane < N;
    const unsigned char* qb = static_cast<const unsigned char*>(a.q) + (tok0 * C + hoff) * sizeof(T);
    // key row j (clamped onto the map) and value chunk c of rows g, g + G, ...
    const int c = lane / G, g = lane % G;
    // bf16 keys stay packed (products of pairs with the query's packed pairs); fp32 keys as floats
    constexpr bool kDot2 = std::is_same<T, bf16>::value;
    uint4 kraw[CH];
    float kf[kDot2 ? 1 : D];
    uint4 vraw[NV];
    {
        const uint4* kp = reinterpret_cast<const uint4*>(static_cast<const unsigned char*>(a.k) +
                                                         ((tok0 + min(lane, N - 1)) * C + hoff) * sizeof(T));
        const unsigned char* vb = static_cast<const unsigned char*>(a.v) + (tok0 * C + hoff) * sizeof(T) + c * 16;
#pragma unroll
        for (int cc = 0; cc < CH; ++cc) kraw[cc] = kp[cc];
#pragma unroll
        for (int u = 0; u < NV; ++u)
            vraw[u] = *reinterpret_cast<const uint4*>(vb + static_cast<size_t>(min(g + u * G, N - 1)) * C * sizeof(T));
        if constexpr (!kDot2) {
#pragma unroll
            for (int cc = 0; cc < CH; ++cc) S::unpack(kraw[cc], kf + cc * E);
        }
    }
    __shared__ float pw[4][kWave];
    __shared__ int sidx[4][kWave];
    __shared__ float skey[4][kWave];
    // the query row: lanes c * G, ... hold its chunk c, read by every lane with readlane; the next
    // row is in flight while this one is used
    auto qchunk = [&](int qi) {
        return reinterpret_cast<const uint4*>(qb + static_cast<size_t>(qi) * C * sizeof(T))[c];
    };
    uint4 qv = qchunk(q0);
    // the previous row's selection and message, stored once this row's query has arrived so that
    // the wait for the query never waits for them
    size_t sel_at = 0, msg_at = 0;
    int sel_i = 0;
    float sel_k = 0.f, msg_v = 0.f;
    bool sel_pending = false, msg_pending = false;
    for (int qi = q0; qi < qend; ++qi) {
        float x = 0.f;
#pragma unroll
        for (int cc = 0; cc < CH; ++cc) {
            uint4 t;
            t.x = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(qv.x), cc * G));
            t.y = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(qv.y), cc * G));
            t.z = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(qv.z), cc * G));
            t.w = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(qv.w), cc * G));
            if constexpr (kDot2) {
                x = dot2_bf16(t.x, kraw[cc].x, x);
                x = dot2_bf16(t.y, kraw[cc].y, x);
                x = dot2_bf16(t.z, kraw[cc].z, x);
                x = dot2_bf16(t.w, kraw[cc].w, x);
            } else {
                float qf[E];
                S::unpack(t, qf);
#pragma unroll
                for (int e = 0; e < E; ++e) x += qf[e] * kf[cc * E + e];
            }
        }
        qv = qchunk(min(qi + 1, qend - 1));
        if (sel_pending) {
            a.sel_idx[sel_at] = sel_i;
            a.sel_key[sel_at] = sel_k;
        }
        if (msg_pending) a.msg[msg_at] = msg_v;
        x = valid ? x * a.scale : -INFINITY;
        const float mx = wave_max_fast(x);
        float p = valid ? __expf(x - mx) : 0.f;
        p *= fast_rcp(wave_sum_fast(p));
        if (a.K > 0) {
            const uint32_t key[1] = {valid ? ordered_bits(x) : 0u};
            const uint32_t name[1] = {static_cast<uint32_t>(lane)};
            bool sel[1];
            const int keff = a.K < N ? a.K : N;
            wave_select_top<1>(key, name, keff, sel);
            const bool kept = sel[0];
            // listed in index order through LDS, then slot o = min(lane, K - 1) written by every lane
            // (lanes past K repeat slot K - 1 with its own values)
            if (kept) {
                const int pos = lanes_below(__ballot(kept));
                sidx[wave][pos] = lane;
                skey[wave][pos] = p;
                if constexpr (VA) p = 0.f;                    // refined at the next level (Omega)
            }
            wave_lds_sync();
            const int o = min(lane, a.K - 1);
            const size_t orow = (static_cast<size_t>(bh) * N + qi) * a.K;
            const int oi = sidx[wave][min(o, kWave - 1)];
            const float ok = skey[wave][min(o, kWave - 1)];
            sel_at = orow + o;
            sel_i = o < keff ? oi : -1;
            sel_k = o < keff ? ok : 0.f;
            sel_pending = true;
        }
        pw[wave][lane] = p;
        wave_lds_sync();
        float acc[E];
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = 0.f;
#pragma unroll
        for (int u = 0; u < NV; ++u) {
            const int jj = g + u * G;
            float pj = pw[wave][jj];
            pj = jj < N ? pj : 0.f;
            float vf[E];
            S::unpack(vraw[u], vf);
#pragma unroll
            for (int e = 0; e < E; ++e) acc[e] += pj * vf[e];
        }
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = group_sum<G>(acc[e]);
        // every lane holds its chunk's sums: lane (g, c) writes channel c * E + g % E (lanes with
        // g >= E repeat a channel with the same value)
        const int ge = g % E;
        float m = acc[0];
#pragma unroll
        for (int e = 1; e < E; ++e) m = ge == e ? acc[e] : m;
        const int ch = c * E + ge;
        if (a.out) {
            float wl = 1.0f;
            if (!VA) wl = a.w ? a.w[((tok0 + qi) * a.heads + h) * a.levels] : 1.0f / a.levels;
            const float pe = a.pe0 ? a.pe0[((tok0 + qi) * a.heads + h) * D + ch] : 0.f;
            S::store1(a.out, (tok0 + qi) * C + hoff + ch, wl * (m + pe));
        } else {
            msg_at = ((tok0 + qi) * a.heads + h) * D + ch;
            msg_v = m;
            msg_pending = true;
        }
    }
    if (sel_pending) {
        a.sel_idx[sel_at] = sel_i;
        a.sel_key[sel_at] = sel_k;
    }
    if (msg_pending) a.msg[msg_at] = msg_v;
}

template <typename T, int D, bool VA>
hipError_t launch_small(const CoarseArgs& a, hipStream_t stream)
{
    // enough query rows per wave that the waves fit the chip's wave slots (at the kernel's
    // occupancy) about once
    // (the occupancy depends on the kernel and the architecture only; racing threads store the same value)
    static std::atomic<int> occupancy{0};
    int blocks_per_cu = occupancy.load(std::memory_order_relaxed);
    if (blocks_per_cu == 0) {
        int n = 0;
        hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &n, reinterpret_cast<const void*>(&coarse_small_kernel<T, D, VA>), 4 * kWave, 0);
        if (e != hipSuccess) return e;
        blocks_per_cu = n > 0 ? n : 1;
        occupancy.store(blocks_per_cu, std::memory_order_relaxed);
    }
    const long long maps = static_cast<long long>(a.B) * a.heads;
    const long long slots = static_cast<long long>(device_cu_count()) * blocks_per_cu * 4;
    long long qpw = std::min<long long>(a.N, std::max<long long>(1, (maps * a.N + slots - 1) / slots));
    while (qpw < a.N && maps * ((a.N + qpw - 1) / qpw) > slots) ++qpw;   // no partial second round
    const long long wpm = (a.N + qpw - 1) / qpw;
    qpw = (a.N + wpm - 1) / wpm;                                          // the rows spread evenly
    const long long waves = maps * wpm;
    if (waves > 0x7FFFFFFFLL - 3) return hipErrorInvalidValue;
    const long long blocks = (waves + 3) / 4;
    hipLaunchKernelGGL((coarse_small_kernel<T, D, VA>), dim3(static_cast<unsigned>(blocks)), dim3(4 * kWave), 0, stream, a,
                       static_cast<int>(qpw));
    return hipGetLastError();
}

// Query rows per workgroup of the coarse kernel (its waves, one per row in the softmax and selection
// phase). Fewer rows per workgroup spread a small map's rows over more compute units, so that the
// selection's scalar work and each phase's latency are shared by fewer rows, at the price of more
// passes over the map's keys and values (from L2) and of MFMA tiles only half filled. Measured on
// MI355X, 8 rows pay where the MFMA phases are cheapest (bf16 with d = 32: one 16-byte chunk per key
// row and k-step pair) and 16 rows elsewhere (fp32, or d = 64).
template <typename T, int D>
constexpr int coarse_rows()
{
    return (sizeof(T) == 2 && D == 32) ? 8 : 16;
}

template <typename T, int D, bool VA, int kPerLane, int Q>
hipError_t launch_rows(const CoarseArgs& a, hipStream_t stream)
{
    const size_t lds = (static_cast<size_t>(Q) * coarse_pitch(a.N) + static_cast<size_t>(Q) * 16 * 16) * sizeof(float);
    if (lds > device_max_lds()) return hipErrorInvalidValue;
    static std::atomic<unsigned long long> configured{0};     // devices whose LDS limit is raised
    if (hipError_t e = set_max_lds_once(reinterpret_cast<const void*>(&coarse_attn_kernel<T, D, VA, kPerLane, Q>), configured);
        e != hipSuccess)
        return e;
    const int tiles = (a.N + Q - 1) / Q;
    const long long blocks = static_cast<long long>(a.B) * a.heads * tiles;
    if (blocks > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((coarse_attn_kernel<T, D, VA, kPerLane, Q>), dim3(static_cast<unsigned>(blocks)), dim3(Q * kWave),
                       lds, stream, a);
    return hipGetLastError();
}

template <typename T, int D, bool VA, int kPerLane>
hipError_t launch_one(const CoarseArgs& a, hipStream_t stream)
{
    return launch_rows<T, D, VA, kPerLane, coarse_rows<T, D>()>(a, stream);
}

template <typename T, int D, bool VA>
hipError_t launch_per_lane(const CoarseArgs& a, hipStream_t stream)
{
    if (a.N <= kWave) {
        if (a.pe_w) return hipErrorInvalidValue;       // the small-map kernel has no fused position encoding
        return launch_small<T, D, VA>(a, stream);
    }
    switch (coarse_per_lane(a.N)) {
    case 1: return launch_one<T, D, VA, 1>(a, stream);
    case 2: return launch_one<T, D, VA, 2>(a, stream);
    case 3: return launch_one<T, D, VA, 3>(a, stream);
    case 4: return launch_one<T, D, VA, 4>(a, stream);
    case 5: return launch_one<T, D, VA, 5>(a, stream);
    case 6: return launch_one<T, D, VA, 6>(a, stream);
    case 8: return launch_one<T, D, VA, 8>(a, stream);
    case 12: return launch_one<T, D, VA, 12>(a, stream);
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
