// Step 1: token pyramids by 2x2 average pooling (Sec. 3.2, pyramid paragraph).
//
// One pass produces up to two coarser levels from a source level. In the two-level pass a
// workgroup owns whole top-level tokens: one thread per 16-byte channel chunk of each of their four
// level-1 children loads that child's 2x2 source chunks (consecutive threads take consecutive
// chunks of a token, so a wave reads whole rows; addresses past the map's edge are clamped onto
// it and the values ignored), writes the level-1 token and stages it in LDS; after a barrier one
// thread in four pools the staged children again for the top token. Tokens too wide for one
// workgroup take the older path in which one thread owns a top-token chunk and loads all 4x4
// source chunks. Deeper pyramids take more passes. Each level is written NHWC or parent-blocked
// as asked.
//
// Arithmetic, fixed so that every implementation stores the same bits: the valid children are
// summed in fp32 as ((c00 + c01) + (c10 + c11)) with missing children left out, multiplied by
// 1/count (a power of two, exact) and rounded to the storage type, nearest-even.
#include "qta_device.h"
#include "qta_internal.h"

namespace qta {

namespace {

template <int E>
__device__ __forceinline__ void pool_children(const float (&c00)[E], const float (&c01)[E], const float (&c10)[E],
                                              const float (&c11)[E], bool right, bool below, float (&out)[E])
{
#pragma clang fp contract(off)
    const float inv = (right && below) ? 0.25f : ((right || below) ? 0.5f : 1.0f);
#pragma unroll
    for (int e = 0; e < E; ++e) {
        float row0 = c00[e];
        if (right) row0 = row0 + c01[e];
        float s = row0;
        if (below) {
            float row1 = c10[e];
            if (right) row1 = row1 + c11[e];
            s = row0 + row1;
        }
        out[e] = s * inv;
    }
}

template <typename T, int NLEV>
__global__ __launch_bounds__(256) void pyramid_pass_kernel(PyramidPassArgs a)
{
    using S = Storage<T>;
    constexpr int E = S::kPer16B;
    constexpr int R = NLEV == 2 ? 4 : 2;                // source rows / columns under one top token
    const int tensor = blockIdx.y;
    const char* __restrict__ src = static_cast<const char*>(a.src[tensor]);
    char* __restrict__ dst1 = static_cast<char*>(a.dst1[tensor]);
    char* __restrict__ dst2 = static_cast<char*>(a.dst2[tensor]);
    const int chunks = a.chunks;                       // 16-byte chunks per token
    const int Ht = NLEV == 2 ? a.H2 : a.H1;
    const int Wt = NLEV == 2 ? a.W2 : a.W1;
    const long long total = static_cast<long long>(a.B) * Ht * Wt * chunks;
    const long long tid = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (tid >= total) return;
    const int ch = static_cast<int>(tid % chunks);
    long long tok = tid / chunks;
    const int X = static_cast<int>(tok % Wt);
    tok /= Wt;
    const int Y = static_cast<int>(tok % Ht);
    const int b = static_cast<int>(tok / Ht);

    // every source chunk under (Y, X), loaded before any is used
    uint4 raw[R][R];
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int y = min(R * Y + i, a.Hs - 1);
#pragma unroll
        for (int j = 0; j < R; ++j) {
            const int x = min(R * X + j, a.Ws - 1);
            raw[i][j] = *reinterpret_cast<const uint4*>(
                src + chunk_offset(a.src_blocked, b, y, x, a.Hs, a.Ws, ch, chunks, a.head_chunks));
        }
    }
    auto store = [&](char* base, bool blocked, int H, int W, int y, int x, const float (&v)[E]) {
        *reinterpret_cast<uint4*>(base + chunk_offset(blocked, b, y, x, H, W, ch, chunks, a.head_chunks)) = S::pack(v);
    };
    // pool the 2x2 source block whose top-left is (i0, j0) of raw into level-1 token (y1, x1)
    auto pool1 = [&](int i0, int j0, int y1, int x1, float (&o)[E]) {
        const bool right = 2 * x1 + 1 < a.Ws, below = 2 * y1 + 1 < a.Hs;
        float c00[E], c01[E], c10[E], c11[E];
        S::unpack(raw[i0][j0], c00);
        S::unpack(raw[i0][j0 + 1], c01);
        S::unpack(raw[i0 + 1][j0], c10);
        S::unpack(raw[i0 + 1][j0 + 1], c11);
        pool_children<E>(c00, c01, c10, c11, right, below, o);
#pragma unroll
        for (int e = 0; e < E; ++e) o[e] = S::round(o[e]);
    };

    if constexpr (NLEV == 1) {
        float o[E];
        pool1(0, 0, Y, X, o);
        store(dst1, a.dst1_blocked, a.H1, a.W1, Y, X, o);
    } else {
        // the four level-1 children of (Y, X), each pooled from its own source children
        float mid[4][E];
        bool mid_ok[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int y1 = 2 * Y + (q >> 1), x1 = 2 * X + (q & 1);
            mid_ok[q] = y1 < a.H1 && x1 < a.W1;
            pool1(2 * (q >> 1), 2 * (q & 1), y1, x1, mid[q]);
            if (mid_ok[q]) store(dst1, a.dst1_blocked, a.H1, a.W1, y1, x1, mid[q]);
        }
        float o[E];
        pool_children<E>(mid[0], mid[1], mid[2], mid[3], mid_ok[1], mid_ok[2], o);
#pragma unroll
        for (int e = 0; e < E; ++e) o[e] = S::round(o[e]);
        store(dst2, a.dst2_blocked, a.H2, a.W2, Y, X, o);
    }
}

// Two-level pass, workgroup = tpb top tokens x 4 children x `chunks` chunks (at most 256 threads).
// ROW (maps of one row): a token has two children, so tpb top tokens x 2 children x `chunks`.
template <typename T, bool ROW>
__global__ __launch_bounds__(256) void pyramid_pass2_kernel(PyramidPassArgs a, int tpb)
{
    using S = Storage<T>;
    constexpr int E = S::kPer16B;
    constexpr int NC = ROW ? 2 : 4;                    // children of a token
    __shared__ uint4 stage[256];
    const int tensor = blockIdx.y;
    const char* __restrict__ src = static_cast<const char*>(a.src[tensor]);
    char* __restrict__ dst1 = static_cast<char*>(a.dst1[tensor]);
    char* __restrict__ dst2 = static_cast<char*>(a.dst2[tensor]);
    const int chunks = a.chunks;
    const int li = threadIdx.x;
    const int ch = li % chunks;
    const int q = (li / chunks) % NC;
    const int t = li / (NC * chunks);
    const long long ntop = static_cast<long long>(a.B) * a.H2 * a.W2;
    const long long top = static_cast<long long>(blockIdx.x) * tpb + t;
    const bool active = top < ntop;                    // inactive threads still reach the barrier
    const long long topc = active ? top : ntop - 1;
    const int X = static_cast<int>(topc % a.W2);
    const int Y = static_cast<int>((topc / a.W2) % a.H2);
    const int b = static_cast<int>(topc / (static_cast<long long>(a.W2) * a.H2));

    const int y1 = ROW ? 0 : 2 * Y + (q >> 1), x1 = 2 * X + (q & 1);
    const bool mid_ok = y1 < a.H1 && x1 < a.W1;
    uint4 raw[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        if (ROW && i == 1) {                               // no row below
            raw[1][0] = raw[0][0];
            raw[1][1] = raw[0][1];
            break;
        }
        const int y = min(2 * y1 + i, a.Hs - 1);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int x = min(2 * x1 + j, a.Ws - 1);
            raw[i][j] = *reinterpret_cast<const uint4*>(
                src + chunk_offset(a.src_blocked, b, y, x, a.Hs, a.Ws, ch, chunks, a.head_chunks));
        }
    }
    float c00[E], c01[E], c10[E], c11[E], mid[E];
    S::unpack(raw[0][0], c00);
    S::unpack(raw[0][1], c01);
    S::unpack(raw[1][0], c10);
    S::unpack(raw[1][1], c11);
    pool_children<E>(c00, c01, c10, c11, 2 * x1 + 1 < a.Ws, 2 * y1 + 1 < a.Hs, mid);
#pragma unroll
    for (int e = 0; e < E; ++e) mid[e] = S::round(mid[e]);
    const uint4 packed = S::pack(mid);
    if (active && mid_ok)
        *reinterpret_cast<uint4*>(dst1 + chunk_offset(a.dst1_blocked, b, y1, x1, a.H1, a.W1, ch, chunks,
                                                      a.head_chunks)) = packed;
    stage[li] = packed;
    __syncthreads();
    if (!active || q != 0) return;
    const int base = t * NC * chunks + ch;
    float m0[E], m1[E], m2[E], m3[E], o[E];
    S::unpack(stage[base], m0);
    S::unpack(stage[base + chunks], m1);
    S::unpack(stage[base + (ROW ? 0 : 2) * chunks], m2);   // ROW: unused (no row below)
    S::unpack(stage[base + (ROW ? 1 : 3) * chunks], m3);
    pool_children<E>(m0, m1, m2, m3, 2 * X + 1 < a.W1, 2 * Y + 1 < a.H1, o);
#pragma unroll
    for (int e = 0; e < E; ++e) o[e] = S::round(o[e]);
    *reinterpret_cast<uint4*>(dst2 + chunk_offset(a.dst2_blocked, b, Y, X, a.H2, a.W2, ch, chunks, a.head_chunks)) =
        S::pack(o);
}

// Three- or four-level pass (NLEV), workgroup = tpb top tokens (level s+NLEV). A unit is one
// 16-byte chunk of one level-1 token under a top token (NC^(NLEV-1) level-1 tokens each); a thread
// takes units tid, tid + 256, ... (at most R), loads the 2x2 source chunks of all of them before
// pooling any, writes the level-1 tokens and stages them in LDS; after each barrier the threads pool
// the staged tokens of one level into the next (written and staged again), up to the top tokens.
// Staged tokens are in hierarchical order (top token, then the child index at each level below
// it), so the NC children of staged token i of one level are tokens NC*i .. NC*i + NC-1 of the level
// below. ROW (maps of one row): two children per token, as in the two-level pass.
template <typename T, bool ROW, int R, int NLEV>
__global__ __launch_bounds__(256) void pyramid_passn_kernel(PyramidPassArgs a, int tpb)
{
    static_assert(NLEV == 3 || NLEV == 4, "three- or four-level pass");
    using S = Storage<T>;
    constexpr int E = S::kPer16B;
    constexpr int NC = ROW ? 2 : 4;
    constexpr int LNC = ROW ? 1 : 2;                   // log2(NC)
    __shared__ uint4 stage1[256 * R];
    __shared__ uint4 stage2[256 * R / NC];
    __shared__ uint4 stage3[NLEV == 4 ? 256 * R / (NC * NC) : 1];
    const int tensor = blockIdx.y;
    const char* __restrict__ src = static_cast<const char*>(a.src[tensor]);
    const int chunks = a.chunks;
    const int L1 = 1 << (LNC * (NLEV - 1));            // level-1 tokens under one top token
    const int U = L1 * chunks;                         // units of one top token
    const int nunits = tpb * U;
    const int Ht = NLEV == 4 ? a.H4 : a.H3, Wt = NLEV == 4 ? a.W4 : a.W3;
    const int ntop = a.B * Ht * Wt;                    // < 2^31, checked by the launcher
    const int top0 = static_cast<int>(blockIdx.x) * tpb;
    // level j's map, destination and layout (j = 1 .. NLEV, compile-time after unrolling)
    auto lvl_H = [&](int j) { return j == 1 ? a.H1 : j == 2 ? a.H2 : j == 3 ? a.H3 : a.H4; };
    auto lvl_W = [&](int j) { return j == 1 ? a.W1 : j == 2 ? a.W2 : j == 3 ? a.W3 : a.W4; };
    auto lvl_dst = [&](int j) {
        return static_cast<char*>(j == 1 ? a.dst1[tensor] : j == 2 ? a.dst2[tensor] : j == 3 ? a.dst3[tensor]
                                                                                                : a.dst4[tensor]);
    };
    auto lvl_blocked = [&](int j) {
        return j == 1 ? a.dst1_blocked : j == 2 ? a.dst2_blocked : j == 3 ? a.dst3_blocked : a.dst4_blocked;
    };
    // (b, y, x) at level j of staged token `tok` of that level (hierarchical order); the top token is
    // clamped onto the last one past the end. Returns whether the top token exists.
    auto level_pos = [&](int j, int tok, int& b, int& y, int& x) {
        const int sh = LNC * (NLEV - j);               // child digits below the top token
        const int t = tok >> sh;
        const int top = min(top0 + t, ntop - 1);
        x = top % Wt;
        y = (top / Wt) % Ht;
        b = top / (Wt * Ht);
#pragma unroll
        for (int k = NLEV - j - 1; k >= 0; --k) {
            const int q = (tok >> (LNC * k)) & (NC - 1);
            y = ROW ? 0 : 2 * y + (q >> 1);
            x = 2 * x + (ROW ? q : (q & 1));
        }
        return top0 + t < ntop;
    };

    int b1[R], y1[R], x1[R], ch1[R];
    bool ok1[R];
    uint4 raw[R][2][2];
#pragma unroll
    for (int it = 0; it < R; ++it) {
        const int u0 = it * 256 + static_cast<int>(threadIdx.x);
        const int u = min(u0, nunits - 1);
        const int tok = u / chunks;
        ch1[it] = u - tok * chunks;
        const bool top_ok = level_pos(1, tok, b1[it], y1[it], x1[it]);
        ok1[it] = u0 < nunits && top_ok && y1[it] < a.H1 && x1[it] < a.W1;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            if (ROW && i == 1) {                           // no row below
                raw[it][1][0] = raw[it][0][0];
                raw[it][1][1] = raw[it][0][1];
                break;
            }
            const int y = min(2 * y1[it] + i, a.Hs - 1);
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int x = min(2 * x1[it] + j, a.Ws - 1);
                raw[it][i][j] = *reinterpret_cast<const uint4*>(
                    src + chunk_offset(a.src_blocked, b1[it], y, x, a.Hs, a.Ws, ch1[it], chunks, a.head_chunks));
            }
        }
    }
    char* __restrict__ dst1 = lvl_dst(1);
#pragma unroll
    for (int it = 0; it < R; ++it) {
        float c00[E], c01[E], c10[E], c11[E], mid[E];
        S::unpack(raw[it][0][0], c00);
        S::unpack(raw[it][0][1], c01);
        S::unpack(raw[it][1][0], c10);
        S::unpack(raw[it][1][1], c11);
        pool_children<E>(c00, c01, c10, c11, 2 * x1[it] + 1 < a.Ws, !ROW && 2 * y1[it] + 1 < a.Hs, mid);
#pragma unroll
        for (int e = 0; e < E; ++e) mid[e] = S::round(mid[e]);
        const uint4 packed = S::pack(mid);
        if (ok1[it])
            *reinterpret_cast<uint4*>(dst1 + chunk_offset(a.dst1_blocked, b1[it], y1[it], x1[it], a.H1, a.W1,
                                                          ch1[it], chunks, a.head_chunks)) = packed;
        stage1[it * 256 + threadIdx.x] = packed;
    }

    // levels 2 .. NLEV: one unit per (staged token, chunk), its children staged at
    // (NC * tok + q) * chunks + ch one level below
#pragma unroll
    for (int j = 2; j <= NLEV; ++j) {
        __syncthreads();
        const uint4* below = j == 2 ? stage1 : j == 3 ? stage2 : stage3;
        uint4* here = j == 2 ? stage2 : stage3;          // (the top level is not staged)
        const int n = (tpb << (LNC * (NLEV - j))) * chunks;
        const int Hb = lvl_H(j - 1), Wb = lvl_W(j - 1), Hj = lvl_H(j), Wj = lvl_W(j);
        char* __restrict__ dst = lvl_dst(j);
        const bool blk = lvl_blocked(j);
        for (int u = threadIdx.x; u < n; u += 256) {
            const int tok = u / chunks, ch = u - tok * chunks;
            int b, y, x;
            const bool top_ok = level_pos(j, tok, b, y, x);
            const int base = NC * tok * chunks + ch;
            float m0[E], m1[E], m2[E], m3[E], o[E];
            S::unpack(below[base], m0);
            S::unpack(below[base + chunks], m1);
            S::unpack(below[base + (ROW ? 0 : 2) * chunks], m2);   // ROW: unused (no row below)
            S::unpack(below[base + (ROW ? 1 : 3) * chunks], m3);
            pool_children<E>(m0, m1, m2, m3, 2 * x + 1 < Wb, !ROW && 2 * y + 1 < Hb, o);
#pragma unroll
            for (int e = 0; e < E; ++e) o[e] = S::round(o[e]);
            const uint4 packed = S::pack(o);
            if (top_ok && y < Hj && x < Wj)
                *reinterpret_cast<uint4*>(dst + chunk_offset(blk, b, y, x, Hj, Wj, ch, chunks, a.head_chunks)) = packed;
            if (j < NLEV) here[u] = packed;
        }
    }
}

}  // namespace

template <typename T, bool ROW, int NLEV>
static hipError_t launch_passn(const PyramidPassArgs& a, int ntensors, hipStream_t stream)
{
    const int U = (1 << ((ROW ? 1 : 2) * (NLEV - 1))) * a.chunks;
    const int tpb = U >= 256 ? 1 : 256 / U;
    const int R = (tpb * U + 255) / 256;
    const long long ntop = static_cast<long long>(a.B) * (NLEV == 4 ? a.H4 : a.H3) * (NLEV == 4 ? a.W4 : a.W3);
    if (ntop <= 0 || ntop > 0x7FFFFFFFLL || R > 4) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>((ntop + tpb - 1) / tpb), ntensors);
    if (R == 1) hipLaunchKernelGGL((pyramid_passn_kernel<T, ROW, 1, NLEV>), grid, dim3(256), 0, stream, a, tpb);
    else if (R == 2) hipLaunchKernelGGL((pyramid_passn_kernel<T, ROW, 2, NLEV>), grid, dim3(256), 0, stream, a, tpb);
    else hipLaunchKernelGGL((pyramid_passn_kernel<T, ROW, 4, NLEV>), grid, dim3(256), 0, stream, a, tpb);
    return hipGetLastError();
}

hipError_t launch_pyramid_pass(const PyramidPassArgs& a, int nlev, int ntensors, bool use_bf16, hipStream_t stream)
{
    if (nlev == 3 || nlev == 4) {
        const bool row = a.Hs == 1;
        if (!pyramid_passn_fits(nlev, a.chunks, row)) return hipErrorInvalidValue;
        if (nlev == 3) {
            if (use_bf16) return row ? launch_passn<bf16, true, 3>(a, ntensors, stream) : launch_passn<bf16, false, 3>(a, ntensors, stream);
            return row ? launch_passn<float, true, 3>(a, ntensors, stream) : launch_passn<float, false, 3>(a, ntensors, stream);
        }
        if (use_bf16) return row ? launch_passn<bf16, true, 4>(a, ntensors, stream) : launch_passn<bf16, false, 4>(a, ntensors, stream);
        return row ? launch_passn<float, true, 4>(a, ntensors, stream) : launch_passn<float, false, 4>(a, ntensors, stream);
    }
    if (nlev == 2 && 4 * a.chunks <= 256) {
        const bool row = a.Hs == 1;                       // maps of one row: two children per token
        const int nc = row ? 2 : 4;
        const int tpb = 256 / (nc * a.chunks);
        const long long ntop = static_cast<long long>(a.B) * a.H2 * a.W2;
        const long long blocks = (ntop + tpb - 1) / tpb;
        if (blocks > 0x7FFFFFFFLL) return hipErrorInvalidValue;
        dim3 grid(static_cast<unsigned>(blocks), ntensors);
        const dim3 block(tpb * nc * a.chunks);
        if (use_bf16) {
            if (row) hipLaunchKernelGGL((pyramid_pass2_kernel<bf16, true>), grid, block, 0, stream, a, tpb);
            else hipLaunchKernelGGL((pyramid_pass2_kernel<bf16, false>), grid, block, 0, stream, a, tpb);
        } else {
            if (row) hipLaunchKernelGGL((pyramid_pass2_kernel<float, true>), grid, block, 0, stream, a, tpb);
            else hipLaunchKernelGGL((pyramid_pass2_kernel<float, false>), grid, block, 0, stream, a, tpb);
        }
        return hipGetLastError();
    }
    const int Ht = nlev == 2 ? a.H2 : a.H1, Wt = nlev == 2 ? a.W2 : a.W1;
    const long long total = static_cast<long long>(a.B) * Ht * Wt * a.chunks;
    const int threads = 256;
    const long long blocks = (total + threads - 1) / threads;
    if (blocks > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    dim3 grid(static_cast<unsigned>(blocks), ntensors);
    if (use_bf16) {
        if (nlev == 2) hipLaunchKernelGGL((pyramid_pass_kernel<bf16, 2>), grid, dim3(threads), 0, stream, a);
        else hipLaunchKernelGGL((pyramid_pass_kernel<bf16, 1>), grid, dim3(threads), 0, stream, a);
    } else {
        if (nlev == 2) hipLaunchKernelGGL((pyramid_pass_kernel<float, 2>), grid, dim3(threads), 0, stream, a);
        else hipLaunchKernelGGL((pyramid_pass_kernel<float, 1>), grid, dim3(threads), 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace qta
