// Step 1: token pyramids by 2x2 average pooling (Sec. 3.2, pyramid paragraph).
//
// One pass produces two to four coarser levels from a source level (pyramid_tree_kernel): a
// workgroup owns a few top-level tokens of one row; threads are (16-byte chunk, token) pairs, so a
// wave reads whole tokens, and each loads the 2x2 source chunks of its level-1 tokens (addresses
// past the map's edge clamped onto it, values ignored), writes them and stages them in LDS; after a
// barrier per level the coarser levels are pooled from LDS. Tokens too wide to stage take the older
// path (pyramid_pass_kernel) in which one thread owns a chunk of a level-1 or level-2 token and
// loads all of its source chunks. Deeper pyramids take more passes. Each level is written NHWC or
// parent-blocked as asked.
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

// Bits of a hierarchical child index: digit k (the finest first) of `tok`, LNC bits each, gives
// bit k of the token's row and column offsets under its ancestor nd levels up (for a 2D map the
// digit's high bit is the row bit; a map of one row has one column bit per digit).
template <bool ROW>
__device__ __forceinline__ void child_offsets(int tok, int nd, int& dy, int& dx)
{
    if constexpr (ROW) {
        dy = 0;
        dx = tok & ((1 << nd) - 1);
    } else {
        dy = 0;
        dx = 0;
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            if (k >= nd) break;
            dx |= ((tok >> (2 * k)) & 1) << k;
            dy |= ((tok >> (2 * k + 1)) & 1) << k;
        }
    }
}

// Pass over NLEV = 2, 3 or 4 levels. A workgroup owns tpb consecutive top-level tokens (level
// s + NLEV) of one row of one batch element and tensor (grid: column block, row, batch x tensor);
// its threads are (chunk, token): thread (c, t) takes chunk c of level-1 tokens t, t + by, ... (at
// most R), loads the 2x2 source chunks of all of them before pooling any, writes the level-1 tokens
// and stages them in LDS; after each barrier the threads pool the staged tokens of one level into
// the next (written and staged again), up to the top tokens. Staged tokens are in hierarchical
// order (top token, then the child index at each level below it), so the NC children of staged
// token i of one level are tokens NC*i .. NC*i + NC-1 of the level below. Every index is a shift,
// a mask or a 24-bit product: the grid gives the top token's coordinates, the thread its chunk,
// and a token's position under its top token is read off the bits of its staged index. Offsets
// are 32-bit within one batch element's map (the launcher checks the sizes). ROW (maps of one
// row): two children per token.
template <typename T, bool ROW, int NLEV, int R>
__global__ __launch_bounds__(1024) void pyramid_tree_kernel(PyramidPassArgs a, int tpb, int ntensors)
{
    static_assert(NLEV >= 2 && NLEV <= 4, "two- to four-level pass");
    using S = Storage<T>;
    constexpr int E = S::kPer16B;
    constexpr int NC = ROW ? 2 : 4;
    constexpr int LNC = ROW ? 1 : 2;                    // log2(NC)
    __shared__ uint4 stage1[kPyramidStage];
    __shared__ uint4 stage2[NLEV >= 3 ? kPyramidStage / NC : 1];
    __shared__ uint4 stage3[NLEV == 4 ? kPyramidStage / (NC * NC) : 1];
    const int ch = threadIdx.x, ty = threadIdx.y, by = blockDim.y;
    const int chunks = a.chunks;
    const int z = blockIdx.z;
    const int b = z / ntensors, tensor = z - b * ntensors;   // uniform
    const int Y = blockIdx.y, X0 = blockIdx.x * tpb;         // first top token of the workgroup
    const uint32_t tok_bytes = static_cast<uint32_t>(chunks) * 16u;
    const int lgh = a.lg_head_chunks;                        // blocked layouts: head and chunk in head
    const uint32_t head = static_cast<uint32_t>(ch) >> lgh, in_head = static_cast<uint32_t>(ch) & ((1u << lgh) - 1u);
    // byte offset of this thread's chunk of token (y, x) within one batch element's H x W map
    auto offset = [&](bool blocked, int H, int W, int y, int x) -> uint32_t {
        if (!blocked) return __umul24(__umul24(y, W) + x, tok_bytes) + ch * 16u;
        const uint32_t Hp = (H + 1) >> 1, Wp = (W + 1) >> 1;
        const uint32_t blk = __umul24(__umul24(head, Hp) + (y >> 1), Wp) + (x >> 1);
        return ((blk * 4u + ((y & 1) * 2 + (x & 1))) << (lgh + 4)) + in_head * 16u;
    };
    auto batch_base = [&](const void* p, bool blocked, int H, int W) {
        const size_t n = blocked ? static_cast<size_t>((H + 1) >> 1) * ((W + 1) >> 1) * 4 : static_cast<size_t>(H) * W;
        return static_cast<const char*>(p) + b * n * tok_bytes;
    };
    auto lvl_H = [&](int j) { return j == 0 ? a.Hs : j == 1 ? a.H1 : j == 2 ? a.H2 : j == 3 ? a.H3 : a.H4; };
    auto lvl_W = [&](int j) { return j == 0 ? a.Ws : j == 1 ? a.W1 : j == 2 ? a.W2 : j == 3 ? a.W3 : a.W4; };
    auto lvl_dst = [&](int j) {
        return j == 1 ? a.dst1[tensor] : j == 2 ? a.dst2[tensor] : j == 3 ? a.dst3[tensor] : a.dst4[tensor];
    };
    auto lvl_blocked = [&](int j) {
        return j == 1 ? a.dst1_blocked : j == 2 ? a.dst2_blocked : j == 3 ? a.dst3_blocked : a.dst4_blocked;
    };

    // level 1 from the source
    constexpr int ND1 = NLEV - 1;                       // child digits of a level-1 token
    const int ntok1 = tpb << (LNC * ND1);
    const char* src = batch_base(a.src[tensor], a.src_blocked, a.Hs, a.Ws);
    int y1[R], x1[R];
    uint4 raw[R][2][2];
#pragma unroll
    for (int it = 0; it < R; ++it) {
        const int tk = min(ty + it * by, ntok1 - 1);
        int dy, dx;
        child_offsets<ROW>(tk, ND1, dy, dx);
        y1[it] = (Y << ND1) + dy;
        x1[it] = ((X0 + (tk >> (LNC * ND1))) << ND1) + dx;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            if (ROW && i == 1) {                           // no row below
                raw[it][1][0] = raw[it][0][0];
                raw[it][1][1] = raw[it][0][1];
                break;
            }
            const int y = min(2 * y1[it] + i, a.Hs - 1);  // clamped onto the map; values ignored
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int x = min(2 * x1[it] + j, a.Ws - 1);
                raw[it][i][j] = load_at<uint4>(src, offset(a.src_blocked, a.Hs, a.Ws, y, x));
            }
        }
    }
    {
        char* dst = const_cast<char*>(batch_base(a.dst1[tensor], a.dst1_blocked, a.H1, a.W1));
#pragma unroll
        for (int it = 0; it < R; ++it) {
            // rows past the last token repeat it (same loads, same value, same staging slot), so the
            // pooling and the staging are unconditional: a pooling under a branch leaves the loads
            // pending on the path that skips it, and the compiler then makes the next level wait for
            // every outstanding memory operation, the global stores of this level included
            const int tk = min(ty + it * by, ntok1 - 1);
            float c00[E], c01[E], c10[E], c11[E], mid[E];
            S::unpack(raw[it][0][0], c00);
            S::unpack(raw[it][0][1], c01);
            S::unpack(raw[it][1][0], c10);
            S::unpack(raw[it][1][1], c11);
            pool_children<E>(c00, c01, c10, c11, 2 * x1[it] + 1 < a.Ws, !ROW && 2 * y1[it] + 1 < a.Hs, mid);
            const uint4 packed = S::pack(mid);               // rounds to the storage type
            stage1[tk * chunks + ch] = packed;
            if (y1[it] < a.H1 && x1[it] < a.W1)
                store_at<uint4>(dst, offset(a.dst1_blocked, a.H1, a.W1, y1[it], x1[it]), packed);
        }
    }

    // levels 2 .. NLEV from the staged level below
#pragma unroll
    for (int j = 2; j <= NLEV; ++j) {
        __syncthreads();
        const uint4* below = j == 2 ? stage1 : j == 3 ? stage2 : stage3;
        uint4* here = j == 2 ? stage2 : stage3;          // (the top level is not staged)
        const int nd = NLEV - j;                         // child digits of a level-j token
        const int ntok = tpb << (LNC * nd);
        const int Hb = lvl_H(j - 1), Wb = lvl_W(j - 1), Hj = lvl_H(j), Wj = lvl_W(j);
        const bool blk = lvl_blocked(j);
        char* dst = const_cast<char*>(batch_base(lvl_dst(j), blk, Hj, Wj));
        for (int tk = ty; tk < ntok; tk += by) {
            int dy, dx;
            child_offsets<ROW>(tk, nd, dy, dx);
            const int y = (Y << nd) + dy, x = ((X0 + (tk >> (LNC * nd))) << nd) + dx;
            const int base = tk * NC * chunks + ch;
            float m0[E], m1[E], m2[E], m3[E], o[E];
            S::unpack(below[base], m0);
            S::unpack(below[base + chunks], m1);
            S::unpack(below[base + (ROW ? 0 : 2) * chunks], m2);   // ROW: unused (no row below)
            S::unpack(below[base + (ROW ? 1 : 3) * chunks], m3);
            pool_children<E>(m0, m1, m2, m3, 2 * x + 1 < Wb, !ROW && 2 * y + 1 < Hb, o);
            const uint4 packed = S::pack(o);
            if (y < Hj && x < Wj) store_at<uint4>(dst, offset(blk, Hj, Wj, y, x), packed);
            if (j < NLEV) here[tk * chunks + ch] = packed;
        }
    }
}

}  // namespace

template <typename T, bool ROW, int NLEV>
static hipError_t launch_tree(const PyramidPassArgs& a, int ntensors, hipStream_t stream)
{
    const PyramidTreeShape g = pyramid_tree_shape(NLEV, a.chunks, ROW);
    if (!g.ok) return hipErrorInvalidValue;
    const int Ht = NLEV == 2 ? a.H2 : NLEV == 3 ? a.H3 : a.H4, Wt = NLEV == 2 ? a.W2 : NLEV == 3 ? a.W3 : a.W4;
    const long long gx = (Wt + g.tpb - 1) / g.tpb, gz = static_cast<long long>(a.B) * ntensors;
    if (Ht <= 0 || Wt <= 0 || Ht > 65535 || gz > 65535 || gx > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(gx), static_cast<unsigned>(Ht), static_cast<unsigned>(gz));
    const dim3 block(a.chunks, g.by);
    if (g.R == 1) hipLaunchKernelGGL((pyramid_tree_kernel<T, ROW, NLEV, 1>), grid, block, 0, stream, a, g.tpb, ntensors);
    else if (g.R == 2) hipLaunchKernelGGL((pyramid_tree_kernel<T, ROW, NLEV, 2>), grid, block, 0, stream, a, g.tpb, ntensors);
    else hipLaunchKernelGGL((pyramid_tree_kernel<T, ROW, NLEV, 4>), grid, block, 0, stream, a, g.tpb, ntensors);
    return hipGetLastError();
}

template <typename T, bool ROW>
static hipError_t launch_tree_n(const PyramidPassArgs& a, int nlev, int ntensors, hipStream_t stream)
{
    if (nlev == 2) return launch_tree<T, ROW, 2>(a, ntensors, stream);
    if (nlev == 3) return launch_tree<T, ROW, 3>(a, ntensors, stream);
    return launch_tree<T, ROW, 4>(a, ntensors, stream);
}


hipError_t launch_pyramid_pass(const PyramidPassArgs& a, int nlev, int ntensors, bool use_bf16, hipStream_t stream)
{
    const bool row = a.Hs == 1;                           // maps of one row: two children per token
    if (nlev >= 2 && nlev <= 4 && pyramid_tree_fits(nlev, a.chunks, a.head_chunks, row, a.Hs, a.Ws)) {
        if (use_bf16) return row ? launch_tree_n<bf16, true>(a, nlev, ntensors, stream) : launch_tree_n<bf16, false>(a, nlev, ntensors, stream);
        return row ? launch_tree_n<float, true>(a, nlev, ntensors, stream) : launch_tree_n<float, false>(a, nlev, ntensors, stream);
    }
    if (nlev > 2) return hipErrorInvalidValue;
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
