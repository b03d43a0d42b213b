// Step 1: token pyramids by 2x2 average pooling (Sec. 3.2, pyramid paragraph).
//
// One pass produces up to two coarser levels from a source level. A thread owns one 16-byte
// channel chunk of one token of the top level it produces: it issues the 16-byte loads of that
// token's (up to) 4x4 source tokens all at once (consecutive threads take consecutive chunks of a
// token, so a wave reads whole rows; addresses past the map's edge are clamped onto it and the
// values ignored), writes the (up to) four intermediate tokens, then pools those rounded values
// again for the top token. Two levels per pass read each map once; deeper pyramids take more
// passes. Each level is written NHWC or parent-blocked as asked.
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

}  // namespace

hipError_t launch_pyramid_pass(const PyramidPassArgs& a, int nlev, int ntensors, bool use_bf16, hipStream_t stream)
{
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
