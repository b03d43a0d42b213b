// Multiscale position encoding (Sec. 3.2, after the locally-enhanced positional encoding the paper
// adopts): at every level an unshared 3x3 depth-wise convolution of V^l, zero outside the map,
// plus a bias. Levels above 0 add it to their message in place; level 0 writes it to a buffer that
// the finest kernel adds to m0 before the levels are combined.
//
// One launch covers every level: a thread owns four channels of four neighbouring tokens of one row
// of one level and reads their 3x6 window once (8- or 16-byte loads; neighbouring threads take the
// other channels of the same tokens), so the encoding costs about one pass over each V level and
// one read-modify-write of each message.
#include <type_traits>

#include "qta_device.h"
#include "qta_internal.h"

namespace qta {

namespace {

// Element offset of channel c of head h of token (y, x) in a level of H x W tokens.
__device__ __forceinline__ size_t elem_offset(bool blocked, int b, int y, int x, int H, int W, int h, int c,
                                              int heads, int d)
{
    if (!blocked) return ((static_cast<size_t>(b) * H + y) * W + x) * heads * d + static_cast<size_t>(h) * d + c;
    const int Hp = (H + 1) / 2, Wp = (W + 1) / 2;
    const size_t blk = ((static_cast<size_t>(b) * heads + h) * Hp + (y >> 1)) * Wp + (x >> 1);
    return (blk * 4 + (y & 1) * 2 + (x & 1)) * d + c;
}

constexpr int kTX = 4;            // tokens along x per thread (their 3x3 windows share columns)
constexpr int kThreads = 256;

// Four consecutive channels of one token as fp32 (one 16-byte fp32 or 8-byte bf16 load).
template <typename T>
__device__ __forceinline__ float4 load4(const void* base, size_t elem)
{
    if constexpr (sizeof(T) == 4) {
        return *reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
    } else {
        const uint2 u = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(base) + elem);
        return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                           __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
    }
}

template <typename T>
__global__ __launch_bounds__(kThreads) void posenc_kernel(PosEncArgs a)
{
    const long long item = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (item >= a.start[a.nlev]) return;
    int l = 0;
    while (item >= a.start[l + 1]) ++l;
    if (item >= a.level_end[l]) return;              // padding between levels
    const PosEncLevel& L = a.lv[l];
    const int C = a.heads * a.d, groups = C / 4;
    const int xtiles = (L.W + kTX - 1) / kTX;
    // within a level the item index fits 32 bits (the launcher checks)
    int r = static_cast<int>(item - a.start[l]);
    const int g = r % groups;
    r /= groups;
    const int x0 = (r % xtiles) * kTX;
    r /= xtiles;
    const int y = r % L.H;
    const int b = r / L.H;
    const int c0 = 4 * g, h = c0 / a.d, c = c0 - h * a.d;
    // every load first: the 3 x (kTX+2) window at clamped (in-bounds) positions, masked when used,
    // so that they are all in flight at once; then the 36 weights of these four channels
    // (contiguous, [C][3][3])
    using Raw = typename std::conditional<sizeof(T) == 4, float4, uint2>::type;
    Raw win[3][kTX + 2];
    bool ok[3][kTX + 2];
#pragma unroll
    for (int ky = 0; ky < 3; ++ky) {
        const int yy = y + ky - 1;
        const int yc = min(max(yy, 0), L.H - 1);
#pragma unroll
        for (int j = 0; j < kTX + 2; ++j) {
            const int xx = x0 + j - 1;
            const int xc = min(max(xx, 0), L.W - 1);
            ok[ky][j] = yy >= 0 && yy < L.H && xx >= 0 && xx < L.W;
            win[ky][j] = *reinterpret_cast<const Raw*>(static_cast<const T*>(L.v) +
                                                       elem_offset(L.blocked != 0, b, yc, xc, L.H, L.W, h, c, a.heads, a.d));
        }
    }
    float wk[36];
    const float4* wp = reinterpret_cast<const float4*>(L.weight + static_cast<size_t>(c0) * 9);
#pragma unroll
    for (int i = 0; i < 9; ++i) {
        const float4 t = wp[i];
        wk[4 * i] = t.x;
        wk[4 * i + 1] = t.y;
        wk[4 * i + 2] = t.z;
        wk[4 * i + 3] = t.w;
    }
    const float4 bias = L.bias ? *reinterpret_cast<const float4*>(L.bias + c0) : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 acc[kTX];
#pragma unroll
    for (int t = 0; t < kTX; ++t) acc[t] = bias;
    // window column j feeds outputs x0 + t with t = j - kx for the three kernel columns kx
#pragma unroll
    for (int ky = 0; ky < 3; ++ky) {
#pragma unroll
        for (int j = 0; j < kTX + 2; ++j) {
            float4 vv;
            if constexpr (sizeof(T) == 4) {
                vv = win[ky][j];
            } else {
                const uint2 u = win[ky][j];
                vv = make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                                 __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
            }
            if (!ok[ky][j]) vv = make_float4(0.f, 0.f, 0.f, 0.f);   // zero outside the map
#pragma unroll
            for (int kx = 0; kx < 3; ++kx) {
                const int t = j - kx;                      // output x0 + t uses column x0 + t + kx - 1
                if (t < 0 || t >= kTX) continue;
                const int k = ky * 3 + kx;
                acc[t].x = fmaf(wk[0 * 9 + k], vv.x, acc[t].x);
                acc[t].y = fmaf(wk[1 * 9 + k], vv.y, acc[t].y);
                acc[t].z = fmaf(wk[2 * 9 + k], vv.z, acc[t].z);
                acc[t].w = fmaf(wk[3 * 9 + k], vv.w, acc[t].w);
            }
        }
    }
    float* const row = L.dst + (static_cast<size_t>(b) * L.H + y) * L.W * C + c0;
    if (L.accumulate) {                                   // uniform: a level's message, read first
        float4 m[kTX];
#pragma unroll
        for (int t = 0; t < kTX; ++t) m[t] = *reinterpret_cast<const float4*>(row + static_cast<size_t>(min(x0 + t, L.W - 1)) * C);
#pragma unroll
        for (int t = 0; t < kTX; ++t) {
            acc[t].x += m[t].x;
            acc[t].y += m[t].y;
            acc[t].z += m[t].z;
            acc[t].w += m[t].w;
        }
    }
#pragma unroll
    for (int t = 0; t < kTX; ++t)
        if (x0 + t < L.W) *reinterpret_cast<float4*>(row + static_cast<size_t>(x0 + t) * C) = acc[t];
}

}  // namespace

hipError_t launch_posenc(const PosEncArgs& a, bool use_bf16, hipStream_t stream)
{
    // item counts per level (one item = 4 channels of kTX tokens of one row)
    PosEncArgs p = a;
    const int cpt = 4;
    const int C = a.heads * a.d;
    if (C % cpt != 0) return hipErrorInvalidValue;
    p.start[0] = 0;
    for (int l = 0; l < a.nlev; ++l) {
        const long long n = static_cast<long long>(a.B) * a.lv[l].H * ((a.lv[l].W + kTX - 1) / kTX) * (C / cpt);
        if (n >= 0x7FFFFFFFLL) return hipErrorInvalidValue;           // items within a level are int
        p.level_end[l] = p.start[l] + n;
        p.start[l + 1] = (p.level_end[l] + kThreads - 1) / kThreads * kThreads;
    }
    const long long total = p.start[p.nlev];
    if (total <= 0) return hipSuccess;
    const long long blocks = total / kThreads;
    if (blocks > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    if (use_bf16) hipLaunchKernelGGL((posenc_kernel<bf16>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream, p);
    else hipLaunchKernelGGL((posenc_kernel<float>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream, p);
    return hipGetLastError();
}

}  // namespace qta
