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

constexpr int kTX = kPosEncTokens;      // tokens along x per thread (their 3x3 windows share columns)
constexpr int kThreads = kPosEncThreads;

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

// Four consecutive channels of dm^0 = scale * dout at one token: scale is w_{i,0} (B with w), 1/L
// (B without w) or 1 (A), one per head.
template <typename T>
__device__ __forceinline__ float4 dm0_load(const PosEncBwdArgs& a, int b, int tok, int N, int C, int c0, int h)
{
    float4 g = load4<T>(a.dout, (static_cast<size_t>(b) * N + tok) * C + c0);
    float s = 1.0f;
    if (a.variant_b) s = a.w ? a.w[((static_cast<size_t>(b) * N + tok) * a.heads + h) * a.nlev] : 1.0f / a.nlev;
    return make_float4(s * g.x, s * g.y, s * g.z, s * g.w);
}

// One thread owns four channels of four neighbouring tokens of one row of one level (as in the
// forward pass). It reads the 3 x 6 windows of dm^l and V^l once, adds to dV at its tokens
// sum over the window of w[tap] * dm(token - tap) (the transposed stencil), and forms its share of the
// kernels' gradient sum_token dm(token) * V(token + tap) and of the bias gradient sum_token dm(token).
// The block then sums those shares per channel through LDS and writes one row of partial sums. At
// level 0 of QuadTree-B with w it also adds <dout_i, encoding_i> to dw_{i,0}: the level-0 message
// that dw_{i,0} multiplies includes the encoding (a head's d/4 threads are consecutive lanes).
template <typename T>
__global__ __launch_bounds__(kThreads) void posenc_bwd_kernel(PosEncBwdArgs a)
{
    constexpr int kPart = 4 * 10;                       // 4 channels x (9 taps + the bias)
    __shared__ float red[kThreads][kPart + 1];
    const long long item = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
    int l = 0;
    while (l + 1 < a.nlev && item >= a.start[l + 1]) ++l;
    const PosEncBwdLevel& L = a.lv[l];
    const int C = a.heads * a.d, groups = C / 4;
    const bool live = item < a.level_end[l];
    const int xtiles = (L.W + kTX - 1) / kTX;
    const long long rel = item - a.start[l];
    int r = live ? static_cast<int>(rel) : 0;
    const int g = r % groups;
    r /= groups;
    const int x0 = (r % xtiles) * kTX;
    r /= xtiles;
    const int y = r % L.H;
    const int b = r / L.H;
    const int c0 = 4 * g, h = c0 / a.d, c = c0 - h * a.d;
    const int N = L.H * L.W;
    float part[kPart];
#pragma unroll
    for (int i = 0; i < kPart; ++i) part[i] = 0.f;
    const bool want_dw = l == 0 && a.dw != nullptr;                   // uniform
    float dwp[kTX] = {};
    if (live) {
        // the windows of dm and V (zero outside the map)
        float4 dmw[3][kTX + 2], vw[3][kTX + 2];
#pragma unroll
        for (int ky = 0; ky < 3; ++ky) {
            const int yy = y + ky - 1;
            const int yc = min(max(yy, 0), L.H - 1);
#pragma unroll
            for (int j = 0; j < kTX + 2; ++j) {
                const int xx = x0 + j - 1;
                const int xc = min(max(xx, 0), L.W - 1);
                const bool ok = yy >= 0 && yy < L.H && xx >= 0 && xx < L.W;
                const int tok = yc * L.W + xc;
                float4 gm = l == 0 ? dm0_load<T>(a, b, tok, N, C, c0, h)
                                   : *reinterpret_cast<const float4*>(L.dm + (static_cast<size_t>(b) * N + tok) * C + c0);
                float4 vv = load4<T>(L.v, elem_offset(L.blocked != 0, b, yc, xc, L.H, L.W, h, c, a.heads, a.d));
                if (!ok) {
                    gm = make_float4(0.f, 0.f, 0.f, 0.f);
                    vv = gm;
                }
                dmw[ky][j] = gm;
                vw[ky][j] = vv;
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
#pragma unroll
        for (int t = 0; t < kTX; ++t) {
            if (x0 + t >= L.W) break;
            const float4 g0 = dmw[1][t + 1];                  // dm at this thread's token (y, x0 + t)
            // the bias and the kernels: dm(token) times V(token + tap)
            part[36 + 0] += g0.x;
            part[36 + 1] += g0.y;
            part[36 + 2] += g0.z;
            part[36 + 3] += g0.w;
            float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int ky = 0; ky < 3; ++ky)
#pragma unroll
                for (int kx = 0; kx < 3; ++kx) {
                    const int k = ky * 3 + kx;
                    const float4 vv = vw[ky][t + kx];
                    part[0 * 9 + k] += g0.x * vv.x;
                    part[1 * 9 + k] += g0.y * vv.y;
                    part[2 * 9 + k] += g0.z * vv.z;
                    part[3 * 9 + k] += g0.w * vv.w;
                    // V at this token fed the message of token - tap + (1, 1) through tap (ky, kx)
                    const float4 gg = dmw[2 - ky][t + 2 - kx];
                    acc.x = fmaf(wk[0 * 9 + k], gg.x, acc.x);
                    acc.y = fmaf(wk[1 * 9 + k], gg.y, acc.y);
                    acc.z = fmaf(wk[2 * 9 + k], gg.z, acc.z);
                    acc.w = fmaf(wk[3 * 9 + k], gg.w, acc.w);
                }
            float4* dst = reinterpret_cast<float4*>(L.dv + (static_cast<size_t>(b) * N + y * L.W + x0 + t) * C + c0);
            const float4 old = *dst;
            *dst = make_float4(old.x + acc.x, old.y + acc.y, old.z + acc.z, old.w + acc.w);
            if (want_dw) {
                // the encoding at this token, against dout there
                float4 e = a.bias0 ? *reinterpret_cast<const float4*>(a.bias0 + c0) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                for (int ky = 0; ky < 3; ++ky)
#pragma unroll
                    for (int kx = 0; kx < 3; ++kx) {
                        const int k = ky * 3 + kx;
                        const float4 vv = vw[ky][t + kx];
                        e.x = fmaf(wk[0 * 9 + k], vv.x, e.x);
                        e.y = fmaf(wk[1 * 9 + k], vv.y, e.y);
                        e.z = fmaf(wk[2 * 9 + k], vv.z, e.z);
                        e.w = fmaf(wk[3 * 9 + k], vv.w, e.w);
                    }
                const float4 go = load4<T>(a.dout, (static_cast<size_t>(b) * N + y * L.W + x0 + t) * C + c0);
                dwp[t] = go.x * e.x + go.y * e.y + go.z * e.z + go.w * e.w;
            }
        }
    }
    if (want_dw) {
        // sum over the head's d/4 threads (aligned groups of consecutive lanes, all of one level and
        // either all live or all past its end), then the first of them adds it to dw_{i,0}
        const int G = a.d / 4;
#pragma unroll
        for (int t = 0; t < kTX; ++t) {
            float s = dwp[t];
            for (int m = 1; m < G; m <<= 1) s += __shfl_xor(s, m, kWave);
            if (live && (g % G) == 0 && x0 + t < L.W) {
                float* dwd = a.dw + ((static_cast<size_t>(b) * N + y * L.W + x0 + t) * a.heads + h) * a.nlev;
                *dwd += s;
            }
        }
    }
#pragma unroll
    for (int i = 0; i < kPart; ++i) red[threadIdx.x][i] = part[i];
    __syncthreads();
    // the block's items start at a multiple of the block size within the level: thread t holds
    // channel group (b0 + t) % groups
    const int b0 = static_cast<int>((static_cast<long long>(blockIdx.x) * blockDim.x - a.start[l]) % groups);
    for (int j = threadIdx.x; j < groups; j += blockDim.x) {
        float s[kPart];
#pragma unroll
        for (int i = 0; i < kPart; ++i) s[i] = 0.f;
        for (int t = ((j - b0) % groups + groups) % groups; t < kThreads; t += groups)
#pragma unroll
            for (int i = 0; i < kPart; ++i) s[i] += red[t][i];
        float* dst = a.part + static_cast<size_t>(blockIdx.x) * C * 10 + static_cast<size_t>(4 * j) * 10;
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
#pragma unroll
            for (int k = 0; k < 9; ++k) dst[cc * 10 + k] = s[cc * 9 + k];
            dst[cc * 10 + 9] = s[36 + cc];
        }
    }
}

// Sums the partial rows of each level: one block per (level, channel group of four), its threads
// taking the level's blocks in turn, then a tree over the threads in LDS.
__global__ __launch_bounds__(kThreads) void posenc_bwd_reduce_kernel(PosEncBwdArgs a)
{
    constexpr int kPart = 40;
    __shared__ float red[kThreads][kPart + 1];
    const int C = a.heads * a.d, groups = C / 4;
    const int l = blockIdx.x / groups, j = blockIdx.x - l * groups;
    const long long first = a.start[l] / kThreads;
    const long long last = (a.level_end[l] + kThreads - 1) / kThreads;
    float s[kPart];
#pragma unroll
    for (int i = 0; i < kPart; ++i) s[i] = 0.f;
    for (long long blk = first + threadIdx.x; blk < last; blk += blockDim.x) {
        const float* src = a.part + static_cast<size_t>(blk) * C * 10 + static_cast<size_t>(4 * j) * 10;
#pragma unroll
        for (int i = 0; i < kPart; ++i) s[i] += src[i];
    }
#pragma unroll
    for (int i = 0; i < kPart; ++i) red[threadIdx.x][i] = s[i];
    __syncthreads();
    for (int half = kThreads / 2; half > 0; half >>= 1) {
        if (static_cast<int>(threadIdx.x) < half)
#pragma unroll
            for (int i = 0; i < kPart; ++i) red[threadIdx.x][i] += red[threadIdx.x + half][i];
        __syncthreads();
    }
    if (threadIdx.x < kPart) {
        const int cc = threadIdx.x / 10, k = threadIdx.x - cc * 10;
        const size_t ch = static_cast<size_t>(l) * C + 4 * j + cc;
        if (k < 9) a.dweight[ch * 9 + k] = red[0][threadIdx.x];
        else if (a.dbias) a.dbias[ch] = red[0][threadIdx.x];
    }
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

namespace qta {

hipError_t launch_posenc_bwd(const PosEncBwdArgs& a, bool use_bf16, hipStream_t stream)
{
    PosEncBwdArgs p = a;
    const int C = a.heads * a.d;
    if (C % 4 != 0 || C / 4 > kThreads) return hipErrorInvalidValue;
    p.start[0] = 0;
    for (int l = 0; l < a.nlev; ++l) {
        const long long n = posenc_items(a.B, a.lv[l].H, a.lv[l].W, C);
        if (n >= 0x7FFFFFFFLL) return hipErrorInvalidValue;           // items within a level are int
        p.level_end[l] = p.start[l] + n;
        p.start[l + 1] = (p.level_end[l] + kThreads - 1) / kThreads * kThreads;
    }
    const long long blocks = p.start[p.nlev] / kThreads;
    if (blocks <= 0) return hipSuccess;
    if (blocks > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    if (use_bf16) hipLaunchKernelGGL((posenc_bwd_kernel<bf16>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream, p);
    else hipLaunchKernelGGL((posenc_bwd_kernel<float>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(posenc_bwd_reduce_kernel, dim3(static_cast<unsigned>(p.nlev * (C / 4))), dim3(kThreads), 0, stream, p);
    return hipGetLastError();
}

}  // namespace qta
