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

constexpr int kBwdRows = kPosEncBwdRows;      // rows one thread sweeps in the encoding's backward

// One thread owns one channel of kTX neighbouring tokens over kBwdRows consecutive rows of one level
// (channel fastest, so a wave reads contiguous channels of a token). It slides a 3-row window of dm^l
// and V^l down the rows (one new row of kTX + 2 values of each per step), adds to dV at its tokens
// sum over the window of w[tap] * dm(token - tap) (the transposed stencil), and accumulates its share
// of the kernel's gradient sum_token dm(token) * V(token + tap) and of the bias gradient
// sum_token dm(token). The block sums those shares per channel through LDS and writes one row of
// partial sums per channel. At level 0 of QuadTree-B with w it also adds <dout_i, encoding_i> to
// dw_{i,0}: the level-0 message that dw_{i,0} multiplies includes the encoding (a head's channels are
// d consecutive lanes).
// One row of the sliding window: dm and V at (y, x0 - 1 .. x0 + kTX) (zero outside the map) and, at
// level 0, dout at the row's own kTX tokens (for the dw term).
struct BwdRow {
    float gm[kTX + 2], vv[kTX + 2], go[kTX];
};

__device__ const float kUnitScale = 1.0f;   // stands in for w when QuadTree-B runs without it


// The work of one block; LEVEL0: a block of level 0 (dm from dout and w), else of a coarser level.
template <typename T, bool LEVEL0>
__device__ __forceinline__ void posenc_bwd_block(const PosEncBwdArgs& a, const long long blk, float (*red)[11])
{
    constexpr int kPart = 10;                          // 9 taps, then the bias
    const long long item = blk * blockDim.x + threadIdx.x;
    int l = 0;
    if constexpr (!LEVEL0)
        while (l + 1 < a.nlev && item >= a.start[l + 1]) ++l;
    const PosEncBwdLevel& L = a.lv[l];
    const int C = a.heads * a.d;
    const bool live = item < a.level_end[l];
    const int xtiles = (L.W + kTX - 1) / kTX, ytiles = (L.H + kBwdRows - 1) / kBwdRows;
    int r = live ? static_cast<int>(item - a.start[l]) : 0;
    const int ch = r % C;
    r /= C;
    const int x0 = (r % xtiles) * kTX;
    r /= xtiles;
    const int y0 = (r % ytiles) * kBwdRows;
    const int b = r / ytiles;
    const int h = ch / a.d, c = ch - h * a.d;
    const int N = L.H * L.W;
    const bool want_dw = LEVEL0 && a.dw != nullptr;   // uniform
    // Column offsets of the window (clamped into the map) and their validity, fixed for the thread:
    // NHWC tensors step C per column; at level 0 w steps heads*L (V there is the caller's, NHWC);
    // at the coarser levels V in the parent-blocked layout ([B][heads][H/2][W/2][2][2][d]) steps 4d
    // per column pair and d within a pair.
    int colc[kTX + 2], colx[kTX + 2];
    unsigned colok[kTX + 2];
    const int wstride = (a.variant_b && a.w) ? a.heads * a.nlev : 0;
#pragma unroll
    for (int j = 0; j < kTX + 2; ++j) {
        const int xx = x0 + j - 1;
        const int xc = min(max(xx, 0), L.W - 1);
        colok[j] = opaque_mask(live && xx >= 0 && xx < L.W);
        colc[j] = xc * C;
        if constexpr (LEVEL0) colx[j] = xc * wstride;
        else colx[j] = L.blocked ? ((xc >> 1) * 4 + (xc & 1)) * a.d : xc * C;
    }
    // level 0 of QuadTree-B scales dout by w_{i,0} (with w) or 1/L (without); QuadTree-A does not
    const float* wsrc = wstride ? a.w + h * a.nlev : &kUnitScale;
    const float sc = (a.variant_b && !a.w) ? 1.0f / a.nlev : 1.0f;
    const int Hp = (L.H + 1) / 2, Wp = (L.W + 1) / 2;
    const T* vbase = static_cast<const T*>(L.v);
    auto load_row = [&](int yy, BwdRow& R) {
        const int yc = min(max(yy, 0), L.H - 1);
        const unsigned rowok = opaque_mask(yy >= 0 && yy < L.H);
        const size_t tokrow = static_cast<size_t>(b) * N + static_cast<size_t>(yc) * L.W;   // token of (b, yc, 0)
        const size_t vrow = (!LEVEL0 && L.blocked)
            ? ((((static_cast<size_t>(b) * a.heads + h) * Hp + (yc >> 1)) * Wp) * 4 + (yc & 1) * 2) * a.d + c
            : tokrow * C + ch;
        const T* vp = vbase + vrow;
        const int* colv = LEVEL0 ? colc : colx;
        if constexpr (LEVEL0) {
            const T* gp = static_cast<const T*>(a.dout) + tokrow * C + ch;
            const float* wp = wsrc + (wstride ? tokrow * wstride : 0);
#pragma unroll
            for (int j = 0; j < kTX + 2; ++j) {
                const float raw = Storage<T>::load1(gp, colc[j]);
                const float g = sc * wp[colx[j]] * raw;
                if (j >= 1 && j <= kTX) R.go[j - 1] = raw;
                R.gm[j] = masked(g, rowok & colok[j]);
            }
        } else {
            const float* gp = L.dm + tokrow * C + ch;
#pragma unroll
            for (int j = 0; j < kTX + 2; ++j) R.gm[j] = masked(gp[colc[j]], rowok & colok[j]);
        }
#pragma unroll
        for (int j = 0; j < kTX + 2; ++j) {
            const float v = Storage<T>::load1(vp, colv[j]);
            R.vv[j] = masked(v, rowok & colok[j]);
        }
    };
    float part[kPart];
#pragma unroll
    for (int i = 0; i < kPart; ++i) part[i] = 0.f;
    float wk[9];
#pragma unroll
    for (int i = 0; i < 9; ++i) wk[i] = L.weight[static_cast<size_t>(ch) * 9 + i];
    const float bias0 = (want_dw && a.bias0) ? a.bias0[ch] : 0.f;
    // Row y of the tile with its window rows above (U), at (M) and below (D): D is loaded here, with
    // dV at the row's tokens, so that the two wait once.
    auto step = [&](int y, const BwdRow& U, const BwdRow& M, BwdRow& D) {
        const int yc = min(y, L.H - 1);
        float* dvp = L.dv + (static_cast<size_t>(b) * N + static_cast<size_t>(yc) * L.W) * C + ch;
        float dvo[kTX];
#pragma unroll
        for (int t = 0; t < kTX; ++t) dvo[t] = dvp[colc[t + 1]];
        load_row(y + 1, D);
        const BwdRow* rows[3] = {&U, &M, &D};
        float dwv[kTX];
#pragma unroll
        for (int t = 0; t < kTX; ++t) {
            // zero dm outside the map makes the partial sums of a token past the edge vanish; only
            // the stores are masked
            const float g0 = M.gm[t + 1];
            part[9] += g0;
            float acc = 0.f, e = bias0;
#pragma unroll
            for (int ky = 0; ky < 3; ++ky)
#pragma unroll
                for (int kx = 0; kx < 3; ++kx) {
                    const int k = ky * 3 + kx;
                    part[k] = fmaf(g0, rows[ky]->vv[t + kx], part[k]);
                    // V at this token fed the message of token - tap + (1, 1) through tap (ky, kx)
                    acc = fmaf(wk[k], rows[2 - ky]->gm[t + 2 - kx], acc);
                    if (want_dw) e = fmaf(wk[k], rows[ky]->vv[t + kx], e);
                }
            if (live && y < L.H && x0 + t < L.W) dvp[colc[t + 1]] = dvo[t] + acc;
            dwv[t] = want_dw ? M.go[t] * e : 0.f;   // the encoding against dout
        }
        if (want_dw) {
            // summed over the head's d channels (d consecutive lanes: the whole wave for d = 64, each
            // half for d = 32), with every lane taking part in the exchanges
#pragma unroll
            for (int t = 0; t < kTX; ++t) {
                const float sum = a.d == 64 ? wave_allreduce(dwv[t], [](float u, float v) { return u + v; })
                                            : half_allreduce(dwv[t], [](float u, float v) { return u + v; });
                if (live && y < L.H && x0 + t < L.W && c == 0)
                    a.dw[((static_cast<size_t>(b) * N + static_cast<size_t>(y) * L.W + x0 + t) * a.heads + h) * a.nlev] += sum;
            }
        }
    };
    // three window slots in rotation (the loop is unrolled by three so that no row is copied)
    BwdRow r0, r1, r2;
    load_row(y0 - 1, r0);
    load_row(y0, r1);
#pragma unroll 1
    for (int dy = 0; dy < kBwdRows; dy += 3) {
        step(y0 + dy, r0, r1, r2);
        if (dy + 1 < kBwdRows) step(y0 + dy + 1, r1, r2, r0);
        if (dy + 2 < kBwdRows) step(y0 + dy + 2, r2, r0, r1);
    }
#pragma unroll
    for (int i = 0; i < kPart; ++i) red[threadIdx.x][i] = part[i];
    __syncthreads();
    // the block's items start at a multiple of the block size within the level: thread t holds
    // channel (b0 + t) % C; thread j < C sums the threads of channel (b0 + j) % C
    const int b0 = static_cast<int>((blk * blockDim.x - a.start[l]) % C);
    if (static_cast<int>(threadIdx.x) < min(C, kThreads)) {
        const int j = threadIdx.x;
        float sum[kPart];
#pragma unroll
        for (int i = 0; i < kPart; ++i) sum[i] = 0.f;
        for (int t = j; t < kThreads; t += C)
#pragma unroll
            for (int i = 0; i < kPart; ++i) sum[i] += red[t][i];
        const int chj = (b0 + j) % C;
        float* dst = a.part + (static_cast<size_t>(blk) * C + chj) * kPart;
#pragma unroll
        for (int i = 0; i < kPart; ++i) dst[i] = sum[i];
    }
}

// One launch for every level: level 0's blocks first (b0 of them), then the coarser levels', which
// run beside them; the two kinds of block take separate code paths (a uniform branch), so neither
// pays for the other's registers.
template <typename T>
__global__ __launch_bounds__(kThreads) void posenc_bwd_kernel(PosEncBwdArgs a, int b0)
{
    __shared__ float red[kThreads][11];
    const long long blk = blockIdx.x;
    if (blk < b0) posenc_bwd_block<T, true>(a, blk, red);
    else posenc_bwd_block<T, false>(a, blk, red);
}

// Sums the partial rows of each level: one block per (level, 64 consecutive entries of the C*10
// row), lane i owning entry i and the block's waves taking the level's blocks in turn (coalesced
// reads), then a sum over the waves in LDS.
constexpr int kReduceWaves = 16;
__global__ __launch_bounds__(kReduceWaves * kWave) void posenc_bwd_reduce_kernel(PosEncBwdArgs a)
{
    __shared__ float red[kReduceWaves][kWave];
    const int C = a.heads * a.d, row = C * 10;
    const int chunks = (row + kWave - 1) / kWave;
    const int l = blockIdx.x / chunks, o = (blockIdx.x - l * chunks) * kWave + (threadIdx.x & (kWave - 1));
    const int wave = threadIdx.x / kWave;
    const long long first = a.start[l] / kThreads;
    const long long last = (a.level_end[l] + kThreads - 1) / kThreads;
    constexpr int kInFlight = 8;                     // independent loads per lane per round
    float s[kInFlight] = {};
    if (o < row) {
        long long blk = first + wave;
        for (; blk + (kInFlight - 1) * kReduceWaves < last; blk += kInFlight * kReduceWaves)
#pragma unroll
            for (int u = 0; u < kInFlight; ++u) s[u] += a.part[static_cast<size_t>(blk + u * kReduceWaves) * row + o];
        for (; blk < last; blk += kReduceWaves) s[0] += a.part[static_cast<size_t>(blk) * row + o];
    }
    float tot = 0.f;
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) tot += s[u];
    red[wave][threadIdx.x & (kWave - 1)] = tot;
    __syncthreads();
    if (wave == 0 && o < row) {
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < kReduceWaves; ++w) s += red[w][threadIdx.x];
        const int chn = o / 10, k = o - chn * 10;
        const size_t cg = static_cast<size_t>(l) * C + chn;
        if (k < 9) a.dweight[cg * 9 + k] = s;
        else if (a.dbias) a.dbias[cg] = s;
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
    if (C > kThreads || (a.d != 32 && a.d != 64)) return hipErrorInvalidValue;
    p.start[0] = 0;
    for (int l = 0; l < a.nlev; ++l) {
        const long long n = posenc_bwd_items(a.B, a.lv[l].H, a.lv[l].W, C);
        if (n >= 0x7FFFFFFFLL) return hipErrorInvalidValue;           // items within a level are int
        p.level_end[l] = p.start[l] + n;
        p.start[l + 1] = (p.level_end[l] + kThreads - 1) / kThreads * kThreads;
    }
    const long long blocks = p.start[p.nlev] / kThreads;
    if (blocks <= 0) return hipSuccess;
    if (blocks > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    const int b0 = static_cast<int>(p.start[1] / kThreads);   // level 0's blocks, then the others
    if (use_bf16) hipLaunchKernelGGL((posenc_bwd_kernel<bf16>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream, p, b0);
    else hipLaunchKernelGGL((posenc_bwd_kernel<float>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream, p, b0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int chunks = (C * 10 + kWave - 1) / kWave;
    hipLaunchKernelGGL(posenc_bwd_reduce_kernel, dim3(static_cast<unsigned>(p.nlev * chunks)), dim3(kReduceWaves * kWave),
                       0, stream, p);
    return hipGetLastError();
}

}  // namespace qta
