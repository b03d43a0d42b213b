// Kernel argument blocks and launchers shared between the HIP kernels and the C-ABI host code.
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <stdint.h>

#include "../../include/qta.h"

namespace qta {

// Storage of one pyramid level (and of the inputs) in HBM:
//  - NHWC:    [B][H][W][heads][d], one token's heads contiguous;
//  - blocked: [B][heads][ceil(H/2)][ceil(W/2)][2][2][d], the 2x2 children of one parent position
//             of one head contiguous (4*d elements; off-map children are unused padding).
// qta_forward keeps every level that is gathered (all but the coarsest) blocked, so a kept key's
// four children are one contiguous run of 4*d*sizeof(dtype) bytes.
struct LevelLayout {
    bool blocked;
};

// Byte offset of the 16-byte chunk `ch` (0 <= ch < C*sizeof(dtype)/16) of token (y, x) in a level
// of H x W tokens; `cpt` chunks per token, `cph` chunks per head row.
__host__ __device__ inline size_t chunk_offset(bool blocked, int b, int y, int x, int H, int W, int ch, int cpt,
                                               int cph)
{
    if (!blocked) return ((static_cast<size_t>(b) * H + y) * W + x) * cpt * 16 + static_cast<size_t>(ch) * 16;
    const int heads = cpt / cph;
    const int h = ch / cph, c2 = ch - h * cph;
    const int Hp = (H + 1) / 2, Wp = (W + 1) / 2;
    const size_t blk = ((static_cast<size_t>(b) * heads + h) * Hp + (y >> 1)) * Wp + (x >> 1);
    const int child = (y & 1) * 2 + (x & 1);
    return ((blk * 4 + child) * cph + c2) * 16;
}

// Bytes of one level of B x H x W tokens with C*tb bytes each.
inline size_t level_bytes(bool blocked, int B, int H, int W, int C, int tb)
{
    if (!blocked) return static_cast<size_t>(B) * H * W * C * tb;
    return static_cast<size_t>(B) * ((H + 1) / 2) * ((W + 1) / 2) * 4 * C * tb;
}

// One pyramid pass over up to three token maps (q, k, v): from a source level produce one, two or
// three coarser levels.
struct PyramidPassArgs {
    const void* src[3];
    void* dst1[3];
    void* dst2[3];
    void* dst3[3];
    void* dst4[3];
    int B, Hs, Ws, H1, W1, H2, W2, H3, W3, H4, W4;
    int chunks;                 // 16-byte chunks per token (C * sizeof(dtype) / 16)
    int head_chunks;            // 16-byte chunks per head row (d * sizeof(dtype) / 16)
    int lg_head_chunks;         // log2(head_chunks) (a power of two for every supported d)
    bool src_blocked, dst1_blocked, dst2_blocked, dst3_blocked, dst4_blocked;
};

// LDS chunks staged per level-1 level of the multi-level pyramid pass (16 KiB).
constexpr int kPyramidStage = 1024;

// Workgroup of the multi-level pyramid pass over nlev levels (2..4): `by` token rows of `chunks`
// threads, each taking up to R level-1 tokens, and tpb top tokens per workgroup (a top token has
// NC^(nlev-1) level-1 tokens, NC = 4, or 2 for maps of one row). About 256 threads, more when a
// top token's level-1 tokens would need more than four per thread.
struct PyramidTreeShape {
    bool ok;
    int by, tpb, R;
};
inline PyramidTreeShape pyramid_tree_shape(int nlev, int chunks, bool row)
{
    PyramidTreeShape g{false, 0, 0, 0};
    if (nlev < 2 || nlev > 4 || chunks <= 0 || chunks > 1024) return g;
    const int L1 = 1 << ((row ? 1 : 2) * (nlev - 1));
    if (static_cast<long long>(L1) * chunks > kPyramidStage) return g;
    int by = 256 / chunks > 1 ? 256 / chunks : 1;
    if (L1 >= by) {
        g.tpb = 1;
        g.R = (L1 + by - 1) / by;
        if (g.R > 4) {
            by = (L1 + 3) / 4;
            g.R = (L1 + by - 1) / by;
        }
    } else {
        g.tpb = by / L1;
        by = g.tpb * L1;
        g.R = 1;
    }
    if (g.R == 3) g.R = 4;                                 // instantiated for 1, 2 and 4
    g.by = by;
    g.ok = static_cast<long long>(by) * chunks <= 1024;
    return g;
}

// Whether the multi-level pyramid pass takes a pass over nlev levels from an Hs x Ws source: the
// shape above exists, head_chunks is a power of two, and one batch element's map of any level of
// the pass (parent-blocked padding included) is addressed with 32-bit offsets and 24-bit products.
inline bool pyramid_tree_fits(int nlev, int chunks, int head_chunks, bool row, int Hs, int Ws)
{
    if (!pyramid_tree_shape(nlev, chunks, row).ok) return false;
    if (head_chunks <= 0 || (head_chunks & (head_chunks - 1)) != 0 || chunks % head_chunks != 0) return false;
    const long long tokens = static_cast<long long>(Hs + 2) * (Ws + 2);
    const long long side = Hs > Ws ? Hs : Ws;
    return tokens < (1LL << 24) && tokens * chunks * 16 < (1LL << 32) && side * chunks < (1LL << 24);
}

struct CoarseArgs {
    const void* q;
    const void* k;
    const void* v;
    int B, heads, N, C;         // N = Hc * Wc tokens at the coarsest level
    int K;                      // 0: no selection
    float scale;
    float* msg;                 // fp32 [B][N][heads][d], or NULL when `out` is written instead
    int32_t* sel_idx;
    float* sel_key;
    void* out;                  // single-level problem: write out = w0 * m (B) or m (A) in dtype
    const float* w;
    const float* pe0;           // single-level problem: position encoding added to m, or NULL
    const float* pe_w;          // or, fused (coarse_attn_kernel): this level's depth-wise kernels fp32 [C][3][3],
                                // applied to v around each query (an Hc x Wc map) and added to m; or NULL
    const float* pe_b;          // its bias fp32 [C], or NULL
    int Wc;                     // map width (with pe_w)
    int levels;
};

// Division of 0 <= n < 2^31 by a fixed divisor d >= 1 with one high multiply and a shift:
// q = (umulhi(n, m) + n) >> s, s = ceil(log2 d), m = floor(2^(32+s) / d) - 2^32 + 1 (the round-up
// method of Granlund and Montgomery, "Division by invariant integers using multiplication",
// PLDI 1994). umulhi(n, m) <= n, so the sum stays below 2^32.
struct FastDiv {
    uint32_t m;
    int s;
    int d;
};

inline FastDiv make_fastdiv(int d)
{
    int s = 0;
    while ((1LL << s) < d) ++s;
    const unsigned __int128 one = 1;
    const uint64_t m = static_cast<uint64_t>(((one << (32 + s)) / static_cast<unsigned>(d)) - (one << 32) + 1);
    return FastDiv{static_cast<uint32_t>(m), s, d};
}

__host__ __device__ __forceinline__ int fast_div(int n, const FastDiv& f)
{
    const uint32_t u = static_cast<uint32_t>(n);
    const uint32_t hi = static_cast<uint32_t>((static_cast<uint64_t>(u) * f.m) >> 32);
    return static_cast<int>((hi + u) >> f.s);
}

struct FineArgs {
    const void* q;
    const void* k;
    const void* v;
    bool q_blocked;             // queries of this level stored blocked (else NHWC)
    bool kv_blocked;            // keys and values of this level stored blocked (else NHWC)
    int B, heads, H, W, Hp, Wp, C;
    int Kp;                     // keys each parent query kept: 4*Kp candidate slots per sibling group
    int Ks;                     // keys this level keeps per query (levels above the finest)
    FastDiv div_Wp;             // division by Wp (flat parent index -> row)
    FastDiv div_heads;          // division by heads (work item -> head); set by the launcher
    FastDiv div_items;          // division by the work items of one (batch, head); set by the launcher
    float scale;
    const int32_t* parent_idx;
    const float* parent_key;
    // intermediate level: outputs
    float* msg;
    int32_t* sel_idx;
    float* sel_key;
    // finest level: fused combination
    void* out;
    const float* w;
    const float* pe0;           // level 0's position encoding, fp32 [B][N][heads][d], added to m0; or NULL
    const float* pe_w;          // or, fused (maps of more than one row): level 0's depth-wise kernels, fp32
                                // [C][3][3], applied to v around each query and added to m0; or NULL
    const float* pe_b;          // its bias, fp32 [C], or NULL
    int levels;
    float inv_levels;           // 1/levels, the weight of every level without w (set by the launcher)
    const float* coarser_msg[QTA_MAX_LEVELS];   // entry j: message of level j (j >= 1)
    int lvl_W[QTA_MAX_LEVELS];                  // map width of level j
    int lvl_N[QTA_MAX_LEVELS];                  // tokens of level j
};

// Multiscale position encoding of one level: dst += (or =, for level 0) the 3x3 depth-wise
// convolution of V at that level with zero padding, plus the bias.
struct PosEncLevel {
    const void* v;              // V at this level (storage type), NHWC or parent-blocked
    int blocked;
    int H, W;
    float* dst;                 // fp32 [B][H*W][heads][d]
    int accumulate;             // 1: dst += encoding (a level's message), 0: dst = encoding
    const float* weight;        // fp32 [C][3][3] for this level
    const float* bias;          // fp32 [C], or NULL
};

struct PosEncArgs {
    PosEncLevel lv[QTA_MAX_LEVELS];
    long long start[QTA_MAX_LEVELS + 1];    // first work item of each level (set by the launcher)
    long long level_end[QTA_MAX_LEVELS];     // one past the last work item of each level
    int nlev;
    int B, heads, d;
};

// Backward of the multiscale position encoding, every level in one launch: with dm^l the gradient of
// level l's message, V^l receives the transposed stencil of dm^l (added to dv), and the kernels and
// bias the per-block partial sums of dm^l correlated with V^l (reduced by launch_posenc_bwd's
// second kernel into dweight / dbias).
struct PosEncBwdLevel {
    const void* v;              // V^l (storage type), NHWC or parent-blocked
    int blocked;
    int H, W;
    const float* dm;            // fp32 [B][H*W][heads][d]; NULL at level 0 (dout and w are used)
    float* dv;                  // fp32 [B][H*W][heads][d]: += the transposed stencil of dm
    const float* weight;        // fp32 [C][3][3] of this level
};

struct PosEncBwdArgs {
    PosEncBwdLevel lv[QTA_MAX_LEVELS];
    long long start[QTA_MAX_LEVELS + 1];    // first work item of each level (set by the launcher)
    long long level_end[QTA_MAX_LEVELS];
    int nlev, B, heads, d;
    int variant_b;
    const void* dout;           // level 0: dm^0 = w_{i,0} * dout_i (B with w), dout_i / L (B without), dout_i (A)
    const float* w;             // fp32 [B][H*W][heads][L] or NULL
    float* part;                // per block of the first kernel: [C][10] partial sums (9 taps, then the bias)
    float* dweight;             // fp32 [L][C][3][3]
    float* dbias;               // fp32 [L][C], or NULL
    const float* bias0;         // level 0's bias fp32 [C], or NULL
    float* dw;                  // B with w: fp32 [B][H*W][heads][L], += <dout_i, level 0's encoding at i>; or NULL
};

// Work items of one level of the encoding's forward pass (4 channels of 4 neighbouring tokens of one
// row), and the 256-thread blocks of the backward's first kernel (every level starts on a block
// boundary).
constexpr int kPosEncTokens = 4;
constexpr int kPosEncThreads = 256;
inline long long posenc_items(int B, int H, int W, int C)
{
    return static_cast<long long>(B) * H * ((W + kPosEncTokens - 1) / kPosEncTokens) * (C / 4);
}
// The backward's items: one channel of kPosEncTokens tokens over kPosEncBwdRows rows.
constexpr int kPosEncBwdRows = 8;
inline long long posenc_bwd_items(int B, int H, int W, int C)
{
    return static_cast<long long>(B) * ((H + kPosEncBwdRows - 1) / kPosEncBwdRows) *
           ((W + kPosEncTokens - 1) / kPosEncTokens) * C;
}
inline long long posenc_bwd_blocks(int B, const int* Hl, const int* Wl, int levels, int C)
{
    long long n = 0;
    for (int l = 0; l < levels; ++l) n += (posenc_bwd_items(B, Hl[l], Wl[l], C) + kPosEncThreads - 1) / kPosEncThreads;
    return n;
}

// ---- backward pass (gradients with the kept-key sets held fixed) ----

// Backward of one finer level l (0 <= l < L-1), in two passes. Query pass: one wave per (parent
// query at l+1, head): dq, each query's softmax statistics, QuadTree-A's parent-score gradients and
// dw_0, and for every key of level l+1 the number of parents that kept it. Key pass: the kept
// (parent, rank) pairs sorted by key, then one wave per chunk of one key's list: dk and dv of the
// key's four children at level l, each row written once.
constexpr int kKeyChunk = 16;       // parents per key-pass chunk

struct BwdLevelArgs {
    const void* q;
    const void* k;
    const void* v;
    bool blocked;               // q, k, v of this level parent-blocked (else NHWC)
    int B, heads, H, W, Hp, Wp, C;
    int Kp;                     // keys each parent kept (4*Kp candidate slots, at most 64)
    int Ks;                     // keys this level keeps (l >= 1)
    FastDiv div_Wp, div_Np, div_heads, div_Kp;   // divisions by Wp, Hp*Wp, heads, Kp; set by the launchers
    float scale;
    const int32_t* parent_idx;  // [B][heads][Np][Kp]
    const float* parent_key;    // QuadTree-A: the parents' scores sigma
    const int32_t* sel_idx;     // QuadTree-A, l >= 1: this level's kept keys [B][heads][N][Ks]
    const float* dsig_in;       // QuadTree-A, l >= 1: dLoss/d(score of each kept key) [B][heads][N][Ks]
    float* dsig_out;            // QuadTree-A: dLoss/d(parent's kept-key scores) [B][heads][Np][Kp]
    const float* dm;            // l >= 1: dLoss/dm^l fp32 [B][N][C]
    const void* dout;           // l == 0: upstream gradient, storage type [B][N][C]
    const float* w;             // l == 0, QuadTree-B: [B][N][heads][L] or NULL (1/L)
    int levels;
    float* dq;                  // fp32 [B][N][C], written
    float* dk;                  // fp32 [B][N][C], written by the key pass
    float* dv;
    float* dw;                  // l == 0, QuadTree-B with w: entry 0 written; or NULL
    float* stats;               // B: [B][heads][N][2] (log-sum-exp, sum p ds); A: [B][heads][N][Kp][2]
    int32_t* count;             // [B*heads*Np] parents that kept each key (zero before the query pass;
                                //   the scan returns it to zero)
    int32_t* slot;              // [B*heads*Np*Kp] place of each kept pair in its key's list
    const int32_t* off;         // [B*heads*Np + 1] start of each key's list in `entries`
    const int32_t* coff;        // [B*heads*Np + 1] first chunk of each key; coff[B*heads*Np] = chunks
    const int32_t* chunk_key;   // [chunks] the key (b*heads + h)*Np + J of each chunk
    int32_t* entries;           // [B*heads*Np*Kp] P*Kp + r of every kept pair, grouped by key
    float* partial;             // [chunks][4][2][d] per-chunk sums of keys with several chunks
    // l == 0: the combination's backward for the coarser levels j >= 1
    float* dm_out[QTA_MAX_LEVELS];          // dLoss/dm^j: j = 1 written, j >= 2 accumulated (zeroed first)
    const float* msg_fwd[QTA_MAX_LEVELS];   // the forward's messages m^j (for dw)
    int lvl_W[QTA_MAX_LEVELS];
    int lvl_N[QTA_MAX_LEVELS];
};

// Scans of the kept-by counts of one level (n = B*heads*Np key slots, blocks of 1024).
struct BwdScanArgs {
    int n, nblocks;
    int32_t* count;
    int32_t* off;
    int32_t* coff;
    int32_t* chunk_key;
    int32_t* block_sums;        // [2 * nblocks]
};

struct BwdFillArgs {
    const int32_t* parent_idx;  // [n][Kp]
    const int32_t* slot;        // [n][Kp]
    long long nentries;         // n * Kp
    int Kp, Np;
    const int32_t* off;
    int32_t* entries;
};

// Backward of the coarsest level (Eq. 1 over all N keys), in two passes: per query (dq and the
// softmax statistics) and per key (dk, dv), both without atomics.
struct BwdCoarseArgs {
    const void* q;
    const void* k;
    const void* v;
    int B, heads, N, C, K;      // K: keys kept per coarse query (0 for a single level)
    float scale;
    const int32_t* sel_idx;     // QuadTree-A with levels > 1
    const float* dsig;          // QuadTree-A with levels > 1: dLoss/d(kept scores)
    const float* dm;            // levels > 1: dLoss/dm fp32 [B][N][C]
    const void* dout;           // single level: upstream gradient (storage type)
    const float* w;             // single level, QuadTree-B: [B][N][heads][1] or NULL
    int variant_b;
    float* stats;               // [B][heads][N][4]: row max, row sum, sum_j p_j ds_j
    float* dq;                  // fp32 [B][N][C], written
    float* dk;
    float* dv;
    float* dw;                  // single level, QuadTree-B with w
};

// Adds to the level-0 gradients every coarser level's, split evenly among valid children.
struct BwdUnpoolArgs {
    int v_pooled;               // 0: V's coarser levels were given (their gradients stay there)
    int B, C, L;
    int H[QTA_MAX_LEVELS], W[QTA_MAX_LEVELS];
    FastDiv div_cpt, div_W1;    // divisions by C/4 and W[1]; set by the launcher
    int bpb;                    // blocks per batch element; set by the launcher
    const float* gq[QTA_MAX_LEVELS];
    const float* gk[QTA_MAX_LEVELS];
    const float* gv[QTA_MAX_LEVELS];
    float* dq;
    float* dk;
    float* dv;
};

struct FillRange {
    float* p;
    size_t n;                   // floats, a multiple of 4, p 16-byte aligned
};

struct TopkArgs {
    const float* keys;
    const int32_t* cand_idx;
    int rows, n, K;
    int32_t* idx_out;
    float* key_out;
};

// Per-device caches: entry `dev` of a table of 64 atomics, filled on first use (several host threads
// may race to fill an entry; they all store the same value).
inline int cached_device_attribute(std::atomic<int> (&cache)[64], hipDeviceAttribute_t attr, int fallback)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return fallback;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        if (hipDeviceGetAttribute(&v, attr, dev) != hipSuccess || v <= 0) v = fallback;
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

// Largest dynamic LDS a workgroup may use on the current device.
inline size_t device_max_lds()
{
    static std::atomic<int> cache[64];
    return static_cast<size_t>(cached_device_attribute(cache, hipDeviceAttributeMaxSharedMemoryPerBlock, 64 * 1024));
}

// Compute units of the current device.
inline int device_cu_count()
{
    static std::atomic<int> cache[64];
    return cached_device_attribute(cache, hipDeviceAttributeMultiprocessorCount, 256);
}

// Raises kernel `fn`'s dynamic-LDS limit to the current device's maximum, once per device: `done` is
// that kernel's set of devices already configured (bit `dev`). Racing threads may both set the
// attribute, which is harmless.
inline hipError_t set_max_lds_once(const void* fn, std::atomic<unsigned long long>& done)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const unsigned long long bit = (dev >= 0 && dev < 64) ? 1ull << dev : 0ull;
    if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
    e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(device_max_lds()));
    if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_release);
    return e;
}

hipError_t launch_pyramid_pass(const PyramidPassArgs& a, int nlev, int ntensors, bool use_bf16, hipStream_t stream);
hipError_t launch_coarse_attn(const CoarseArgs& a, int d, bool variant_a, bool use_bf16, hipStream_t stream);
hipError_t launch_posenc(const PosEncArgs& a, bool use_bf16, hipStream_t stream);
hipError_t launch_posenc_bwd(const PosEncBwdArgs& a, bool use_bf16, hipStream_t stream);
hipError_t launch_fine_attn(const FineArgs& a, int d, bool variant_a, bool use_bf16, bool finest, hipStream_t stream);
hipError_t launch_topk(const TopkArgs& a, hipStream_t stream);
// Orders each of `rows` selection rows of K entries (idx int32, key fp32, in place) by (key descending,
// index ascending), empty slots (index -1) last.
hipError_t launch_sort_rows(int32_t* idx, float* key, long long rows, int K, hipStream_t stream);
hipError_t launch_fill_zero(const FillRange* r, int n, hipStream_t stream);
hipError_t launch_bwd_level(const BwdLevelArgs& a, int d, bool variant_a, bool use_bf16, bool finest,
                            hipStream_t stream);
hipError_t launch_bwd_keys(const BwdLevelArgs& a, const BwdScanArgs& sc, int d, bool variant_a, bool use_bf16,
                           bool finest, hipStream_t stream);
hipError_t launch_bwd_coarse(const BwdCoarseArgs& a, int d, bool variant_a, bool use_bf16, hipStream_t stream);
hipError_t launch_bwd_unpool(const BwdUnpoolArgs& a, hipStream_t stream);

}  // namespace qta
