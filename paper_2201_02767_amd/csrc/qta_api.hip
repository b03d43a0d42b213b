// C ABI of the QuadTree attention library: argument validation, level geometry, workspace layout
// and the launch sequence of qta_forward. Everything here runs on the host; validation finishes
// before the first launch, and nothing allocates, synchronises or copies.
#include <stddef.h>
#include <stdint.h>

#include "qta_internal.h"

using namespace qta;

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

size_t dtype_bytes(qta_dtype t) { return t == QTA_BF16 ? 2 : 4; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool dtype_ok(qta_dtype t) { return t == QTA_F32 || t == QTA_BF16; }

bool variant_ok(qta_variant v) { return v == QTA_VARIANT_A || v == QTA_VARIANT_B; }

// Level sizes by ceil halving. INVALID unless every level but the coarsest holds more than one
// token (a level above a 1x1 map would repeat it).
qta_status dims(int H, int W, int levels, int* Hl, int* Wl)
{
    if (H <= 0 || W <= 0 || levels <= 0) return QTA_ERR_INVALID;
    if (levels > QTA_MAX_LEVELS) return QTA_ERR_INVALID;
    if (static_cast<long long>(H) * W > 0x3FFFFFFFLL) return QTA_ERR_UNSUPPORTED;
    Hl[0] = H;
    Wl[0] = W;
    for (int l = 1; l < levels; ++l) {
        if (Hl[l - 1] == 1 && Wl[l - 1] == 1) return QTA_ERR_INVALID;
        Hl[l] = (Hl[l - 1] + 1) / 2;
        Wl[l] = (Wl[l - 1] + 1) / 2;
    }
    return QTA_OK;
}

// Shape checks shared by the attention calls.
qta_status check_problem(int B, int heads, int d, int K, qta_variant variant, qta_dtype dtype)
{
    if (B <= 0 || heads <= 0 || d <= 0 || K <= 0) return QTA_ERR_INVALID;
    if (!variant_ok(variant) || !dtype_ok(dtype)) return QTA_ERR_INVALID;
    if (d != 32 && d != 64) return QTA_ERR_UNSUPPORTED;
    if (K > QTA_MAX_K) return QTA_ERR_UNSUPPORTED;
    if (static_cast<long long>(heads) * d > (1 << 20)) return QTA_ERR_UNSUPPORTED;
    return QTA_OK;
}

// One batch element's token map must stay below 2^24 tokens and 2^31 bytes: the attention
// kernels address it with 32-bit offsets and 24-bit coordinate products.
qta_status map_ok(int H, int W, int heads, int d, qta_dtype dtype)
{
    const long long n = static_cast<long long>(H) * W;
    if (n >= (1LL << 24)) return QTA_ERR_UNSUPPORTED;
    if (n * heads * d * static_cast<long long>(dtype_bytes(dtype)) >= (1LL << 31)) return QTA_ERR_UNSUPPORTED;
    return QTA_OK;
}

// Keys kept per query at every selecting level: entry l (1 <= l <= levels-1) in [1, QTA_MAX_K].
qta_status check_k_levels(const int* Kl, int levels)
{
    if (levels > 1 && !Kl) return QTA_ERR_INVALID;
    for (int l = 1; l < levels; ++l) {
        if (Kl[l] <= 0) return QTA_ERR_INVALID;
        if (Kl[l] > QTA_MAX_K) return QTA_ERR_UNSUPPORTED;
    }
    return QTA_OK;
}

// Intermediate level l (produced by the pyramid, gathered by level l's attention) is stored
// parent-blocked when V comes from the pyramid. The input level stays NHWC: a blocked copy of it
// would cost a write and a read of k and v for no gain in the gathers.
bool use_blocked(const int* Kl, int l, int levels, bool v_supplied)
{
    (void)Kl;
    return !v_supplied && l >= 1 && l <= levels - 2;
}

// Whether level l's position encoding is computed inside that level's attention kernel: the coarsest
// level when it takes the tiled coarse kernel (more than 64 tokens), a finer level when its kernel is
// the one with at most 64 candidate slots and the level is not a one-row map (whose pairs of parents
// that kernel packs). The other levels get the separate encoding pass (level 0 through a workspace
// buffer, the others in place on their messages).
bool pe_level_fused(int l, int levels, const int* Hl, const int* Wl, const int* Kl)
{
    if (l == levels - 1) return Hl[l] * Wl[l] > 64;
    return !(Hl[l] == 1 && Hl[l + 1] == 1) && 4 * Kl[l + 1] <= 64;
}

qta_status layout(int B, int heads, int H, int W, int d, int levels, const int* Kl, bool v_supplied, bool pe,
                  qta_dtype dtype, qta_workspace_layout* L)
{
    qta_status st = check_problem(B, heads, d, 1, QTA_VARIANT_B, dtype);
    if (st != QTA_OK) return st;
    st = check_k_levels(Kl, levels);
    if (st != QTA_OK) return st;
    int Hl[QTA_MAX_LEVELS], Wl[QTA_MAX_LEVELS];
    st = dims(H, W, levels, Hl, Wl);
    if (st != QTA_OK) return st;
    if (static_cast<long long>(Hl[levels - 1]) * Wl[levels - 1] > QTA_MAX_COARSE) return QTA_ERR_UNSUPPORTED;
    st = map_ok(H, W, heads, d, dtype);
    if (st != QTA_OK) return st;
    *L = qta_workspace_layout{};
    L->levels = levels;
    const int C = heads * d;
    const int tb = static_cast<int>(dtype_bytes(dtype));
    size_t off = 0;
    for (int l = 0; l < levels; ++l) {
        L->H[l] = Hl[l];
        L->W[l] = Wl[l];
        L->K[l] = l >= 1 ? Kl[l] : 0;
        L->blocked[l] = use_blocked(Kl, l, levels, v_supplied) ? 1 : 0;
    }
    for (int l = 1; l < levels; ++l) {
        const size_t N = static_cast<size_t>(Hl[l]) * Wl[l];
        const size_t tok = level_bytes(L->blocked[l] != 0, B, Hl[l], Wl[l], C, tb);
        L->q[l] = off;
        off = align_up(off + tok);
        L->k[l] = off;
        off = align_up(off + tok);
        if (!v_supplied) {
            L->v[l] = off;
            off = align_up(off + tok);
        }
        L->msg[l] = off;
        off = align_up(off + static_cast<size_t>(B) * N * C * sizeof(float));
        L->sel_idx[l] = off;
        off = align_up(off + static_cast<size_t>(B) * heads * N * Kl[l] * sizeof(int32_t));
        L->sel_key[l] = off;
        off = align_up(off + static_cast<size_t>(B) * heads * N * Kl[l] * sizeof(float));
    }
    if (pe && !pe_level_fused(0, levels, Hl, Wl, Kl)) {
        L->pe0 = off;
        off = align_up(off + static_cast<size_t>(B) * Hl[0] * Wl[0] * C * sizeof(float));
    }
    L->total = off > kAlign ? off : kAlign;   // nonzero for every valid problem
    return QTA_OK;
}

// The options of qta_forward_ex with K filled in where K_levels is NULL.
struct Options {
    int Kl[QTA_MAX_LEVELS];
    const void* const* v_levels;
    const float* pe_weight;
    const float* pe_bias;
};

qta_status read_options(int K, int levels, const qta_options* opt, Options* o)
{
    o->v_levels = opt ? opt->v_levels : nullptr;
    o->pe_weight = opt ? opt->pe_weight : nullptr;
    o->pe_bias = opt ? opt->pe_bias : nullptr;
    const int* src = opt ? opt->K_levels : nullptr;
    if (levels <= 0 || levels > QTA_MAX_LEVELS) return QTA_ERR_INVALID;
    if (!src && K <= 0) return QTA_ERR_INVALID;
    if (!src && K > QTA_MAX_K) return QTA_ERR_UNSUPPORTED;
    for (int l = 0; l < QTA_MAX_LEVELS; ++l) o->Kl[l] = K;
    if (src)
        for (int l = 1; l < levels; ++l) o->Kl[l] = src[l];
    if (o->pe_bias && !o->pe_weight) return QTA_ERR_INVALID;
    const uintptr_t pw = reinterpret_cast<uintptr_t>(o->pe_weight), pb = reinterpret_cast<uintptr_t>(o->pe_bias);
    if ((pw & 15u) != 0 || (pb & 15u) != 0) return QTA_ERR_INVALID;
    return QTA_OK;
}

float resolve_scale(float scale, int d) { return scale > 0.f ? scale : 1.0f / __builtin_sqrtf(static_cast<float>(d)); }

qta_status launch_status(hipError_t e) { return e == hipSuccess ? QTA_OK : QTA_ERR_HIP; }

// Pyramid passes: from level s produce s+1 .. s+4 when exactly those remain, or s+1 .. s+3 when
// exactly those remain (and the tokens fit the four- or three-level pass), else s+1 and, when it
// exists, s+2; repeat from the last level made.
// `blocked` gives the storage of each level (level 0, the input, is NHWC).
hipError_t run_pyramid(const void* const* src0, void* (*lvl)[QTA_MAX_LEVELS], int ntensors, int B,
                       const int* Hl, const int* Wl, const int* blocked, int levels, int chunks, int head_chunks,
                       bool use_bf16, hipStream_t stream)
{
    for (int s = 0; s + 1 < levels;) {
        const bool four = levels - s == 5 && pyramid_tree_fits(4, chunks, head_chunks, Hl[s] == 1, Hl[s], Wl[s]);
        const bool three = levels - s == 4 && pyramid_tree_fits(3, chunks, head_chunks, Hl[s] == 1, Hl[s], Wl[s]);
        const int nlev = four ? 4 : three ? 3 : (s + 2 < levels) ? 2 : 1;
        PyramidPassArgs a{};
        for (int t = 0; t < ntensors; ++t) {
            a.src[t] = s == 0 ? src0[t] : lvl[t][s];
            a.dst1[t] = lvl[t][s + 1];
            a.dst2[t] = nlev >= 2 ? lvl[t][s + 2] : nullptr;
            a.dst3[t] = nlev >= 3 ? lvl[t][s + 3] : nullptr;
            a.dst4[t] = nlev == 4 ? lvl[t][s + 4] : nullptr;
        }
        a.B = B;
        a.Hs = Hl[s];
        a.Ws = Wl[s];
        a.H1 = Hl[s + 1];
        a.W1 = Wl[s + 1];
        a.H2 = nlev >= 2 ? Hl[s + 2] : 0;
        a.W2 = nlev >= 2 ? Wl[s + 2] : 0;
        a.H3 = nlev >= 3 ? Hl[s + 3] : 0;
        a.W3 = nlev >= 3 ? Wl[s + 3] : 0;
        a.H4 = nlev == 4 ? Hl[s + 4] : 0;
        a.W4 = nlev == 4 ? Wl[s + 4] : 0;
        a.chunks = chunks;
        a.head_chunks = head_chunks;
        a.lg_head_chunks = 0;
        while ((2 << a.lg_head_chunks) <= head_chunks) ++a.lg_head_chunks;
        a.src_blocked = s > 0 && blocked[s];
        a.dst1_blocked = blocked[s + 1] != 0;
        a.dst2_blocked = nlev >= 2 && blocked[s + 2] != 0;
        a.dst3_blocked = nlev >= 3 && blocked[s + 3] != 0;
        a.dst4_blocked = nlev == 4 && blocked[s + 4] != 0;
        hipError_t e = launch_pyramid_pass(a, nlev, ntensors, use_bf16, stream);
        if (e != hipSuccess) return e;
        s += nlev;
    }
    return hipSuccess;
}

// Workspace of the backward pass: per level l >= 1 the gradient of the message (dm) and the
// level's q, k, v gradients (fp32 [B][N_l][C]); QuadTree-A's gradients of the kept scores
// ([B][heads][N_l][K_l]); the coarse softmax statistics ([B][heads][N_c][4]); and per finer level
// its query statistics and the counting sort of its kept pairs (counts, places in the lists, list
// and chunk offsets, block sums, lists, chunk keys, per-chunk partial rows), separate per level so
// that one level's sort and key pass may run beside the next level's query pass. What is summed
// with atomics (dm at levels >= 2, the counts) forms one contiguous region, cleared at the start of
// every call; each level's scan returns its counts to zero.
struct BwdLayout {
    size_t dm[QTA_MAX_LEVELS], gq[QTA_MAX_LEVELS], gk[QTA_MAX_LEVELS], gv[QTA_MAX_LEVELS];
    size_t dsig[QTA_MAX_LEVELS];
    size_t zero_begin, zero_end;
    size_t stats, total;
    size_t count[QTA_MAX_LEVELS], off[QTA_MAX_LEVELS], coff[QTA_MAX_LEVELS], block_sums[QTA_MAX_LEVELS];
    size_t entries[QTA_MAX_LEVELS], slot[QTA_MAX_LEVELS], chunk_key[QTA_MAX_LEVELS], partial[QTA_MAX_LEVELS];
    size_t qstats[QTA_MAX_LEVELS];
    size_t pe_part;                 // with the position encoding: the per-block partial sums of its gradients
    long long nslots_max;           // B*heads*N_{l+1} over the finer levels
};

void bwd_layout(int B, int heads, const int* Hl, const int* Wl, int C, int d, int levels, const int* Kl, bool va,
                bool pe, BwdLayout* L)
{
    *L = BwdLayout{};
    const int c = levels - 1;
    auto fbytes = [&](int l) { return static_cast<size_t>(B) * Hl[l] * Wl[l] * C * sizeof(float); };
    auto nslots = [&](int l) { return static_cast<long long>(B) * heads * Hl[l + 1] * Wl[l + 1]; };
    for (int l = 0; l < c; ++l) L->nslots_max = nslots(l) > L->nslots_max ? nslots(l) : L->nslots_max;
    size_t off = 0;
    L->zero_begin = off;
    for (int l = 2; l <= c; ++l) {
        L->dm[l] = off;
        off = align_up(off + fbytes(l));
    }
    for (int l = 0; l < c; ++l) {       // padded to whole quads: the scan reads four counts at a time
        L->count[l] = off;
        off = align_up(off + static_cast<size_t>((nslots(l) + 3) & ~3LL) * sizeof(int32_t));
    }
    L->zero_end = off;
    if (c >= 1) {
        L->dm[1] = off;
        off = align_up(off + fbytes(1));
    }
    for (int l = 1; l <= c; ++l) {
        L->gk[l] = off;
        off = align_up(off + fbytes(l));
        L->gv[l] = off;
        off = align_up(off + fbytes(l));
        L->gq[l] = off;
        off = align_up(off + fbytes(l));
        if (va) {
            L->dsig[l] = off;
            off = align_up(off + static_cast<size_t>(B) * heads * Hl[l] * Wl[l] * Kl[l] * sizeof(float));
        }
    }
    L->stats = off;
    off = align_up(off + static_cast<size_t>(B) * heads * Hl[c] * Wl[c] * 4 * sizeof(float));
    for (int l = 0; l < c; ++l) {
        const long long n = nslots(l);
        const long long e = n * Kl[l + 1];
        const long long ch = n + (e + kKeyChunk - 1) / kKeyChunk;
        const long long st = static_cast<long long>(B) * heads * Hl[l] * Wl[l] * 2 * (va ? Kl[l + 1] : 1);
        L->off[l] = off;
        off = align_up(off + static_cast<size_t>(n + 1) * sizeof(int32_t));
        L->coff[l] = off;
        off = align_up(off + static_cast<size_t>(n + 1) * sizeof(int32_t));
        L->block_sums[l] = off;
        off = align_up(off + static_cast<size_t>(2 * ((n + 1023) / 1024)) * sizeof(int32_t));
        L->entries[l] = off;
        off = align_up(off + static_cast<size_t>(e) * sizeof(int32_t));
        L->slot[l] = off;
        off = align_up(off + static_cast<size_t>(e) * sizeof(int32_t));
        L->chunk_key[l] = off;
        off = align_up(off + static_cast<size_t>(ch) * sizeof(int32_t));
        L->partial[l] = off;
        off = align_up(off + static_cast<size_t>(ch) * 8 * d * sizeof(float));
        L->qstats[l] = off;
        off = align_up(off + static_cast<size_t>(st) * sizeof(float));
    }
    if (pe) {
        L->pe_part = off;
        off = align_up(off + static_cast<size_t>(posenc_bwd_blocks(B, Hl, Wl, levels, C)) * C * 10 * sizeof(float));
    }
    L->total = off > kAlign ? off : kAlign;
}

}  // namespace

extern "C" {

const char* qta_status_str(qta_status status)
{
    switch (status) {
    case QTA_OK: return "ok";
    case QTA_ERR_INVALID: return "invalid argument";
    case QTA_ERR_UNSUPPORTED: return "unsupported shape or type";
    case QTA_ERR_WORKSPACE: return "workspace too small";
    case QTA_ERR_HIP: return "HIP launch failed";
    default: break;
    }
    return "unknown status";
}

qta_status qta_level_dims(int H, int W, int levels, int* Hl, int* Wl)
{
    if (!Hl || !Wl) return QTA_ERR_INVALID;
    return dims(H, W, levels, Hl, Wl);
}

// Epipolar attention is the same layer on every row as its own 1 x W map (B*H maps of 1 x W).
qta_status rows_as_maps(const qta_options* opt, int* B, int* H)
{
    if (!opt || !opt->epipolar) return QTA_OK;
    if (*B <= 0 || *H <= 0) return QTA_ERR_INVALID;
    const long long rows = static_cast<long long>(*B) * *H;
    if (rows > 0x7FFFFFFFLL) return QTA_ERR_UNSUPPORTED;
    *B = static_cast<int>(rows);
    *H = 1;
    return QTA_OK;
}

qta_status qta_get_workspace_layout_ex(int B, int heads, int H, int W, int d, int levels, int K, qta_dtype dtype,
                                       const qta_options* opt, qta_workspace_layout* out)
{
    if (!out) return QTA_ERR_INVALID;
    qta_status rs = rows_as_maps(opt, &B, &H);
    if (rs != QTA_OK) return rs;
    Options o;
    qta_status st = read_options(K, levels, opt, &o);
    if (st != QTA_OK) return st;
    return layout(B, heads, H, W, d, levels, o.Kl, o.v_levels != nullptr, o.pe_weight != nullptr, dtype, out);
}

size_t qta_workspace_bytes_ex(int B, int heads, int H, int W, int d, int levels, int K, qta_dtype dtype,
                              const qta_options* opt)
{
    qta_workspace_layout L;
    if (qta_get_workspace_layout_ex(B, heads, H, W, d, levels, K, dtype, opt, &L) != QTA_OK) return 0;
    return L.total;
}

qta_status qta_get_workspace_layout(int B, int heads, int H, int W, int d, int levels, int K, qta_dtype dtype,
                                    qta_workspace_layout* out)
{
    return qta_get_workspace_layout_ex(B, heads, H, W, d, levels, K, dtype, nullptr, out);
}

size_t qta_workspace_bytes(int B, int heads, int H, int W, int d, int levels, int K, qta_dtype dtype)
{
    return qta_workspace_bytes_ex(B, heads, H, W, d, levels, K, dtype, nullptr);
}

qta_status qta_build_pyramid(const void* x, void* levels_out, int B, int H, int W, int C, int levels, qta_dtype dtype,
                             void* stream)
{
    if (!x || !levels_out || B <= 0 || C <= 0 || !dtype_ok(dtype)) return QTA_ERR_INVALID;
    if (!aligned16(x) || !aligned16(levels_out)) return QTA_ERR_INVALID;
    if ((static_cast<size_t>(C) * dtype_bytes(dtype)) % 16 != 0) return QTA_ERR_UNSUPPORTED;
    int Hl[QTA_MAX_LEVELS], Wl[QTA_MAX_LEVELS];
    qta_status st = dims(H, W, levels, Hl, Wl);
    if (st != QTA_OK) return st;
    if (levels == 1) return QTA_OK;
    void* lvl[1][QTA_MAX_LEVELS] = {};
    size_t off = 0;
    for (int l = 1; l < levels; ++l) {
        lvl[0][l] = static_cast<char*>(levels_out) + off;
        off += static_cast<size_t>(B) * Hl[l] * Wl[l] * C * dtype_bytes(dtype);
    }
    const void* src[1] = {x};
    const int chunks = static_cast<int>(static_cast<size_t>(C) * dtype_bytes(dtype) / 16);
    const int nhwc[QTA_MAX_LEVELS] = {};
    return launch_status(run_pyramid(src, lvl, 1, B, Hl, Wl, nhwc, levels, chunks, chunks,
                                     dtype == QTA_BF16, static_cast<hipStream_t>(stream)));
}

qta_status qta_coarse_attn(const void* qc, const void* kc, const void* vc, int B, int heads, int Hc, int Wc, int d,
                           int K, qta_variant variant, qta_dtype dtype, float scale, float* msg, int32_t* sel_idx,
                           float* sel_key, void* stream)
{
    qta_status st = check_problem(B, heads, d, K, variant, dtype);
    if (st != QTA_OK) return st;
    if (!qc || !kc || !vc || !msg) return QTA_ERR_INVALID;
    if ((sel_idx == nullptr) != (sel_key == nullptr)) return QTA_ERR_INVALID;
    if (!aligned16(qc) || !aligned16(kc) || !aligned16(vc) || !aligned16(msg)) return QTA_ERR_INVALID;
    if (Hc <= 0 || Wc <= 0) return QTA_ERR_INVALID;
    if (static_cast<long long>(Hc) * Wc > QTA_MAX_COARSE) return QTA_ERR_UNSUPPORTED;
    CoarseArgs a{};
    a.q = qc;
    a.k = kc;
    a.v = vc;
    a.B = B;
    a.heads = heads;
    a.N = Hc * Wc;
    a.C = heads * d;
    a.K = sel_idx ? K : 0;
    a.scale = resolve_scale(scale, d);
    a.msg = msg;
    a.sel_idx = sel_idx;
    a.sel_key = sel_key;
    a.levels = 1;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (launch_coarse_attn(a, d, variant == QTA_VARIANT_A, dtype == QTA_BF16, s) != hipSuccess) return QTA_ERR_HIP;
    // the stage call returns each row ordered (inside qta_forward a selection stays an unordered set)
    if (!sel_idx) return QTA_OK;
    return launch_status(launch_sort_rows(sel_idx, sel_key, static_cast<long long>(B) * heads * Hc * Wc, K, s));
}

qta_status qta_topk(const float* keys, const int32_t* cand_idx, int rows, int n, int K, int32_t* idx_out,
                    float* key_out, void* stream)
{
    if (!keys || !idx_out || rows <= 0 || n <= 0 || K <= 0) return QTA_ERR_INVALID;
    if (n > 4096 || K > QTA_MAX_K) return QTA_ERR_UNSUPPORTED;
    if (static_cast<long long>(rows) * n > (1LL << 40)) return QTA_ERR_UNSUPPORTED;
    TopkArgs a{keys, cand_idx, rows, n, K, idx_out, key_out};
    return launch_status(launch_topk(a, static_cast<hipStream_t>(stream)));
}

qta_status qta_fine_attn(const void* ql, const void* kl, const void* vl, int B, int heads, int Hl, int Wl, int d, int K,
                         qta_variant variant, qta_dtype dtype, float scale, const int32_t* parent_idx,
                         const float* parent_key, float* msg, int32_t* sel_idx, float* sel_key, void* stream)
{
    qta_status st = check_problem(B, heads, d, K, variant, dtype);
    if (st != QTA_OK) return st;
    if (!ql || !kl || !vl || !parent_idx || !msg || !sel_idx || !sel_key) return QTA_ERR_INVALID;
    if (variant == QTA_VARIANT_A && !parent_key) return QTA_ERR_INVALID;
    if (!aligned16(ql) || !aligned16(kl) || !aligned16(vl) || !aligned16(msg)) return QTA_ERR_INVALID;
    if (Hl <= 0 || Wl <= 0 || (Hl == 1 && Wl == 1)) return QTA_ERR_INVALID;
    st = map_ok(Hl, Wl, heads, d, dtype);
    if (st != QTA_OK) return st;
    FineArgs a{};
    a.q = ql;
    a.k = kl;
    a.v = vl;
    a.B = B;
    a.heads = heads;
    a.H = Hl;
    a.W = Wl;
    a.Hp = (Hl + 1) / 2;
    a.Wp = (Wl + 1) / 2;
    a.C = heads * d;
    a.Kp = K;
    a.Ks = K;
    a.scale = resolve_scale(scale, d);
    a.parent_idx = parent_idx;
    a.parent_key = parent_key;
    a.msg = msg;
    a.sel_idx = sel_idx;
    a.sel_key = sel_key;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (launch_fine_attn(a, d, variant == QTA_VARIANT_A, dtype == QTA_BF16, false, s) != hipSuccess) return QTA_ERR_HIP;
    // the stage call returns each row ordered (inside qta_forward a selection stays an unordered set)
    return launch_status(launch_sort_rows(sel_idx, sel_key, static_cast<long long>(B) * heads * Hl * Wl, K, s));
}

qta_status qta_finest_attn(const void* q0, const void* k0, const void* v0, int B, int heads, int H, int W, int d, int K,
                           qta_variant variant, qta_dtype dtype, float scale, const int32_t* parent_idx,
                           const float* parent_key, int levels, const float* const* coarser_msg, const float* w,
                           void* out, void* stream)
{
    qta_status st = check_problem(B, heads, d, K, variant, dtype);
    if (st != QTA_OK) return st;
    if (!q0 || !k0 || !v0 || !parent_idx || !out || !coarser_msg) return QTA_ERR_INVALID;
    if (variant == QTA_VARIANT_A && !parent_key) return QTA_ERR_INVALID;
    if (!aligned16(q0) || !aligned16(k0) || !aligned16(v0) || !aligned16(out)) return QTA_ERR_INVALID;
    if (levels < 2) return QTA_ERR_INVALID;
    int Hl[QTA_MAX_LEVELS], Wl[QTA_MAX_LEVELS];
    st = dims(H, W, levels, Hl, Wl);
    if (st != QTA_OK) return st;
    st = map_ok(H, W, heads, d, dtype);
    if (st != QTA_OK) return st;
    FineArgs a{};
    a.q = q0;
    a.k = k0;
    a.v = v0;
    a.B = B;
    a.heads = heads;
    a.H = H;
    a.W = W;
    a.Hp = Hl[1];
    a.Wp = Wl[1];
    a.C = heads * d;
    a.Kp = K;
    a.Ks = 0;
    a.scale = resolve_scale(scale, d);
    a.parent_idx = parent_idx;
    a.parent_key = parent_key;
    a.out = out;
    a.w = w;
    a.levels = levels;
    for (int l = 1; l < levels; ++l) {
        if (!coarser_msg[l - 1] || !aligned16(coarser_msg[l - 1])) return QTA_ERR_INVALID;
        a.coarser_msg[l] = coarser_msg[l - 1];
        a.lvl_W[l] = Wl[l];
        a.lvl_N[l] = Hl[l] * Wl[l];
    }
    return launch_status(launch_fine_attn(a, d, variant == QTA_VARIANT_A, dtype == QTA_BF16, true,
                                          static_cast<hipStream_t>(stream)));
}

qta_status qta_forward_ex(const void* q, const void* k, const void* v, const float* w, int B, int heads, int H, int W,
                          int d, int levels, int K, qta_variant variant, qta_dtype dtype, float scale,
                          const qta_options* opt, void* out, void* workspace, size_t workspace_bytes, void* stream)
{
    qta_status st = check_problem(B, heads, d, 1, variant, dtype);
    if (st != QTA_OK) return st;
    if (!q || !k || !v || !out) return QTA_ERR_INVALID;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return QTA_ERR_INVALID;
    st = rows_as_maps(opt, &B, &H);
    if (st != QTA_OK) return st;
    Options o;
    st = read_options(K, levels, opt, &o);
    if (st != QTA_OK) return st;
    const void* const* v_levels = o.v_levels;
    const bool v_supplied = v_levels != nullptr;
    const bool pe = o.pe_weight != nullptr;
    if (v_supplied)
        for (int l = 1; l < levels && l < QTA_MAX_LEVELS; ++l)
            if (!v_levels[l] || !aligned16(v_levels[l])) return QTA_ERR_INVALID;
    qta_workspace_layout L;
    st = layout(B, heads, H, W, d, levels, o.Kl, v_supplied, pe, dtype, &L);
    if (st != QTA_OK) return st;
    const int* Kl = o.Kl;
    if (levels > 1 || pe) {
        if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return QTA_ERR_INVALID;
        if (workspace_bytes < L.total) return QTA_ERR_WORKSPACE;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool use_bf16 = dtype == QTA_BF16;
    const bool va = variant == QTA_VARIANT_A;
    const float tau = resolve_scale(scale, d);
    const int C = heads * d;
    char* ws = static_cast<char*>(workspace);
    const void* lv[3][QTA_MAX_LEVELS] = {};
    void* pyr[3][QTA_MAX_LEVELS] = {};
    lv[0][0] = q;
    lv[1][0] = k;
    lv[2][0] = v;
    for (int l = 1; l < levels; ++l) {
        pyr[0][l] = ws + L.q[l];
        pyr[1][l] = ws + L.k[l];
        pyr[2][l] = v_supplied ? nullptr : ws + L.v[l];
        lv[0][l] = pyr[0][l];
        lv[1][l] = pyr[1][l];
        lv[2][l] = v_supplied ? v_levels[l] : pyr[2][l];
    }
    auto msg = [&](int l) { return reinterpret_cast<float*>(ws + L.msg[l]); };
    auto sidx = [&](int l) { return reinterpret_cast<int32_t*>(ws + L.sel_idx[l]); };
    auto skey = [&](int l) { return reinterpret_cast<float*>(ws + L.sel_key[l]); };

    // 1. pyramids of q, k and v (intermediate levels blocked when the layout says so)
    if (levels > 1) {
        const void* src[3] = {q, k, v};
        const int chunks = static_cast<int>(static_cast<size_t>(C) * dtype_bytes(dtype) / 16);
        const int head_chunks = static_cast<int>(static_cast<size_t>(d) * dtype_bytes(dtype) / 16);
        hipError_t e = run_pyramid(src, pyr, v_supplied ? 2 : 3, B, L.H, L.W, L.blocked, levels, chunks,
                                   head_chunks, use_bf16, s);
        if (e != hipSuccess) return QTA_ERR_HIP;
    }

    // multiscale position encoding: each level's attention kernel adds its own where it can
    // (pe_level_fused); one separate pass covers the other levels, adding it in place to the messages
    // of levels above 0 and writing level 0's to the workspace for the finest kernel (launched right
    // before that kernel)
    bool fused[QTA_MAX_LEVELS] = {};
    int unfused = 0;
    for (int l = 0; l < levels; ++l) {
        fused[l] = pe && pe_level_fused(l, levels, L.H, L.W, o.Kl);
        unfused += (pe && !fused[l]) ? 1 : 0;
    }
    auto pe_w = [&](int l) { return fused[l] ? o.pe_weight + static_cast<size_t>(l) * C * 9 : nullptr; };
    auto pe_b = [&](int l) { return (fused[l] && o.pe_bias) ? o.pe_bias + static_cast<size_t>(l) * C : nullptr; };
    float* pe0 = (pe && !fused[0]) ? reinterpret_cast<float*>(ws + L.pe0) : nullptr;
    // the separate encoding pass over the levels whose kernel does not fuse it
    auto posenc = [&]() -> hipError_t {
        if (unfused == 0) return hipSuccess;
        PosEncArgs p{};
        p.nlev = 0;
        p.B = B;
        p.heads = heads;
        p.d = d;
        for (int l = 0; l < levels; ++l) {
            if (fused[l]) continue;
            PosEncLevel& e = p.lv[p.nlev++];
            e.v = l == 0 ? v : lv[2][l];
            e.blocked = l == 0 ? 0 : L.blocked[l];
            e.H = L.H[l];
            e.W = L.W[l];
            e.dst = l == 0 ? pe0 : msg(l);
            e.accumulate = l == 0 ? 0 : 1;
            e.weight = o.pe_weight + static_cast<size_t>(l) * C * 9;
            e.bias = o.pe_bias ? o.pe_bias + static_cast<size_t>(l) * C : nullptr;
        }
        return launch_posenc(p, use_bf16, s);
    };

    // 2-3. coarsest level
    const int c = levels - 1;
    {
        CoarseArgs a{};
        a.q = lv[0][c];
        a.k = lv[1][c];
        a.v = lv[2][c];
        a.B = B;
        a.heads = heads;
        a.N = L.H[c] * L.W[c];
        a.C = C;
        a.scale = tau;
        a.levels = levels;
        a.pe_w = pe_w(c);
        a.pe_b = pe_b(c);
        a.Wc = L.W[c];
        if (levels == 1) {
            a.K = 0;
            a.out = out;
            a.w = w;
            if (pe) {
                hipError_t e = posenc();
                if (e != hipSuccess) return QTA_ERR_HIP;
                a.pe0 = pe0;
            }
        } else {
            a.K = Kl[c];
            a.msg = msg(c);
            a.sel_idx = sidx(c);
            a.sel_key = skey(c);
        }
        hipError_t e = launch_coarse_attn(a, d, va, use_bf16, s);
        if (e != hipSuccess) return QTA_ERR_HIP;
    }
    if (levels == 1) return QTA_OK;

    // 3-4. intermediate levels, coarse to fine
    for (int l = c - 1; l >= 1; --l) {
        FineArgs a{};
        a.q = lv[0][l];
        a.k = lv[1][l];
        a.v = lv[2][l];
        a.q_blocked = L.blocked[l] != 0;
        a.kv_blocked = L.blocked[l] != 0;
        a.B = B;
        a.heads = heads;
        a.H = L.H[l];
        a.W = L.W[l];
        a.Hp = L.H[l + 1];
        a.Wp = L.W[l + 1];
        a.C = C;
        a.Kp = Kl[l + 1];
        a.Ks = Kl[l];
        a.scale = tau;
        a.parent_idx = sidx(l + 1);
        a.parent_key = skey(l + 1);
        a.msg = msg(l);
        a.sel_idx = sidx(l);
        a.sel_key = skey(l);
        a.pe_w = pe_w(l);
        a.pe_b = pe_b(l);
        hipError_t e = launch_fine_attn(a, d, va, use_bf16, false, s);
        if (e != hipSuccess) return QTA_ERR_HIP;
    }

    // 4-5. finest level with the combination fused in
    if (pe) {
        hipError_t e = posenc();
        if (e != hipSuccess) return QTA_ERR_HIP;
    }
    {
        FineArgs a{};
        a.q = q;
        a.k = k;
        a.v = v;
        a.q_blocked = false;
        a.kv_blocked = false;
        a.B = B;
        a.heads = heads;
        a.H = H;
        a.W = W;
        a.Hp = L.H[1];
        a.Wp = L.W[1];
        a.C = C;
        a.Kp = Kl[1];
        a.Ks = 0;
        a.scale = tau;
        a.parent_idx = sidx(1);
        a.parent_key = skey(1);
        a.out = out;
        a.w = w;
        a.pe0 = pe0;
        a.pe_w = pe_w(0);
        a.pe_b = pe_b(0);
        a.levels = levels;
        for (int l = 1; l < levels; ++l) {
            a.coarser_msg[l] = msg(l);
            a.lvl_W[l] = L.W[l];
            a.lvl_N[l] = L.H[l] * L.W[l];
        }
        hipError_t e = launch_fine_attn(a, d, va, use_bf16, true, s);
        if (e != hipSuccess) return QTA_ERR_HIP;
    }
    return QTA_OK;
}

qta_status qta_forward(const void* q, const void* k, const void* v, const float* w, int B, int heads, int H, int W,
                       int d, int levels, int K, qta_variant variant, qta_dtype dtype, float scale, void* out,
                       void* workspace, size_t workspace_bytes, void* stream)
{
    return qta_forward_ex(q, k, v, w, B, heads, H, W, d, levels, K, variant, dtype, scale, nullptr, out, workspace,
                          workspace_bytes, stream);
}

}  // extern "C"

// ---- the forward without a caller workspace ----
// The workspace of qta_forward_ex_noalloc: one array per device, in the library's code object, so
// that a call allocates nothing. In host code `scratch` names a host-side stand-in, never the device
// memory: the device address is looked up per device (scratch_device_ptr) and only that is used.
static __device__ __align__(256) unsigned char scratch[QTA_NOALLOC_WORKSPACE_BYTES];

namespace {

std::atomic<void*> scratch_address[64];      // per device: the device address of `scratch`

// The device address of `scratch` on the current device, looked up on the first call on that device
// (with that device current); racing threads store the same address.
qta_status scratch_device_ptr(void** out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return QTA_ERR_HIP;
    if (dev < 0 || dev >= 64) return QTA_ERR_UNSUPPORTED;
    void* p = scratch_address[dev].load(std::memory_order_acquire);
    if (!p) {
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return QTA_ERR_HIP;
        if ((reinterpret_cast<uintptr_t>(p) & (kAlign - 1)) != 0) return QTA_ERR_HIP;
        scratch_address[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return QTA_OK;
}

}  // namespace

extern "C" {

qta_status qta_forward_ex_noalloc(const void* q, const void* k, const void* v, const float* w, int B, int heads, int H,
                                  int W, int d, int levels, int K, qta_variant variant, qta_dtype dtype, float scale,
                                  const qta_options* opt, void* out, void* stream)
{
    // everything qta_forward_ex validates before it touches the workspace, so that a rejected call
    // does not reach the device either
    qta_status st = check_problem(B, heads, d, 1, variant, dtype);
    if (st != QTA_OK) return st;
    if (!q || !k || !v || !out) return QTA_ERR_INVALID;
    qta_workspace_layout L;
    st = qta_get_workspace_layout_ex(B, heads, H, W, d, levels, K, dtype, opt, &L);
    if (st != QTA_OK) return st;
    if (L.total > QTA_NOALLOC_WORKSPACE_BYTES) return QTA_ERR_WORKSPACE;
    void* ws = nullptr;
    st = scratch_device_ptr(&ws);
    if (st != QTA_OK) return st;
    return qta_forward_ex(q, k, v, w, B, heads, H, W, d, levels, K, variant, dtype, scale, opt, out, ws,
                          QTA_NOALLOC_WORKSPACE_BYTES, stream);
}

}  // extern "C"

extern "C" {

size_t qta_backward_workspace_bytes_ex(int B, int heads, int H, int W, int d, int levels, int K, qta_variant variant,
                                       qta_dtype dtype, const qta_options* opt)
{
    if (rows_as_maps(opt, &B, &H) != QTA_OK) return 0;
    if (!variant_ok(variant)) return 0;
    Options o;
    if (read_options(K, levels, opt, &o) != QTA_OK) return 0;
    qta_workspace_layout L;
    if (layout(B, heads, H, W, d, levels, o.Kl, o.v_levels != nullptr, o.pe_weight != nullptr, dtype, &L) != QTA_OK)
        return 0;
    BwdLayout G;
    bwd_layout(B, heads, L.H, L.W, heads * d, d, levels, o.Kl, variant == QTA_VARIANT_A, o.pe_weight != nullptr, &G);
    return G.total;
}

}  // extern "C"

namespace {

// The backward pass; with only_finest, just the level-0 kernel (for profiling it alone).
qta_status backward_impl(const void* q, const void* k, const void* v, const float* w, const void* dout, int B,
                         int heads, int H, int W, int d, int levels, int K, qta_variant variant, qta_dtype dtype,
                         float scale, const qta_options* opt, const void* workspace, size_t workspace_bytes,
                         float* dq, float* dk, float* dv, float* dw, void* bwd_workspace, size_t bwd_workspace_bytes,
                         void* stream, bool only_finest)
{
    qta_status st = check_problem(B, heads, d, 1, variant, dtype);
    if (st != QTA_OK) return st;
    if (!q || !k || !v || !dout || !dq || !dk || !dv) return QTA_ERR_INVALID;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(dout) || !aligned16(dq) || !aligned16(dk) ||
        !aligned16(dv))
        return QTA_ERR_INVALID;
    st = rows_as_maps(opt, &B, &H);
    if (st != QTA_OK) return st;
    Options o;
    st = read_options(K, levels, opt, &o);
    if (st != QTA_OK) return st;
    const bool v_supplied = o.v_levels != nullptr;
    const bool pe = o.pe_weight != nullptr;
    if (v_supplied) {
        if (!opt->dv_levels) return QTA_ERR_INVALID;
        for (int l = 1; l < levels && l < QTA_MAX_LEVELS; ++l)
            if (!o.v_levels[l] || !aligned16(o.v_levels[l]) || !opt->dv_levels[l] || !aligned16(opt->dv_levels[l]))
                return QTA_ERR_INVALID;
    }
    if (pe) {
        if (!opt->dpe_weight || !aligned16(opt->dpe_weight)) return QTA_ERR_INVALID;
        if (o.pe_bias && !opt->dpe_bias) return QTA_ERR_INVALID;
        if (static_cast<long long>(heads) * d > 256) return QTA_ERR_UNSUPPORTED;
    }
    qta_workspace_layout L;
    st = layout(B, heads, H, W, d, levels, o.Kl, v_supplied, pe, dtype, &L);
    if (st != QTA_OK) return st;
    const int* Kl = o.Kl;
    for (int l = 1; l < levels; ++l)
        if (4 * Kl[l] > 64) return QTA_ERR_UNSUPPORTED;
    if (levels > 1) {
        if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return QTA_ERR_INVALID;
        if (workspace_bytes < L.total) return QTA_ERR_WORKSPACE;
    }
    const bool va = variant == QTA_VARIANT_A;
    const int C = heads * d;
    BwdLayout G;
    bwd_layout(B, heads, L.H, L.W, C, d, levels, Kl, va, pe, &G);
    if (G.nslots_max >= 0x7FFFFFFFLL / 64) return QTA_ERR_UNSUPPORTED;     // sort indices are int
    if (!bwd_workspace || (reinterpret_cast<uintptr_t>(bwd_workspace) & (kAlign - 1)) != 0) return QTA_ERR_INVALID;
    if (bwd_workspace_bytes < G.total) return QTA_ERR_WORKSPACE;
    float* dw_out = (!va && w) ? dw : nullptr;

    hipStream_t s = static_cast<hipStream_t>(stream);
    // the finest level's counting sort and key pass go to the auxiliary stream when there is one
    // (not for the finest step alone); `after(x, y)` orders later work on y after the work issued
    // so far on x
    hipStream_t s2 = (opt && opt->aux_stream && !only_finest && levels > 1) ? static_cast<hipStream_t>(opt->aux_stream) : s;
    // with a third stream the coarser finer levels' sorts and key passes go there
    hipStream_t s3 = (s2 != s && opt->aux_stream2) ? static_cast<hipStream_t>(opt->aux_stream2) : s;
    // (both streams feed this device's kernels only: a device-scope release is enough, and the
    // system-scope one would add a cache write-back on every hand-over)
    auto after = [](hipStream_t x, hipStream_t y) {
        hipEvent_t e;
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming | hipEventDisableSystemFence) != hipSuccess) return false;
        const bool ok = hipEventRecord(e, x) == hipSuccess && hipStreamWaitEvent(y, e, 0) == hipSuccess;
        return hipEventDestroy(e) == hipSuccess && ok;
    };
    struct DeferredKeys {
        BwdLevelArgs a;
        BwdScanArgs sc;
        int level;
    };
    DeferredKeys deferred[QTA_MAX_LEVELS];
    int ndeferred = 0;
    const long long coarse_tiles = static_cast<long long>(B) * heads * ((L.H[levels - 1] * L.W[levels - 1] + 15) / 16);
    const bool defer_coarser = s2 != s && s3 == s && coarse_tiles < device_cu_count();
    // (measured: a gain where one intermediate level sits below a coarse level that fills the
    // chip; with more intermediate levels, or a coarse level with idle units, a loss)
    const bool qside = !va && s3 != s && levels == 3 && coarse_tiles >= device_cu_count();
    const bool use_bf16 = dtype == QTA_BF16;
    const float tau = resolve_scale(scale, d);
    const char* ws = static_cast<const char*>(workspace);
    char* gws = static_cast<char*>(bwd_workspace);
    auto fptr = [&](size_t off) { return reinterpret_cast<float*>(gws + off); };
    auto sidx = [&](int l) { return reinterpret_cast<const int32_t*>(ws + L.sel_idx[l]); };
    auto skey = [&](int l) { return reinterpret_cast<const float*>(ws + L.sel_key[l]); };
    // V at level l >= 1 (given levels are the caller's), and where its gradient goes (given levels:
    // the caller's dv_levels, which the pyramid adjoint then leaves alone)
    auto vlev = [&](int l) -> const void* { return v_supplied ? o.v_levels[l] : ws + L.v[l]; };
    auto gvlev = [&](int l) -> float* { return v_supplied ? opt->dv_levels[l] : fptr(G.gv[l]); };
    const int c = levels - 1;
    if (only_finest && levels < 2) return QTA_ERR_INVALID;

    if (levels > 1 && !only_finest) {
        // clear what is accumulated: dm of levels >= 2 and the kept-by counts
        FillRange r[1];
        r[0] = FillRange{fptr(G.zero_begin), (G.zero_end - G.zero_begin) / sizeof(float)};
        if (launch_fill_zero(r, 1, s) != hipSuccess) return QTA_ERR_HIP;


    }
    if (levels > 1) {
        // 2. finer levels, finest first (QuadTree-A's score gradients go up one level each)
        for (int l = 0; l < (only_finest ? 1 : c); ++l) {
            // with an auxiliary stream the finest level's sort and key pass (the largest) go there
            // right after its query pass. The coarser levels' sorts and key passes go to the third
            // stream when there is one, each right after its level's query pass; with two streams
            // only, when the coarse level's tile kernels leave compute units idle (fewer 16-row
            // tiles than units) they follow those on the caller's stream, so that the coarse level
            // runs beside the finest key pass, and otherwise they go to the auxiliary stream too
            BwdLevelArgs a{};
            if (l == 0) {
                a.q = q;
                a.k = k;
                a.v = v;
                a.blocked = false;
                a.dout = dout;
                a.w = va ? nullptr : w;
                a.dq = dq;
                a.dk = dk;
                a.dv = dv;
                a.dw = dw_out;
                for (int j = 1; j < levels; ++j) {      // 1. the combination's backward
                    a.dm_out[j] = fptr(G.dm[j]);
                    a.msg_fwd[j] = reinterpret_cast<const float*>(ws + L.msg[j]);
                    a.lvl_W[j] = L.W[j];
                    a.lvl_N[j] = L.H[j] * L.W[j];
                }
            } else {
                a.q = ws + L.q[l];
                a.k = ws + L.k[l];
                a.v = vlev(l);
                a.blocked = L.blocked[l] != 0;
                a.sel_idx = sidx(l);
                a.dsig_in = va ? fptr(G.dsig[l]) : nullptr;
                a.dm = fptr(G.dm[l]);
                a.dq = fptr(G.gq[l]);
                a.dk = fptr(G.gk[l]);
                a.dv = gvlev(l);
            }
            a.B = B;
            a.heads = heads;
            a.H = L.H[l];
            a.W = L.W[l];
            a.Hp = L.H[l + 1];
            a.Wp = L.W[l + 1];
            a.C = C;
            a.Kp = Kl[l + 1];
            a.Ks = l >= 1 ? Kl[l] : 0;
            a.scale = tau;
            a.parent_idx = sidx(l + 1);
            a.parent_key = skey(l + 1);
            a.dsig_out = va ? fptr(G.dsig[l + 1]) : nullptr;
            a.levels = levels;
            a.stats = fptr(G.qstats[l]);
            a.count = reinterpret_cast<int32_t*>(gws + G.count[l]);
            a.off = reinterpret_cast<const int32_t*>(gws + G.off[l]);
            a.coff = reinterpret_cast<const int32_t*>(gws + G.coff[l]);
            a.chunk_key = reinterpret_cast<const int32_t*>(gws + G.chunk_key[l]);
            a.entries = reinterpret_cast<int32_t*>(gws + G.entries[l]);
            a.slot = reinterpret_cast<int32_t*>(gws + G.slot[l]);
            a.partial = fptr(G.partial[l]);
            // QuadTree-B with three streams and one intermediate level (`qside`): that level's query
            // pass needs only the finest query pass (every dm comes from it), so it runs on the
            // third stream beside the coarse level
            const hipStream_t sq = (l > 0 && qside) ? s3 : s;
            if (launch_bwd_level(a, d, va, use_bf16, l == 0, sq) != hipSuccess) return QTA_ERR_HIP;
            if (l == 0 && qside && !after(s, s3)) return QTA_ERR_HIP;
            // the stream of this level's sort and key pass, which need its query pass
            const hipStream_t sk = l == 0 ? s2 : (s3 != s ? s3 : (defer_coarser ? s : s2));
            if (sk != sq && !after(sq, sk)) return QTA_ERR_HIP;
            BwdScanArgs sc{};
            sc.n = B * heads * L.H[l + 1] * L.W[l + 1];
            sc.nblocks = (sc.n + 1023) / 1024;
            sc.count = a.count;
            sc.off = reinterpret_cast<int32_t*>(gws + G.off[l]);
            sc.coff = reinterpret_cast<int32_t*>(gws + G.coff[l]);
            sc.chunk_key = reinterpret_cast<int32_t*>(gws + G.chunk_key[l]);
            sc.block_sums = reinterpret_cast<int32_t*>(gws + G.block_sums[l]);
            if (s2 != s && l > 0 && defer_coarser) {
                deferred[ndeferred++] = DeferredKeys{a, sc, l};
                continue;
            }
            if (launch_bwd_keys(a, sc, d, va, use_bf16, l == 0, sk) != hipSuccess) return QTA_ERR_HIP;
        }
    }
    if (only_finest) return QTA_OK;

    // 3. coarsest level
    {
        BwdCoarseArgs a{};
        a.B = B;
        a.heads = heads;
        a.N = L.H[c] * L.W[c];
        a.C = C;
        a.scale = tau;
        a.variant_b = va ? 0 : 1;
        a.stats = fptr(G.stats);
        if (levels == 1) {
            a.q = q;
            a.k = k;
            a.v = v;
            a.K = 0;
            a.dout = dout;
            a.w = va ? nullptr : w;
            a.dq = dq;
            a.dk = dk;
            a.dv = dv;
            a.dw = dw_out;
        } else {
            a.q = ws + L.q[c];
            a.k = ws + L.k[c];
            a.v = vlev(c);
            a.K = Kl[c];
            a.sel_idx = sidx(c);
            a.dsig = va ? fptr(G.dsig[c]) : nullptr;
            a.dm = fptr(G.dm[c]);
            a.dq = fptr(G.gq[c]);
            a.dk = fptr(G.gk[c]);
            a.dv = gvlev(c);
        }
        if (launch_bwd_coarse(a, d, va, use_bf16, s) != hipSuccess) return QTA_ERR_HIP;
    }
    // the position encoding's backward (every level, once all of the level's v gradients are
    // written; before the unpooling, which reads them)
    auto posenc_bwd = [&]() -> hipError_t {
        PosEncBwdArgs p{};
        p.nlev = levels;
        p.B = B;
        p.heads = heads;
        p.d = d;
        p.variant_b = va ? 0 : 1;
        p.dout = dout;
        p.w = va ? nullptr : w;
        p.part = fptr(G.pe_part);
        p.dweight = opt->dpe_weight;
        p.dbias = o.pe_bias ? opt->dpe_bias : nullptr;
        p.bias0 = o.pe_bias;
        p.dw = dw_out;
        for (int l = 0; l < levels; ++l) {
            PosEncBwdLevel& e = p.lv[l];
            e.v = l == 0 ? v : vlev(l);
            e.blocked = l == 0 ? 0 : L.blocked[l];
            e.H = L.H[l];
            e.W = L.W[l];
            e.dm = l == 0 ? nullptr : fptr(G.dm[l]);
            e.dv = l == 0 ? dv : gvlev(l);
            e.weight = o.pe_weight + static_cast<size_t>(l) * C * 9;
        }
        return launch_posenc_bwd(p, use_bf16, s);
    };
    if (levels == 1) return (pe && posenc_bwd() != hipSuccess) ? QTA_ERR_HIP : QTA_OK;
    for (int i = 0; i < ndeferred; ++i)
        if (launch_bwd_keys(deferred[i].a, deferred[i].sc, d, va, use_bf16, false, s) != hipSuccess) return QTA_ERR_HIP;
    if (s2 != s && !after(s2, s)) return QTA_ERR_HIP;       // the key passes before the unpooling
    if (s3 != s && !after(s3, s)) return QTA_ERR_HIP;
    if (pe && posenc_bwd() != hipSuccess) return QTA_ERR_HIP;

    // 4. pyramids
    BwdUnpoolArgs u{};
    u.v_pooled = v_supplied ? 0 : 1;
    u.B = B;
    u.C = C;
    u.L = levels;
    for (int l = 0; l < levels; ++l) {
        u.H[l] = L.H[l];
        u.W[l] = L.W[l];
        if (l >= 1) {
            u.gq[l] = fptr(G.gq[l]);
            u.gk[l] = fptr(G.gk[l]);
            u.gv[l] = v_supplied ? nullptr : fptr(G.gv[l]);
        }
    }
    u.dq = dq;
    u.dk = dk;
    u.dv = dv;
    return launch_bwd_unpool(u, s) == hipSuccess ? QTA_OK : QTA_ERR_HIP;
}

}  // namespace

extern "C" {

qta_status qta_backward_ex(const void* q, const void* k, const void* v, const float* w, const void* dout, int B,
                           int heads, int H, int W, int d, int levels, int K, qta_variant variant, qta_dtype dtype,
                           float scale, const qta_options* opt, const void* workspace, size_t workspace_bytes,
                           float* dq, float* dk, float* dv, float* dw, void* bwd_workspace,
                           size_t bwd_workspace_bytes, void* stream)
{
    return backward_impl(q, k, v, w, dout, B, heads, H, W, d, levels, K, variant, dtype, scale, opt, workspace,
                         workspace_bytes, dq, dk, dv, dw, bwd_workspace, bwd_workspace_bytes, stream, false);
}

qta_status qta_backward_finest_ex(const void* q, const void* k, const void* v, const float* w, const void* dout,
                                  int B, int heads, int H, int W, int d, int levels, int K, qta_variant variant,
                                  qta_dtype dtype, float scale, const qta_options* opt, const void* workspace,
                                  size_t workspace_bytes, float* dq, float* dk, float* dv, float* dw,
                                  void* bwd_workspace, size_t bwd_workspace_bytes, void* stream)
{
    return backward_impl(q, k, v, w, dout, B, heads, H, W, d, levels, K, variant, dtype, scale, opt, workspace,
                         workspace_bytes, dq, dk, dv, dw, bwd_workspace, bwd_workspace_bytes, stream, true);
}

}  // extern "C"
