/*
 * qta.h - QuadTree attention forward on AMD Instinct MI355X (gfx950): the C ABI.
 *
 * The method is QuadTree attention (Tang et al., "QuadTree Attention for Vision Transformers",
 * ICLR 2022), Sec. 3.2. For every query token it computes a message from all key tokens in a
 * coarse-to-fine manner:
 *   1. L-level pyramids of Q, K and V by 2x2 average pooling (Sec. 3.2, pyramid paragraph);
 *   2. at the coarsest level every query attends to every key, Eq. (1);
 *   3. each query keeps the K keys with the highest attention scores (Sec. 3.2, Fig. 1);
 *   4. at each finer level a query attends only to the 2x2 children of its parent query's kept
 *      keys; the four sibling queries of one parent share that candidate set (Fig. 1 caption);
 *   5. the per-level messages are combined: QuadTree-A sums partial messages over the disjoint
 *      regions Omega^l (Eqs. 2-4), QuadTree-B takes a weighted sum of per-level attention over
 *      the overlapping regions Gamma^l (Eqs. 5-6).
 *
 * Conventions shared by every call
 *   - Level l = 0 is the finest level (the input map), l = L-1 the coarsest. Level l+1 has
 *     ceil(H_l/2) x ceil(W_l/2) tokens; token (y,x) at level l+1 averages its children
 *     (2y+dy, 2x+dx) at level l that lie inside the map (a missing child is not counted).
 *   - Token tensors are NHWC, [B][H][W][heads][d] contiguous (C = heads*d channels), in the
 *     storage type `dtype` (fp32 or bf16). Pyramid levels use the same layout at their size.
 *   - Flat token index at level l: y*W_l + x.
 *   - Messages are fp32 [B][N_l][heads][d]. Selections are int32 [B][heads][N_l][K] holding the
 *     flat key indices of level l that a query keeps: the first min(K, number of candidates)
 *     entries are the kept keys, the rest are -1. Scores are fp32 in the same shape, aligned with
 *     the indices (0 where the index is -1): QuadTree-B stores the softmax probability, QuadTree-A
 *     the recursive score s. The stage calls (qta_coarse_attn, qta_fine_attn) return every row
 *     ordered by (score descending, index ascending); the selections qta_forward keeps in its
 *     workspace are sets in an unspecified but deterministic order (no consumer needs them sorted).
 *   - Each head is an independent quadtree. Softmax temperature: `scale` if > 0, else 1/sqrt(d).
 *   - A query keeps the K candidates of highest score; ties at the cut go to the lower flat index.
 *
 * Memory and errors
 *   - Every tensor pointer is a DEVICE pointer that the caller owns; the library never
 *     allocates, frees, synchronises or copies back. Every call is asynchronous on `stream`
 *     (a hipStream_t; NULL is the null stream).
 *   - Arguments are validated on the host before any launch. Invalid shapes or null pointers
 *     return QTA_ERR_INVALID, shapes the kernels do not support QTA_ERR_UNSUPPORTED, a too-small
 *     workspace QTA_ERR_WORKSPACE; a failed launch returns QTA_ERR_HIP. Faults that happen on
 *     the device surface at the caller's next synchronisation.
 *   - Supported: d in {32, 64}; 1 <= K <= QTA_MAX_K; coarsest level N_{L-1} <= QTA_MAX_COARSE;
 *     1 <= L <= QTA_MAX_LEVELS with no level above a 1x1 map; token pointers 16-byte aligned;
 *     per batch element fewer than 2^24 tokens and 2^31 bytes in the token map (attention calls).
 *   - K larger than a query's candidate count is not an error: min(K, count) keys are kept.
 *   - Inputs must be finite; outputs must not alias inputs. Calls are re-entrant and may come from
 *     several host threads: the library keeps no data between calls. Its only process-wide state
 *     is per-device caches (device attributes, and each kernel's raised LDS limit, set once per
 *     device), filled with atomic operations on first use.
 */
#ifndef QTA_H
#define QTA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define QTA_MAX_LEVELS 16
#define QTA_MAX_K 64
#define QTA_MAX_COARSE 1024

/* Each enum ends with a sentinel at INT_MAX so that its range covers every int: a caller may pass
 * any int, and values other than the listed ones are rejected as QTA_ERR_INVALID. */
typedef enum {
    QTA_OK = 0,
    QTA_ERR_INVALID = 1,
    QTA_ERR_UNSUPPORTED = 2,
    QTA_ERR_WORKSPACE = 3,
    QTA_ERR_HIP = 4,
    QTA_STATUS_MAX_ENUM = 0x7FFFFFFF
} qta_status;

typedef enum { QTA_VARIANT_A = 0, QTA_VARIANT_B = 1, QTA_VARIANT_MAX_ENUM = 0x7FFFFFFF } qta_variant;

typedef enum { QTA_F32 = 0, QTA_BF16 = 1, QTA_DTYPE_MAX_ENUM = 0x7FFFFFFF } qta_dtype;

/* Byte offsets of the regions qta_forward keeps in its workspace. Entries for levels that do not
 * exist (and level 0 of q/k/v, msg, sel_idx, sel_key, which live outside it) are 0.
 * Intermediate pyramid levels (1 <= l <= levels-2: produced by pooling and gathered by level l's
 * attention) are stored parent-blocked when blocked[l] is 1:
 * [B][heads][ceil(H_l/2)][ceil(W_l/2)][2][2][d], i.e. the 2x2 children of one parent position of
 * one head are 4*d contiguous elements (off-map children are unused padding). The input level 0
 * and the coarsest level are NHWC. Blocking is used unless V's coarser levels are the caller's
 * (qta_options.v_levels). */
typedef struct {
    int levels;
    int H[QTA_MAX_LEVELS];
    int W[QTA_MAX_LEVELS];
    int blocked[QTA_MAX_LEVELS];    /* 1: pyramid level l is parent-blocked, 0: NHWC         */
    int K[QTA_MAX_LEVELS];          /* keys kept per query at level l >= 1 (0 at level 0)     */
    size_t q[QTA_MAX_LEVELS];       /* pyramid level l >= 1, dtype                          */
    size_t k[QTA_MAX_LEVELS];
    size_t v[QTA_MAX_LEVELS];
    size_t msg[QTA_MAX_LEVELS];     /* level l >= 1, fp32 [B][N_l][heads][d]                 */
    size_t sel_idx[QTA_MAX_LEVELS]; /* level l >= 1, int32 [B][heads][N_l][K_l]              */
    size_t sel_key[QTA_MAX_LEVELS]; /* level l >= 1, fp32  [B][heads][N_l][K_l]              */
    size_t pe0;                     /* level 0's position encoding when not fused, fp32 [B][N][heads][d] */
    size_t total;                   /* bytes; every region starts on a 256-byte boundary     */
} qta_workspace_layout;

/* Human-readable name of a status code (static storage). */
const char* qta_status_str(qta_status status);

/* Level sizes for an H x W map with `levels` levels (ceil halving). Hl, Wl: host arrays of at
 * least `levels` ints. */
qta_status qta_level_dims(int H, int W, int levels, int* Hl, int* Wl);

/* Workspace regions used by qta_forward for this problem (host struct, filled in). */
qta_status qta_get_workspace_layout(int B, int heads, int H, int W, int d, int levels, int K,
                                    qta_dtype dtype, qta_workspace_layout* layout);

/* Bytes of workspace qta_forward needs (at least 256 for every valid problem); 0 if the arguments
 * are invalid or unsupported. */
size_t qta_workspace_bytes(int B, int heads, int H, int W, int d, int levels, int K, qta_dtype dtype);

qta_status qta_forward(const void* q, const void* k, const void* v, const float* w,
                       int B, int heads, int H, int W, int d, int levels, int K,
                       qta_variant variant, qta_dtype dtype, float scale,
                       void* out, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Options of the *_ex calls. A NULL pointer to this struct, or NULL members, select the defaults.
 *   K_levels   host array; entry l (1 <= l <= levels-1) is the number of keys every query of level
 *              l keeps (1..QTA_MAX_K); entry 0 is not read. Level l-1's candidates are the 2x2
 *              children of the parent's K_levels[l] keys. The feature-matching setting of the
 *              paper keeps 8 at the finest selecting level and doubles K at each coarser level
 *              (Sec. 4.1.1). NULL: the call's K at every level.
 *   v_levels   host array of device pointers; entry l (1 <= l <= levels-1) is V at level l,
 *              [B][H_l][W_l][heads][d] dtype, 16-byte aligned, used as given (the paper builds V's
 *              levels with a stride-2 conv-norm-act layer for self-attention, Sec. 3.2; that layer
 *              is the caller's). Entry 0 is not read: level 0 is `v`. Every level is then stored
 *              NHWC in the workspace. NULL: V's levels are average-pooled like Q's and K's.
 *   pe_weight  device fp32 [levels][heads*d][3][3], 16-byte aligned: the multiscale position
 *              encoding (Sec. 3.2, the locally-enhanced positional encoding applied at every
 *              level): level l's message at a query gets the 3x3 depth-wise cross-correlation of
 *              V^l around the query's token (zero outside the map), channel by channel, before the
 *              levels are combined. NULL: no position encoding.
 *   pe_bias    device fp32 [levels][heads*d], 16-byte aligned, added with it; NULL: none.
 *              Requires pe_weight.
 *   epipolar   nonzero: attention along the rows only, as in stereo matching where both self- and
 *              cross attention stay on epipolar lines (Sec. 4.1.2). Every row of every batch
 *              element is then an independent 1 x W map: the pyramids pool pairs along the row
 *              (the quadtree becomes a binary tree) and a query meets the 2 children of each kept
 *              key. Shapes, layouts and w are unchanged; the result is the call on B*H maps of
 *              1 x W, which is also how the workspace and v_levels are laid out
 *              ([B*H][1][W_l][heads][d]) and how `levels` is validated (by W alone).
 *   aux_stream a second hipStream_t (caller-owned, default priority) on which qta_backward_ex may
 *              run work that does not feed the next level: the finest level's counting sort and
 *              key pass overlap the coarser levels' work, which stays on `stream`. The
 *              call orders both streams itself (events recorded on one and waited for on the
 *              other); when it returns, all its work is ordered before later work on `stream`,
 *              and nothing later on aux_stream depends on it. NULL: everything on `stream`. The
 *              forward ignores it.
 *   aux_stream2 a third hipStream_t (caller-owned, default priority, distinct from the other two),
 *              used only with aux_stream: the coarser finer levels' counting sorts and key passes
 *              run there, each right after its level's query pass, beside the finest key pass on
 *              aux_stream and the coarse level on `stream`; ordered and joined like aux_stream.
 *              NULL: those go to aux_stream or `stream`, whichever keeps the coarse level busier.
 *   dpe_weight, dpe_bias, dv_levels  outputs of qta_backward_ex only (the forward ignores them): with
 *              pe_weight, dpe_weight (device fp32 [levels][heads*d][3][3], 16-byte aligned) receives the
 *              gradient of the encoding's kernels, and with pe_bias, dpe_bias (device fp32
 *              [levels][heads*d]) that of its bias; with v_levels, dv_levels (host array of device
 *              pointers, entry l >= 1 fp32 [B][H_l][W_l][heads][d], 16-byte aligned) receives the
 *              gradient of each given V level. Required when their input is given; overwritten.
 */
typedef struct {
    const int* K_levels;
    const void* const* v_levels;
    const float* pe_weight;
    const float* pe_bias;
    int epipolar;
    void* aux_stream;
    void* aux_stream2;
    float* dpe_weight;
    float* dpe_bias;
    float* const* dv_levels;
} qta_options;

/* Workspace of qta_forward_ex with these options (layout and byte count as for qta_forward). With a
 * position encoding, level 0's encoding is computed inside the finest level's kernel on maps of more
 * than one row when 4*K_1 <= 64; otherwise (a single level, one-row maps or epipolar attention,
 * 4*K_1 > 64) the workspace also holds it, fp32 [B][H*W][heads][d], at layout.pe0. */
qta_status qta_get_workspace_layout_ex(int B, int heads, int H, int W, int d, int levels, int K,
                                       qta_dtype dtype, const qta_options* opt, qta_workspace_layout* layout);
size_t qta_workspace_bytes_ex(int B, int heads, int H, int W, int d, int levels, int K, qta_dtype dtype,
                              const qta_options* opt);

/*
 * qta_forward_ex - qta_forward with the options above (NULL opt: exactly qta_forward). K is read
 * only where opt->K_levels is NULL. With a position encoding the workspace is needed also for a
 * single level.
 */
qta_status qta_forward_ex(const void* q, const void* k, const void* v, const float* w, int B, int heads,
                          int H, int W, int d, int levels, int K, qta_variant variant, qta_dtype dtype,
                          float scale, const qta_options* opt, void* out, void* workspace,
                          size_t workspace_bytes, void* stream);

/*
 * qta_forward_ex_noalloc - qta_forward_ex for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the same computation and
 * results, with the workspace taken from an array of QTA_NOALLOC_WORKSPACE_BYTES inside the library,
 * one per device, which the runtime places in device memory when it loads the library's code on that
 * device and which stays there until the process ends. The call allocates and frees nothing; its
 * first call on a device looks the array's address up (hipGetSymbolAddress) with that device current.
 *   Problems whose workspace (qta_workspace_bytes_ex with the same arguments) exceeds
 *   QTA_NOALLOC_WORKSPACE_BYTES return QTA_ERR_WORKSPACE before any launch; other errors as in
 *   qta_forward_ex.
 *   Every call on one device uses that device's one array: calls that may run at the same time on
 *   one device (different streams, or host threads without an order between their streams) race and
 *   give wrong results; calls issued in order on one stream are safe. No part of the array needs to
 *   start cleared (each call writes every region it reads), and its contents after a call are
 *   unspecified.
 */
#define QTA_NOALLOC_WORKSPACE_BYTES ((size_t)64 << 20)
qta_status qta_forward_ex_noalloc(const void* q, const void* k, const void* v, const float* w, int B, int heads,
                                  int H, int W, int d, int levels, int K, qta_variant variant, qta_dtype dtype,
                                  float scale, const qta_options* opt, void* out, void* stream);

/*
 * qta_backward_ex - gradients of the layer for training (the paper trains every model with it,
 * Sec. 4): given dout = dLoss/dout, the gradients of q, k, v and, for QuadTree-B with w, of w. The
 * kept-key sets are those the forward chose and are held fixed: top-K is a selection and has no
 * gradient; everything computed from the kept keys is differentiated, including QuadTree-A's
 * scores s = s_parent * t (Eq. 4), whose gradient flows back to the level that produced
 * s_parent. Pyramid levels are means of their valid children, so each child receives 1/n of a
 * pooled token's gradient (the rounding of pooled values to the storage type is taken as exact).
 *   q, k, v, w   the forward's inputs, unchanged since qta_forward_ex.
 *   workspace    the workspace that qta_forward_ex filled for these inputs and options, unchanged
 *                (read only: pyramids, messages, kept keys and their scores).
 *   dout         [B][H][W][heads][d] dtype.
 *   dq, dk, dv   fp32 [B][H][W][heads][d], overwritten.
 *   dw           fp32 [B][H*W][heads][levels], overwritten for QuadTree-B when w is given (NULL:
 *                not computed); not touched otherwise.
 *   bwd_workspace  device memory of qta_backward_workspace_bytes_ex bytes, 256-byte aligned; its
 *                contents need not be preserved between calls.
 * With caller-supplied V levels (opt->v_levels) their gradients go to opt->dv_levels and do not
 * flow into dv; with the position encoding (opt->pe_weight, Sec. 3.2) V's gradient also receives the
 * encoding's transposed stencil at every level, and opt->dpe_weight / opt->dpe_bias the gradients of
 * its kernels and bias. Unsupported (QTA_ERR_UNSUPPORTED): K_l with 4*K_l > 64 at any level, and the
 * encoding with heads*d > 256. Some sums (the message gradients of levels >= 2, and each key's list
 * of the parents that kept it) are ordered by atomics, so the last bits may vary between runs.
 * Options as in qta_forward_ex.
 */
size_t qta_backward_workspace_bytes_ex(int B, int heads, int H, int W, int d, int levels, int K,
                                       qta_variant variant, qta_dtype dtype, const qta_options* opt);
qta_status qta_backward_ex(const void* q, const void* k, const void* v, const float* w, const void* dout,
                           int B, int heads, int H, int W, int d, int levels, int K, qta_variant variant,
                           qta_dtype dtype, float scale, const qta_options* opt, const void* workspace,
                           size_t workspace_bytes, float* dq, float* dk, float* dv, float* dw,
                           void* bwd_workspace, size_t bwd_workspace_bytes, void* stream);

/*
 * qta_backward_finest_ex - the level-0 step of qta_backward_ex alone (the attention backward at the
 * finest level: its query pass and its key pass), for timing it: same arguments, and the workspaces a
 * qta_backward_ex call on the same inputs left behind. It overwrites dq, dk, dv and, for QuadTree-B
 * with w, dw[..][0] with that step's values, so the gradients are no longer those of the layer
 * afterwards. levels >= 2.
 */
qta_status qta_backward_finest_ex(const void* q, const void* k, const void* v, const float* w, const void* dout,
                                  int B, int heads, int H, int W, int d, int levels, int K, qta_variant variant,
                                  qta_dtype dtype, float scale, const qta_options* opt, const void* workspace,
                                  size_t workspace_bytes, float* dq, float* dk, float* dv, float* dw,
                                  void* bwd_workspace, size_t bwd_workspace_bytes, void* stream);

/*
 * qta_build_pyramid - step 1: levels 1..levels-1 of one token map by 2x2 average pooling
 * (Sec. 3.2). Each level is pooled from the stored level below it: the valid children are summed
 * in fp32 as ((c00 + c01) + (c10 + c11)), missing children left out, multiplied by 1/count and
 * rounded to nearest-even in dtype.
 *   x           [B][H][W][C] dtype, C*sizeof(dtype) a multiple of 16 bytes.
 *   levels_out  levels 1..levels-1 back to back, level l at element offset
 *               sum_{1<=j<l} B*H_j*W_j*C, each [B][H_l][W_l][C] dtype.
 */
qta_status qta_build_pyramid(const void* x, void* levels_out, int B, int H, int W, int C, int levels,
                             qta_dtype dtype, void* stream);

/*
 * qta_coarse_attn - steps 2-3 at the coarsest level (Eq. 1 over the whole Hc x Wc map).
 *   qc, kc, vc  coarsest pyramid level, [B][Hc][Wc][heads][d] dtype; Hc*Wc <= QTA_MAX_COARSE.
 *   msg         fp32 [B][Hc*Wc][heads][d].
 *   sel_idx, sel_key  [B][heads][Hc*Wc][K]: the min(K, Hc*Wc) keys of highest probability, each
 *               row ordered by (probability descending, index ascending), then the -1 slots.
 *               Both NULL: no selection (a single-level problem) and msg is full attention for
 *               either variant. Otherwise both must be given; QuadTree-A's msg then leaves out
 *               the kept keys (they are refined at the next level, Omega = Gamma - Gamma'),
 *               QuadTree-B's msg covers all keys.
 */
qta_status qta_coarse_attn(const void* qc, const void* kc, const void* vc,
                           int B, int heads, int Hc, int Wc, int d, int K,
                           qta_variant variant, qta_dtype dtype, float scale,
                           float* msg, int32_t* sel_idx, float* sel_key, void* stream);

/*
 * qta_topk - step 3 as a standalone row-wise selection.
 *   keys      fp32 [rows][n]; cand_idx int32 [rows][n] naming each candidate (entries < 0 are not
 *             candidates), or NULL for the column index. 1 <= n <= 4096, 1 <= K <= QTA_MAX_K.
 *   idx_out   int32 [rows][K]: the names of the min(K, #candidates) largest keys, ordered by
 *             (key descending, name ascending), padded with -1.
 *   key_out   fp32 [rows][K] (may be NULL): their keys, 0 in padded slots.
 */
qta_status qta_topk(const float* keys, const int32_t* cand_idx, int rows, int n, int K,
                    int32_t* idx_out, float* key_out, void* stream);

/*
 * qta_fine_attn - steps 3-4 at an intermediate level l (0 < l < L-1): every query of the
 * Hl x Wl map attends to the 2x2 children of the keys its parent kept at level l+1.
 *   ql, kl, vl  level l, [B][Hl][Wl][heads][d] dtype.
 *   parent_idx  int32 [B][heads][Np][K] selections of level l+1 (Np = ceil(Hl/2)*ceil(Wl/2)).
 *   parent_key  fp32 same shape: the parents' scores; required for QuadTree-A, ignored by B.
 *   msg         fp32 [B][Hl*Wl][heads][d]. B: softmax over all candidates, Eq. (6).
 *               A: s = s_parent * t with t a softmax over the 2x2 children of one kept key
 *               (Eq. 4); the message sums s*v over the candidates this query does not keep
 *               (Eq. 3 over Omega).
 *   sel_idx, sel_key  [B][heads][Hl*Wl][K]: this level's selections (B by probability, A by s),
 *               each row ordered by (score descending, index ascending), then the -1 slots.
 */
qta_status qta_fine_attn(const void* ql, const void* kl, const void* vl,
                         int B, int heads, int Hl, int Wl, int d, int K,
                         qta_variant variant, qta_dtype dtype, float scale,
                         const int32_t* parent_idx, const float* parent_key,
                         float* msg, int32_t* sel_idx, float* sel_key, void* stream);

/*
 * qta_finest_attn - steps 4-5 at level 0, with the combination fused in (Eqs. 2 and 5).
 *   q0, k0, v0  [B][H][W][heads][d] dtype (the inputs of qta_forward).
 *   parent_idx, parent_key  selections of level 1 as in qta_fine_attn.
 *   coarser_msg host array of levels-1 device pointers: entry j-1 is the fp32 message of level j,
 *               [B][N_j][heads][d], j = 1..levels-1.
 *   w           as in qta_forward (B only; NULL means 1/levels).
 *   out         [B][H][W][heads][d] dtype. Each query adds its own level-0 message and the
 *               messages of its ancestors (y >> j, x >> j) at every coarser level j.
 */
qta_status qta_finest_attn(const void* q0, const void* k0, const void* v0,
                           int B, int heads, int H, int W, int d, int K,
                           qta_variant variant, qta_dtype dtype, float scale,
                           const int32_t* parent_idx, const float* parent_key,
                           int levels, const float* const* coarser_msg, const float* w,
                           void* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* QTA_H */
