/*
 * QuadTree attention forward: plain, slow CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the correctness reference for the GPU library. Only the
 * test suite, the smoke check and the benchmark's CPU-baseline leg may load it. The product path
 * never calls it, and it shares no code, header, table or helper with the GPU library.
 *
 * It follows Tang et al., "QuadTree Attention for Vision Transformers" (ICLR 2022), Sec. 3.2:
 *   - L-level token pyramids of Q, K and V by 2x2 average pooling (Sec. 3.2, pyramid paragraph);
 *   - plain softmax attention, Eq. (1), at the coarsest level, where every query sees every key;
 *   - per query, the K keys with the highest attention scores are kept (Sec. 3.2, Fig. 1);
 *   - at each finer level a query only meets the 2x2 children of its parent's kept keys;
 *   - QuadTree-A: scores s^l = s^{l-1} t^l with t a softmax over the 2x2 children of one kept key,
 *     partial messages over Omega^l = Gamma^l - Gamma^{l+1}, summed over levels (Eqs. 2-4);
 *   - QuadTree-B: per-level attention over the whole region Gamma^l, combined with per-query
 *     level weights w (Eqs. 5-6).
 *
 * Level numbering: l = 0 is the finest level (the input map) and l = L-1 the coarsest. (The paper's
 * Sec. 3.2 counts from the coarsest, its complexity appendix from the finest.)
 *
 * Readings where the paper is silent (each also listed in the design notes of the repository):
 *   - ceil pooling: a level-(l+1) token (y,x) averages its valid children (2y+dy, 2x+dx) at level
 *     l, dividing by their count; the sum is taken in fp32 as ((c00 + c01) + (c10 + c11)) with
 *     missing children left out, then multiplied by 1/n and rounded to the storage type;
 *   - the recursion base is s = 1 above the coarsest level, so coarse scores are the full softmax;
 *   - t is normalised over the valid 2x2 children of one kept parent key;
 *   - A ranks candidates by s, B by its softmax probability; ties go to the lower flat index;
 *   - A's message at a level that selects leaves out that query's own kept keys; at l = 0 (no
 *     further level) every candidate contributes;
 *   - temperature tau = 1/sqrt(d) (head dimension) at every level unless a scale is given;
 *   - w is used as given, [B][H*W][heads][L]; NULL means 1/L everywhere;
 *   - every head is an independent quadtree;
 *   - K may differ per level (the paper's matching setting keeps K = 8 at the finest selecting
 *     level and doubles it at each coarser one, Sec. 4.1.1): K_l keys are kept by every query of
 *     level l, and a query of level l-1 meets the 2x2 children of its parent's K_l keys;
 *   - V's coarser levels may be supplied by the caller instead of pooled (the paper builds them
 *     with a conv-norm-act layer for self-attention, Sec. 3.2); they are then used as given;
 *   - multiscale position encoding (Sec. 3.2, after the locally-enhanced positional encoding it
 *     cites): an unshared 3x3 depth-wise convolution of V^l (zero padding, optional bias) at each
 *     level, added to level l's message at the query's own position before the levels are
 *     combined.
 *
 * Arithmetic: every dot product, softmax and message sum is in double, from the stored (already
 * rounded) pyramid values. Pyramids are computed in fp32 exactly as stated above.
 *
 * Teacher forcing: a caller may supply the kept-key lists of every selecting level. The oracle then
 * uses them instead of its own choices (for A, with its own scores of the supplied keys), so a
 * GPU run whose selections differ at near-ties can still be compared level by level.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define QO_MAX_LEVELS 16

enum { QO_F32 = 0, QO_BF16 = 1 };
enum { QO_A = 0, QO_B = 1 };

typedef struct {
    /* inputs: NHWC, [B][H][W][heads*d]; values must be representable in `dtype` */
    const float* q;
    const float* k;
    const float* v;
    const float* w;               /* variant B only: [B][H*W][heads][L]; NULL means 1/L */
    int B, heads, H, W, d, L, K, variant, dtype;
    const int* K_levels;          /* NULL (K at every level), or entry l in 1..L-1: K_l */
    const float* const* v_levels; /* NULL (pooled V), or entry l in 1..L-1: V at level l, [B][H_l][W_l][C] */
    const float* pe_weight;       /* NULL (no position encoding), or [L][C][3][3] depth-wise kernels */
    const float* pe_bias;         /* NULL (no bias), or [L][C]; used only with pe_weight */
    double scale;                 /* <= 0 means 1/sqrt(d) */
    const int32_t* const* forced; /* NULL, or per level l in 1..L-1: [B][heads][N_l][K_l] */
    /* outputs, all optional (NULL pointers or NULL entries are skipped) */
    double* out;                  /* [B][H][W][heads][d] */
    float* const* pyr_q;          /* per level l in 1..L-1: [B][H_l][W_l][C] */
    float* const* pyr_k;
    float* const* pyr_v;
    double* const* msg;           /* per level l in 0..L-1: [B][N_l][heads][d] */
    int32_t* const* sel_idx;      /* per level l in 1..L-1: [B][heads][N_l][K_l], -1 padded */
    double* const* sel_key;       /* same shape; 0 where idx is -1 */
    int32_t* const* cand_idx;     /* per level l in 0..L-1: [B][heads][N_l][ncand_l] */
    double* const* cand_key;      /*   ncand = N_{L-1} at the coarsest level, 4 K_{l+1} elsewhere */
} qo_forward_args;

/* ----------------------------------------------------------------------------------------- */
/* geometry                                                                                   */
/* ----------------------------------------------------------------------------------------- */

/* Level sizes: each level halves the previous one, rounding up (Sec. 3.2; App. A.1 gives
 * HW/4^l tokens at level l for maps that divide exactly). */
int qo_level_dims(int H, int W, int L, int* Hl, int* Wl)
{
    if (H <= 0 || W <= 0 || L <= 0 || L > QO_MAX_LEVELS) return -1;
    Hl[0] = H;
    Wl[0] = W;
    for (int l = 1; l < L; ++l) {
        Hl[l] = (Hl[l - 1] + 1) / 2;
        Wl[l] = (Wl[l - 1] + 1) / 2;
    }
    return 0;
}

/* ----------------------------------------------------------------------------------------- */
/* storage rounding                                                                           */
/* ----------------------------------------------------------------------------------------- */

/* Round an fp32 value to the nearest bfloat16 (ties to even) and return it as fp32. */
static float round_to_bf16(float x)
{
    uint32_t u;
    memcpy(&u, &x, 4);
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7FFFu + lsb;
    u &= 0xFFFF0000u;
    float y;
    memcpy(&y, &u, 4);
    return y;
}

static float round_to_dtype(float x, int dtype)
{
    return dtype == QO_BF16 ? round_to_bf16(x) : x;
}

/* ----------------------------------------------------------------------------------------- */
/* pyramid                                                                                    */
/* ----------------------------------------------------------------------------------------- */

/* One pooling step (Sec. 3.2: query, key and value pyramids by average pooling; QuadTree-A uses
 * it for all three). dst[b][y][x][c] is the mean of the valid children of (y,x) in src. */
int qo_pool_level(const float* src, int B, int Hs, int Ws, int C, int dtype, float* dst)
{
    if (!src || !dst || B <= 0 || Hs <= 0 || Ws <= 0 || C <= 0) return -1;
    const int Hd = (Hs + 1) / 2, Wd = (Ws + 1) / 2;
    for (int b = 0; b < B; ++b)
        for (int y = 0; y < Hd; ++y)
            for (int x = 0; x < Wd; ++x) {
                const int has_right = (2 * x + 1) < Ws;
                const int has_below = (2 * y + 1) < Hs;
                const int n = (1 + has_right) * (1 + has_below);
                const float inv_n = 1.0f / (float)n;
                for (int c = 0; c < C; ++c) {
                    const float c00 = src[(((size_t)b * Hs + 2 * y) * Ws + 2 * x) * C + c];
                    float row0 = c00;
                    if (has_right) row0 = row0 + src[(((size_t)b * Hs + 2 * y) * Ws + 2 * x + 1) * C + c];
                    float sum = row0;
                    if (has_below) {
                        float row1 = src[(((size_t)b * Hs + 2 * y + 1) * Ws + 2 * x) * C + c];
                        if (has_right)
                            row1 = row1 + src[(((size_t)b * Hs + 2 * y + 1) * Ws + 2 * x + 1) * C + c];
                        sum = row0 + row1;
                    }
                    const float mean = sum * inv_n;
                    dst[(((size_t)b * Hd + y) * Wd + x) * C + c] = round_to_dtype(mean, dtype);
                }
            }
    return 0;
}

/* ----------------------------------------------------------------------------------------- */
/* small helpers                                                                              */
/* ----------------------------------------------------------------------------------------- */

/* <q_i, k_j> over one head's d channels, in double. */
static double dot_head(const float* qrow, const float* krow, int d)
{
    double acc = 0.0;
    for (int c = 0; c < d; ++c) acc += (double)qrow[c] * (double)krow[c];
    return acc;
}

/* Is candidate a ranked before candidate b? Higher key first, then lower flat index. */
static int ranks_before(double key_a, int idx_a, double key_b, int idx_b)
{
    if (key_a != key_b) return key_a > key_b;
    return idx_a < idx_b;
}

/* Top-K by plain repeated selection: out_pos[r] is the candidate position of the r-th kept key,
 * for r < min(K, number of valid candidates); returns that count. valid[] marks candidates. */
static int select_top_k(const double* key, const int* idx, const int* valid, int n, int K, int* out_pos,
                        char* taken)
{
    for (int j = 0; j < n; ++j) taken[j] = 0;
    int kept = 0;
    for (int r = 0; r < K; ++r) {
        int best = -1;
        for (int j = 0; j < n; ++j) {
            if (!valid[j] || taken[j]) continue;
            if (best < 0 || ranks_before(key[j], idx[j], key[best], idx[best])) best = j;
        }
        if (best < 0) break;
        taken[best] = 1;
        out_pos[kept++] = best;
    }
    return kept;
}

/* ----------------------------------------------------------------------------------------- */
/* forward                                                                                    */
/* ----------------------------------------------------------------------------------------- */

/* Return codes: 0 ok, -1 bad arguments, -2 a forced selection is not a candidate of its query,
 * -3 out of memory. */
int qo_forward(const qo_forward_args* a)
{
    if (!a || !a->q || !a->k || !a->v) return -1;
    const int B = a->B, NH = a->heads, H = a->H, W = a->W, d = a->d, L = a->L, K = a->K;
    if (B <= 0 || NH <= 0 || d <= 0 || K <= 0) return -1;
    if (a->variant != QO_A && a->variant != QO_B) return -1;
    if (a->dtype != QO_F32 && a->dtype != QO_BF16) return -1;
    int Hl[QO_MAX_LEVELS], Wl[QO_MAX_LEVELS];
    if (qo_level_dims(H, W, L, Hl, Wl) != 0) return -1;
    const int C = NH * d;
    const double tau = a->scale > 0.0 ? a->scale : 1.0 / sqrt((double)d);
    const int isB = a->variant == QO_B;
    size_t Nl[QO_MAX_LEVELS] = {0};
    for (int l = 0; l < L; ++l) Nl[l] = (size_t)Hl[l] * (size_t)Wl[l];
    const int Lc = L - 1;           /* coarsest level */
    const int nc_coarse = (int)Nl[Lc];
    int Kl[QO_MAX_LEVELS];          /* keys kept per query at level l (l >= 1) */
    int Kmax = 0;
    for (int l = 0; l < L; ++l) {
        Kl[l] = a->K_levels ? a->K_levels[l] : K;
        if (l >= 1 && Kl[l] <= 0) return -1;
        if (l >= 1 && Kl[l] > Kmax) Kmax = Kl[l];
    }
    if (a->v_levels)
        for (int l = 1; l < L; ++l)
            if (!a->v_levels[l]) return -1;

    int rc = 0;
    float* pq[QO_MAX_LEVELS] = {0};
    float* pk[QO_MAX_LEVELS] = {0};
    float* pv[QO_MAX_LEVELS] = {0};
    double* msg[QO_MAX_LEVELS] = {0};
    int32_t* sel[QO_MAX_LEVELS] = {0};
    double* key[QO_MAX_LEVELS] = {0};
    int ncand_max = nc_coarse > 4 * Kmax ? nc_coarse : 4 * Kmax;
    double* ck = malloc(sizeof(double) * ncand_max);
    int* ci = malloc(sizeof(int) * ncand_max);
    int* cv = malloc(sizeof(int) * ncand_max);
    double* cx = malloc(sizeof(double) * ncand_max);
    int* pos = malloc(sizeof(int) * (Kmax + 1));
    char* taken = malloc(ncand_max);
    char* in_sel = malloc(ncand_max);
    double* acc = malloc(sizeof(double) * d);
    if (!ck || !ci || !cv || !cx || !pos || !taken || !in_sel || !acc) { rc = -3; goto done; }

    /* level 0 of each pyramid is the input as stored */
    for (int l = 0; l < L; ++l) {
        const size_t n = (size_t)B * Nl[l] * C;
        pq[l] = malloc(sizeof(float) * n);
        pk[l] = malloc(sizeof(float) * n);
        pv[l] = malloc(sizeof(float) * n);
        msg[l] = malloc(sizeof(double) * (size_t)B * Nl[l] * NH * d);
        if (!pq[l] || !pk[l] || !pv[l] || !msg[l]) { rc = -3; goto done; }
        if (l >= 1) {
            sel[l] = malloc(sizeof(int32_t) * (size_t)B * NH * Nl[l] * Kl[l]);
            key[l] = malloc(sizeof(double) * (size_t)B * NH * Nl[l] * Kl[l]);
            if (!sel[l] || !key[l]) { rc = -3; goto done; }
        }
    }
    for (size_t i = 0; i < (size_t)B * Nl[0] * C; ++i) {
        pq[0][i] = round_to_dtype(a->q[i], a->dtype);
        pk[0][i] = round_to_dtype(a->k[i], a->dtype);
        pv[0][i] = round_to_dtype(a->v[i], a->dtype);
    }
    for (int l = 1; l < L; ++l) {
        qo_pool_level(pq[l - 1], B, Hl[l - 1], Wl[l - 1], C, a->dtype, pq[l]);
        qo_pool_level(pk[l - 1], B, Hl[l - 1], Wl[l - 1], C, a->dtype, pk[l]);
        if (a->v_levels) {
            for (size_t i = 0; i < (size_t)B * Nl[l] * C; ++i) pv[l][i] = round_to_dtype(a->v_levels[l][i], a->dtype);
        } else {
            qo_pool_level(pv[l - 1], B, Hl[l - 1], Wl[l - 1], C, a->dtype, pv[l]);
        }
    }

    for (int b = 0; b < B; ++b)
        for (int h = 0; h < NH; ++h) {
            /* ---- coarsest level: every query against every key (Eq. 1) ---- */
            {
                const int l = Lc;
                const size_t N = Nl[l];
                for (size_t i = 0; i < N; ++i) {
                    const float* qi = pq[l] + ((size_t)b * N + i) * C + (size_t)h * d;
                    double mx = -INFINITY;
                    for (size_t j = 0; j < N; ++j) {
                        const float* kj = pk[l] + ((size_t)b * N + j) * C + (size_t)h * d;
                        cx[j] = tau * dot_head(qi, kj, d);
                        if (cx[j] > mx) mx = cx[j];
                    }
                    double den = 0.0;
                    for (size_t j = 0; j < N; ++j) { ck[j] = exp(cx[j] - mx); den += ck[j]; }
                    for (size_t j = 0; j < N; ++j) { ck[j] /= den; ci[j] = (int)j; cv[j] = 1; in_sel[j] = 0; }

                    if (L > 1) {
                        const int Ks = Kl[l];
                        int kept;
                        int32_t* srow = sel[l] + (((size_t)b * NH + h) * N + i) * Ks;
                        double* krow = key[l] + (((size_t)b * NH + h) * N + i) * Ks;
                        if (a->forced && a->forced[l]) {
                            const int32_t* frow = a->forced[l] + (((size_t)b * NH + h) * N + i) * Ks;
                            kept = 0;
                            for (int r = 0; r < Ks; ++r) {
                                if (frow[r] < 0) break;
                                if (frow[r] >= (int32_t)N) { rc = -2; goto done; }
                                pos[kept++] = frow[r];
                            }
                        } else {
                            kept = select_top_k(ck, ci, cv, (int)N, Ks, pos, taken);
                        }
                        for (int r = 0; r < Ks; ++r) {
                            srow[r] = r < kept ? ci[pos[r]] : -1;
                            krow[r] = r < kept ? ck[pos[r]] : 0.0;
                        }
                        /* QuadTree-A: the kept keys are refined at the next level, so this level's
                         * message covers only the rest of the map (Omega = Gamma - Gamma'). */
                        if (!isB)
                            for (int r = 0; r < kept; ++r) in_sel[pos[r]] = 1;
                    }
                    for (int c = 0; c < d; ++c) acc[c] = 0.0;
                    for (size_t j = 0; j < N; ++j) {
                        if (in_sel[j]) continue;
                        const float* vj = pv[l] + ((size_t)b * N + j) * C + (size_t)h * d;
                        for (int c = 0; c < d; ++c) acc[c] += ck[j] * (double)vj[c];
                    }
                    double* m = msg[l] + (((size_t)b * N + i) * NH + h) * d;
                    for (int c = 0; c < d; ++c) m[c] = acc[c];
                    if (a->cand_key && a->cand_key[l]) {
                        double* o = a->cand_key[l] + (((size_t)b * NH + h) * N + i) * N;
                        for (size_t j = 0; j < N; ++j) o[j] = ck[j];
                    }
                    if (a->cand_idx && a->cand_idx[l]) {
                        int32_t* o = a->cand_idx[l] + (((size_t)b * NH + h) * N + i) * N;
                        for (size_t j = 0; j < N; ++j) o[j] = (int32_t)j;
                    }
                }
            }

            /* ---- finer levels: a query meets the children of its parent's kept keys ---- */
            for (int l = Lc - 1; l >= 0; --l) {
                const size_t N = Nl[l], Np = Nl[l + 1];
                const int Hh = Hl[l], Ww = Wl[l], Wp = Wl[l + 1];
                const int Kp = Kl[l + 1];      /* the parent's kept keys */
                const int ncand = 4 * Kp;
                for (int y = 0; y < Hh; ++y)
                    for (int x = 0; x < Ww; ++x) {
                        const size_t i = (size_t)y * Ww + x;
                        const size_t P = (size_t)(y >> 1) * Wp + (size_t)(x >> 1);
                        const int32_t* psel = sel[l + 1] + (((size_t)b * NH + h) * Np + P) * Kp;
                        const double* pkey = key[l + 1] + (((size_t)b * NH + h) * Np + P) * Kp;
                        const float* qi = pq[l] + ((size_t)b * N + i) * C + (size_t)h * d;
                        /* candidate slot 4r+c: child c (order (0,0),(0,1),(1,0),(1,1)) of the parent's
                         * r-th kept key; slots of missing keys or off-map children are invalid */
                        for (int r = 0; r < Kp; ++r) {
                            const int J = psel[r];
                            for (int c = 0; c < 4; ++c) {
                                const int s = 4 * r + c;
                                cv[s] = 0;
                                ci[s] = -1;
                                ck[s] = 0.0;
                                in_sel[s] = 0;
                                if (J < 0) continue;
                                const int cy = 2 * (J / Wp) + (c >> 1);
                                const int cxx = 2 * (J % Wp) + (c & 1);
                                if (cy >= Hh || cxx >= Ww) continue;
                                cv[s] = 1;
                                ci[s] = cy * Ww + cxx;
                                const float* kj = pk[l] + ((size_t)b * N + ci[s]) * C + (size_t)h * d;
                                cx[s] = tau * dot_head(qi, kj, d);
                            }
                        }
                        if (isB) {
                            /* Eq. (6): softmax over every key of the region Gamma */
                            double mx = -INFINITY, den = 0.0;
                            for (int s = 0; s < ncand; ++s) if (cv[s] && cx[s] > mx) mx = cx[s];
                            for (int s = 0; s < ncand; ++s) if (cv[s]) { ck[s] = exp(cx[s] - mx); den += ck[s]; }
                            for (int s = 0; s < ncand; ++s) if (cv[s]) ck[s] /= den;
                        } else {
                            /* Eq. (4): s = s_parent * t, t a softmax over the children of one kept key */
                            for (int r = 0; r < Kp; ++r) {
                                double mx = -INFINITY, den = 0.0;
                                for (int c = 0; c < 4; ++c) { const int s = 4 * r + c; if (cv[s] && cx[s] > mx) mx = cx[s]; }
                                for (int c = 0; c < 4; ++c) { const int s = 4 * r + c; if (cv[s]) { ck[s] = exp(cx[s] - mx); den += ck[s]; } }
                                for (int c = 0; c < 4; ++c) { const int s = 4 * r + c; if (cv[s]) ck[s] = pkey[r] * (ck[s] / den); }
                            }
                        }
                        if (l >= 1) {
                            const int Ks = Kl[l];
                            int kept;
                            int32_t* srow = sel[l] + (((size_t)b * NH + h) * N + i) * Ks;
                            double* krow = key[l] + (((size_t)b * NH + h) * N + i) * Ks;
                            if (a->forced && a->forced[l]) {
                                const int32_t* frow = a->forced[l] + (((size_t)b * NH + h) * N + i) * Ks;
                                kept = 0;
                                for (int r = 0; r < Ks; ++r) {
                                    if (frow[r] < 0) break;
                                    int found = -1;
                                    for (int s = 0; s < ncand; ++s) if (cv[s] && ci[s] == frow[r]) found = s;
                                    if (found < 0) { rc = -2; goto done; }
                                    pos[kept++] = found;
                                }
                            } else {
                                kept = select_top_k(ck, ci, cv, ncand, Ks, pos, taken);
                            }
                            for (int r = 0; r < Ks; ++r) {
                                srow[r] = r < kept ? ci[pos[r]] : -1;
                                krow[r] = r < kept ? ck[pos[r]] : 0.0;
                            }
                            if (!isB)
                                for (int r = 0; r < kept; ++r) in_sel[pos[r]] = 1;
                        }
                        for (int c = 0; c < d; ++c) acc[c] = 0.0;
                        for (int s = 0; s < ncand; ++s) {
                            if (!cv[s] || in_sel[s]) continue;
                            const float* vj = pv[l] + ((size_t)b * N + ci[s]) * C + (size_t)h * d;
                            for (int c = 0; c < d; ++c) acc[c] += ck[s] * (double)vj[c];
                        }
                        double* m = msg[l] + (((size_t)b * N + i) * NH + h) * d;
                        for (int c = 0; c < d; ++c) m[c] = acc[c];
                        if (a->cand_key && a->cand_key[l]) {
                            double* o = a->cand_key[l] + (((size_t)b * NH + h) * N + i) * ncand;
                            for (int s = 0; s < ncand; ++s) o[s] = cv[s] ? ck[s] : 0.0;
                        }
                        if (a->cand_idx && a->cand_idx[l]) {
                            int32_t* o = a->cand_idx[l] + (((size_t)b * NH + h) * N + i) * ncand;
                            for (int s = 0; s < ncand; ++s) o[s] = ci[s];
                        }
                    }
            }
        }

    /* ---- multiscale position encoding: m^l_i += sum over the 3x3 window of w_l[c] * V^l[c] (+ b_l[c]),
     * zero outside the map, for every level and channel ---- */
    if (a->pe_weight) {
        for (int l = 0; l < L; ++l) {
            const int Hh = Hl[l], Ww = Wl[l];
            for (int b = 0; b < B; ++b)
                for (int y = 0; y < Hh; ++y)
                    for (int x = 0; x < Ww; ++x)
                        for (int c = 0; c < C; ++c) {
                            const float* kw = a->pe_weight + ((size_t)l * C + c) * 9;
                            double acc2 = a->pe_bias ? (double)a->pe_bias[(size_t)l * C + c] : 0.0;
                            for (int ky = 0; ky < 3; ++ky)
                                for (int kx = 0; kx < 3; ++kx) {
                                    const int yy = y + ky - 1, xx = x + kx - 1;
                                    if (yy < 0 || yy >= Hh || xx < 0 || xx >= Ww) continue;
                                    acc2 += (double)kw[ky * 3 + kx] * (double)pv[l][(((size_t)b * Hh + yy) * Ww + xx) * C + c];
                                }
                            msg[l][((size_t)b * Nl[l] + (size_t)y * Ww + x) * C + c] += acc2;
                        }
        }
    }

    /* ---- combination: Eq. (2) for A, Eq. (5) for B; a finest query takes the message of its
     * ancestor at every level, since sub-patches share their parent's coarse messages ---- */
    if (a->out) {
        for (int b = 0; b < B; ++b)
            for (int y = 0; y < H; ++y)
                for (int x = 0; x < W; ++x)
                    for (int h = 0; h < NH; ++h) {
                        const size_t i = (size_t)y * W + x;
                        double* o = a->out + (((size_t)b * Nl[0] + i) * NH + h) * d;
                        for (int c = 0; c < d; ++c) o[c] = 0.0;
                        for (int l = 0; l < L; ++l) {
                            const size_t anc = (size_t)(y >> l) * Wl[l] + (size_t)(x >> l);
                            double wl = 1.0;
                            if (isB) wl = a->w ? (double)a->w[(((size_t)b * Nl[0] + i) * NH + h) * L + l] : 1.0 / L;
                            const double* m = msg[l] + (((size_t)b * Nl[l] + anc) * NH + h) * d;
                            for (int c = 0; c < d; ++c) o[c] += wl * m[c];
                        }
                    }
    }

    /* ---- copy requested intermediates ---- */
    for (int l = 0; l < L; ++l) {
        const size_t n = (size_t)B * Nl[l] * C;
        if (l >= 1) {
            if (a->pyr_q && a->pyr_q[l]) memcpy(a->pyr_q[l], pq[l], sizeof(float) * n);
            if (a->pyr_k && a->pyr_k[l]) memcpy(a->pyr_k[l], pk[l], sizeof(float) * n);
            if (a->pyr_v && a->pyr_v[l]) memcpy(a->pyr_v[l], pv[l], sizeof(float) * n);
            if (a->sel_idx && a->sel_idx[l]) memcpy(a->sel_idx[l], sel[l], sizeof(int32_t) * (size_t)B * NH * Nl[l] * Kl[l]);
            if (a->sel_key && a->sel_key[l]) memcpy(a->sel_key[l], key[l], sizeof(double) * (size_t)B * NH * Nl[l] * Kl[l]);
        }
        if (a->msg && a->msg[l]) memcpy(a->msg[l], msg[l], sizeof(double) * (size_t)B * Nl[l] * NH * d);
    }

done:
    for (int l = 0; l < QO_MAX_LEVELS; ++l) {
        free(pq[l]); free(pk[l]); free(pv[l]); free(msg[l]); free(sel[l]); free(key[l]);
    }
    free(ck); free(ci); free(cv); free(cx); free(pos); free(taken); free(in_sel); free(acc);
    return rc;
}

/* ----------------------------------------------------------------------------------------- */
/* backward                                                                                   */
/* ----------------------------------------------------------------------------------------- */

/*
 * Gradients of the layer output with respect to q, k, v and (QuadTree-B) w, for an upstream
 * gradient dout = dLoss/dout. The kept-key sets are held fixed: they are the forward's (or the
 * forced ones), and the gradient flows through everything computed from them. The chain rule is
 * taken step by step through the forward above:
 *   - combination (Eqs. 2 and 5): dm^l at a level-l token is the sum over its finest descendants i
 *     of w_{i,l} dout_i (1 for A); dw_{i,l} = <dout_i, m^l of the ancestor>;
 *   - QuadTree-B at a level (Eq. 6): m = sum_j p_j v_j with p a softmax over the candidates, so
 *     dv_j += p_j dm, g_j = <dm, v_j>, dlogit_j = p_j (g_j - sum_j' p_j' g_j');
 *   - QuadTree-A at a level (Eqs. 3-4): m = sum over Omega of s_j v_j with s_j = sigma_r t_j, t a
 *     softmax over the children of kept key r and sigma_r that key's score at the parent level. The
 *     gradient of s_j is <dm, v_j> on Omega and, for a key this query keeps, the gradient of its
 *     score that the next finer level sends back (its children's s are sigma times their t). Then
 *     dsigma_r = sum over r's children of t_j ds_j goes up to the parent, dt_j = sigma_r ds_j, and
 *     dlogit_j = t_j (dt_j - sum over r's children of t_j' dt_j');
 *   - logits tau <q, k_j>: dq += tau dlogit_j k_j, dk_j += tau dlogit_j q;
 *   - pyramid (Sec. 3.2): a pooled token is the mean of its n valid children, so each child
 *     receives 1/n of the pooled token's gradient (the storage rounding of pooled values is taken
 *     as the identity).
 *   - multiscale position encoding (Sec. 3.2): each level's message received the 3x3 depth-wise
 *     cross-correlation of V^l plus a bias, so its kernels and bias get the gradient dm^l correlated
 *     with V^l (and summed), and V^l gets dm^l convolved with the kernels (the transposed stencil);
 *   - caller-supplied V levels are inputs of their own: their gradients are returned per level and
 *     do not flow down the V pyramid.
 * The levels are processed finest first, so that QuadTree-A's score gradients reach the coarser
 * level that produced the scores.
 *
 * Return codes as qo_forward.
 */
typedef struct {
    qo_forward_args fwd;          /* the forward problem; its output pointers are ignored        */
    const float* dout;            /* [B][H][W][heads*d]                                           */
    double* dq;                   /* [B][H][W][heads*d] each                                      */
    double* dk;
    double* dv;
    double* dw;                   /* B with w given: [B][H*W][heads][L]; otherwise not written    */
    double* dpe_weight;           /* with a position encoding: [L][C][3][3], or NULL              */
    double* dpe_bias;             /* with a position encoding: [L][C], or NULL                    */
    double* const* dv_levels;     /* with given V levels: entry l in 1..L-1, [B][H_l][W_l][C]     */
} qo_backward_args;

int qo_backward(const qo_backward_args* ba)
{
    if (!ba || !ba->dout || !ba->dq || !ba->dk || !ba->dv) return -1;
    const qo_forward_args* a = &ba->fwd;
    if (a->v_levels && !ba->dv_levels) return -1;
    const int B = a->B, NH = a->heads, H = a->H, W = a->W, d = a->d, L = a->L, K = a->K;
    if (B <= 0 || NH <= 0 || d <= 0 || K <= 0) return -1;
    int Hl[QO_MAX_LEVELS], Wl[QO_MAX_LEVELS];
    if (qo_level_dims(H, W, L, Hl, Wl) != 0) return -1;
    const int C = NH * d;
    const double tau = a->scale > 0.0 ? a->scale : 1.0 / sqrt((double)d);
    const int isB = a->variant == QO_B;
    size_t Nl[QO_MAX_LEVELS] = {0};
    int Kl[QO_MAX_LEVELS] = {0};
    int Kmax = 1;
    for (int l = 0; l < L; ++l) {
        Nl[l] = (size_t)Hl[l] * (size_t)Wl[l];
        Kl[l] = a->K_levels ? a->K_levels[l] : K;
        if (l >= 1 && Kl[l] > Kmax) Kmax = Kl[l];
    }
    const int Lc = L - 1;

    int rc = 0;
    float* pq[QO_MAX_LEVELS] = {0};
    float* pk[QO_MAX_LEVELS] = {0};
    float* pv[QO_MAX_LEVELS] = {0};
    double* msg[QO_MAX_LEVELS] = {0};
    int32_t* sel[QO_MAX_LEVELS] = {0};
    double* key[QO_MAX_LEVELS] = {0};
    double* dm[QO_MAX_LEVELS] = {0};     /* dLoss/dm^l, [B][N_l][heads][d] */
    double* dQ[QO_MAX_LEVELS] = {0};     /* gradients at each level, [B][N_l][C] */
    double* dK[QO_MAX_LEVELS] = {0};
    double* dV[QO_MAX_LEVELS] = {0};
    double* dsig[QO_MAX_LEVELS] = {0};   /* A: dLoss/d(kept score), [B][heads][N_l][K_l] */
    const int ncand_max = (int)Nl[Lc] > 4 * Kmax ? (int)Nl[Lc] : 4 * Kmax;
    double* cx = malloc(sizeof(double) * ncand_max);   /* logits */
    double* cp = malloc(sizeof(double) * ncand_max);   /* B: p; A: t */
    double* cs = malloc(sizeof(double) * ncand_max);   /* A: s = sigma t */
    double* cg = malloc(sizeof(double) * ncand_max);   /* dLoss/d(weight) */
    double* cd = malloc(sizeof(double) * ncand_max);   /* dLoss/d(logit) */
    int* ci = malloc(sizeof(int) * ncand_max);
    int* cv = malloc(sizeof(int) * ncand_max);
    int* kpos = malloc(sizeof(int) * ncand_max);       /* position in the query's own kept list, or -1 */
    if (!cx || !cp || !cs || !cg || !cd || !ci || !cv || !kpos) { rc = -3; goto done; }

    for (int l = 0; l < L; ++l) {
        const size_t n = (size_t)B * Nl[l] * C;
        pq[l] = malloc(sizeof(float) * n);
        pk[l] = malloc(sizeof(float) * n);
        pv[l] = malloc(sizeof(float) * n);
        msg[l] = malloc(sizeof(double) * n);
        dm[l] = calloc(n, sizeof(double));
        dQ[l] = calloc(n, sizeof(double));
        dK[l] = calloc(n, sizeof(double));
        dV[l] = calloc(n, sizeof(double));
        if (!pq[l] || !pk[l] || !pv[l] || !msg[l] || !dm[l] || !dQ[l] || !dK[l] || !dV[l]) { rc = -3; goto done; }
        if (l >= 1) {
            const size_t ns = (size_t)B * NH * Nl[l] * Kl[l];
            sel[l] = malloc(sizeof(int32_t) * ns);
            key[l] = malloc(sizeof(double) * ns);
            dsig[l] = calloc(ns, sizeof(double));
            if (!sel[l] || !key[l] || !dsig[l]) { rc = -3; goto done; }
        }
    }

    /* the forward, for its pyramids, messages, kept keys and their scores */
    {
        qo_forward_args f = *a;
        f.out = NULL;
        f.pyr_q = pq;
        f.pyr_k = pk;
        f.pyr_v = pv;
        f.msg = msg;
        f.sel_idx = sel;
        f.sel_key = key;
        f.cand_idx = NULL;
        f.cand_key = NULL;
        rc = qo_forward(&f);
        if (rc != 0) goto done;
        for (size_t i = 0; i < (size_t)B * Nl[0] * C; ++i) {
            pq[0][i] = round_to_dtype(a->q[i], a->dtype);
            pk[0][i] = round_to_dtype(a->k[i], a->dtype);
            pv[0][i] = round_to_dtype(a->v[i], a->dtype);
        }
    }

    /* combination: dm^l and dw */
    for (int b = 0; b < B; ++b)
        for (int y = 0; y < H; ++y)
            for (int x = 0; x < W; ++x)
                for (int h = 0; h < NH; ++h) {
                    const size_t i = (size_t)y * W + x;
                    const float* go = ba->dout + ((size_t)b * Nl[0] + i) * C + (size_t)h * d;
                    for (int l = 0; l < L; ++l) {
                        const size_t anc = (size_t)(y >> l) * Wl[l] + (size_t)(x >> l);
                        const size_t widx = (((size_t)b * Nl[0] + i) * NH + h) * L + l;
                        double wl = 1.0;
                        if (isB) wl = a->w ? (double)a->w[widx] : 1.0 / L;
                        double* g = dm[l] + (((size_t)b * Nl[l] + anc) * NH + h) * d;
                        const double* m = msg[l] + (((size_t)b * Nl[l] + anc) * NH + h) * d;
                        double dot = 0.0;
                        for (int c = 0; c < d; ++c) {
                            g[c] += wl * (double)go[c];
                            dot += (double)go[c] * m[c];
                        }
                        if (isB && a->w && ba->dw) ba->dw[widx] = dot;
                    }
                }

    for (int b = 0; b < B; ++b)
        for (int h = 0; h < NH; ++h) {
            /* ---- finer levels, finest first ---- */
            for (int l = 0; l < Lc; ++l) {
                const size_t N = Nl[l], Np = Nl[l + 1];
                const int Hh = Hl[l], Ww = Wl[l], Wp = Wl[l + 1];
                const int Kp = Kl[l + 1];
                const int ncand = 4 * Kp;
                for (int y = 0; y < Hh; ++y)
                    for (int x = 0; x < Ww; ++x) {
                        const size_t i = (size_t)y * Ww + x;
                        const size_t P = (size_t)(y >> 1) * Wp + (size_t)(x >> 1);
                        const size_t prow = ((size_t)b * NH + h) * Np + P;
                        const int32_t* psel = sel[l + 1] + prow * Kp;
                        const double* pkey = key[l + 1] + prow * Kp;
                        double* pdsig = dsig[l + 1] + prow * Kp;
                        const float* qi = pq[l] + ((size_t)b * N + i) * C + (size_t)h * d;
                        const double* gm = dm[l] + (((size_t)b * N + i) * NH + h) * d;
                        /* candidates as in the forward: slot 4r+c is child c of kept key r */
                        for (int r = 0; r < Kp; ++r)
                            for (int c = 0; c < 4; ++c) {
                                const int s = 4 * r + c;
                                cv[s] = 0;
                                ci[s] = -1;
                                kpos[s] = -1;
                                const int J = psel[r];
                                if (J < 0) continue;
                                const int cy = 2 * (J / Wp) + (c >> 1), cxx = 2 * (J % Wp) + (c & 1);
                                if (cy >= Hh || cxx >= Ww) continue;
                                cv[s] = 1;
                                ci[s] = cy * Ww + cxx;
                                cx[s] = tau * dot_head(qi, pk[l] + ((size_t)b * N + ci[s]) * C + (size_t)h * d, d);
                            }
                        /* the keys this query keeps (A: their score gradients come from level l-1) */
                        if (l >= 1) {
                            const int32_t* srow = sel[l] + (((size_t)b * NH + h) * N + i) * Kl[l];
                            for (int r = 0; r < Kl[l]; ++r) {
                                if (srow[r] < 0) continue;
                                for (int s = 0; s < ncand; ++s)
                                    if (cv[s] && ci[s] == srow[r]) kpos[s] = r;
                            }
                        }
                        /* forward weights */
                        if (isB) {
                            double mx = -INFINITY, den = 0.0;
                            for (int s = 0; s < ncand; ++s) if (cv[s] && cx[s] > mx) mx = cx[s];
                            for (int s = 0; s < ncand; ++s) if (cv[s]) { cp[s] = exp(cx[s] - mx); den += cp[s]; }
                            for (int s = 0; s < ncand; ++s) if (cv[s]) cp[s] /= den;
                        } else {
                            for (int r = 0; r < Kp; ++r) {
                                double mx = -INFINITY, den = 0.0;
                                for (int c = 0; c < 4; ++c) { const int s = 4 * r + c; if (cv[s] && cx[s] > mx) mx = cx[s]; }
                                for (int c = 0; c < 4; ++c) { const int s = 4 * r + c; if (cv[s]) { cp[s] = exp(cx[s] - mx); den += cp[s]; } }
                                for (int c = 0; c < 4; ++c) { const int s = 4 * r + c; if (cv[s]) { cp[s] /= den; cs[s] = pkey[r] * cp[s]; } }
                            }
                        }
                        /* gradient of each weight, and the values' gradients */
                        for (int s = 0; s < ncand; ++s) {
                            if (!cv[s]) continue;
                            const float* vj = pv[l] + ((size_t)b * N + ci[s]) * C + (size_t)h * d;
                            double* dvj = dV[l] + ((size_t)b * N + ci[s]) * C + (size_t)h * d;
                            const int in_omega = isB || l == 0 || kpos[s] < 0;
                            if (in_omega) {
                                double g = 0.0;
                                for (int c = 0; c < d; ++c) g += gm[c] * (double)vj[c];
                                cg[s] = g;
                                const double wgt = isB ? cp[s] : cs[s];
                                for (int c = 0; c < d; ++c) dvj[c] += wgt * gm[c];
                            } else {
                                cg[s] = dsig[l][(((size_t)b * NH + h) * N + i) * Kl[l] + kpos[s]];
                            }
                        }
                        /* logit gradients */
                        if (isB) {
                            double D = 0.0;
                            for (int s = 0; s < ncand; ++s) if (cv[s]) D += cp[s] * cg[s];
                            for (int s = 0; s < ncand; ++s) if (cv[s]) cd[s] = cp[s] * (cg[s] - D);
                        } else {
                            for (int r = 0; r < Kp; ++r) {
                                double dsr = 0.0, D = 0.0;
                                for (int c = 0; c < 4; ++c) {
                                    const int s = 4 * r + c;
                                    if (!cv[s]) continue;
                                    dsr += cp[s] * cg[s];            /* d sigma_r */
                                    D += cp[s] * (pkey[r] * cg[s]);  /* sum t dt */
                                }
                                if (psel[r] >= 0) pdsig[r] += dsr;
                                for (int c = 0; c < 4; ++c) {
                                    const int s = 4 * r + c;
                                    if (cv[s]) cd[s] = cp[s] * (pkey[r] * cg[s] - D);
                                }
                            }
                        }
                        /* through the logits */
                        double* dqi = dQ[l] + ((size_t)b * N + i) * C + (size_t)h * d;
                        for (int s = 0; s < ncand; ++s) {
                            if (!cv[s]) continue;
                            const float* kj = pk[l] + ((size_t)b * N + ci[s]) * C + (size_t)h * d;
                            double* dkj = dK[l] + ((size_t)b * N + ci[s]) * C + (size_t)h * d;
                            for (int c = 0; c < d; ++c) {
                                dqi[c] += tau * cd[s] * (double)kj[c];
                                dkj[c] += tau * cd[s] * (double)qi[c];
                            }
                        }
                    }
            }

            /* ---- coarsest level: every key (Eq. 1) ---- */
            {
                const int l = Lc;
                const size_t N = Nl[l];
                for (size_t i = 0; i < N; ++i) {
                    const float* qi = pq[l] + ((size_t)b * N + i) * C + (size_t)h * d;
                    const double* gm = dm[l] + (((size_t)b * N + i) * NH + h) * d;
                    double mx = -INFINITY, den = 0.0;
                    for (size_t j = 0; j < N; ++j) {
                        cx[j] = tau * dot_head(qi, pk[l] + ((size_t)b * N + j) * C + (size_t)h * d, d);
                        if (cx[j] > mx) mx = cx[j];
                        kpos[j] = -1;
                    }
                    for (size_t j = 0; j < N; ++j) { cp[j] = exp(cx[j] - mx); den += cp[j]; }
                    for (size_t j = 0; j < N; ++j) cp[j] /= den;
                    if (L > 1 && !isB) {
                        const int32_t* srow = sel[l] + (((size_t)b * NH + h) * N + i) * Kl[l];
                        for (int r = 0; r < Kl[l]; ++r)
                            if (srow[r] >= 0) kpos[srow[r]] = r;
                    }
                    double D = 0.0;
                    for (size_t j = 0; j < N; ++j) {
                        const float* vj = pv[l] + ((size_t)b * N + j) * C + (size_t)h * d;
                        double* dvj = dV[l] + ((size_t)b * N + j) * C + (size_t)h * d;
                        if (kpos[j] < 0) {
                            double g = 0.0;
                            for (int c = 0; c < d; ++c) g += gm[c] * (double)vj[c];
                            cg[j] = g;
                            for (int c = 0; c < d; ++c) dvj[c] += cp[j] * gm[c];
                        } else {
                            cg[j] = dsig[l][(((size_t)b * NH + h) * N + i) * Kl[l] + kpos[j]];
                        }
                        D += cp[j] * cg[j];
                    }
                    double* dqi = dQ[l] + ((size_t)b * N + i) * C + (size_t)h * d;
                    for (size_t j = 0; j < N; ++j) {
                        const double dl = cp[j] * (cg[j] - D);
                        const float* kj = pk[l] + ((size_t)b * N + j) * C + (size_t)h * d;
                        double* dkj = dK[l] + ((size_t)b * N + j) * C + (size_t)h * d;
                        for (int c = 0; c < d; ++c) {
                            dqi[c] += tau * dl * (double)kj[c];
                            dkj[c] += tau * dl * (double)qi[c];
                        }
                    }
                }
            }
        }

    /* multiscale position encoding: the message of every level-l token received
     * e_i[c] = b[c] + sum over the window of w[c][tap] * V^l(i + tap)[c] (zero outside the map), so
     * db[c] = sum_i dm_i[c], dw[c][tap] = sum_i dm_i[c] * V^l(i + tap)[c] and each window token
     * receives w[c][tap] * dm_i[c] in its value gradient */
    if (a->pe_weight) {
        if (ba->dpe_weight) memset(ba->dpe_weight, 0, sizeof(double) * (size_t)L * C * 9);
        if (ba->dpe_bias) memset(ba->dpe_bias, 0, sizeof(double) * (size_t)L * C);
        for (int l = 0; l < L; ++l) {
            const int Hh = Hl[l], Ww = Wl[l];
            for (int b = 0; b < B; ++b)
                for (int y = 0; y < Hh; ++y)
                    for (int x = 0; x < Ww; ++x)
                        for (int c = 0; c < C; ++c) {
                            const double g = dm[l][((size_t)b * Nl[l] + (size_t)y * Ww + x) * C + c];
                            const float* kw = a->pe_weight + ((size_t)l * C + c) * 9;
                            if (ba->dpe_bias) ba->dpe_bias[(size_t)l * C + c] += g;
                            for (int ky = 0; ky < 3; ++ky)
                                for (int kx = 0; kx < 3; ++kx) {
                                    const int yy = y + ky - 1, xx = x + kx - 1;
                                    if (yy < 0 || yy >= Hh || xx < 0 || xx >= Ww) continue;
                                    const size_t j = (((size_t)b * Hh + yy) * Ww + xx) * C + c;
                                    if (ba->dpe_weight)
                                        ba->dpe_weight[((size_t)l * C + c) * 9 + ky * 3 + kx] += g * (double)pv[l][j];
                                    dV[l][j] += (double)kw[ky * 3 + kx] * g;
                                }
                        }
        }
    }

    /* pyramid: each pooled token hands 1/n of its gradient to each of its n valid children (V only
     * when its levels were pooled; given V levels keep their gradients) */
    for (int l = Lc; l >= 1; --l) {
        const int Hs = Hl[l - 1], Ws = Wl[l - 1];
        for (int b = 0; b < B; ++b)
            for (int y = 0; y < Hl[l]; ++y)
                for (int x = 0; x < Wl[l]; ++x) {
                    const int ny = (2 * y + 1 < Hs) ? 2 : 1, nx = (2 * x + 1 < Ws) ? 2 : 1;
                    const double inv_n = 1.0 / (double)(ny * nx);
                    const size_t src = ((size_t)b * Nl[l] + (size_t)y * Wl[l] + x) * C;
                    for (int cy = 0; cy < ny; ++cy)
                        for (int cxx = 0; cxx < nx; ++cxx) {
                            const size_t dst = ((size_t)b * Nl[l - 1] + (size_t)(2 * y + cy) * Ws + (2 * x + cxx)) * C;
                            for (int c = 0; c < C; ++c) {
                                dQ[l - 1][dst + c] += dQ[l][src + c] * inv_n;
                                dK[l - 1][dst + c] += dK[l][src + c] * inv_n;
                                if (!a->v_levels) dV[l - 1][dst + c] += dV[l][src + c] * inv_n;
                            }
                        }
                }
    }
    memcpy(ba->dq, dQ[0], sizeof(double) * (size_t)B * Nl[0] * C);
    memcpy(ba->dk, dK[0], sizeof(double) * (size_t)B * Nl[0] * C);
    memcpy(ba->dv, dV[0], sizeof(double) * (size_t)B * Nl[0] * C);
    if (a->v_levels)
        for (int l = 1; l < L; ++l)
            if (ba->dv_levels[l]) memcpy(ba->dv_levels[l], dV[l], sizeof(double) * (size_t)B * Nl[l] * C);

done:
    for (int l = 0; l < QO_MAX_LEVELS; ++l) {
        free(pq[l]); free(pk[l]); free(pv[l]); free(msg[l]); free(sel[l]); free(key[l]);
        free(dm[l]); free(dQ[l]); free(dK[l]); free(dV[l]); free(dsig[l]);
    }
    free(cx); free(cp); free(cs); free(cg); free(cd); free(ci); free(cv); free(kpos);
    return rc;
}
