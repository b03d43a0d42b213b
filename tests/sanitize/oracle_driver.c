/*
 * Sanitizer driver for the CPU oracle (test infrastructure): runs the oracle's forward and backward
 * on small problems that reach its edge cases (odd and one-row maps, K above the candidate count,
 * both variants, both storage types, per-level K, caller-supplied V levels, the position encoding,
 * teacher forcing with its own choice), so that AddressSanitizer and UndefinedBehaviorSanitizer see
 * every indexing path. Built and run by tests/test_sanitizers.py; exits 0 when every call returns 0
 * and the results are finite.
 */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

#include "../../oracle/oracle.c"

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;

/* splitmix64, mapped to a float in [-2, 2) with a step of 1/64 (exact in bf16 and fp32) */
static float draw(void)
{
    uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    return (float)((int)(z % 256) - 128) / 64.0f;
}

static float* alloc_fill(size_t n)
{
    float* p = (float*)malloc(n * sizeof(float));
    for (size_t i = 0; i < n; ++i) p[i] = draw();
    return p;
}

static int all_finite(const double* p, size_t n)
{
    for (size_t i = 0; i < n; ++i)
        if (!isfinite(p[i])) return 0;
    return 1;
}

typedef struct {
    int B, heads, H, W, d, L, K, variant, dtype;
    int ksched, vgiven, pe, with_w, forced;
} Case;

static int run_case(const Case* c)
{
    const int C = c->heads * c->d;
    int Hl[QO_MAX_LEVELS], Wl[QO_MAX_LEVELS];
    if (qo_level_dims(c->H, c->W, c->L, Hl, Wl) != 0) return 1;
    const size_t n0 = (size_t)c->B * c->H * c->W * C;
    float* q = alloc_fill(n0);
    float* k = alloc_fill(n0);
    float* v = alloc_fill(n0);
    float* dout = alloc_fill(n0);
    float* w = NULL;
    if (c->with_w) {
        w = alloc_fill((size_t)c->B * c->H * c->W * c->heads * c->L);
        for (size_t i = 0; i < (size_t)c->B * c->H * c->W * c->heads * c->L; ++i) w[i] = fabsf(w[i]) / c->L;
    }
    int Kl[QO_MAX_LEVELS];
    for (int l = 0; l < QO_MAX_LEVELS; ++l) Kl[l] = c->K;
    if (c->ksched)
        for (int l = 1; l < c->L; ++l) Kl[l] = c->K << (l - 1);
    float* vl[QO_MAX_LEVELS] = {0};
    if (c->vgiven)
        for (int l = 1; l < c->L; ++l) vl[l] = alloc_fill((size_t)c->B * Hl[l] * Wl[l] * C);
    float* pw = c->pe ? alloc_fill((size_t)c->L * C * 9) : NULL;
    float* pb = c->pe ? alloc_fill((size_t)c->L * C) : NULL;

    double* out = (double*)calloc(n0, sizeof(double));
    double* msg[QO_MAX_LEVELS] = {0};
    int32_t* sidx[QO_MAX_LEVELS] = {0};
    double* skey[QO_MAX_LEVELS] = {0};
    float* pq[QO_MAX_LEVELS] = {0};
    float* pk[QO_MAX_LEVELS] = {0};
    float* pv[QO_MAX_LEVELS] = {0};
    int32_t* cidx[QO_MAX_LEVELS] = {0};
    double* ckey[QO_MAX_LEVELS] = {0};
    for (int l = 0; l < c->L; ++l) {
        const size_t N = (size_t)Hl[l] * Wl[l];
        msg[l] = (double*)calloc((size_t)c->B * N * C, sizeof(double));
        const int ncand = l == c->L - 1 ? (int)N : 4 * Kl[l + 1];
        cidx[l] = (int32_t*)calloc((size_t)c->B * c->heads * N * ncand, sizeof(int32_t));
        ckey[l] = (double*)calloc((size_t)c->B * c->heads * N * ncand, sizeof(double));
        if (l >= 1) {
            sidx[l] = (int32_t*)calloc((size_t)c->B * c->heads * N * Kl[l], sizeof(int32_t));
            skey[l] = (double*)calloc((size_t)c->B * c->heads * N * Kl[l], sizeof(double));
            pq[l] = (float*)calloc((size_t)c->B * N * C, sizeof(float));
            pk[l] = (float*)calloc((size_t)c->B * N * C, sizeof(float));
            pv[l] = (float*)calloc((size_t)c->B * N * C, sizeof(float));
        }
    }
    qo_forward_args a = {0};
    a.q = q;
    a.k = k;
    a.v = v;
    a.w = w;
    a.B = c->B;
    a.heads = c->heads;
    a.H = c->H;
    a.W = c->W;
    a.d = c->d;
    a.L = c->L;
    a.K = c->K;
    a.variant = c->variant;
    a.dtype = c->dtype;          /* the inputs (multiples of 1/64 in [-2, 2)) are exact in bf16 */
    a.K_levels = Kl;
    a.v_levels = c->vgiven ? (const float* const*)vl : NULL;
    a.pe_weight = pw;
    a.pe_bias = pb;
    a.out = out;
    a.pyr_q = pq;
    a.pyr_k = pk;
    a.pyr_v = pv;
    a.msg = msg;
    a.sel_idx = sidx;
    a.sel_key = skey;
    a.cand_idx = cidx;
    a.cand_key = ckey;
    int bad = qo_forward(&a) != 0 || !all_finite(out, n0);
    if (!bad && c->forced && c->L > 1) {        /* teacher forcing with the oracle's own choice */
        a.forced = (const int32_t* const*)sidx;
        bad = qo_forward(&a) != 0 || !all_finite(out, n0);
        a.forced = NULL;
    }
    if (!bad && !c->vgiven && !c->pe) {
        double* dq = (double*)calloc(n0, sizeof(double));
        double* dk = (double*)calloc(n0, sizeof(double));
        double* dv = (double*)calloc(n0, sizeof(double));
        double* dw = (double*)calloc((size_t)c->B * c->H * c->W * c->heads * c->L, sizeof(double));
        qo_backward_args ba = {0};
        ba.fwd = a;
        ba.fwd.cand_idx = NULL;
        ba.fwd.cand_key = NULL;
        ba.dout = dout;
        ba.dq = dq;
        ba.dk = dk;
        ba.dv = dv;
        ba.dw = dw;
        bad = qo_backward(&ba) != 0 || !all_finite(dq, n0) || !all_finite(dk, n0) || !all_finite(dv, n0);
        free(dq);
        free(dk);
        free(dv);
        free(dw);
    }
    for (int l = 0; l < c->L; ++l) {
        free(msg[l]);
        free(cidx[l]);
        free(ckey[l]);
        free(sidx[l]);
        free(skey[l]);
        free(pq[l]);
        free(pk[l]);
        free(pv[l]);
        free(vl[l]);
    }
    free(out);
    free(q);
    free(k);
    free(v);
    free(dout);
    free(w);
    free(pw);
    free(pb);
    return bad;
}

int main(void)
{
    static const Case cases[] = {
        /* B heads  H   W  d  L  K var   dtype   ksched vgiven pe w forced */
        {2, 2, 9, 11, 8, 3, 2, QO_A, QO_F32, 0, 0, 0, 0, 1},
        {1, 1, 13, 7, 4, 4, 3, QO_B, QO_F32, 0, 0, 0, 1, 1},
        {1, 2, 1, 21, 8, 4, 2, QO_B, QO_F32, 0, 0, 0, 1, 0},      /* one-row map */
        {1, 1, 5, 5, 8, 3, 9, QO_A, QO_F32, 0, 0, 0, 0, 0},       /* K above the candidate count */
        {2, 1, 8, 8, 4, 1, 3, QO_B, QO_F32, 0, 0, 0, 1, 0},       /* one level */
        {1, 2, 12, 10, 8, 3, 2, QO_B, QO_BF16, 1, 0, 0, 1, 1},    /* K schedule, bf16 storage */
        {1, 1, 11, 9, 8, 3, 2, QO_A, QO_F32, 0, 1, 0, 0, 0},      /* given V levels */
        {1, 2, 10, 7, 4, 4, 2, QO_B, QO_F32, 0, 1, 1, 1, 0},      /* given V levels and encoding */
        {1, 1, 7, 13, 8, 3, 3, QO_A, QO_F32, 1, 0, 1, 0, 0},      /* encoding, K schedule */
    };
    int failures = 0;
    for (size_t i = 0; i < sizeof cases / sizeof cases[0]; ++i) {
        if (run_case(&cases[i])) {
            fprintf(stderr, "case %zu failed\n", i);
            ++failures;
        }
    }
    printf("%zu cases, %d failures\n", sizeof cases / sizeof cases[0], failures);
    return failures != 0;
}
