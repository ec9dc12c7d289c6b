/*
 * ALTR visual-token reduction: plain fp64 CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the checker the GPU path is measured
 * against.  Only the test suite, the package smoke check and the CPU-baseline
 * leg of the benchmark may load it; the product path never does.  It shares no
 * source, header, table or helper with the HIP library.
 *
 * Every function follows the paper's definitions in the order the paper gives
 * them, in double precision, with no blocking, fusion or reordering:
 *   - Stage I (Sec. "Stage I: Importance-Aware Token Selection via Renyi
 *     Entropy"): magnitude normalisation, Eq. (3); second-order Renyi
 *     entropy, Eq. (4); the K1 highest-entropy tokens form X^imp.
 *   - Stage II (Sec. "Stage II: Diversity-Aware Token Selection via Feature
 *     Variation Consistency"): cosine between the pre- and post-MLP states,
 *     Eq. (6); ascending sort of the remainder; stride sampling.
 *   - Overall pipeline (Sec. "Overall Token Reduction Pipeline", Eq. (7),
 *     Algorithm 1): budget split K1 = floor(lambda*K), K2 = K - K1; the stride
 *     t = max(1, floor(|X^rem| / K2)); X* = X^imp U X^div.
 *
 * Readings of points the paper leaves open (each is also listed in the design
 * notes of the repository):
 *   - natural logarithm in Eq. (4);
 *   - an all-zero row (Eq. (3) is 0/0) gets H2 = 0, the bottom of [0, log D];
 *   - a zero-norm pre- or post-MLP state gets s = 0;
 *   - ties in Stage I go to the lower token index, ties in the Stage II sort
 *     keep index order (a stable ascending sort);
 *   - the "1, 1+t, ..." positions of Algorithm 1 are 1-based, i.e. sorted
 *     positions 0, t, 2t, ... counted from 0;
 *   - X* is returned in ascending original token index.
 *
 * Inputs are rows of IEEE binary32 (dtype 0), bfloat16 (dtype 1, the upper
 * half of a binary32) or binary64 (dtype 2, e.g. an exact product computed
 * in double).  All widen to double exactly.
 *
 * Parity pins: every function here is checked by the CPU test suite against
 * closed forms, invariants, library routines (numpy lexsort) and brute-force
 * enumeration on tiny inputs; see tests/test_oracle_pins.py.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_DTYPE_F32 0
#define ORACLE_DTYPE_BF16 1
#define ORACLE_DTYPE_F64 2

/* ---- element access --------------------------------------------------- */

/* bfloat16 is the high 16 bits of a binary32 value: shifting the stored
 * pattern up by 16 bits gives that binary32 exactly. */
static double elem(const void* base, int dtype, size_t i)
{
    if (dtype == ORACLE_DTYPE_BF16) {
        uint16_t h = ((const uint16_t*)base)[i];
        uint32_t w = ((uint32_t)h) << 16;
        float f;
        memcpy(&f, &w, sizeof f);
        return (double)f;
    }
    if (dtype == ORACLE_DTYPE_F64)
        return ((const double*)base)[i];
    return (double)((const float*)base)[i];
}

static size_t elem_bytes(int dtype)
{
    return dtype == ORACLE_DTYPE_BF16 ? 2u : dtype == ORACLE_DTYPE_F64 ? 8u : 4u;
}

/* ---- Stage I: Eq. (3) and Eq. (4) ------------------------------------- */

/* H2(x) = -log sum_j p_j^2 with p_j = |x_j| / sum_k |x_k|.
 * Written exactly as the two equations read: first the normaliser, then the
 * distribution, then the sum of squares, then the negative log. */
double altr_oracle_renyi2(const void* row, int dtype, int D)
{
    double norm = 0.0;
    for (int k = 0; k < D; ++k)
        norm += fabs(elem(row, dtype, (size_t)k));
    if (norm == 0.0)
        return 0.0; /* reading: an all-zero row has H2 = 0 */
    double sum_p2 = 0.0;
    for (int j = 0; j < D; ++j) {
        double p = fabs(elem(row, dtype, (size_t)j)) / norm;
        sum_p2 += p * p;
    }
    return -log(sum_p2);
}

/* Self-check form of the same quantity.  With m the mean of |x| and V the
 * population variance of |x| over the D channels,
 *   sum_j p_j^2 = D (V + m^2) / (D m)^2 = (1 + V/m^2) / D,
 * so H2 = log D - log(1 + V/m^2).  The variance is taken two-pass.  Used by
 * the tests to cross-check altr_oracle_renyi2 (agreement to ~1e-12). */
double altr_oracle_renyi2_cv(const void* row, int dtype, int D)
{
    double s1 = 0.0;
    for (int k = 0; k < D; ++k)
        s1 += fabs(elem(row, dtype, (size_t)k));
    if (s1 == 0.0)
        return 0.0;
    double m = s1 / D;
    double v = 0.0;
    for (int k = 0; k < D; ++k) {
        double d = fabs(elem(row, dtype, (size_t)k)) - m;
        v += d * d;
    }
    v /= D;
    return log((double)D) - log1p(v / (m * m));
}

/* ---- Variant: Shannon entropy of the same distribution ----------------- */

/* H1(x) = -sum_j p_j log p_j with p_j = |x_j| / sum_k |x_k| (Eq. (3)) and
 * 0 log 0 = 0; an all-zero row has H1 = 0, the same reading as for H2.  The
 * paper names Shannon entropy only as the measure its Renyi score improves
 * on (Sec. "Stage I"); it is a selectable variant of the Stage I score. */
double altr_oracle_shannon(const void* row, int dtype, int D)
{
    double norm = 0.0;
    for (int k = 0; k < D; ++k)
        norm += fabs(elem(row, dtype, (size_t)k));
    if (norm == 0.0)
        return 0.0; /* reading: an all-zero row has H1 = 0 */
    double h = 0.0;
    for (int j = 0; j < D; ++j) {
        double q = fabs(elem(row, dtype, (size_t)j)) / norm;
        if (q > 0.0)
            h -= q * log(q);
    }
    return h;
}

/* ---- Stage II: Eq. (6) ------------------------------------------------ */

/* s = <a, b> / (||a||_2 ||b||_2); s = 0 when either norm is zero (reading).
 * The denominator is taken as sqrt(||a||^2 ||b||^2), the same number in exact
 * arithmetic; one square root keeps exact ties exact when the product of the
 * squared norms is a perfect square (cos(x, c x) = 1 for integer rows). */
double altr_oracle_cosine(const void* a, const void* b, int dtype, int Dc)
{
    double dot = 0.0, na = 0.0, nb = 0.0;
    for (int j = 0; j < Dc; ++j) {
        double u = elem(a, dtype, (size_t)j);
        double w = elem(b, dtype, (size_t)j);
        dot += u * w;
        na += u * u;
        nb += w * w;
    }
    if (na == 0.0 || nb == 0.0)
        return 0.0;
    return dot / sqrt(na * nb);
}

/* Per-token scores for a packed block of rows.  entropy selects the Stage I
 * score: 2 = Renyi-2 (Eq. (4), the method), 1 = Shannon (the variant). */
void altr_oracle_scores(const void* X, const void* Xpre, const void* Xpost,
                        int dtype, int64_t rows, int D, int Dc, int entropy,
                        double* h2, double* s)
{
    size_t eb = elem_bytes(dtype);
    for (int64_t i = 0; i < rows; ++i) {
        const void* xr = (const char*)X + (size_t)i * D * eb;
        if (h2)
            h2[i] = entropy == 1 ? altr_oracle_shannon(xr, dtype, D)
                                 : altr_oracle_renyi2(xr, dtype, D);
        if (s)
            s[i] = altr_oracle_cosine((const char*)Xpre + (size_t)i * Dc * eb,
                                      (const char*)Xpost + (size_t)i * Dc * eb,
                                      dtype, Dc);
    }
}

/* ---- Algorithm 1: budget split and stride ------------------------------ */

/* K1 = floor(lambda K) evaluated in double, K2 = K - K1; the stride over the
 * remainder of R = N - K1 tokens is t = max(1, floor(R / K2)) (0 when K2 = 0).
 * Returns 0 on success, -1 when the inputs are outside 1 <= K <= N,
 * 0 <= lambda <= 1. */
int altr_oracle_budget(int N, int K, double lambda, int* K1, int* K2, int* t)
{
    if (N < 1 || K < 1 || K > N || !(lambda >= 0.0 && lambda <= 1.0))
        return -1;
    int k1 = (int)floor(lambda * (double)K);
    int k2 = K - k1;
    int r = N - k1;
    int tt = 0;
    if (k2 > 0) {
        tt = r / k2;
        if (tt < 1)
            tt = 1;
    }
    if (K1) *K1 = k1;
    if (K2) *K2 = k2;
    if (t) *t = tt;
    return 0;
}

/* ---- Algorithm 1: selection from scores -------------------------------- */

typedef struct {
    double key;
    int32_t idx;
} keyed;

/* Stage I order: higher entropy first; equal entropy, lower index first. */
static int by_h2_desc(const void* pa, const void* pb)
{
    const keyed* a = (const keyed*)pa;
    const keyed* b = (const keyed*)pb;
    if (a->key > b->key) return -1;
    if (a->key < b->key) return 1;
    return (a->idx > b->idx) - (a->idx < b->idx);
}

/* Stage II order: ascending consistency; equal values keep index order. */
static int by_s_asc(const void* pa, const void* pb)
{
    const keyed* a = (const keyed*)pa;
    const keyed* b = (const keyed*)pb;
    if (a->key < b->key) return -1;
    if (a->key > b->key) return 1;
    return (a->idx > b->idx) - (a->idx < b->idx);
}

/* One image.  h2[N] ranks Stage I (higher kept first), s[N] orders Stage II.
 * given_imp, when not NULL, replaces Stage I with a caller-supplied X^imp
 * (given_imp[i] != 0 marks token i); its size must equal floor(lambda K).
 * This conditional form lets a Stage II comparison start from another
 * implementation's X^imp without a Stage I near-tie cascading into Stage II.
 * stride_mode 0 is Algorithm 1's floor stride; stride_mode 1 is the prose
 * variant (a real-valued interval R/K2, position floor(j R / K2)).
 * Writes K indices ascending into out_idx and 0 (X^imp) / 1 (X^div) into
 * out_src (may be NULL).  Returns 0, or -1 on invalid arguments. */
int altr_oracle_select(int N, int K, double lambda, const double* h2,
                       const double* s, const uint8_t* given_imp,
                       int stride_mode, int32_t* out_idx, uint8_t* out_src)
{
    int K1, K2, t;
    if (altr_oracle_budget(N, K, lambda, &K1, &K2, &t) != 0)
        return -1;
    uint8_t* role = (uint8_t*)calloc((size_t)N, 1); /* 0 none, 1 imp, 2 div */
    keyed* v = (keyed*)malloc(sizeof(keyed) * (size_t)N);
    if (!role || !v) {
        free(role);
        free(v);
        return -1;
    }

    /* Stage I: X^imp <- Top-K1 tokens by H2. */
    if (given_imp) {
        int cnt = 0;
        for (int i = 0; i < N; ++i)
            if (given_imp[i]) {
                role[i] = 1;
                ++cnt;
            }
        if (cnt != K1) {
            free(role);
            free(v);
            return -1;
        }
    } else {
        for (int i = 0; i < N; ++i) {
            v[i].key = h2[i];
            v[i].idx = i;
        }
        qsort(v, (size_t)N, sizeof(keyed), by_h2_desc);
        for (int r = 0; r < K1; ++r)
            role[v[r].idx] = 1;
    }

    /* Stage II: X^rem <- X \ X^imp, sorted by s ascending; stride picks. */
    if (K2 > 0) {
        int R = 0;
        for (int i = 0; i < N; ++i)
            if (role[i] == 0) {
                v[R].key = s[i];
                v[R].idx = i;
                ++R;
            }
        qsort(v, (size_t)R, sizeof(keyed), by_s_asc);
        for (int j = 0; j < K2; ++j) {
            long pos;
            if (stride_mode == 1)
                pos = (long)floor((double)j * (double)R / (double)K2);
            else
                pos = (long)j * t;
            role[v[pos].idx] = 2;
        }
    }

    /* X* <- X^imp U X^div, listed in ascending token index. */
    int k = 0;
    for (int i = 0; i < N; ++i)
        if (role[i]) {
            out_idx[k] = i;
            if (out_src)
                out_src[k] = (uint8_t)(role[i] == 2);
            ++k;
        }
    free(role);
    free(v);
    return k == K ? 0 : -1;
}

/* ---- the whole module over a packed batch ------------------------------ */

/* Rows of image b start at sum_{b'<b} N[b'] in X, Xpre and Xpost, and its
 * outputs at sum_{b'<b} K[b'] in out_idx, out_src and out.  out_idx is
 * image-local.  out (may be NULL) receives the kept rows of X byte for byte.
 * h2 and s (may be NULL) receive the per-token scores of all rows.
 * given_imp (may be NULL) is the packed per-token X^imp mask of the
 * conditional form.  entropy: 2 = Renyi-2 (the method), 1 = Shannon (h2 then
 * receives H1).  Returns 0, or -(1 + b) for the first failing image. */
int altr_oracle_reduce(const void* X, const void* Xpre, const void* Xpost,
                       int dtype, int B, const int32_t* N, const int32_t* K,
                       int D, int Dc, double lambda, int stride_mode,
                       int entropy, const uint8_t* given_imp, int32_t* out_idx,
                       uint8_t* out_src, void* out, double* h2, double* s)
{
    size_t eb = elem_bytes(dtype);
    int64_t row0 = 0, out0 = 0;
    for (int b = 0; b < B; ++b) {
        int n = N[b];
        double* hb = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
        double* sb = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
        if (!hb || !sb) {
            free(hb);
            free(sb);
            return -(1 + b);
        }
        altr_oracle_scores((const char*)X + (size_t)row0 * D * eb,
                           (const char*)Xpre + (size_t)row0 * Dc * eb,
                           (const char*)Xpost + (size_t)row0 * Dc * eb,
                           dtype, n, D, Dc, entropy, hb, sb);
        if (h2) memcpy(h2 + row0, hb, sizeof(double) * (size_t)n);
        if (s) memcpy(s + row0, sb, sizeof(double) * (size_t)n);
        int rc = altr_oracle_select(n, K[b], lambda, hb, sb,
                                    given_imp ? given_imp + row0 : NULL,
                                    stride_mode, out_idx + out0,
                                    out_src ? out_src + out0 : NULL);
        free(hb);
        free(sb);
        if (rc != 0)
            return -(1 + b);
        if (out) {
            for (int k = 0; k < K[b]; ++k)
                memcpy((char*)out + (size_t)(out0 + k) * D * eb,
                       (const char*)X + (size_t)(row0 + out_idx[out0 + k]) * D * eb,
                       (size_t)D * eb);
        }
        row0 += n;
        out0 += K[b];
    }
    return 0;
}
