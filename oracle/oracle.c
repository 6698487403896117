/*
 * oracle.c -- plain, slow CPU oracle for the Aspis detect-and-aggregate step.
 *
 * TEST INFRASTRUCTURE ONLY: used by the test suite, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path.  It shares no
 * code with the HIP library.  Each function restates one definition of
 * Konstantinidis & Ramamoorthy, "Aspis: Robust Detection for Distributed
 * Learning" (MLSys 2022) in the most direct form: no blocking, no fusion,
 * no reordering beyond what the definition states.
 *
 * Parity unpinned (conventions only): the vote's tie-break when no replica
 * value has a majority, and the lower median / totalOrder convention for an
 * even number of selected files and for -0, +0 and NaN.
 */
#include "oracle.h"

#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* Combinatorics (Section 3: f = C(K,r), l = C(K-1,r-1), Remark 1).     */
/* ------------------------------------------------------------------ */

int64_t oracle_binom(int64_t n, int64_t k)
{
    if (n < 0 || k < 0 || k > n) return 0;
    if (k > n - k) k = n - k;
    /* After step j the running value equals C(n-k+j, j): an integer. */
    __int128 c = 1;
    for (int64_t j = 1; j <= k; ++j) {
        c = c * (n - k + j) / j;
        if (c > (__int128)INT64_MAX) return -1;
    }
    return (int64_t)c;
}

/* Algorithm 2: every r-subset of the K workers, one file each.  Example 1
 * fixes file 0 <-> {U1,U2,U3}, i.e. lexicographic order over ascending
 * member lists (0-based worker ids here). */
int64_t oracle_assign(int32_t K, int32_t r, int32_t *subsets, int64_t cap)
{
    if (K < 1 || r < 1 || r > K || subsets == NULL) return -1;
    int64_t f = oracle_binom(K, r);
    if (f < 0 || f > cap) return -1;
    int32_t c[128];
    if (r > 128) return -1;
    for (int32_t s = 0; s < r; ++s) c[s] = s;
    for (int64_t i = 0; i < f; ++i) {
        for (int32_t s = 0; s < r; ++s) subsets[i * r + s] = c[s];
        /* lexicographic successor: bump the rightmost entry that can grow,
         * then reset the entries after it to consecutive values */
        int32_t j = r - 1;
        while (j >= 0 && c[j] == K - r + j) --j;
        if (j < 0) break;
        c[j] += 1;
        for (int32_t t = j + 1; t < r; ++t) c[t] = c[t - 1] + 1;
    }
    return f;
}

/* Index of slot pair (s,t), s<t, in the lexicographic list of pairs. */
static int32_t pair_index(int32_t r, int32_t s, int32_t t)
{
    int32_t p = 0;
    for (int32_t a = 0; a < r; ++a)
        for (int32_t b = a + 1; b < r; ++b) {
            if (a == s && b == t) return p;
            ++p;
        }
    return -1;
}

/* ------------------------------------------------------------------ */
/* Detection (Section 4, Eq. 4, Eq. 5, Algorithm 3).                    */
/* ------------------------------------------------------------------ */

static uint32_t bits_of(float x)
{
    uint32_t b;
    memcpy(&b, &x, sizeof b);
    return b;
}

/* Eq. (4): two returned gradients agree iff they are the same vector; the
 * paper's honest workers return exactly the same gradient, so equality is
 * bitwise equality of every coordinate. */
void oracle_pair_agreement(const float *g, int64_t f, int32_t r, int64_t n,
                           int64_t pitch, uint8_t *alpha)
{
    int32_t P = r * (r - 1) / 2;
    for (int64_t i = 0; i < f; ++i) {
        int32_t p = 0;
        for (int32_t s = 0; s < r; ++s)
            for (int32_t t = s + 1; t < r; ++t) {
                const float *a = g + (i * r + s) * pitch;
                const float *b = g + (i * r + t) * pitch;
                uint8_t equal = 1;
                for (int64_t k = 0; k < n; ++k)
                    if (bits_of(a[k]) != bits_of(b[k])) { equal = 0; break; }
                alpha[i * P + p] = equal;
                ++p;
            }
    }
}

/* Eq. (5): total agreements of a worker pair over its common files. */
void oracle_agreement_counts(const uint8_t *alpha, const int32_t *subsets,
                             int64_t f, int32_t r, int32_t K,
                             int64_t *agree_count)
{
    int32_t P = r * (r - 1) / 2;
    for (int32_t u = 0; u < K; ++u)
        for (int32_t v = 0; v < K; ++v) {
            int64_t count = 0;
            if (u != v) {
                for (int64_t i = 0; i < f; ++i) {
                    int32_t su = -1, sv = -1;
                    for (int32_t s = 0; s < r; ++s) {
                        if (subsets[i * r + s] == u) su = s;
                        if (subsets[i * r + s] == v) sv = s;
                    }
                    if (su < 0 || sv < 0) continue;  /* not a common file */
                    int32_t lo = su < sv ? su : sv, hi = su < sv ? sv : su;
                    count += alpha[i * P + pair_index(r, lo, hi)];
                }
            }
            agree_count[u * K + v] = count;
        }
}

/* Algorithm 3, first loop: connect U_u and U_v iff they agree on all of
 * their C(K-2, r-2) common files. */
void oracle_graph(const int64_t *agree_count, int32_t K, int32_t r,
                  uint8_t *adj)
{
    int64_t common = oracle_binom(K - 2, r - 2);
    for (int32_t u = 0; u < K; ++u)
        for (int32_t v = 0; v < K; ++v)
            adj[u * K + v] = (u != v && agree_count[u * K + v] == common);
}

/* Algorithm 3, clique step.  Bron-Kerbosch with the Tomita pivot rule (the
 * algorithm behind the enumeration the paper uses) lists every maximal clique
 * exactly once; the maximum ones are those of the largest size. */
typedef struct {
    const uint8_t *adj;
    int32_t K;
    oracle_clique_result *res;
} bk_state;

static void bk_report(bk_state *st, const uint8_t *R, int32_t size)
{
    oracle_clique_result *res = st->res;
    res->n_maximal += 1;
    if (size > res->omega) {
        res->omega = size;
        res->n_maximum = 0;
        res->n_stored = 0;
    }
    if (size == res->omega) {
        if (res->n_stored < 16) {
            memset(res->member[res->n_stored], 0, 128);
            for (int32_t u = 0; u < st->K; ++u)
                res->member[res->n_stored][u] = R[u];
            res->n_stored += 1;
        }
        res->n_maximum += 1;
    }
}

static void bk(bk_state *st, const uint8_t *R, int32_t rsize,
               const uint8_t *P, const uint8_t *X)
{
    int32_t K = st->K;
    const uint8_t *adj = st->adj;
    int32_t any = 0;
    for (int32_t u = 0; u < K; ++u) any |= P[u] | X[u];
    if (!any) { bk_report(st, R, rsize); return; }

    /* pivot: the vertex of P u X with the most neighbours in P */
    int32_t pivot = -1, best = -1;
    for (int32_t u = 0; u < K; ++u) {
        if (!(P[u] | X[u])) continue;
        int32_t c = 0;
        for (int32_t v = 0; v < K; ++v) c += P[v] & adj[u * K + v];
        if (c > best) { best = c; pivot = u; }
    }

    uint8_t cand[128], Pl[128], Xl[128], Rn[128], Pn[128], Xn[128];
    for (int32_t v = 0; v < K; ++v) {
        cand[v] = P[v] && !adj[pivot * K + v];
        Pl[v] = P[v];
        Xl[v] = X[v];
    }
    for (int32_t v = 0; v < K; ++v) {
        if (!cand[v]) continue;
        for (int32_t w = 0; w < K; ++w) {
            Rn[w] = R[w];
            Pn[w] = Pl[w] & adj[v * K + w];
            Xn[w] = Xl[w] & adj[v * K + w];
        }
        Rn[v] = 1;
        bk(st, Rn, rsize + 1, Pn, Xn);
        Pl[v] = 0;
        Xl[v] = 1;
    }
}

int oracle_cliques(const uint8_t *adj, int32_t K, int32_t q,
                   oracle_clique_result *res)
{
    if (K < 1 || K > 128 || adj == NULL || res == NULL) return -1;
    memset(res, 0, sizeof *res);
    uint8_t R[128], P[128], X[128];
    for (int32_t u = 0; u < K; ++u) { R[u] = 0; P[u] = 1; X[u] = 0; }
    bk_state st = { adj, K, res };
    bk(&st, R, 0, P, X);
    res->success = (res->n_maximum == 1 && res->omega >= K - q);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Aggregation (Section 2 Case 1 / Case 2, Eq. 3, Algorithm 1).         */
/* ------------------------------------------------------------------ */

/* Eq. (3): the majority value among the r replicas.  Equal replicas form
 * classes; the slot of the largest class wins (first slot on ties). */
void oracle_vote(const uint8_t *alpha, int64_t f, int32_t r, int8_t *vote,
                 uint8_t *has_majority)
{
    int32_t P = r * (r - 1) / 2;
    int32_t r_major = (r + 1) / 2;
    for (int64_t i = 0; i < f; ++i) {
        int32_t best_slot = 0, best_count = 0;
        for (int32_t s = 0; s < r; ++s) {
            int32_t count = 1; /* itself */
            for (int32_t t = 0; t < r; ++t) {
                if (t == s) continue;
                int32_t lo = s < t ? s : t, hi = s < t ? t : s;
                count += alpha[i * P + pair_index(r, lo, hi)];
            }
            if (count > best_count) { best_count = count; best_slot = s; }
        }
        vote[i] = (int8_t)best_slot;
        has_majority[i] = (uint8_t)(best_count >= r_major);
    }
}

/* Algorithm 1: Case 1 keeps, per file, the gradient of a worker in
 * N(B_i) n H (the first such slot), and drops files with none; Case 2
 * keeps the majority value of every file. */
int64_t oracle_select(const int32_t *subsets, int64_t f, int32_t r,
                      const int8_t *vote, int32_t success,
                      const uint8_t *honest, int32_t *sel)
{
    int64_t kept = 0;
    for (int64_t i = 0; i < f; ++i) {
        int32_t s_sel = -1;
        if (success) {
            for (int32_t s = 0; s < r; ++s)
                if (honest[subsets[i * r + s]]) { s_sel = s; break; }
        } else {
            s_sel = vote[i];
        }
        sel[i] = s_sel;
        if (s_sel >= 0) ++kept;
    }
    return kept;
}

/* IEEE-754 totalOrder on binary32 bit patterns: negatives (sign set) come
 * first and order by decreasing magnitude bits; non-negatives follow in
 * increasing magnitude bits.  -NaN < -inf < ... < -0 < +0 < ... < +inf < +NaN */
static int total_order_cmp(const void *pa, const void *pb)
{
    uint32_t a = bits_of(*(const float *)pa), b = bits_of(*(const float *)pb);
    uint32_t sa = a >> 31, sb = b >> 31;
    if (sa != sb) return sa ? -1 : 1;
    if (a == b) return 0;
    if (sa == 0) return a < b ? -1 : 1;
    return a > b ? -1 : 1;
}

/* Case 2: coordinate-wise median of the selected file gradients; for an
 * even count the lower of the two middle elements. */
int oracle_median(const float *g, int64_t f, int32_t r, int64_t n,
                  int64_t pitch, const int32_t *sel, float *out)
{
    int64_t m = 0;
    for (int64_t i = 0; i < f; ++i) m += sel[i] >= 0;
    if (m == 0) return -1;
    float *col = (float *)malloc((size_t)m * sizeof(float));
    if (!col) return -2;
    for (int64_t k = 0; k < n; ++k) {
        int64_t c = 0;
        for (int64_t i = 0; i < f; ++i)
            if (sel[i] >= 0) col[c++] = g[(i * r + sel[i]) * pitch + k];
        qsort(col, (size_t)m, sizeof(float), total_order_cmp);
        out[k] = col[(m - 1) / 2];
    }
    free(col);
    return 0;
}

/* Case 1: average of the chosen gradients, summed in file order. */
int oracle_mean(const float *g, int64_t f, int32_t r, int64_t n,
                int64_t pitch, const int32_t *sel, float *out)
{
    int64_t m = 0;
    for (int64_t i = 0; i < f; ++i) m += sel[i] >= 0;
    if (m == 0) return -1;
    for (int64_t k = 0; k < n; ++k) {
        double sum = 0.0;
        for (int64_t i = 0; i < f; ++i)
            if (sel[i] >= 0) sum += (double)g[(i * r + sel[i]) * pitch + k];
        out[k] = (float)(sum / (double)m);
    }
    return 0;
}
