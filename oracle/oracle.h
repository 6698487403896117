/*
 * oracle.h -- plain, slow CPU oracle for the Aspis detect-and-aggregate step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library includes, links or
 * calls this code; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg do.  It shares no source with the HIP path.
 *
 * Every function follows one passage of Konstantinidis & Ramamoorthy,
 * "Aspis: Robust Detection for Distributed Learning" (MLSys 2022), cited at
 * the definition.  All functions are single-threaded and allocate only
 * small temporaries.
 *
 * Parity-unpinned conventions (the paper leaves them open; any consistent
 * choice would be "correct"):
 *   - vote when no replica value reaches a majority (plurality, lowest slot
 *     wins ties);
 *   - median of an even count (lower median) and the order of -0/+0/NaN
 *     (IEEE-754 totalOrder).
 */
#ifndef ASPIS_ORACLE_H
#define ASPIS_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Binomial coefficient C(n,k) computed exactly; -1 if it exceeds int64. */
int64_t oracle_binom(int64_t n, int64_t k);

/* Algorithm 2 / Example 1: the f = C(K,r) r-subsets of {0..K-1} in
 * lexicographic order, each listed with ascending members.  Writes
 * subsets[i*r + s] = s-th worker of file i.  Returns f, or -1 if f > cap
 * or the arguments are invalid. */
int64_t oracle_assign(int32_t K, int32_t r, int32_t *subsets, int64_t cap);

/* Eq. (4): alpha[i*P + p] = 1 iff the two replicas of slot pair p of file i
 * are equal (bitwise, on every one of the n coordinates given), else 0.
 * Slot pairs p enumerate (s,t), s<t, lexicographically: P = r(r-1)/2.
 * Element (i,s,k) is read at g[(i*r+s)*pitch + k].  Over a split coordinate
 * range the caller ANDs the per-range results. */
void oracle_pair_agreement(const float *g, int64_t f, int32_t r, int64_t n,
                           int64_t pitch, uint8_t *alpha);

/* Eq. (5): agree_count[u*K+v] = sum over the files common to workers u and v
 * of the per-file agreement of their two replicas (u != v; diagonal = 0). */
void oracle_agreement_counts(const uint8_t *alpha, const int32_t *subsets,
                             int64_t f, int32_t r, int32_t K,
                             int64_t *agree_count);

/* Algorithm 3, first loop: adj[u*K+v] = 1 iff agree_count == C(K-2, r-2). */
void oracle_graph(const int64_t *agree_count, int32_t K, int32_t r,
                  uint8_t *adj);

typedef struct {
    int32_t omega;            /* size of a maximum clique                     */
    int32_t n_maximum;        /* number of distinct maximum cliques           */
    int64_t n_maximal;        /* number of maximal cliques enumerated         */
    int32_t success;          /* unique maximum clique and omega >= K - q     */
    int32_t n_stored;         /* maximum cliques stored below (<= 16)         */
    uint8_t member[16][128];  /* member[c][u] = 1 iff worker u in clique c    */
} oracle_clique_result;

/* Algorithm 3, clique step: enumerate every maximal clique of the graph by
 * Bron-Kerbosch with Tomita pivoting, count the maximum ones; success iff
 * exactly one maximum clique exists and its size is >= K - q.  K <= 128. */
int oracle_cliques(const uint8_t *adj, int32_t K, int32_t q,
                   oracle_clique_result *res);

/* Eq. (3): majority of the r replicas of each file from the equality
 * relation alpha.  vote[i] = the slot whose value is held by the most slots
 * (ties -> lowest slot); has_majority[i] = that count >= (r+1)/2. */
void oracle_vote(const uint8_t *alpha, int64_t f, int32_t r, int8_t *vote,
                 uint8_t *has_majority);

/* Algorithm 1, aggregation input.  Success: sel[i] = lowest slot whose
 * worker is honest (honest[u] = 1), -1 if none (file ignored).
 * Failure: sel[i] = vote[i].  Returns the number of selected files. */
int64_t oracle_select(const int32_t *subsets, int64_t f, int32_t r,
                      const int8_t *vote, int32_t success,
                      const uint8_t *honest, int32_t *sel);

/* Algorithm 1, Case 2 reduction: out[k] = lower median (rank floor((m-1)/2),
 * m = number of selected files) of {g[i][sel[i]][k] : sel[i] >= 0} under
 * IEEE-754 totalOrder, for k in [0,n).  Returns -1 if nothing is selected. */
int oracle_median(const float *g, int64_t f, int32_t r, int64_t n,
                  int64_t pitch, const int32_t *sel, float *out);

/* Algorithm 1, Case 1 reduction: out[k] = (float)( (sum over selected files
 * in ascending order, in double) / m ).  Returns -1 if nothing selected. */
int oracle_mean(const float *g, int64_t f, int32_t r, int64_t n,
                int64_t pitch, const int32_t *sel, float *out);

#ifdef __cplusplus
}
#endif
#endif
