// aspis_sim.cpp -- distortion-fraction simulator (Section 5 and the appendix
// tables): the detect-and-aggregate step run on symbolic replicas instead of
// gradients, to count the files whose aggregation input is distorted under
// the attacks of Section 4.1 (weak) and Section 4.2 (optimal, Theorem 1),
// plus the DETOX group-majority scheme the paper compares against.
//
// A replica is symbolic: it is either the file's true value or the one value
// all adversaries agree on (colluding adversaries send identical
// distortions, which is what both attacks of Section 4 assume).  The
// simulation follows the same steps as the GPU path: per-file pairwise
// agreement (Eq. 4), the K x K disagreement rows (Eq. 5), the per-file vote
// (Eq. 3), the clique of Algorithm 3 (aspis_clique), and the selection of
// Algorithm 1.  Files are enumerated on the fly in lexicographic order
// (Algorithm 2), split over host threads by rank.
#include <algorithm>
#include <chrono>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <thread>
#include <vector>

#include "../../include/aspis.h"

namespace aspis {
aspis_status host_fail(aspis_status st, const char *msg);
void host_clear_error();
}  // namespace aspis

namespace {

constexpr int kMaxSimR = 15;
constexpr int64_t kMaxSimFiles = int64_t(1) << 31;

int64_t choose(int64_t n, int64_t k) {
    if (k < 0 || n < 0 || k > n) return 0;
    k = std::min(k, n - k);
    unsigned __int128 v = 1;
    for (int64_t j = 0; j < k; ++j) {
        v = v * (unsigned __int128)(n - j) / (unsigned __int128)(j + 1);
        if (v > (unsigned __int128)INT64_MAX) return -1;
    }
    return (int64_t)v;
}

struct Set128 {
    uint64_t w[2] = {0, 0};
    bool has(int u) const { return (w[u >> 6] >> (u & 63)) & 1u; }
    void add(int u) { w[u >> 6] |= 1ull << (u & 63); }
};

// The r-subset of rank `rank` in lexicographic order (combinatorial number
// system): the first member is the smallest u whose block of subsets
// starting with u contains the rank, and so on.
void unrank(int K, int r, int64_t rank, int *s) {
    int u = 0;
    for (int j = 0; j < r; ++j) {
        for (;; ++u) {
            const int64_t block = choose(K - u - 1, r - j - 1);
            if (rank < block) break;
            rank -= block;
        }
        s[j] = u++;
    }
}

// Lexicographic successor; false after the last subset.
bool next_subset(int K, int r, int *s) {
    int j = r - 1;
    while (j >= 0 && s[j] == K - r + j) --j;
    if (j < 0) return false;
    ++s[j];
    for (int k = j + 1; k < r; ++k) s[k] = s[k - 1] + 1;
    return true;
}

struct Scenario {
    int K, r, q;
    aspis_attack attack;
    Set128 adv, dis;   // A and, for the optimal attack, D
    int need;          // r' = (r+1)/2
};

// Slot classes of a file: bit s set iff slot s holds the adversaries' value.
uint32_t classes(const Scenario &sc, const int *s) {
    uint32_t cls = 0;
    int n_adv = 0;
    bool others_in_d = true;
    for (int j = 0; j < sc.r; ++j) {
        if (sc.adv.has(s[j])) {
            cls |= 1u << j;
            ++n_adv;
        } else if (!sc.dis.has(s[j])) {
            others_in_d = false;
        }
    }
    if (sc.attack == ASPIS_ATTACK_OPTIMAL && !(n_adv >= sc.need && others_in_d)) return 0u;
    return cls;
}

unsigned sim_threads(int64_t f) {
    unsigned n = std::thread::hardware_concurrency();
    n = n == 0 ? 1 : std::min(n, 16u);
    const int64_t per = 1 << 16;   // no thread for fewer files than this
    return (unsigned)std::max<int64_t>(1, std::min<int64_t>(n, (f + per - 1) / per));
}

// Run body(first_subset, count, thread_index) over [0, f) in contiguous rank
// ranges, one per thread.
template <typename Body>
void for_ranges(const Scenario &sc, int64_t f, unsigned nt, Body body) {
    std::vector<std::thread> th;
    for (unsigned t = 0; t < nt; ++t) {
        const int64_t lo = f * t / nt, hi = f * (t + 1) / nt;
        th.emplace_back([&, lo, hi, t]() {
            int s[kMaxSimR];
            unrank(sc.K, sc.r, lo, s);
            body(s, hi - lo, t);
        });
    }
    for (auto &x : th) x.join();
}

double ms_since(std::chrono::steady_clock::time_point t0) {
    return std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
}

aspis_status read_set(const int32_t *ids, int n, int K, Set128 *out, const char *what) {
    static thread_local char msg[128];
    for (int j = 0; j < n; ++j) {
        if (ids[j] < 0 || ids[j] >= K || out->has(ids[j])) {
            snprintf(msg, sizeof msg, "aspis_simulate: %s must be %d distinct workers in [0,K)", what, n);
            return aspis::host_fail(ASPIS_ERR_INVALID_ARG, msg);
        }
        out->add(ids[j]);
    }
    return ASPIS_OK;
}

}  // namespace

extern "C" {

aspis_status aspis_simulate(int32_t K, int32_t r, int32_t q, aspis_attack attack,
                            const int32_t *adversaries, const int32_t *disagree_set,
                            aspis_sim_result *res, uint64_t *disagree_rows) {
    if (!res) return aspis::host_fail(ASPIS_ERR_INVALID_ARG, "aspis_simulate: NULL result");
    if (K < 3 || K > ASPIS_MAX_K_CLIQUE || r < 3 || r > K || r > kMaxSimR || r % 2 == 0)
        return aspis::host_fail(ASPIS_ERR_INVALID_ARG,
                                "aspis_simulate: need 3 <= K <= 128 and odd 3 <= r <= min(K,15)");
    if (q < 0 || 2 * q >= K)
        return aspis::host_fail(ASPIS_ERR_INVALID_ARG, "aspis_simulate: need 0 <= q < K/2");
    if (attack != ASPIS_ATTACK_WEAK && attack != ASPIS_ATTACK_OPTIMAL)
        return aspis::host_fail(ASPIS_ERR_INVALID_ARG, "aspis_simulate: unknown attack");
    const int64_t f = choose(K, r);
    if (f < 0 || f > kMaxSimFiles)
        return aspis::host_fail(ASPIS_ERR_OVERFLOW, "aspis_simulate: C(K,r) exceeds 2^31 files");
    Scenario sc{K, r, q, attack, {}, {}, (r + 1) / 2};
    aspis_status st;
    if (adversaries) {
        if ((st = read_set(adversaries, q, K, &sc.adv, "adversaries")) != ASPIS_OK) return st;
    } else {
        for (int u = 0; u < q; ++u) sc.adv.add(u);
    }
    if (attack == ASPIS_ATTACK_OPTIMAL) {
        if (disagree_set) {
            if ((st = read_set(disagree_set, q, K, &sc.dis, "disagree_set")) != ASPIS_OK) return st;
            for (int u = 0; u < K; ++u)
                if (sc.dis.has(u) && sc.adv.has(u))
                    return aspis::host_fail(ASPIS_ERR_INVALID_ARG,
                                            "aspis_simulate: disagree_set must be honest workers");
        } else {
            int taken = 0;   // the q lowest-indexed honest workers
            for (int u = 0; u < K && taken < q; ++u)
                if (!sc.adv.has(u)) {
                    sc.dis.add(u);
                    ++taken;
                }
        }
    }
    const auto t0 = std::chrono::steady_clock::now();
    const unsigned nt = sim_threads(f);
    const int nw = (K + 63) / 64;

    // pass 1: disagreement rows and the Case 2 count (files whose vote is
    // the adversaries' value: they hold the plurality of the slots)
    std::vector<uint64_t> rows((size_t)nt * K * 2, 0ull);
    std::vector<int64_t> case2(nt, 0);
    for_ranges(sc, f, nt, [&](int *s, int64_t n, unsigned t) {
        uint64_t *my = &rows[(size_t)t * K * 2];
        int64_t c2 = 0;
        for (int64_t k = 0; k < n; ++k) {
            const uint32_t cls = classes(sc, s);
            if (cls) {
                const int n_adv = __builtin_popcount(cls);
                c2 += 2 * n_adv > r ? 1 : 0;
                for (int a = 0; a < r; ++a)
                    for (int b = a + 1; b < r; ++b)
                        if (((cls >> a) ^ (cls >> b)) & 1u) {
                            my[s[a] * 2 + (s[b] >> 6)] |= 1ull << (s[b] & 63);
                            my[s[b] * 2 + (s[a] >> 6)] |= 1ull << (s[a] & 63);
                        }
            }
            next_subset(K, r, s);
        }
        case2[t] = c2;
    });
    std::vector<uint64_t> dis((size_t)K * nw, 0ull);
    for (unsigned t = 0; t < nt; ++t)
        for (int u = 0; u < K; ++u)
            for (int w = 0; w < nw; ++w) dis[(size_t)u * nw + w] |= rows[((size_t)t * K + u) * 2 + w];
    int64_t distorted_case2 = 0;
    for (auto c : case2) distorted_case2 += c;
    double ms_files = ms_since(t0);

    // Algorithm 3 on the host
    const auto t1 = std::chrono::steady_clock::now();
    aspis_clique_result cl;
    if ((st = aspis_clique(dis.data(), K, q, &cl)) != ASPIS_OK) return st;
    const double ms_clique = ms_since(t1);

    int64_t distorted = distorted_case2, dropped = 0;
    if (cl.success) {
        // pass 2 (Case 1): the lowest slot held by a member of H, or none
        const auto t2 = std::chrono::steady_clock::now();
        Set128 h;
        h.w[0] = cl.honest[0];
        h.w[1] = cl.honest[1];
        std::vector<int64_t> bad(nt, 0), drop(nt, 0);
        for_ranges(sc, f, nt, [&](int *s, int64_t n, unsigned t) {
            int64_t b = 0, dr = 0;
            for (int64_t k = 0; k < n; ++k) {
                int slot = -1;
                for (int j = 0; j < r; ++j)
                    if (h.has(s[j])) {
                        slot = j;
                        break;
                    }
                if (slot < 0) {
                    ++dr;
                } else if ((classes(sc, s) >> slot) & 1u) {
                    ++b;
                }
                next_subset(K, r, s);
            }
            bad[t] = b;
            drop[t] = dr;
        });
        distorted = 0;
        for (unsigned t = 0; t < nt; ++t) {
            distorted += bad[t] + drop[t];
            dropped += drop[t];
        }
        ms_files += ms_since(t2);
    }

    std::memset(res, 0, sizeof *res);
    res->files = f;
    res->distorted = distorted;
    res->dropped = dropped;
    res->success = cl.success;
    res->omega = cl.omega;
    res->n_maximum = cl.n_maximum;
    res->n_maximal = cl.n_maximal;
    res->epsilon = (double)distorted / (double)f;
    res->epsilon_baseline = (double)q / (double)K;
    res->ms_files = ms_files;
    res->ms_clique = ms_clique;
    if (disagree_rows) std::memcpy(disagree_rows, dis.data(), dis.size() * sizeof(uint64_t));
    aspis::host_clear_error();
    return ASPIS_OK;
}

aspis_status aspis_detox(int32_t K, int32_t r, int32_t q, aspis_attack attack,
                         int64_t *distorted_groups, double *epsilon) {
    if (!distorted_groups || !epsilon)
        return aspis::host_fail(ASPIS_ERR_INVALID_ARG, "aspis_detox: NULL output");
    if (r < 1 || r % 2 == 0 || K < r || K % r != 0 || q < 0 || q > K)
        return aspis::host_fail(ASPIS_ERR_INVALID_ARG,
                                "aspis_detox: need odd r dividing K and 0 <= q <= K");
    if (attack != ASPIS_ATTACK_WEAK && attack != ASPIS_ATTACK_OPTIMAL)
        return aspis::host_fail(ASPIS_ERR_INVALID_ARG, "aspis_detox: unknown attack");
    const int groups = K / r, need = (r + 1) / 2;
    std::vector<int> per_group(groups, 0);
    for (int i = 0; i < q; ++i) {
        int grp;
        if (attack == ASPIS_ATTACK_WEAK) {
            // Section 5, weak attack on DETOX: the i-th adversary comes from
            // group i mod (K/r) while that group still has honest workers
            grp = i % groups;
            while (per_group[grp] == r) grp = (grp + 1) % groups;
        } else {
            // the worst-case choice: r' adversaries per group, group after
            // group, the remainder in the next group
            grp = std::min(i / need, groups - 1);
            while (per_group[grp] == r) grp = (grp + 1) % groups;
        }
        ++per_group[grp];
    }
    int64_t c = 0;
    for (int g = 0; g < groups; ++g) c += per_group[g] >= need ? 1 : 0;
    *distorted_groups = c;
    *epsilon = (double)c * r / (double)K;   // each group votes on r/K of the batch
    aspis::host_clear_error();
    return ASPIS_OK;
}

}  // extern "C"
