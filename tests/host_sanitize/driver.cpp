// Exercises the host entry points of libaspis and the oracle under
// AddressSanitizer / UndefinedBehaviorSanitizer: assignment, worker row
// tables, clique enumeration on random and structured graphs up to K = 128,
// the distortion-fraction simulator (multithreaded) and DETOX, the argument
// checks of the device entry points, and the oracle's C functions.  Prints
// "ok" and exits 0 when every check holds.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "../../include/aspis.h"

extern "C" {
#include "../../oracle/oracle.h"
}

#define CHECK(c)                                                        \
    do {                                                                \
        if (!(c)) {                                                     \
            std::fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            std::exit(1);                                               \
        }                                                               \
    } while (0)

int main() {
    // assignment and worker rows against the oracle's assignment
    for (int K : {3, 7, 15, 25}) {
        for (int r : {3, 5}) {
            if (r > K) continue;
            const int64_t f = aspis_num_files(K, r);
            std::vector<int32_t> a((size_t)f * r), b((size_t)f * r), rows((size_t)f * r);
            CHECK(aspis_assign(K, r, a.data(), f) == ASPIS_OK);
            CHECK(oracle_assign(K, r, b.data(), f) == f);
            CHECK(a == b);
            CHECK(aspis_worker_rows(K, r, rows.data(), f * r) == ASPIS_OK);
            std::vector<int> seen((size_t)f * r, 0);
            for (auto x : rows) {
                CHECK(x >= 0 && x < f * r);
                ++seen[x];
            }
            for (auto c : seen) CHECK(c == 1);
            CHECK(aspis_assign(K, r, a.data(), f - 1) == ASPIS_ERR_BUFFER_SMALL);
        }
    }
    // cliques: random graphs, compared with the oracle, up to two words
    std::mt19937_64 rng(7);
    for (int trial = 0; trial < 200; ++trial) {
        // small K: the number of maximal cliques of a random graph grows
        // exponentially with K; the two-word paths are covered by the
        // simulator runs below (K = 60 and 128)
        const int K = 3 + (int)(rng() % 26);
        const int nw = (K + 63) / 64;
        const double p = 0.05 + 0.45 * (double)(rng() % 100) / 100.0;   // disagreement density
        std::vector<uint64_t> rows((size_t)K * nw, 0);
        std::vector<uint8_t> adj((size_t)K * K, 0);
        for (int u = 0; u < K; ++u)
            for (int v = u + 1; v < K; ++v) {
                const bool dis = (double)(rng() % 10000) / 10000.0 < p;
                if (dis) {
                    rows[(size_t)u * nw + v / 64] |= 1ull << (v % 64);
                    rows[(size_t)v * nw + u / 64] |= 1ull << (u % 64);
                } else {
                    adj[(size_t)u * K + v] = adj[(size_t)v * K + u] = 1;
                }
            }
        aspis_clique_result res;
        CHECK(aspis_clique(rows.data(), K, 0, &res) == ASPIS_OK);
        oracle_clique_result ref;
        CHECK(oracle_cliques(adj.data(), K, 0, &ref) == 0);
        CHECK(res.omega == ref.omega && res.n_maximum == ref.n_maximum);
        CHECK(res.n_maximal == ref.n_maximal);
    }
    // simulator and DETOX, including a threaded K=60 run and bad arguments
    aspis_sim_result sr;
    CHECK(aspis_simulate(15, 3, 4, ASPIS_ATTACK_OPTIMAL, nullptr, nullptr, &sr, nullptr) == ASPIS_OK);
    CHECK(sr.distorted == 28 && !sr.success);
    std::vector<uint64_t> dis(60);
    CHECK(aspis_simulate(60, 5, 20, ASPIS_ATTACK_WEAK, nullptr, nullptr, &sr, dis.data()) == ASPIS_OK);
    CHECK(sr.success && sr.distorted == 15504);   // C(20,5)
    CHECK(aspis_simulate(128, 3, 40, ASPIS_ATTACK_OPTIMAL, nullptr, nullptr, &sr, nullptr) == ASPIS_OK);
    CHECK(!sr.success && sr.n_maximum == 2 && sr.distorted == 41080);   // C(80,3)/2
    const int32_t bad_a[2] = {1, 1};
    CHECK(aspis_simulate(15, 3, 2, ASPIS_ATTACK_WEAK, bad_a, nullptr, &sr, nullptr) == ASPIS_ERR_INVALID_ARG);
    int64_t groups = 0;
    double eps = 0;
    CHECK(aspis_detox(15, 3, 6, ASPIS_ATTACK_WEAK, &groups, &eps) == ASPIS_OK && groups == 1);
    CHECK(aspis_detox(16, 3, 6, ASPIS_ATTACK_WEAK, &groups, &eps) == ASPIS_ERR_INVALID_ARG);
    // device entry points reject bad shapes before any HIP call
    aspis_detect_out det{(uint32_t *)16, (int8_t *)16, (uint8_t *)16, (uint64_t *)16};
    CHECK(aspis_detect((const float *)16, 7, 4, 10, (const int32_t *)16, &det, nullptr) == ASPIS_ERR_INVALID_ARG);
    CHECK(aspis_detect(nullptr, 7, 3, 10, (const int32_t *)16, &det, nullptr) == ASPIS_ERR_INVALID_ARG);
    // the oracle's median and mean on a small case
    const int64_t f = 5, r = 3, n = 4;
    std::vector<float> g((size_t)f * r * n);
    for (size_t i = 0; i < g.size(); ++i) g[i] = (float)((int)(rng() % 200) - 100) * 0.25f;
    std::vector<int32_t> sel = {0, 1, 2, -1, 0};
    std::vector<float> med(n), mean(n);
    CHECK(oracle_median(g.data(), f, (int32_t)r, n, n, sel.data(), med.data()) == 0);
    CHECK(oracle_mean(g.data(), f, (int32_t)r, n, n, sel.data(), mean.data()) == 0);
    std::puts("ok");
    return 0;
}
