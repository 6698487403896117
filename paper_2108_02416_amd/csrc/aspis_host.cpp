// aspis_host.cpp -- C ABI of libaspis: argument checking, the host steps of
// the method (Algorithm 2 assignment, Algorithm 3 clique enumeration) and the
// orchestration of the gfx950 kernels (aspis_kernels.hip).
#include <hip/hip_runtime.h>

#include <atomic>
#include <chrono>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "../../include/aspis.h"
#include "aspis_internal.h"

namespace {

thread_local char g_err[512] = "";

aspis_status fail(aspis_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
aspis_status fail(aspis_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

#define ASPIS_HIP(call)                                                                  \
    do {                                                                                 \
        hipError_t e_ = (call);                                                          \
        if (e_ != hipSuccess)                                                            \
            return fail(ASPIS_ERR_DEVICE, "%s failed: %s", #call, hipGetErrorString(e_)); \
    } while (0)

// C(n,k) exactly, -1 when it exceeds int64.
int64_t binom(int64_t n, int64_t k) {
    if (k < 0 || n < 0 || k > n) return 0;
    k = k < n - k ? k : n - k;
    unsigned __int128 v = 1;
    for (int64_t j = 0; j < k; ++j) {
        v = v * (unsigned __int128)(n - j) / (unsigned __int128)(j + 1);
        if (v > (unsigned __int128)INT64_MAX) return -1;
    }
    return (int64_t)v;
}

// Depth-first enumeration of r-subsets of {0..K-1}: emits them in
// lexicographic order (smaller first member first, then recursively).
void emit_subsets(int32_t K, int32_t r, int32_t depth, int32_t next, int32_t *cur,
                  int32_t *&dst) {
    if (depth == r) {
        std::memcpy(dst, cur, sizeof(int32_t) * r);
        dst += r;
        return;
    }
    for (int32_t u = next; u <= K - (r - depth); ++u) {
        cur[depth] = u;
        emit_subsets(K, r, depth + 1, u + 1, cur, dst);
    }
}

// ---- bitset clique enumeration (K <= 128) -------------------------------

struct Bits {
    uint64_t w[2];
};
inline Bits band(Bits a, Bits b) { return {{a.w[0] & b.w[0], a.w[1] & b.w[1]}}; }
inline Bits bandnot(Bits a, Bits b) { return {{a.w[0] & ~b.w[0], a.w[1] & ~b.w[1]}}; }
inline bool empty(Bits a) { return (a.w[0] | a.w[1]) == 0; }
inline int popcount(Bits a) { return __builtin_popcountll(a.w[0]) + __builtin_popcountll(a.w[1]); }
inline bool has(Bits a, int u) { return (a.w[u >> 6] >> (u & 63)) & 1u; }
inline void set(Bits &a, int u) { a.w[u >> 6] |= 1ull << (u & 63); }
inline void clr(Bits &a, int u) { a.w[u >> 6] &= ~(1ull << (u & 63)); }

struct CliqueSearch {
    int K;
    Bits nbr[128];
    int omega = 0;
    int n_max = 0;
    int64_t n_maximal = 0;
    Bits first{{0, 0}};

    void report(Bits R) {
        ++n_maximal;
        const int sz = popcount(R);
        if (sz > omega) {
            omega = sz;
            n_max = 0;
            first = R;
        }
        if (sz == omega) ++n_max;
    }

    // Bron-Kerbosch with Tomita pivoting: every maximal clique once.
    void expand(Bits R, Bits P, Bits X) {
        if (empty(P) && empty(X)) {
            report(R);
            return;
        }
        int pivot = -1, best = -1;
        for (int half = 0; half < 2; ++half) {
            uint64_t cand = P.w[half] | X.w[half];
            while (cand) {
                const int u = half * 64 + __builtin_ctzll(cand);
                cand &= cand - 1;
                const int c = popcount(band(P, nbr[u]));
                if (c > best) {
                    best = c;
                    pivot = u;
                }
            }
        }
        Bits todo = bandnot(P, nbr[pivot]);
        for (int half = 0; half < 2; ++half) {
            uint64_t bits = todo.w[half];
            while (bits) {
                const int v = half * 64 + __builtin_ctzll(bits);
                bits &= bits - 1;
                Bits R2 = R;
                set(R2, v);
                expand(R2, band(P, nbr[v]), band(X, nbr[v]));
                clr(P, v);
                set(X, v);
            }
        }
    }
};

aspis_status check_device_shape(int32_t K, int32_t r, int64_t d, int64_t *f_out) {
    if (K < 2 || K > ASPIS_MAX_K_DEVICE)
        return fail(ASPIS_ERR_INVALID_ARG, "K=%d outside [2,%d]", K, ASPIS_MAX_K_DEVICE);
    if (r < 3 || r > ASPIS_MAX_R || r > K || (r % 2) == 0)
        return fail(ASPIS_ERR_INVALID_ARG, "r=%d must be odd, 3 <= r <= min(K,%d)", r,
                    ASPIS_MAX_R);
    if (d < 1) return fail(ASPIS_ERR_INVALID_ARG, "d=%lld must be >= 1", (long long)d);
    const int64_t f = binom(K, r);
    if (f < 0) return fail(ASPIS_ERR_OVERFLOW, "C(%d,%d) overflows int64", K, r);
    if (f * r > INT32_MAX)
        return fail(ASPIS_ERR_OVERFLOW, "f*r=%lld exceeds int32 row indexing", (long long)(f * r));
    if ((__int128)f * r * d > (__int128)INT64_MAX / 4)
        return fail(ASPIS_ERR_OVERFLOW, "f*r*d overflows int64 bytes");
    *f_out = f;
    return ASPIS_OK;
}

uint64_t honest_mask(const aspis_clique_result *res) { return res->success ? res->honest[0] : 0ull; }

// m = number of kept files, from the host-side clique outcome alone: on
// success a file is dropped iff all its r workers are outside H, i.e. it is
// one of the C(K-|H|, r) subsets of the detected set; otherwise every file
// keeps its vote.
int64_t kept_files(int32_t K, int32_t r, int64_t f, const aspis_clique_result *res) {
    if (!res->success) return f;
    const int h = __builtin_popcountll(res->honest[0]) + __builtin_popcountll(res->honest[1]);
    return f - binom(K - h, r);
}

bool use_mean(aspis_reduce mode, const aspis_clique_result *res) {
    return mode == ASPIS_REDUCE_MEAN || (mode == ASPIS_REDUCE_PAPER && res->success);
}

// Full-key tiles when on average over the probed coordinates at least this
// many files share the high 16-bit key half of the median.  The half-key
// tiles read back the low half of every such file, so their extra time
// follows the mean count: 28 files tied with the median (ALIE colluders
// sending the honest mean, K = 15) cost the half-key single pass about as
// much as the full-key tiles cost, and data tied on a fraction x of the
// coordinates (455 files each there) costs about x times the fully tied
// case.  The mean, unlike a typical coordinate's count, sees ties that
// cover less than half of the coordinates.
constexpr uint32_t kTieFullKeys = 16;

// The tie estimate: the mean, rounded up, over the probed coordinates of
// the number of files tied with the median's high key half
// (launch_tie_probe).
uint32_t tie_estimate(const uint32_t *counts, int n) {
    uint64_t sum = 0;
    for (int j = 0; j < n; ++j) sum += counts[j];
    return n > 0 ? (uint32_t)((sum + (uint64_t)n - 1) / (uint64_t)n) : 0u;
}

aspis_status check_detect_out(const aspis_detect_out *o) {
    if (!o || !o->pair_diff || !o->vote || !o->has_majority || !o->disagree)
        return fail(ASPIS_ERR_INVALID_ARG, "detect outputs must all be non-NULL");
    return ASPIS_OK;
}

}  // namespace

namespace aspis {
// error reporting for the other host sources of the library
aspis_status host_fail(aspis_status st, const char *msg) { return fail(st, "%s", msg); }
void host_clear_error() { g_err[0] = 0; }
}  // namespace aspis

extern "C" {

const char *aspis_last_error(void) { return g_err; }

int64_t aspis_num_files(int32_t K, int32_t r) {
    if (K < 1 || r < 1 || r > K) return -1;
    return binom(K, r);
}

aspis_status aspis_assign(int32_t K, int32_t r, int32_t *subsets, int64_t cap_files) {
    if (K < 1 || r < 1 || r > K || subsets == nullptr)
        return fail(ASPIS_ERR_INVALID_ARG, "aspis_assign: need 1 <= r <= K and a buffer");
    const int64_t f = binom(K, r);
    if (f < 0) return fail(ASPIS_ERR_OVERFLOW, "C(%d,%d) overflows int64", K, r);
    if (f > cap_files)
        return fail(ASPIS_ERR_BUFFER_SMALL, "need %lld files, buffer holds %lld", (long long)f,
                    (long long)cap_files);
    std::vector<int32_t> cur(r);
    int32_t *dst = subsets;
    emit_subsets(K, r, 0, 0, cur.data(), dst);
    return ASPIS_OK;
}

aspis_status aspis_clique(const uint64_t *rows, int32_t K, int32_t q, aspis_clique_result *res) {
    if (!rows || !res) return fail(ASPIS_ERR_INVALID_ARG, "aspis_clique: NULL argument");
    if (K < 1 || K > ASPIS_MAX_K_CLIQUE)
        return fail(ASPIS_ERR_INVALID_ARG, "aspis_clique: K=%d outside [1,%d]", K, ASPIS_MAX_K_CLIQUE);
    if (q < 0 || 2 * q >= K)
        return fail(ASPIS_ERR_INVALID_ARG, "aspis_clique: q=%d outside [0,K/2)", q);
    const int nw = (K + 63) / 64;
    auto bit = [&](int u, int v) { return (rows[u * nw + (v >> 6)] >> (v & 63)) & 1ull; };
    for (int u = 0; u < K; ++u) {
        if (bit(u, u)) return fail(ASPIS_ERR_INVALID_ARG, "aspis_clique: diagonal bit %d set", u);
        for (int w = 0; w < nw; ++w) {
            const int hi = K - 64 * w;
            const uint64_t valid = hi >= 64 ? ~0ull : ((1ull << hi) - 1ull);
            if (rows[u * nw + w] & ~valid)
                return fail(ASPIS_ERR_INVALID_ARG, "aspis_clique: bits beyond K in row %d", u);
        }
        for (int v = u + 1; v < K; ++v)
            if (bit(u, v) != bit(v, u))
                return fail(ASPIS_ERR_INVALID_ARG, "aspis_clique: matrix not symmetric at (%d,%d)", u, v);
    }
    CliqueSearch cs;
    cs.K = K;
    Bits all{{0, 0}};
    for (int u = 0; u < K; ++u) set(all, u);
    for (int u = 0; u < K; ++u) {
        Bits dis{{rows[u * nw], nw > 1 ? rows[u * nw + 1] : 0ull}};
        Bits n = bandnot(all, dis);
        clr(n, u);
        cs.nbr[u] = n;
    }
    cs.expand(Bits{{0, 0}}, all, Bits{{0, 0}});
    std::memset(res, 0, sizeof *res);
    res->omega = cs.omega;
    res->n_maximum = cs.n_max;
    res->n_words = nw;
    res->n_maximal = cs.n_maximal;
    res->first[0] = cs.first.w[0];
    res->first[1] = cs.first.w[1];
    res->success = (cs.n_max == 1 && cs.omega >= K - q) ? 1 : 0;
    if (res->success) {
        res->honest[0] = cs.first.w[0];
        res->honest[1] = cs.first.w[1];
        Bits det = bandnot(all, cs.first);
        res->detected[0] = det.w[0];
        res->detected[1] = det.w[1];
    }
    g_err[0] = 0;
    return ASPIS_OK;
}

size_t aspis_aggregate_workspace(int32_t K, int32_t r, int64_t d) {
    int64_t f = 0;
    if (check_device_shape(K, r, d, &f) != ASPIS_OK) return 0;
    return aspis::workspace_bytes(f, r);
}

}  // extern "C"

namespace {

// Coordinates the single pass guesses its selection from: about 2^24
// replica words (200 MB; 0.3 % of the bytes at f = 455, d = 11.2M), between
// 4,096 and 32,768 coordinates.  Any disagreement there is caught; one
// elsewhere only costs redoing the reduction (or the tiles it touches).
int64_t probe_coords(int64_t f, int64_t d) {
    int64_t p = (int64_t(1) << 24) / (f > 0 ? f : 1);
    p = p < 4096 ? 4096 : p > 32768 ? 32768 : p;
    return d < p ? d : p;
}

// The seed of a probe drawn for this call: SplitMix64 of a per-process
// random base and a call counter (never 0, which denotes the prefix).
uint64_t probe_seed() {
    static const uint64_t base = []() -> uint64_t {
        // the system's entropy source; the clock if it cannot be opened
        try {
            std::random_device rd;
            return ((uint64_t)rd() << 32) ^ (uint64_t)rd();
        } catch (...) {
            return (uint64_t)std::chrono::steady_clock::now().time_since_epoch().count();
        }
    }();
    static std::atomic<uint64_t> calls{0};
    const uint64_t x = aspis::splitmix64(base + calls.fetch_add(1, std::memory_order_relaxed));
    return x ? x : 1u;
}

// The probe of a call: the whole vector when d is no longer than the probe,
// the prefix when asked, else blocks at positions drawn for the call.
aspis::ProbeSet make_probe(int64_t f, int64_t d, uint32_t flags) {
    const int64_t n = probe_coords(f, d);
    aspis::ProbeSet p;
    if (n >= d || (flags & ASPIS_FLAG_PROBE_PREFIX)) {
        p.kend = n;
        p.nb = (n + aspis::kProbeBlockCols - 1) / aspis::kProbeBlockCols;
    } else {
        p.nb = n / aspis::kProbeBlockCols;   // 4 to 32: n is 4,096 to 32,768 here
        p.seed = probe_seed();
        for (int64_t j = 0; j < p.nb; ++j) p.start[j] = aspis::probe_block_start(p.seed, j, d);
    }
    return p;
}

// The worker-major upload of Algorithm 1: worker u returns the gradients of
// its l = C(K-1,r-1) files in ascending file order, so replica (i,s) is row
// u*l + k of the upload, where u is slot s's worker and file i is the k-th
// file of u.
void worker_row_table(int32_t K, int32_t r, int32_t *row_of) {
    const int64_t f = binom(K, r), l = binom(K - 1, r - 1);
    std::vector<int32_t> subsets((size_t)f * r), cur(r), next_local(K, 0);
    int32_t *dst = subsets.data();
    emit_subsets(K, r, 0, 0, cur.data(), dst);
    for (int64_t i = 0; i < f; ++i)
        for (int s = 0; s < r; ++s) {
            const int32_t u = subsets[(size_t)i * r + s];
            row_of[(size_t)i * r + s] = (int32_t)(u * l + next_local[u]++);
        }
}

aspis_status detect_impl(const float *grads, const int32_t *row_of, int32_t K, int32_t r,
                         int64_t d, const int32_t *subsets_dev, const aspis_detect_out *out,
                         void *stream) {
    int64_t f = 0;
    aspis_status st = check_device_shape(K, r, d, &f);
    if (st != ASPIS_OK) return st;
    if (!grads || !subsets_dev) return fail(ASPIS_ERR_INVALID_ARG, "aspis_detect: NULL input");
    if ((st = check_detect_out(out)) != ASPIS_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    ASPIS_HIP(aspis::launch_fill_u32(out->pair_diff, f, 0u, s));
    ASPIS_HIP(aspis::launch_fill_u64(out->disagree, K, 0ull, s));
    ASPIS_HIP(aspis::launch_agree(grads, row_of, f, r, d, d, out->pair_diff, s));
    ASPIS_HIP(aspis::launch_vote(out->pair_diff, subsets_dev, f, r, out->vote, out->has_majority,
                                 out->disagree, s));
    return ASPIS_OK;
}

aspis_status aggregate_impl(const float *grads, const int32_t *row_of, int32_t K, int32_t r,
                            int64_t d, const int32_t *subsets_dev, const aspis_detect_out *det,
                            const aspis_clique_result *res, aspis_reduce mode, float *out,
                            int32_t *sel_out, int64_t *n_selected, void *workspace,
                            size_t ws_bytes, void *stream, aspis::TileUse *use = nullptr,
                            bool full_keys = false) {
    int64_t f = 0;
    aspis_status st = check_device_shape(K, r, d, &f);
    if (st != ASPIS_OK) return st;
    if (!grads || !subsets_dev || !det || !det->vote || !res || !out || !workspace)
        return fail(ASPIS_ERR_INVALID_ARG, "aspis_aggregate: NULL argument");
    if (mode != ASPIS_REDUCE_MEDIAN && mode != ASPIS_REDUCE_MEAN && mode != ASPIS_REDUCE_PAPER)
        return fail(ASPIS_ERR_INVALID_ARG, "aspis_aggregate: unknown mode %d", (int)mode);
    if (ws_bytes < aspis::workspace_bytes(f, r))
        return fail(ASPIS_ERR_BUFFER_SMALL, "workspace needs %zu bytes", aspis::workspace_bytes(f, r));
    if (((uintptr_t)workspace & 255u) != 0)
        return fail(ASPIS_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    if (res->success && (res->honest[1] != 0 || K > 64))
        return fail(ASPIS_ERR_INVALID_ARG, "honest set beyond worker 63");
    const int64_t m = kept_files(K, r, f, res);
    if (n_selected) *n_selected = m;
    const bool mean = use_mean(mode, res);
    hipStream_t s = static_cast<hipStream_t>(stream);
    aspis::Workspace ws = aspis::carve_workspace(workspace, f, r);
    ASPIS_HIP(aspis::launch_select(subsets_dev, det->vote, f, r, res->success, honest_mask(res),
                                   row_of, ws, sel_out, nullptr, 0, s));
    if (m == 0) return fail(ASPIS_ERR_NO_FILES, "selection kept no file");
    if (mean)
        ASPIS_HIP(aspis::launch_mean(grads, d, ws, out, s));
    else
        ASPIS_HIP(aspis::launch_median(grads, d, ws, f, out, s, use, full_keys));
    return ASPIS_OK;
}

aspis_status detect_aggregate_impl(const float *grads, bool worker_major, int32_t K, int32_t r,
                                   int32_t q, int64_t d, const int32_t *subsets_dev,
                                   const aspis_detect_out *det, aspis_reduce mode, float *out,
                                   int32_t *sel_out, aspis_clique_result *res,
                                   int64_t *n_selected, void *workspace, size_t ws_bytes,
                                   uint32_t flags, aspis_run_stats *stats, void *stream) {
    using clk = std::chrono::steady_clock;
    const auto t0 = clk::now();
    int64_t f = 0;
    aspis_status st = check_device_shape(K, r, d, &f);
    if (st != ASPIS_OK) return st;
    if (!grads || !subsets_dev || !out || !res || !workspace)
        return fail(ASPIS_ERR_INVALID_ARG, "aspis_detect_aggregate: NULL argument");
    if ((st = check_detect_out(det)) != ASPIS_OK) return st;
    if (q < 0 || 2 * q >= K) return fail(ASPIS_ERR_INVALID_ARG, "q=%d outside [0,K/2)", q);
    if (mode != ASPIS_REDUCE_MEDIAN && mode != ASPIS_REDUCE_MEAN && mode != ASPIS_REDUCE_PAPER)
        return fail(ASPIS_ERR_INVALID_ARG, "unknown mode %d", (int)mode);
    if (ws_bytes < aspis::workspace_bytes(f, r))
        return fail(ASPIS_ERR_BUFFER_SMALL, "workspace needs %zu bytes", aspis::workspace_bytes(f, r));
    if (((uintptr_t)workspace & 255u) != 0)
        return fail(ASPIS_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool timing = stats && (flags & ASPIS_FLAG_TIMING);
    aspis_run_stats local{};
    // timing events, released on every return (error returns included)
    struct Events {
        hipEvent_t e[6] = {};
        ~Events() {
            for (hipEvent_t x : e)
                if (x) (void)hipEventDestroy(x);
        }
    } events;
    hipEvent_t *ev = events.e;
    if (timing)
        for (int i = 0; i < 6; ++i) ASPIS_HIP(hipEventCreate(&ev[i]));
    aspis::Workspace ws = aspis::carve_workspace(workspace, f, r);
    // key tiles: full keys when asked, half keys when asked, else chosen
    // from the tie probe run with the first agreement pass
    bool full_keys = (flags & ASPIS_FLAG_FULL_KEYS) != 0;
    const bool tie_probe =
        (flags & (ASPIS_FLAG_FULL_KEYS | ASPIS_FLAG_HALF_KEYS)) == 0 && mode != ASPIS_REDUCE_MEAN;
    const aspis::ProbeSet probe = make_probe(f, d, flags);
    const int n_tie = (int)(probe.coords() < aspis::kTieCols ? probe.coords() : aspis::kTieCols);
    uint32_t *tie_dev = reinterpret_cast<uint32_t *>(ws.stage + aspis::kStageTie);
    local.tie_rows = -1;
    local.repair_groups = -1;
    local.probe_blocks = probe.seed ? (int32_t)probe.nb : 0;
    auto decide_keys = [&](const uint64_t *staged_words) {
        if (!tie_probe) return;
        const uint32_t t = tie_estimate(
            reinterpret_cast<const uint32_t *>(staged_words + aspis::kStageTie), n_tie);
        local.tie_rows = (int32_t)t;
        full_keys = t >= kTieFullKeys;
    };
    // the two-pass path: the disagreement rows and the tie counts, one sync
    uint64_t rows[aspis::kStageWords] = {};
    auto graph_to_host = [&](aspis_clique_result *out_res) -> aspis_status {
        ASPIS_HIP(hipMemcpyAsync(rows, det->disagree, sizeof(uint64_t) * K,
                                 hipMemcpyDeviceToHost, s));
        if (tie_probe)
            ASPIS_HIP(hipMemcpyAsync(rows + aspis::kStageTie, tie_dev, sizeof(uint32_t) * n_tie,
                                     hipMemcpyDeviceToHost, s));
        ASPIS_HIP(hipStreamSynchronize(s));
        decide_keys(rows);
        return aspis_clique(rows, K, q, out_res);
    };
    // the row of every replica in a worker-major upload, in the workspace,
    // and the repair's group count copied back.  The host memory must
    // outlive the asynchronous copies: the guard, declared after it and so
    // destroyed before it, waits for the stream on every return once armed
    // (a no-op after the synchronisations of a normal return)
    std::vector<int32_t> host_rows;
    int32_t groups = -1;
    struct DrainStream {
        hipStream_t s;
        bool armed = false;
        ~DrainStream() {
            if (armed) (void)hipStreamSynchronize(s);
        }
    } drain{s};
    const int32_t *row_of = nullptr;
    if (worker_major) {
        drain.armed = true;
        host_rows.resize((size_t)f * r);
        worker_row_table(K, r, host_rows.data());
        ASPIS_HIP(hipMemcpyAsync(ws.row_of, host_rows.data(), host_rows.size() * sizeof(int32_t),
                                 hipMemcpyHostToDevice, s));
        row_of = ws.row_of;
    }

    const bool try_fused = !(flags & ASPIS_FLAG_TWO_PASS) && f <= aspis::kVoteRowsMaxFiles &&
                           (aspis::fused_supported(f, r) || aspis::fused_mean_supported(f, r));
    if (try_fused) {
        // the detection rows of the last vote, staged in the workspace by
        // vote_rows_kernel, with stage[64] = "some vote changed"
        uint64_t staged[aspis::kStageWords] = {};
        auto staged_clique = [&](aspis_clique_result *out_res, int words) -> aspis_status {
            ASPIS_HIP(hipMemcpyAsync(staged, ws.stage, sizeof(uint64_t) * words,
                                     hipMemcpyDeviceToHost, s));
            ASPIS_HIP(hipStreamSynchronize(s));
            return aspis_clique(staged, K, q, out_res);
        };
        // 1) agreement on the probed coordinates -> provisional clique and
        //    selection; the tie probe rides on the same copy to the host
        local.probe_coords = probe.coords();
        if (timing) ASPIS_HIP(hipEventRecord(ev[0], s));
        ASPIS_HIP(aspis::launch_agree_file(grads, row_of, f, r, d, probe, det->pair_diff, s));
        ASPIS_HIP(aspis::launch_vote_rows(det->pair_diff, subsets_dev, f, r, K, det->vote,
                                          det->has_majority, det->disagree, ws.stage, s));
        if (tie_probe)
            ASPIS_HIP(aspis::launch_tie_probe(grads, row_of, f, r, d, probe, tie_dev, s));
        if (timing) ASPIS_HIP(hipEventRecord(ev[1], s));
        aspis_clique_result guess{};
        if ((st = staged_clique(&guess, tie_probe ? aspis::kStageWords : 65)) != ASPIS_OK)
            return st;
        decide_keys(staged);
        // the reduction the guess calls for: the median (Case 2, or MEDIAN
        // mode) or the mean (Case 1 in PAPER mode, or MEAN mode)
        const bool guess_mean = use_mean(mode, &guess);
        if (guess_mean ? aspis::fused_mean_supported(f, r) : aspis::fused_supported(f, r)) {
            local.fused = 1;
            aspis::TileUse fused_tile{};   // stays empty for the mean
            // the guessed selection; the same launch zeroes pair_diff for
            // the main pass
            ASPIS_HIP(aspis::launch_select(subsets_dev, det->vote, f, r, guess.success,
                                           honest_mask(&guess), row_of, ws, nullptr,
                                           det->pair_diff, f, s));
            // 2) one pass: agreement on every coordinate + the reduction with
            //    the guessed selection
            if (timing) ASPIS_HIP(hipEventRecord(ev[2], s));
            if (guess_mean)
                ASPIS_HIP(aspis::launch_fused_mean(grads, row_of, f, r, d, ws, det->pair_diff, out, s));
            else
                ASPIS_HIP(aspis::launch_fused(grads, row_of, f, r, d, ws, det->pair_diff, out, s,
                                              &fused_tile, full_keys));
            if (timing) ASPIS_HIP(hipEventRecord(ev[3], s));
            ASPIS_HIP(aspis::launch_vote_rows(det->pair_diff, subsets_dev, f, r, K, det->vote,
                                              det->has_majority, det->disagree, ws.stage, s));
            if ((st = staged_clique(res, 65)) != ASPIS_OK) return st;
            const bool vote_changed = staged[64] != 0;
            // 3) the final selection.  The guess selected the same replica of
            //    every file iff both detections took the same case and
            //    Case 1 found the same H (the selection depends on H alone),
            //    or Case 2 voted the same slot for every file (it keeps the
            //    vote); it holds iff that is so and the reduction is the same
            const int64_t m = kept_files(K, r, f, res);
            if (n_selected) *n_selected = m;
            const bool same_sel =
                guess.success == res->success &&
                (res->success ? honest_mask(&guess) == honest_mask(res) : !vote_changed);
            const bool hit = same_sel && use_mean(mode, res) == guess_mean;
            local.speculation_hit = hit ? 1 : 0;
            if (m == 0) return fail(ASPIS_ERR_NO_FILES, "selection kept no file");
            // a wrong guess that asked for the same reduction as the final
            // detection is repaired tile by tile (every tile when the kept
            // files differ): the guessed selection is saved for the compare
            const bool final_mean = use_mean(mode, res);
            const bool repair = !hit && guess_mean == final_mean;
            if (timing) ASPIS_HIP(hipEventRecord(ev[4], s));
            if (repair) ASPIS_HIP(aspis::launch_save_sel(ws, f, s));
            // the workspace describes the final selection from here on (the
            // rows and positions a rerun of the reduction reads)
            if (!hit || sel_out)
                ASPIS_HIP(aspis::launch_select(subsets_dev, det->vote, f, r, res->success,
                                               honest_mask(res), row_of, ws, sel_out, nullptr, 0,
                                               s));
            if (!hit) {
                fused_tile = aspis::TileUse{};
                if (repair) {
                    const int cols = aspis::reduce_tile_cols(grads, f, d, final_mean, full_keys);
                    ASPIS_HIP(aspis::launch_dirty_tiles(grads, row_of, f, r, d, ws, det->pair_diff,
                                                        cols, s));
                    if (final_mean)
                        ASPIS_HIP(aspis::launch_mean(grads, d, ws, out, s, true));
                    else
                        ASPIS_HIP(aspis::launch_median(grads, d, ws, f, out, s, &fused_tile,
                                                       full_keys, true));
                    drain.armed = true;
                    ASPIS_HIP(hipMemcpyAsync(&groups, ws.repair, sizeof(int32_t),
                                             hipMemcpyDeviceToHost, s));
                } else if (final_mean) {
                    ASPIS_HIP(aspis::launch_mean(grads, d, ws, out, s));
                } else {
                    ASPIS_HIP(aspis::launch_median(grads, d, ws, f, out, s, &fused_tile, full_keys));
                }
            }
            local.tile_cols = fused_tile.cols;
            local.half_keys = fused_tile.half;
            if (timing) ASPIS_HIP(hipEventRecord(ev[5], s));
            ASPIS_HIP(hipStreamSynchronize(s));
            local.repair_groups = groups;
            if (timing) {
                ASPIS_HIP(hipEventElapsedTime(&local.ms_probe, ev[0], ev[1]));
                ASPIS_HIP(hipEventElapsedTime(&local.ms_main, ev[2], ev[3]));
                ASPIS_HIP(hipEventElapsedTime(&local.ms_fallback, ev[4], ev[5]));
            }
            local.ms_total = std::chrono::duration<float, std::milli>(clk::now() - t0).count();
            if (stats) *stats = local;
            return ASPIS_OK;
        }
    }
    // two-pass: full agreement, clique, then selection and reduction
    if (timing) ASPIS_HIP(hipEventRecord(ev[2], s));
    if ((st = detect_impl(grads, row_of, K, r, d, subsets_dev, det, stream)) != ASPIS_OK) return st;
    if (tie_probe)
        ASPIS_HIP(aspis::launch_tie_probe(grads, row_of, f, r, d, probe, tie_dev, s));
    if ((st = graph_to_host(res)) != ASPIS_OK) return st;
    aspis::TileUse tile{};
    st = aggregate_impl(grads, row_of, K, r, d, subsets_dev, det, res, mode, out, sel_out,
                        n_selected, workspace, ws_bytes, stream, &tile, full_keys);
    local.tile_cols = tile.cols;
    local.half_keys = tile.half;
    if (timing) ASPIS_HIP(hipEventRecord(ev[3], s));
    ASPIS_HIP(hipStreamSynchronize(s));
    if (timing) ASPIS_HIP(hipEventElapsedTime(&local.ms_main, ev[2], ev[3]));
    local.ms_total = std::chrono::duration<float, std::milli>(clk::now() - t0).count();
    if (stats) *stats = local;
    return st;
}


}  // namespace

extern "C" {

aspis_status aspis_detect(const float *grads, int32_t K, int32_t r, int64_t d,
                          const int32_t *subsets_dev, const aspis_detect_out *out, void *stream) {
    return detect_impl(grads, nullptr, K, r, d, subsets_dev, out, stream);
}

aspis_status aspis_aggregate(const float *grads, int32_t K, int32_t r, int64_t d,
                             const int32_t *subsets_dev, const aspis_detect_out *det,
                             const aspis_clique_result *res, aspis_reduce mode, float *out,
                             int32_t *sel_out, int64_t *n_selected, void *workspace,
                             size_t ws_bytes, void *stream) {
    return aggregate_impl(grads, nullptr, K, r, d, subsets_dev, det, res, mode, out, sel_out,
                          n_selected, workspace, ws_bytes, stream);
}

aspis_status aspis_detect_aggregate(const float *grads, int32_t K, int32_t r, int32_t q, int64_t d,
                                    const int32_t *subsets_dev, const aspis_detect_out *det,
                                    aspis_reduce mode, float *out, int32_t *sel_out,
                                    aspis_clique_result *res, int64_t *n_selected, void *workspace,
                                    size_t ws_bytes, uint32_t flags, aspis_run_stats *stats,
                                    void *stream) {
    return detect_aggregate_impl(grads, false, K, r, q, d, subsets_dev, det, mode, out, sel_out,
                                 res, n_selected, workspace, ws_bytes, flags, stats, stream);
}

aspis_status aspis_detect_aggregate_noalloc(const float *grads, int32_t K, int32_t r, int32_t q,
                                            int64_t d, const int32_t *subsets_dev,
                                            const aspis_detect_out *det, aspis_reduce mode,
                                            float *out, int32_t *sel_out,
                                            aspis_clique_result *res, int64_t *n_selected,
                                            uint32_t flags, aspis_run_stats *stats,
                                            void *stream) {
    int64_t f = 0;
    aspis_status st = check_device_shape(K, r, d, &f);
    if (st != ASPIS_OK) return st;
    if (flags & ASPIS_FLAG_TIMING)
        return fail(ASPIS_ERR_INVALID_ARG,
                    "aspis_detect_aggregate_noalloc: ASPIS_FLAG_TIMING creates timing events; "
                    "not available here");
    const size_t need = aspis::workspace_bytes(f, r);
    if (need > aspis::kScratchBytes)
        return fail(ASPIS_ERR_BUFFER_SMALL,
                    "aspis_detect_aggregate_noalloc: K=%d r=%d needs %zu bytes of scratch, the "
                    "static scratch holds %zu (use aspis_detect_aggregate with a workspace)",
                    K, r, need, aspis::kScratchBytes);
    void *scratch = nullptr;
    ASPIS_HIP(aspis::scratch_ptr(&scratch));
    return detect_aggregate_impl(grads, false, K, r, q, d, subsets_dev, det, mode, out, sel_out,
                                 res, n_selected, scratch, aspis::kScratchBytes, flags, stats,
                                 stream);
}

aspis_status aspis_detect_aggregate_wm(const float *grads_wm, int32_t K, int32_t r, int32_t q,
                                       int64_t d, const int32_t *subsets_dev,
                                       const aspis_detect_out *det, aspis_reduce mode, float *out,
                                       int32_t *sel_out, aspis_clique_result *res,
                                       int64_t *n_selected, void *workspace, size_t ws_bytes,
                                       uint32_t flags, aspis_run_stats *stats, void *stream) {
    return detect_aggregate_impl(grads_wm, true, K, r, q, d, subsets_dev, det, mode, out, sel_out,
                                 res, n_selected, workspace, ws_bytes, flags, stats, stream);
}

aspis_status aspis_worker_rows(int32_t K, int32_t r, int32_t *row_of, int64_t cap_entries) {
    if (K < 1 || r < 1 || r > K || row_of == nullptr)
        return fail(ASPIS_ERR_INVALID_ARG, "aspis_worker_rows: need 1 <= r <= K and a buffer");
    const int64_t f = binom(K, r);
    if (f < 0 || f > INT32_MAX / r) return fail(ASPIS_ERR_OVERFLOW, "C(%d,%d)*r overflows int32", K, r);
    if (f * r > cap_entries)
        return fail(ASPIS_ERR_BUFFER_SMALL, "need %lld entries, buffer holds %lld",
                    (long long)(f * r), (long long)cap_entries);
    worker_row_table(K, r, row_of);
    return ASPIS_OK;
}

static_assert(ASPIS_NOALLOC_SCRATCH_BYTES == aspis::kScratchBytes, "scratch size of aspis.h");
static_assert(ASPIS_KERNEL_NONE == aspis::kKernelNone && ASPIS_KERNEL_FUSED_WS == aspis::kKernelFusedWs &&
                  ASPIS_KERNEL_FUSED == aspis::kKernelFused &&
                  ASPIS_KERNEL_MEDIAN_WS == aspis::kKernelMedianWs &&
                  ASPIS_KERNEL_MEDIAN_TILE == aspis::kKernelMedianTile &&
                  ASPIS_KERNEL_MEDIAN_RADIX == aspis::kKernelMedianRadix,
              "kernel kinds of aspis.h and the launchers");

static void to_abi(const aspis::KernelPlan &k, aspis_kernel_plan *out) {
    out->kernel = k.kind;
    out->tile_cols = k.tile_cols;
    out->sweeps = k.sweeps;
    out->half_keys = k.half_keys;
    out->stream_threads = k.stream_threads;
    out->row_table = k.row_table;
    out->block = k.block;
    out->reserved = 0;
    out->lds_bytes = k.lds_bytes;
}

aspis_status aspis_plan(int32_t K, int32_t r, int64_t d, int32_t worker_major, uint32_t flags,
                        aspis_kernel_plan *single_pass, aspis_kernel_plan *median) {
    int64_t f = 0;
    aspis_status st = check_device_shape(K, r, d, &f);
    if (st != ASPIS_OK) return st;
    if (!single_pass || !median) return fail(ASPIS_ERR_INVALID_ARG, "aspis_plan: NULL output");
    const bool vec = d % 4 == 0;
    const bool full_keys = (flags & ASPIS_FLAG_FULL_KEYS) != 0;
    aspis::KernelPlan fused{}, med{};
    if (f <= aspis::kVoteRowsMaxFiles)
        aspis::plan_fused(f, r, vec, worker_major != 0, &fused, full_keys);
    aspis::plan_median(f, vec, &med, full_keys);
    to_abi(fused, single_pass);
    to_abi(med, median);
    if (fused.kind == aspis::kKernelUnbuilt || med.kind == aspis::kKernelUnbuilt)
        return fail(ASPIS_ERR_INVALID_ARG, "aspis_plan: K=%d r=%d d=%lld: a planned kernel is not built",
                    K, r, (long long)d);
    g_err[0] = 0;
    return ASPIS_OK;
}

size_t aspis_read_probe_sink_words(void) { return aspis::read_probe_sink_words(); }

aspis_status aspis_read_probe(const void *buf, size_t nbytes, uint32_t *sink, void *stream) {
    if (!buf || !sink || nbytes % 16 != 0 || ((uintptr_t)buf & 15u))
        return fail(ASPIS_ERR_INVALID_ARG, "aspis_read_probe: need 16-byte aligned buffer and size");
    ASPIS_HIP(aspis::launch_read_probe(buf, nbytes, sink, static_cast<hipStream_t>(stream)));
    return ASPIS_OK;
}

}  // extern "C"
