// aspis_kernels.hip -- gfx950 kernels of the Aspis detect-and-aggregate step.
//
// The replicas are float32 rows of d coordinates: row (i,s) holds the
// gradient the worker in slot s returned for file i, either at row i*r+s of
// a file-major [f][r][d] tensor or through a row table (the workers' own
// [K][l][d] uploads).  Everything here is integer work on the 32-bit
// patterns (bitwise comparison, order-preserving keys) except the fp64 sums
// of the mean, so nothing is a dense contraction and no MFMA is used; the
// kernels are bound by HBM reads.
//
//   agree_kernel       Eq. (4): per file, OR over coordinates of "slot pair p
//                      differs"; one coalesced stream over the r rows.
//   agree_file_kernel  the same over a coordinate prefix, one workgroup per
//                      file (the probe of the single pass).
//   vote_kernel        Eq. (3) majority per file and the K x K disagreement
//                      rows (Section 4: edge iff the pair agrees on all
//                      common files).
//   vote_rows_kernel   the same in one workgroup, rows built in LDS and
//                      staged for the host (the single pass).
//   select_kernel      Algorithm 1 selection (Case 1 honest replica / Case 2
//                      majority) and the ordered list of kept rows.
//   median_kernel      Algorithm 1 Case 2 coordinate-wise median: a tile of T
//                      coordinates x all kept rows is staged in LDS as
//                      totalOrder keys, and each column's lower median is
//                      found by G lanes of one wave (select_tile: one LDS
//                      histogram round, then a bitwise radix finish).
//   median_ws_kernel   the same median, warp-specialised like the single
//                      pass (two-pass path, and the rerun after a wrong guess).
//   fused_ws_kernel    agreement + median in one read, warp-specialised: some
//                      waves stream the next tile while the others select on
//                      the current one (the headline path, r = 3).  For
//                      hundreds of rows or more the LDS tile keeps only the
//                      high 16 bits of each key (select_half_tile), which
//                      doubles the tile width; the low halves of the rows
//                      that tie with the median's high half are read back.
//   fused_kernel       agreement + median in one read for r = 5, 7 and
//                      unaligned rows (load, then select, per tile).
//   fused_mean_kernel  agreement + Case 1 mean in one read.
//   mean_kernel        Algorithm 1 Case 1 mean, fp64 accumulation in file
//                      order.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>

#include "aspis_internal.h"

namespace aspis {

namespace {

// ---------------------------------------------------------------------------
// helpers

// Order-preserving map of a binary32 bit pattern to an unsigned key:
// unsigned order of keys == IEEE-754 totalOrder of the floats.
__device__ __forceinline__ uint32_t to_key(uint32_t b) {
    return b ^ ((uint32_t)((int32_t)b >> 31) | 0x80000000u);
}
__device__ __forceinline__ uint32_t from_key(uint32_t k) {
    return (k & 0x80000000u) ? (k ^ 0x80000000u) : ~k;
}

// Reductions over groups of G consecutive lanes (G a power of two <= 64).
// Offsets below 16 use DPP row permutations: after the two quad steps every
// lane of a quad holds the quad's value, and the half-row / row mirrors pair
// each lane with one lane of the other half.
enum class Op { And, Or, Add, Max, Min };

template <Op OP>
__device__ __forceinline__ uint32_t combine(uint32_t a, uint32_t b) {
    if constexpr (OP == Op::And) return a & b;
    if constexpr (OP == Op::Or) return a | b;
    if constexpr (OP == Op::Max) return a > b ? a : b;
    if constexpr (OP == Op::Min) return a < b ? a : b;
    return a + b;
}

// Two 16-bit unsigned lanes of a word at once (v_pk_min_u16, v_pk_max_u16,
// v_pk_add_u16: integer lanes, no carry between them).
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pk_min_u16(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_min(__builtin_bit_cast(u16x2, a),
                                                                  __builtin_bit_cast(u16x2, b)));
}
__device__ __forceinline__ uint32_t pk_max_u16(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(u16x2, a),
                                                                  __builtin_bit_cast(u16x2, b)));
}
__device__ __forceinline__ uint32_t pk_add_u16(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, a) + __builtin_bit_cast(u16x2, b));
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

template <int G, Op OP>
__device__ __forceinline__ uint32_t group_reduce(uint32_t v) {
    static_assert(G >= 1 && G <= 64 && (G & (G - 1)) == 0, "group size");
    if constexpr (G >= 2) v = combine<OP>(v, dpp<0xB1>(v));    // quad_perm [1,0,3,2]
    if constexpr (G >= 4) v = combine<OP>(v, dpp<0x4E>(v));    // quad_perm [2,3,0,1]
    if constexpr (G >= 8) v = combine<OP>(v, dpp<0x141>(v));   // row_half_mirror
    if constexpr (G >= 16) v = combine<OP>(v, dpp<0x140>(v));  // row_mirror
    if constexpr (G >= 32) v = combine<OP>(v, (uint32_t)__shfl_xor((int)v, 16, 64));
    if constexpr (G >= 64) v = combine<OP>(v, (uint32_t)__shfl_xor((int)v, 32, 64));
    return v;
}

// Inclusive prefix sum over groups of G consecutive lanes; g = lane index
// within the group.  A group inside one 16-lane row shifts with DPP row_shr;
// row_shr does not cross rows, so wider groups shift through ds_bpermute.
template <int G>
__device__ __forceinline__ uint32_t group_scan(uint32_t v, int g) {
#pragma unroll
    for (int k = 1; k < G; k <<= 1) {
        uint32_t y;
        if constexpr (G <= 16) {
            if (k == 1) y = dpp<0x111>(v);
            else if (k == 2) y = dpp<0x112>(v);
            else if (k == 4) y = dpp<0x114>(v);
            else y = dpp<0x118>(v);
        } else {
            y = (uint32_t)__shfl_up((int)v, k, 64);
        }
        v += (g >= k) ? y : 0u;
    }
    return v;
}

// Threads per workgroup of the tile kernels for tile width T: 1024 down to
// 16-wide tiles, then one wave (64 lanes) per column.
template <int T>
constexpr int tile_block() { return T >= 16 ? 1024 : 64 * T; }

// LDS layout of a [rows x T] key tile read by G lanes per column.  Row j
// lives at j*T; within the row, column c is stored at c ^ swz(j % G).  The
// G lanes of a column read rows j == g (mod G); the swizzle puts the 32
// lanes of every half-wave in 32 distinct banks.
template <int T, int G>
__host__ __device__ constexpr int tile_swz_of(int g) {
    static_assert(T == 4 || T == 8 || T == 16 || T == 32 || T == 64 || T == 128, "tile width");
    static_assert(G >= 1 && G <= 64 && (G & (G - 1)) == 0, "lanes per column");
    if constexpr (T >= 32) {
        static_assert(G <= 32, "swizzle needs at most 32 lanes per wide column");
        return g * (32 / G);
    } else {
        return (g / (32 / T)) & (T - 1);
    }
}

// The promise above, checked at compile time for every (T, G) the kernels
// instantiate: the first word each lane of a half-wave reads lies in a bank
// (of 32) of its own.  A lane's later rows lie G*T words further, a multiple
// of 32, so they keep the same banks.
template <int T, int G>
constexpr bool tile_swz_conflict_free() {
    for (int h = 0; h < T * G; h += 32) {
        uint32_t used = 0;
        for (int i = h; i < h + 32 && i < T * G; ++i) {
            const int c = i / G, g = i % G;
            const int bank = (g * T + (c ^ tile_swz_of<T, G>(g))) % 32;
            if (used & (1u << bank)) return false;
            used |= 1u << bank;
        }
    }
    return true;
}

template <int T, int G>
__device__ __forceinline__ int tile_swz(int g) {
    static_assert(tile_swz_conflict_free<T, G>(), "tile swizzle leaves a bank conflict");
    return tile_swz_of<T, G>(g);
}

// Store the keys of row j, columns 4cq..4cq+3.
template <int T, int G>
__device__ __forceinline__ void put_keys(uint32_t *tile, int j, int cq, const uint32_t k[4]) {
    const int sw = tile_swz<T, G>(j % G);
    if constexpr (T >= 32 && (32 / G) % 4 == 0) {
        // the swizzle keeps each aligned group of four columns together
        *reinterpret_cast<uint4 *>(&tile[j * T + ((4 * cq) ^ sw)]) = make_uint4(k[0], k[1], k[2], k[3]);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) tile[j * T + ((4 * cq + e) ^ sw)] = k[e];
    }
}

constexpr int kSelBatch = 8;   // LDS reads in flight per lane

// Per-column histogram of the selection (kHistBuckets buckets plus one
// overflow bucket); the column stride of kHistStride words keeps each
// column's bucket block 16-byte aligned and puts equal buckets of
// neighbouring columns in different banks.
constexpr int kHistWindow = 7;   // key bits resolved by one histogram round
static_assert(kHistBuckets == 1 << kHistWindow && kHistStride > kHistBuckets, "histogram");

__host__ __device__ constexpr int64_t hist_words(int T) { return (int64_t)T * kHistStride; }

// One pass over a lane's candidates, in batches of kSelBatch LDS reads.
template <int STRIDE, typename F>
__device__ __forceinline__ void for_each_candidate(const uint32_t *base, int cnt, F &&fn) {
    int x = 0;
    for (; x + kSelBatch <= cnt; x += kSelBatch) {
        uint32_t v[kSelBatch];
#pragma unroll
        for (int u = 0; u < kSelBatch; ++u) v[u] = base[(x + u) * STRIDE];
#pragma unroll
        for (int u = 0; u < kSelBatch; ++u) fn(v[u]);
    }
    for (; x < cnt; ++x) fn(base[x * STRIDE]);
}

// In-place compaction of a lane's candidates: keeps the values for which
// keep(v) holds, in order.  Every value is stored at the write cursor, which
// advances only for kept values; a batch is read before any of its slots is
// overwritten and the cursor never passes the read point.  Returns the
// number kept.
template <int STRIDE, typename F>
__device__ __forceinline__ int compact(uint32_t *base, int cnt, F &&keep) {
    int w = 0, x = 0;
    for (; x + kSelBatch <= cnt; x += kSelBatch) {
        uint32_t v[kSelBatch];
#pragma unroll
        for (int u = 0; u < kSelBatch; ++u) v[u] = base[(x + u) * STRIDE];
#pragma unroll
        for (int u = 0; u < kSelBatch; ++u) {
            base[w * STRIDE] = v[u];
            w += keep(v[u]) ? 1 : 0;
        }
    }
    for (; x < cnt; ++x) {
        const uint32_t v = base[x * STRIDE];
        base[w * STRIDE] = v;
        w += keep(v) ? 1 : 0;
    }
    return w;
}

// Lower median (rank floor((n-1)/2)) of each of the T columns of the LDS key
// tile holding n rows, found by the G lanes stid = c*G + g of each column c;
// written to out[k0 + c] for k0 + c < d.  hist: the workgroup's histogram
// block (hist_words(T) words, zero on entry; left zero on exit except for
// the overflow buckets).
//
// Exact selection on the keys in two stages:
//  1. histogram rounds while many candidates remain: the bits above the
//     highest bit where the candidates differ are common to all of them, so
//     the next kHistWindow bits below it split the candidates into ordered
//     buckets; an LDS histogram and a prefix scan over the buckets give the
//     bucket holding the sought rank, and only its members are kept
//     (compacted in place).  The first round decides the sign from the
//     count of sign-clear keys and works on the magnitude bits (the keys of
//     negative values hold them complemented); keys of the other sign land
//     in the overflow bucket or past every bucket of the sought sign.
//  2. bitwise MSB radix select on the few survivors: split on the highest
//     differing bit, keep the side holding the rank, until all are equal.
// Lane g owns rows g, g+G, ...; its x-th candidate lives at base[x*STRIDE].
template <int T, int G>
__device__ __forceinline__ void select_tile(uint32_t *tile, uint32_t *hist, int n, int64_t k0,
                                            int64_t d, float *out, int stid) {
    constexpr int STRIDE = G * T;
    constexpr int BPL = kHistBuckets / G;   // buckets scanned per lane
    static_assert(BPL >= 2 && BPL % 2 == 0, "buckets per lane");
    const int g = stid % G;
    const int c = stid / G;
    uint32_t *base = tile + g * T + (c ^ tile_swz<T, G>(g));
    uint32_t *hcol = hist + c * kHistStride;
    int cnt = (n > g) ? (n - g + G - 1) / G : 0;
    int total = n;
    uint32_t m = (uint32_t)(n - 1) / 2;

    // first pass: common magnitude bits and the count of sign-clear keys
    uint32_t am = 0xFFFFFFFFu, om = 0u, z = 0u;
    for_each_candidate<STRIDE>(base, cnt, [&](uint32_t v) {
        const uint32_t mag = (v ^ ~(uint32_t)((int32_t)v >> 31)) & 0x7FFFFFFFu;
        am &= mag;
        om |= mag;
        z += v >> 31;
    });
    am = group_reduce<G, Op::And>(am);
    om = group_reduce<G, Op::Or>(om);
    z = (uint32_t)total - group_reduce<G, Op::Add>(z);   // keys with the top bit clear

    auto and_or = [&](uint32_t &a, uint32_t &o) {
        a = 0xFFFFFFFFu;
        o = 0u;
        for_each_candidate<STRIDE>(base, cnt, [&](uint32_t v) {
            a &= v;
            o |= v;
        });
        a = group_reduce<G, Op::And>(a);
        o = group_reduce<G, Op::Or>(o);
    };
    // one histogram round over the candidates whose keys lie in
    // [bias, bias + 2^(hb+1)); keeps the bucket holding rank m
    auto hist_round = [&](uint32_t bias, int hb) {
        const int sh = hb >= kHistWindow - 1 ? hb - (kHistWindow - 1) : 0;
        for_each_candidate<STRIDE>(base, cnt, [&](uint32_t v) {
            const uint32_t b = min((v - bias) >> sh, (uint32_t)kHistBuckets);
            atomicAdd(&hcol[b], 1u);
        });
        // bucket holding rank m: B = number of buckets whose inclusive
        // prefix count is <= m, below = the largest such prefix
        uint32_t h[BPL];
#pragma unroll
        for (int q = 0; q < BPL; q += 2) {
            const uint2 w2 = *reinterpret_cast<const uint2 *>(&hcol[g * BPL + q]);
            h[q] = w2.x;
            h[q + 1] = w2.y;
        }
#pragma unroll
        for (int q = 0; q < BPL; q += 2)
            *reinterpret_cast<uint2 *>(&hcol[g * BPL + q]) = make_uint2(0u, 0u);
        uint32_t tot = 0u;
#pragma unroll
        for (int q = 0; q < BPL; ++q) tot += h[q];
        uint32_t run = group_scan<G>(tot, g) - tot;
        uint32_t le = 0u, below = 0u;
#pragma unroll
        for (int q = 0; q < BPL; ++q) {
            run += h[q];
            const bool ok = run <= m;
            le += ok ? 1u : 0u;
            below = ok ? run : below;
        }
        le = group_reduce<G, Op::Add>(le);
        below = group_reduce<G, Op::Max>(below);
        m -= below;
        const uint32_t lo = bias + (le << sh);
        const uint32_t width = 1u << sh;
        cnt = compact<STRIDE>(base, cnt, [&](uint32_t v) { return v - lo < width; });
        total = (int)group_reduce<G, Op::Add>((uint32_t)cnt);
    };

    uint32_t a, o, varying;
    bool have_count = false;
    if (total > 2 * G) {
        uint32_t sgn = 0x80000000u;
        if (m < z) sgn = 0u;
        else m -= z;
        const uint32_t vm = am ^ om;
        if (vm == 0u) {   // every candidate has the same magnitude
            a = sgn ? (0x80000000u | am) : (~am & 0x7FFFFFFFu);
            varying = 0u;
        } else {
            const int hb = 31 - __clz(vm);
            const uint32_t hi = 0x7FFFFFFFu & ~((2u << hb) - 1u);
            hist_round(sgn ? (0x80000000u | (am & hi)) : (~am & hi), hb);
            and_or(a, o);
            varying = a ^ o;
            // the sign is settled now; every round settles the bits from the
            // highest differing one down to the window's lowest, so the next
            // round starts strictly lower (at most 31 / kHistWindow more)
            for (int round = 0; varying != 0u && total > 2 * G && round < 5; ++round) {
                const int hb2 = 31 - __clz(varying);
                hist_round(a & ~((2u << hb2) - 1u), hb2);
                and_or(a, o);
                varying = a ^ o;
            }
        }
    } else {
        and_or(a, o);
        varying = a ^ o;
        have_count = (varying >> 31) != 0u;   // z counts zeros of the top bit
    }

    // each step settles the highest differing bit: at most 32 steps
    for (int step = 0; varying != 0u && step < 32; ++step) {
        const uint32_t bit = 1u << (31 - __clz(varying));
        if (!have_count) {
            z = 0u;
            for_each_candidate<STRIDE>(base, cnt, [&](uint32_t v) { z += (v & bit) == 0u; });
            z = group_reduce<G, Op::Add>(z);
        }
        have_count = false;
        uint32_t want;
        if (m < z) {
            want = 0u;
        } else {
            want = bit;
            m -= z;
        }
        cnt = compact<STRIDE>(base, cnt, [&](uint32_t v) { return (v & bit) == want; });
        and_or(a, o);
        varying = a ^ o;
    }
    if (g == 0 && k0 + c < d) out[k0 + c] = __uint_as_float(from_key(a));
}

// ---------------------------------------------------------------------------
// Half-key tiles.  The LDS tile holds only the high 16 bits of every key,
// two rows per word, so a tile of the same LDS size is twice as wide (and
// the row segments read from HBM twice as long).  The high half of the
// sought key is selected exactly on the tile; the low halves are then read
// back from the replica rows, only for the rows whose high half equals it
// (about one row per column on continuous data; every row when all high
// halves of a column are equal, which costs speed, not exactness).
//
// Layout for a streaming role of RPI rows per sweep: rows j and j + RPI,
// which one lane loads in two consecutive sweeps, share the word of
// pair-row p = (j / 2RPI) * RPI + j % RPI (j / RPI even: low half), stored
// at p*T + (c ^ swz(p % G)), so a lane writes whole words.  Rows without a
// kept value (past the last row, or a dropped file) hold the largest key,
// 0xFFFF, as do the low halves read back for them: appending elements that
// are not below any other leaves every rank below the kept count in place.

constexpr int kHalfWindow = 6;                  // key bits per histogram round
constexpr int kHalfBuckets = 1 << kHalfWindow;
constexpr int kHalfStride = kHalfBuckets + 2;   // words per column block
constexpr uint32_t kHalfTop = 0xFFFFu;          // largest key: padding rows

__host__ __device__ constexpr int64_t half_hist_words(int T) { return (int64_t)T * kHalfStride; }
// streaming rows per sweep of a tile T columns wide, for `fill` streaming
// threads of four columns each
__host__ __device__ constexpr int half_rpi(int T, int fill) { return fill * 4 / T; }
// pair-rows of a tile of `rows` rows: whole pairs of sweeps
__host__ __device__ constexpr int64_t half_pair_rows(int64_t rows, int T, int fill) {
    return (rows + 2 * half_rpi(T, fill) - 1) / (2 * half_rpi(T, fill)) * half_rpi(T, fill);
}
__host__ __device__ constexpr int64_t half_tile_words(int64_t rows, int T, int fill) {
    return half_pair_rows(rows, T, fill) * T;
}

// Row held by half h of pair-row p.
template <int RPI>
__device__ __forceinline__ int half_row(int p, int h) {
    return (p / RPI) * 2 * RPI + h * RPI + p % RPI;
}

// The high halves of two full keys, packed (a's in the low 16 bits).
__device__ __forceinline__ uint32_t pack_high(uint32_t a, uint32_t b) {
    return (a >> 16) | (b & 0xFFFF0000u);
}

// Store pair-row p, columns 4cq..4cq+3, from the packed high halves of the
// even sweep (lo: columns 0,1 and 2,3 in two registers) and of the odd one.
template <int T, int G>
__device__ __forceinline__ void put_pairs(uint32_t *tile, int p, int cq, const uint32_t lo[2],
                                          const uint32_t hi[2]) {
    uint32_t w[4];
    w[0] = (lo[0] & 0xFFFFu) | (hi[0] << 16);
    w[1] = (lo[0] >> 16) | (hi[0] & 0xFFFF0000u);
    w[2] = (lo[1] & 0xFFFFu) | (hi[1] << 16);
    w[3] = (lo[1] >> 16) | (hi[1] & 0xFFFF0000u);
    const int sw = tile_swz<T, G>(p % G);
    if constexpr (T >= 64 && (32 / G) % 4 == 0) {
        // the swizzle keeps each aligned group of four columns together
        *reinterpret_cast<uint4 *>(&tile[p * T + ((4 * cq) ^ sw)]) = make_uint4(w[0], w[1], w[2], w[3]);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) tile[p * T + ((4 * cq + e) ^ sw)] = w[e];
    }
}

// Lower median of each of the T columns of a half-key tile of np pair-rows
// holding nk kept values (1 <= nk, 2*np <= 65536), by the G lanes
// stid = c*G + g of column c, written to out[k0 + c] for k0 + c < d.
// row(j) gives the replica row of g behind tile row j, or -1 for a padding
// row.  hist: half_hist_words(T) words, zero on entry and on exit.  The
// tile is overwritten.  With REG > 0 (np a multiple of G, np / G <= REG)
// the lane's words are read from the tile once, into registers, and every
// later pass over the keys reads those (the median kernel measured 4-5 %
// faster at 455 rows; the single pass, whose registers are taken by its
// own state, keeps reading the tile).
//
//  1. one pass: the least key, the greatest key below 0xFFFF, the least
//     sign-set and the greatest sign-clear key, and the count of sign-set
//     keys (packed 16-bit min / max / add, two keys an instruction); settles
//     the sign and the window [lo, hi] of the keys of that sign;
//  2. histogram rounds over the window, each resolving kHalfWindow bits,
//     until the sought high half H is known (at most 3 rounds; H = 0xFFFF
//     when the rank falls past a sign-set window); nothing is compacted,
//     every round reads all keys;
//  3. one pass collecting the rows whose high half is H into the lane's
//     16-bit slots (in place), then their low halves are read from g;
//  4. bitwise radix select on those low halves for the remaining rank.
template <int T, int G, int RPI, int REG = 0, typename RowFn>
__device__ __forceinline__ void select_half_tile(uint32_t *tile, uint32_t *hist, int np, int nk,
                                                 int64_t k0, int64_t d, float *out, int stid,
                                                 const float *__restrict__ g, RowFn &&row) {
    constexpr int STRIDE = G * T;   // words between a lane's pair-rows
    constexpr int BPL = kHalfBuckets / G;
    static_assert(BPL >= 2 && BPL % 2 == 0, "buckets per lane");
    const int gl = stid % G;
    const int c = stid / G;
    uint32_t *base = tile + gl * T + (c ^ tile_swz<T, G>(gl));
    uint16_t *base16 = reinterpret_cast<uint16_t *>(base);
    uint32_t *hcol = hist + c * kHalfStride;
    const int cnt = np > gl ? (np - gl + G - 1) / G : 0;   // words of this lane
    uint32_t m = (uint32_t)(nk - 1) / 2;
    // REG > 0: the lane's words are read once, into registers.  The caller
    // passes np = half_pair_rows(...), a multiple of RPI = 4G, so every lane
    // of the wave holds the same count, a multiple of 4, at most REG
    static_assert(REG == 0 || RPI == 4 * G, "register mode needs RPI = 4G");
    uint32_t kw[REG > 0 ? REG : 1];
    const int cw = __builtin_amdgcn_readfirstlane(cnt);

    // every key of the lane: fn(key, word x, half h) for pair-row gl + x*G
    auto each = [&](auto &&fn) __attribute__((always_inline)) {
        if constexpr (REG > 0) {
            // cw is a multiple of 4 (np is a multiple of RPI = 4G)
#pragma unroll
            for (int xb = 0; xb < REG; xb += 4) {
                if (xb < cw) {
#pragma unroll
                    for (int x = xb; x < xb + 4 && x < REG; ++x) {
                        fn(kw[x] & 0xFFFFu, x, 0);
                        fn(kw[x] >> 16, x, 1);
                    }
                }
            }
            return;
        }
        int x = 0;
        for (; x + kSelBatch <= cnt; x += kSelBatch) {
            uint32_t v[kSelBatch];
#pragma unroll
            for (int u = 0; u < kSelBatch; ++u) v[u] = base[(x + u) * STRIDE];
#pragma unroll
            for (int u = 0; u < kSelBatch; ++u) {
                fn(v[u] & 0xFFFFu, x + u, 0);
                fn(v[u] >> 16, x + u, 1);
            }
        }
        for (; x < cnt; ++x) {
            const uint32_t v = base[x * STRIDE];
            fn(v & 0xFFFFu, x, 0);
            fn(v >> 16, x, 1);
        }
    };
    // the lane's x-th 16-bit slot (step 3 on)
    auto slot = [&](int x) __attribute__((always_inline)) -> uint16_t & {
        return base16[(x >> 1) * 2 * STRIDE + (x & 1)];
    };

    // 1. extremes and the sign count, both keys of a word at once in 16-bit
    //    lanes: the least key, the greatest key below 0xFFFF (the greatest
    //    key + 1, which wraps 0xFFFF to 0), and with the sign bit flipped the
    //    least sign-set key and the greatest sign-clear key; the number of
    //    sign-set keys
    uint32_t mn2 = 0xFFFFFFFFu, mt2 = 0u, ms2 = 0xFFFFFFFFu, mc2 = 0u, ns = 0u;
    auto stats = [&](uint32_t w) __attribute__((always_inline)) {
        const uint32_t x = w ^ 0x80008000u;
        mn2 = pk_min_u16(mn2, w);
        mt2 = pk_max_u16(mt2, pk_add_u16(w, 0x00010001u));
        ms2 = pk_min_u16(ms2, x);
        mc2 = pk_max_u16(mc2, x);
        ns += (uint32_t)__builtin_popcount(w & 0x80008000u);
    };
    if constexpr (REG > 0) {
#pragma unroll
        for (int xb = 0; xb < REG; xb += 4) {
            if (xb < cw) {
#pragma unroll
                for (int x = xb; x < xb + 4 && x < REG; ++x) kw[x] = base[x * STRIDE];
            }
        }
#pragma unroll
        for (int xb = 0; xb < REG; xb += 4) {
            if (xb < cw) {
#pragma unroll
                for (int x = xb; x < xb + 4 && x < REG; ++x) stats(kw[x]);
            }
        }
    } else {
        int x = 0;
        for (; x + kSelBatch <= cnt; x += kSelBatch) {
            uint32_t v[kSelBatch];
#pragma unroll
            for (int u = 0; u < kSelBatch; ++u) v[u] = base[(x + u) * STRIDE];
#pragma unroll
            for (int u = 0; u < kSelBatch; ++u) stats(v[u]);
        }
        for (; x < cnt; ++x) stats(base[x * STRIDE]);
    }
    auto lo16 = [](uint32_t v2, bool lower) __attribute__((always_inline)) {
        const uint32_t a = v2 & 0xFFFFu, b = v2 >> 16;
        return lower ? (a < b ? a : b) : (a > b ? a : b);
    };
    const uint32_t mn = group_reduce<G, Op::Min>(lo16(mn2, true));                // least key
    const uint32_t mt = group_reduce<G, Op::Max>(lo16(mt2, false));               // greatest below 0xFFFF, + 1
    const uint32_t ms = group_reduce<G, Op::Min>(lo16(ms2, true)) ^ 0x8000u;      // least sign-set
    const uint32_t mc = group_reduce<G, Op::Max>(lo16(mc2, false)) ^ 0x8000u;     // greatest sign-clear
    const uint32_t z = (uint32_t)(2 * np) - group_reduce<G, Op::Add>(ns);         // sign-clear count

    // 2. the window [lo, hi] of the keys of the sought key's sign (below
    //    0xFFFF); histogram rounds split it into kHalfBuckets buckets of
    //    2^sh keys and keep the one holding rank m, until sh = 0 (16 bits:
    //    three rounds at most).  A key above hi inside the window (0xFFFF, or
    //    a sign-set key in a sign-clear window) is counted like any other:
    //    it is above the sought key.  The rank past a sign-set window is a
    //    0xFFFF key.
    //    The round of single keys (sh = 0) also lists the lane's keys in its
    //    window as (word, half, bucket) codes in the lane's 16-bit slots, in
    //    place (the write cursor never passes the read cursor), and keeps
    //    those of the sought bucket as row numbers: step 3 then has its rows
    //    without another pass.  Not in a first round that may find the rank
    //    past a sign-set window (the tile must stay whole for the 0xFFFF
    //    pass), nor when a lane holds 512 words or more (9 bits of word).
    uint32_t H = kHalfTop;
    bool settled = false, collected = false;
    int w = 0;
    uint32_t lo, hi;
    const bool clear_sign = m < z;
    if (clear_sign) {
        lo = mn;
        hi = mc;
    } else {
        m -= z;
        lo = ms;
        hi = mt - 1u;
        if (mt == 0u || hi < lo) settled = true;   // no sign-set key below 0xFFFF
    }
    if (!settled) {
        uint32_t bias = lo;
        const int width = 32 - __clz(hi - lo);   // bits of hi - lo (0 when equal)
        int sh = width > kHalfWindow ? width - kHalfWindow : 0;
        for (int round = 0; round < 3; ++round) {
            const uint32_t span = (uint32_t)kHalfBuckets << sh;
            const bool list = sh == 0 && (round > 0 || clear_sign) && np <= 511 * G;
            if (list) {
                each([&](uint32_t k, int x, int hf) {
                    const uint32_t o = k - bias;
                    if (o < span) {
                        atomicAdd(&hcol[o], 1u);
                        slot(w) = (uint16_t)(((uint32_t)x << 7) | ((uint32_t)hf << 6) | o);
                        ++w;
                    }
                });
            } else {
                each([&](uint32_t k, int, int) {
                    const uint32_t o = k - bias;
                    if (o < span) atomicAdd(&hcol[o >> sh], 1u);
                });
            }
            uint32_t h[BPL];
#pragma unroll
            for (int q = 0; q < BPL; q += 2) {
                const uint2 w2 = *reinterpret_cast<const uint2 *>(&hcol[gl * BPL + q]);
                h[q] = w2.x;
                h[q + 1] = w2.y;
            }
#pragma unroll
            for (int q = 0; q < BPL; q += 2)
                *reinterpret_cast<uint2 *>(&hcol[gl * BPL + q]) = make_uint2(0u, 0u);
            uint32_t tot = 0u;
#pragma unroll
            for (int q = 0; q < BPL; ++q) tot += h[q];
            uint32_t run = group_scan<G>(tot, gl) - tot;
            uint32_t le = 0u, below = 0u;
#pragma unroll
            for (int q = 0; q < BPL; ++q) {
                run += h[q];
                const bool ok = run <= m;
                le += ok ? 1u : 0u;
                below = ok ? run : below;
            }
            le = group_reduce<G, Op::Add>(le);
            below = group_reduce<G, Op::Max>(below);
            m -= below;
            if (le == (uint32_t)kHalfBuckets) {   // past the window: a 0xFFFF key
                settled = true;
                break;
            }
            bias += le << sh;
            if (sh == 0) {
                if (list) {   // the listed keys of bucket le, as row numbers
                    int n2 = 0;
                    for (int j = 0; j < w; ++j) {
                        const uint32_t v = slot(j);
                        if ((v & 63u) == le) {
                            slot(n2) = (uint16_t)half_row<RPI>(gl + (int)(v >> 7) * G, (int)(v >> 6) & 1);
                            ++n2;
                        }
                    }
                    w = n2;
                    collected = true;
                }
                break;
            }
            sh = sh > kHalfWindow ? sh - kHalfWindow : 0;
        }
        if (!settled) H = bias;
    }

    // 3. rows whose high half is H, as row numbers in the lane's slots (the
    //    write cursor never passes the read cursor), then their low halves
    if (!collected) {
        w = 0;
        each([&](uint32_t k, int x, int hf) {
            if (k == H) {
                slot(w) = (uint16_t)half_row<RPI>(gl + x * G, hf);
                ++w;
            }
        });
    }
    const bool valid = k0 + c < d;
    constexpr int kGather = 4;   // row reads in flight per lane
    for (int x0 = 0; x0 < w; x0 += kGather) {
        uint32_t v[kGather];
#pragma unroll
        for (int u = 0; u < kGather; ++u) {
            v[u] = 0xFFFFFFFFu;   // a padding row: the largest key
            if (x0 + u < w) {
                const int64_t rr = row(slot(x0 + u));
                if (rr >= 0 && valid) v[u] = to_key(__float_as_uint(g[rr * d + k0 + c]));
            }
        }
#pragma unroll
        for (int u = 0; u < kGather; ++u)
            if (x0 + u < w) slot(x0 + u) = (uint16_t)(v[u] & 0xFFFFu);
    }

    // 4. bitwise radix select of rank m among the low halves
    auto and_or = [&](uint32_t &a, uint32_t &o) __attribute__((always_inline)) {
        a = 0xFFFFu;
        o = 0u;
        for (int x = 0; x < w; ++x) {
            const uint32_t v = slot(x);
            a &= v;
            o |= v;
        }
        a = group_reduce<G, Op::And>(a);
        o = group_reduce<G, Op::Or>(o);
    };
    uint32_t a, o;
    and_or(a, o);
    uint32_t varying = a ^ o;
    for (int step = 0; varying != 0u && step < 16; ++step) {
        const uint32_t bit = 1u << (31 - __clz(varying));
        uint32_t zc = 0u;
        for (int x = 0; x < w; ++x) zc += (slot(x) & bit) == 0u;
        zc = group_reduce<G, Op::Add>(zc);
        uint32_t want;
        if (m < zc) {
            want = 0u;
        } else {
            want = bit;
            m -= zc;
        }
        int nw = 0;
        for (int x = 0; x < w; ++x) {
            const uint16_t v = slot(x);
            slot(nw) = v;
            nw += (v & bit) == want ? 1 : 0;
        }
        w = nw;
        and_or(a, o);
        varying = a ^ o;
    }
    if (gl == 0 && valid) out[k0 + c] = __uint_as_float(from_key((H << 16) | a));
}

// One 16-byte load (16-byte aligned) from a replica row that the pass
// reads once: a non-temporal load, which streams past the caches instead of
// filling them with lines nothing reads again (measured 3-6 % faster than a
// plain load on the 61 GB single pass).
__device__ __forceinline__ uint4 load_stream(const float *p) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Load four consecutive coordinates [k, k+4) of one row as bit patterns;
// coordinates at or beyond kend read as 0.
template <bool VEC>
__device__ __forceinline__ void load4(const float *row, int64_t k, int64_t kend,
                                      uint32_t v[4]) {
    if (VEC && k + 3 < kend) {
        const uint4 q = load_stream(row + k);
        v[0] = q.x;
        v[1] = q.y;
        v[2] = q.z;
        v[3] = q.w;
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            v[e] = (k + e < kend) ? __float_as_uint(row[k + e]) : 0u;
    }
}

// ---------------------------------------------------------------------------
// utility kernels

__global__ void fill_u32_kernel(uint32_t *p, int64_t n, uint32_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}
__global__ void fill_u64_kernel(uint64_t *p, int64_t n, uint64_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// ---------------------------------------------------------------------------
// agreement: Eq. (4) for every file and slot pair, over coordinates [0,kend)

constexpr int kAgreeUnroll = 4;                       // float4 per thread
constexpr int64_t kAgreeChunk = (int64_t)kBlock * 4 * kAgreeUnroll;

// Row of replica (i,s): i*R+s in the file-major tensor, or row_of[i*R+s]
// when a row table is given.
__device__ __forceinline__ int64_t replica_row(const int32_t *row_of, int64_t i, int R, int s) {
    return row_of ? (int64_t)row_of[i * R + s] : i * R + s;
}

template <int R, bool VEC>
__global__ void __launch_bounds__(kBlock)
agree_kernel(const float *__restrict__ g, const int32_t *__restrict__ row_of, int64_t f,
             int64_t d, int64_t kend, int64_t nchunks, uint32_t *__restrict__ pair_diff) {
    const int64_t nwork = f * nchunks;
    for (int64_t w = blockIdx.x; w < nwork; w += gridDim.x) {
        const int64_t i = w / nchunks;
        const int64_t chunk = w - i * nchunks;
        const float *rows[R];
#pragma unroll
        for (int s = 0; s < R; ++s) rows[s] = g + replica_row(row_of, i, R, s) * d;
        uint32_t diff = 0u;
#pragma unroll
        for (int u = 0; u < kAgreeUnroll; ++u) {
            const int64_t k = chunk * kAgreeChunk + (int64_t)u * kBlock * 4 +
                              (int64_t)threadIdx.x * 4;
            if (k < kend) {
                uint32_t v[R][4];
#pragma unroll
                for (int s = 0; s < R; ++s) load4<VEC>(rows[s], k, kend, v[s]);
                int p = 0;
#pragma unroll
                for (int s = 0; s < R; ++s)
#pragma unroll
                    for (int t = s + 1; t < R; ++t) {
                        const uint32_t x = (v[s][0] ^ v[t][0]) | (v[s][1] ^ v[t][1]) |
                                           (v[s][2] ^ v[t][2]) | (v[s][3] ^ v[t][3]);
                        diff |= (x != 0u ? 1u : 0u) << p;
                        ++p;
                    }
            }
        }
        // OR over the wave; one atomic per wave only when something differs
        uint32_t wdiff = 0u;
        constexpr int P = R * (R - 1) / 2;
#pragma unroll
        for (int p = 0; p < P; ++p)
            if (__ballot((diff >> p) & 1u)) wdiff |= 1u << p;
        // the word already holds the bits after the first chunks of a file
        // that differs: read it first, so that the other chunks' waves of
        // that file do not all queue atomics on one address
        if ((threadIdx.x & 63) == 0 && wdiff && (wdiff & ~__atomic_load_n(&pair_diff[i], __ATOMIC_RELAXED)))
            atomicOr(&pair_diff[i], wdiff);
    }
}

// Agreement of one file per workgroup over coordinates [0,kend) (the
// prefix probe of the single pass): the workgroup ORs its lanes' bits and
// stores the file's word, so pair_diff needs no zero fill and no atomics.
template <int R, bool VEC>
__global__ void __launch_bounds__(kBlock)
agree_file_kernel(const float *__restrict__ g, const int32_t *__restrict__ row_of, int64_t f,
                  int64_t d, ProbeSet probe, uint32_t *__restrict__ pair_diff) {
    static_assert(kProbeBlockCols == kBlock * 4, "one float4 per thread and probe block");
    __shared__ uint32_t wave_bits[kBlock / 64];
    constexpr int P = R * (R - 1) / 2;
    for (int64_t i = blockIdx.x; i < f; i += gridDim.x) {
        const float *rows[R];
#pragma unroll
        for (int s = 0; s < R; ++s) rows[s] = g + replica_row(row_of, i, R, s) * d;
        uint32_t diff = 0u;
        for (int64_t j0 = 0; j0 < probe.nb; j0 += kAgreeUnroll) {
            uint32_t v[kAgreeUnroll][R][4];
#pragma unroll
            for (int u = 0; u < kAgreeUnroll; ++u) {
                // block j0+u: the thread's four coordinates (none past its end)
                int64_t k = 0, kend = 0;
                if (j0 + u < probe.nb) {
                    const int64_t b = probe.block_start(j0 + u);
                    k = b + (int64_t)threadIdx.x * 4;
                    kend = probe.block_end(b);
                }
#pragma unroll
                for (int s = 0; s < R; ++s) {
                    if (k < kend)
                        load4<VEC>(rows[s], k, kend, v[u][s]);
                    else
                        v[u][s][0] = v[u][s][1] = v[u][s][2] = v[u][s][3] = 0u;
                }
            }
#pragma unroll
            for (int u = 0; u < kAgreeUnroll; ++u) {
                int p = 0;
#pragma unroll
                for (int s = 0; s < R; ++s)
#pragma unroll
                    for (int t = s + 1; t < R; ++t) {
                        const uint32_t x = (v[u][s][0] ^ v[u][t][0]) | (v[u][s][1] ^ v[u][t][1]) |
                                           (v[u][s][2] ^ v[u][t][2]) | (v[u][s][3] ^ v[u][t][3]);
                        diff |= (x != 0u ? 1u : 0u) << p;
                        ++p;
                    }
            }
        }
        uint32_t wdiff = 0u;
#pragma unroll
        for (int p = 0; p < P; ++p)
            if (__ballot((diff >> p) & 1u)) wdiff |= 1u << p;
        if ((threadIdx.x & 63) == 0) wave_bits[threadIdx.x >> 6] = wdiff;
        __syncthreads();
        if (threadIdx.x == 0) {
            uint32_t b = 0u;
#pragma unroll
            for (int w = 0; w < kBlock / 64; ++w) b |= wave_bits[w];
            pair_diff[i] = b;
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// vote and disagreement rows

// Eq. (3) for one file from its pair-difference word: the lowest slot of the
// largest class of bitwise-equal replicas and that class's size.  Calls
// differ(s, t) for every slot pair whose replicas differ.
template <typename DiffFn>
__device__ __forceinline__ void file_vote(uint32_t pd, int r, int *vote_slot, int *class_size,
                                          DiffFn differ) {
    // same[s] = bitmask of slots whose replica equals slot s's
    uint32_t same[8];
    for (int s = 0; s < r; ++s) same[s] = 1u << s;
    int p = 0;
    for (int s = 0; s < r; ++s)
        for (int t = s + 1; t < r; ++t, ++p) {
            if (pd >> p & 1u) {
                differ(s, t);
            } else {
                same[s] |= 1u << t;
                same[t] |= 1u << s;
            }
        }
    int best = 0, best_n = 0;
    for (int s = 0; s < r; ++s) {
        const int c = __popc(same[s]);
        if (c > best_n) {
            best_n = c;
            best = s;
        }
    }
    *vote_slot = best;
    *class_size = best_n;
}

__global__ void vote_kernel(const uint32_t *__restrict__ pair_diff,
                            const int32_t *__restrict__ subsets, int64_t f,
                            int r, int8_t *__restrict__ vote,
                            uint8_t *__restrict__ has_majority,
                            uint64_t *__restrict__ disagree) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < f;
         i += (int64_t)gridDim.x * blockDim.x) {
        int best = 0, best_n = 0;
        file_vote(pair_diff[i], r, &best, &best_n, [&](int s, int t) {
            const int us = subsets[i * r + s], ut = subsets[i * r + t];
            atomicOr((unsigned long long *)&disagree[us], 1ull << ut);
            atomicOr((unsigned long long *)&disagree[ut], 1ull << us);
        });
        vote[i] = (int8_t)best;
        has_majority[i] = (uint8_t)(best_n >= (r + 1) / 2);
    }
}

// The same in one workgroup, for the single pass (f is at most a few
// thousand there): the K rows are built in LDS and stored whole (no zero
// fill), and a copy goes to stage[0..K) for the host, with stage[64] = 1 if
// any file's vote differs from the one vote[] held before the call.
__global__ void __launch_bounds__(1024)
vote_rows_kernel(const uint32_t *__restrict__ pair_diff, const int32_t *__restrict__ subsets,
                 int64_t f, int r, int K, int8_t *__restrict__ vote,
                 uint8_t *__restrict__ has_majority, uint64_t *__restrict__ disagree,
                 uint64_t *__restrict__ stage) {
    __shared__ unsigned long long rows[64];
    __shared__ int changed;
    const int tid = threadIdx.x;
    if (tid < 64) rows[tid] = 0ull;
    if (tid == 0) changed = 0;
    __syncthreads();
    for (int64_t i = tid; i < f; i += blockDim.x) {
        int best = 0, best_n = 0;
        file_vote(pair_diff[i], r, &best, &best_n, [&](int s, int t) {
            const int us = subsets[i * r + s], ut = subsets[i * r + t];
            atomicOr(&rows[us], 1ull << ut);
            atomicOr(&rows[ut], 1ull << us);
        });
        if (vote[i] != (int8_t)best) changed = 1;
        vote[i] = (int8_t)best;
        has_majority[i] = (uint8_t)(best_n >= (r + 1) / 2);
    }
    __syncthreads();
    if (tid < K) {
        disagree[tid] = rows[tid];
        stage[tid] = rows[tid];
    }
    if (tid == 0) stage[64] = (uint64_t)changed;
}

// ---------------------------------------------------------------------------
// selection (one workgroup of 1024 threads; f is at most a few thousand)

__global__ void __launch_bounds__(1024)
select_kernel(const int32_t *__restrict__ subsets,
              const int8_t *__restrict__ vote, int64_t f, int r,
              int success, uint64_t honest, const int32_t *__restrict__ row_of,
              int32_t *__restrict__ sel, int32_t *__restrict__ pos, int32_t *__restrict__ rows,
              int32_t *__restrict__ n_sel, int32_t *__restrict__ sel_out,
              uint32_t *__restrict__ zero, int64_t n_zero) {
    __shared__ int wave_tot[16];
    __shared__ int carry;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (zero)
        for (int64_t i = tid; i < n_zero; i += 1024) zero[i] = 0u;
    if (tid == 0) carry = 0;
    __syncthreads();
    for (int64_t b = 0; b < f; b += 1024) {
        const int64_t i = b + tid;
        int s = -1;
        if (i < f) {
            if (success) {
                for (int x = 0; x < r; ++x)
                    if (honest >> subsets[i * r + x] & 1ull) {
                        s = x;
                        break;
                    }
            } else {
                s = vote[i];
            }
        }
        const bool keep = s >= 0;
        const uint64_t bal = __ballot(keep);
        const int in_wave = __popcll(bal & ((1ull << lane) - 1ull));
        if (lane == 0) wave_tot[wave] = __popcll(bal);
        __syncthreads();
        int before = carry;
        for (int w = 0; w < wave; ++w) before += wave_tot[w];
        if (i < f) {
            const int p = keep ? before + in_wave : -1;
            sel[i] = s;
            pos[i] = p;
            if (sel_out) sel_out[i] = s;
            if (keep) rows[p] = row_of ? row_of[i * r + s] : (int32_t)(i * r + s);
        }
        __syncthreads();
        if (tid == 0) {
            int tot = 0;
            for (int w = 0; w < 16; ++w) tot += wave_tot[w];
            carry += tot;
        }
        __syncthreads();
    }
    if (tid == 0) *n_sel = carry;
}

// ---------------------------------------------------------------------------
// median of the kept rows

constexpr int kMedianBatch = 8;   // row loads per thread issued as one burst

// The tiles a median launch computes: every tile, or (a repair after a
// wrong guess) the tiles of the groups whose bit is set, bit b for tiles
// [b << gshift, (b + 1) << gshift).  Uniform per workgroup.
struct TileMask {
    const uint32_t *bits = nullptr;
    const int32_t *count = nullptr;   // groups set (no tile at all when 0)
    int gshift = 0;
    __device__ __forceinline__ bool has(int64_t t) const {
        const int64_t b = t >> gshift;
        return ((bits[b >> 5] >> (b & 31)) & 1u) != 0u;
    }
    // the first computed tile of t, t + step, ..., or one >= ntiles: t
    // itself when its bit is set, else the bits of eight candidates at once
    __device__ __forceinline__ int64_t next(int64_t t, int64_t step, int64_t ntiles) const {
        if (bits == nullptr || t >= ntiles) return t;
        if (*count == 0) return ntiles;
        if (has(t)) return t;
        for (t += step; t < ntiles; t += 8 * step) {
            uint32_t hit = 0u;
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int64_t tu = t + u * step;
                if (tu < ntiles && has(tu)) hit |= 1u << u;
            }
            if (hit) return t + (int64_t)(__ffs(hit) - 1) * step;
        }
        return ntiles;
    }
};

template <int T, bool VEC>
__global__ void __launch_bounds__(tile_block<T>())
median_kernel(const float *__restrict__ g, int64_t d,
              const int32_t *__restrict__ rows, const int32_t *__restrict__ n_sel,
              int64_t ntiles, float *__restrict__ out, TileMask mask) {
    extern __shared__ uint32_t smem[];
    constexpr int BLOCK = tile_block<T>();
    uint32_t *hist = smem;
    uint32_t *tile = smem + hist_words(T);
    constexpr int G = BLOCK / T;
    constexpr int CPR = T / 4;           // float4 chunks per row segment
    constexpr int RPI = BLOCK / CPR;     // rows filled per sweep
    const int n = *n_sel;
    if (n <= 0) return;
    const int tid = threadIdx.x;
    for (int i = tid; i < hist_words(T); i += BLOCK) hist[i] = 0u;
    const int cq = tid % CPR, j0 = tid / CPR;
    for (int64_t t = mask.next(blockIdx.x, gridDim.x, ntiles); t < ntiles;
         t = mask.next(t + gridDim.x, gridDim.x, ntiles)) {
        const int64_t k0 = t * T;
        for (int jb = 0; jb < n; jb += RPI * kMedianBatch) {
            uint32_t v[kMedianBatch][4];
#pragma unroll
            for (int b = 0; b < kMedianBatch; ++b) {
                const int j = jb + b * RPI + j0;
                if (j < n) load4<VEC>(g + (int64_t)rows[j] * d, k0 + 4 * cq, d, v[b]);
            }
#pragma unroll
            for (int b = 0; b < kMedianBatch; ++b) {
                const int j = jb + b * RPI + j0;
                if (j < n) {
                    uint32_t k[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) k[e] = to_key(v[b][e]);
                    put_keys<T, G>(tile, j, cq, k);
                }
            }
        }
        __syncthreads();
        select_tile<T, G>(tile, hist, n, k0, d, out, tid);
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// fused agreement + median (one read of all r replicas)

template <int R>
constexpr int fused_batch() { return R == 3 ? 4 : (R == 5 ? 2 : 1); }

template <int T, int R, bool VEC>
__global__ void __launch_bounds__(tile_block<T>())
fused_kernel(const float *__restrict__ g, const int32_t *__restrict__ row_of, int64_t f, int64_t d,
             const int32_t *__restrict__ sel, const int32_t *__restrict__ pos,
             const int32_t *__restrict__ n_sel, int64_t ntiles,
             uint32_t *__restrict__ pair_diff, float *__restrict__ out) {
    extern __shared__ uint32_t smem[];
    constexpr int BLOCK = tile_block<T>();
    constexpr int G = BLOCK / T;
    constexpr int CPR = T / 4;
    constexpr int RPI = BLOCK / CPR;
    constexpr int B = fused_batch<R>();
    const int n = *n_sel;
    uint32_t *hist = smem;
    uint32_t *tile = smem + hist_words(T);
    uint32_t *pd = tile + f * T;         // [f] per-workgroup pair-difference bits
    const int tid = threadIdx.x;
    for (int64_t i = tid; i < f; i += BLOCK) pd[i] = 0u;
    for (int i = tid; i < hist_words(T); i += BLOCK) hist[i] = 0u;
    __syncthreads();
    const int cq = tid % CPR, j0 = tid / CPR;
    for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const int64_t k0 = t * T;
        for (int64_t ib = 0; ib < f; ib += (int64_t)RPI * B) {
            uint32_t v[B][R][4];
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const int64_t i = ib + b * RPI + j0;
                if (i < f) {
#pragma unroll
                    for (int s = 0; s < R; ++s)
                        load4<VEC>(g + replica_row(row_of, i, R, s) * d, k0 + 4 * cq, d, v[b][s]);
                }
            }
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const int64_t i = ib + b * RPI + j0;
                if (i >= f) continue;
                uint32_t diff = 0u;
                int p = 0;
#pragma unroll
                for (int s = 0; s < R; ++s)
#pragma unroll
                    for (int u = s + 1; u < R; ++u) {
                        const uint32_t x = (v[b][s][0] ^ v[b][u][0]) | (v[b][s][1] ^ v[b][u][1]) |
                                           (v[b][s][2] ^ v[b][u][2]) | (v[b][s][3] ^ v[b][u][3]);
                        diff |= (x != 0u ? 1u : 0u) << p;
                        ++p;
                    }
                if (diff) atomicOr(&pd[i], diff);
                const int j = pos[i];
                if (j >= 0) {
                    const int s_sel = sel[i];
                    uint32_t w[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        w[e] = v[b][0][e];
#pragma unroll
                        for (int s = 1; s < R; ++s) w[e] = (s_sel == s) ? v[b][s][e] : w[e];
                    }
#pragma unroll
                    for (int e = 0; e < 4; ++e) w[e] = to_key(w[e]);
                    put_keys<T, G>(tile, j, cq, w);
                }
            }
        }
        __syncthreads();
        if (n > 0) select_tile<T, G>(tile, hist, n, k0, d, out, tid);
        __syncthreads();
    }
    for (int64_t i = tid; i < f; i += BLOCK)
        if (pd[i]) atomicOr(&pair_diff[i], pd[i]);
}

// ---------------------------------------------------------------------------
// fused agreement + median, warp-specialised: waves 0-7 stream tile t+1 into
// registers (compare the r replicas, keep the guessed replica's keys) while
// waves 8-15 run the selection on tile t in LDS; the keys are handed over
// between two barriers.  The row loads and the selection overlap inside one
// workgroup, so a single [f x T] tile of LDS per CU is enough.

constexpr int kWsThreads = 1024;   // threads of a warp-specialised workgroup
constexpr int kWsFill = 512;       // threads of the streaming role (default split)

// sweeps per burst of loads: as many as the streaming role's registers hold
// next to the tile's keys (SW x 4 registers, or SW x 2 with half keys).  The
// 36-sweep tile spills either way; one sweep per burst spills least
template <int R, int SW>
constexpr int ws_batch() { return R == 3 ? (SW > 32 ? 1 : SW > 12 ? 2 : 3) : 1; }

template <int T, int R, int SW, bool IND, bool HALF, int FILL, bool RTG = false>
__global__ void __launch_bounds__(kWsThreads)
fused_ws_kernel(const float *__restrict__ g, const int32_t *__restrict__ row_of, int64_t f, int64_t d,
                const int32_t *__restrict__ sel, const int32_t *__restrict__ pos,
                const int32_t *__restrict__ n_sel, int64_t ntiles,
                uint32_t *__restrict__ pair_diff, float *__restrict__ out) {
    extern __shared__ uint32_t smem[];
    constexpr int G = (kWsThreads - FILL) / T;   // selection lanes per column
    constexpr int CPR = T / 4;           // float4 chunks per row segment
    constexpr int RPI = FILL / CPR;      // rows per sweep of the streaming role
    constexpr int B = ws_batch<R, SW>(); // sweeps per burst of loads
    // key registers per sweep: 4 keys, or (HALF) 4 high halves packed in 2;
    // a half-key tile's rows are the files themselves
    constexpr int KW = HALF ? 2 : 4;
    static_assert(!HALF || (SW % 2 == 0 && RPI == half_rpi(T, FILL) && RPI % 8 == 0 && R <= 7),
                  "half-key sweeps");
    // a file's pair-difference bits fit a nibble only at r = 3 (3 bits)
    constexpr bool PDN = HALF && R == 3;
    const int n = *n_sel;
    const int64_t hwords = HALF ? half_hist_words(T) : hist_words(T);
    const int64_t f8 = (f + 7) / 8;
    uint32_t *hist = smem;               // selection histograms
    uint32_t *tile = smem + hwords;
    // per-file words.  Full keys: pd [f] pair-difference bits, ps [f]
    // (tile row << 3) | slot or -1.  Half keys (tile row = file): ps [f/8],
    // one nibble per file, 8 | slot or 0; pd [f/8] pair-difference nibbles
    // at r = 3, else pd [f] words
    uint32_t *pd = tile + (HALF ? half_tile_words(f, T, FILL) : f * T);
    int32_t *ps = reinterpret_cast<int32_t *>(pd + (PDN ? f8 : f));
    // [f*R] row table (IND): staged in LDS, or (RTG) read from global
    // memory, where it stays cached, when LDS is needed for a wider tile
    int32_t *rt_lds = ps + (HALF ? f8 : f);
    const int32_t *rt = RTG ? row_of : rt_lds;
    const int tid = threadIdx.x;
    if constexpr (HALF) {
        for (int64_t w = tid; w < f8; w += kWsThreads) {
            uint32_t v = 0u;
            for (int e = 0; e < 8; ++e) {
                const int64_t i = 8 * w + e;
                if (i < f && pos[i] >= 0) v |= (8u | (uint32_t)sel[i]) << (4 * e);
            }
            ps[w] = (int32_t)v;
        }
        for (int64_t w = tid; w < (PDN ? f8 : f); w += kWsThreads) pd[w] = 0u;
    } else {
        for (int64_t i = tid; i < f; i += kWsThreads) {
            pd[i] = 0u;
            ps[i] = pos[i] >= 0 ? (pos[i] << 3) | sel[i] : -1;
        }
    }
    // the slot nibble of file i (HALF): 8 | slot when kept, else 0
    auto nib = [&](int i) __attribute__((always_inline)) {
        return ((uint32_t)ps[i >> 3] >> ((i & 7) * 4)) & 15u;
    };
    if constexpr (IND && !RTG)
        for (int64_t i = tid; i < f * R; i += kWsThreads) rt_lds[i] = row_of[i];
    for (int i = tid; i < hwords; i += kWsThreads) hist[i] = 0u;
    __syncthreads();
    // roles are whole waves: the first FILL/64 waves stream, the rest
    // select; every wave executes the same number of barriers (1 + 2 per
    // tile)
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    if (wave < FILL / 64) {
        const int cq = tid % CPR, j0 = tid / CPR;
        const int64_t sweep = (int64_t)RPI * R * d;   // elements between sweeps
        uint32_t keys[SW][KW];
        // pair-difference bits of the lane's files (sweep x: bits
        // NP*(x % PER) of word x / PER), ORed over every tile in registers
        // and merged into LDS once at the end
        constexpr int NPB = R * (R - 1) / 2;
        constexpr int PER = 32 / NPB;
        uint32_t pdacc[(SW + PER - 1) / PER];
#pragma unroll
        for (int a = 0; a < (SW + PER - 1) / PER; ++a) pdacc[a] = 0u;
        // the r replica chunks of one sweep, kept in registers (a value
        // type, so that no per-lane indexing can turn it into memory)
        struct Chunks {
            uint4 q[R];
        };
        // issue the row loads of sweep x of tile t.  Every load is in bounds:
        // a lane past the end of the rows (tail tile; d % 4 == 0) reads the
        // last chunk of its row instead (a repeated chunk changes neither
        // the agreement bits nor any written median), and a lane past the
        // last file loads nothing (proc_sweep ignores it).
        auto load_sweep = [&](int64_t t, int x) __attribute__((always_inline)) {
            const int64_t col = min(t * T + 4 * cq, d - 4);
            if constexpr (IND) {
                int i = j0 + x * RPI;
                asm volatile("" : "+v"(i));   // row addresses recomputed per tile
                Chunks c;
                if (i < f) {
#pragma unroll
                    for (int s = 0; s < R; ++s)
                        c.q[s] = load_stream(g + (int64_t)rt[i * R + s] * d + col);
                } else {
#pragma unroll
                    for (int s = 0; s < R; ++s) c.q[s] = make_uint4(0u, 0u, 0u, 0u);
                }
                return c;
            }
            const float *base = g + (int64_t)j0 * R * d + col;
            int lim = (int)(f - j0);   // sweeps x with x * RPI < lim hold a file
            // opaque copies of the tile's base address, the limit and the
            // sweep stride: every row address and check below is recomputed
            // from them, instead of the compiler carrying one pointer, one
            // lane mask and one offset per sweep across tiles
            int64_t stride = sweep;
            asm volatile("" : "+v"(base), "+v"(lim), "+s"(stride));
            Chunks c;
            if (x * RPI < lim) {
                const float *rows = base + x * stride;
#pragma unroll
                for (int s = 0; s < R; ++s) c.q[s] = load_stream(rows + s * d);
            } else {
#pragma unroll
                for (int s = 0; s < R; ++s) c.q[s] = make_uint4(0u, 0u, 0u, 0u);
            }
            return c;
        };
        // compare the replicas of sweep x and keep the guessed replica's keys
        // (HALF: its high key halves, packed two to a register, 0xFFFF for a
        // file past the last or dropped)
        auto proc_sweep = [&](int x, Chunks c) __attribute__((always_inline)) {
            const int i = j0 + x * RPI;   // f <= C(64,3) here
            if constexpr (HALF) {
                keys[x][0] = 0xFFFFFFFFu;
                keys[x][1] = 0xFFFFFFFFu;
            }
            if (i < f) {
                uint32_t diff = 0u;
                int p = 0;
#pragma unroll
                for (int s = 0; s < R; ++s)
#pragma unroll
                    for (int u = s + 1; u < R; ++u) {
                        const uint32_t y = (c.q[s].x ^ c.q[u].x) | (c.q[s].y ^ c.q[u].y) |
                                           (c.q[s].z ^ c.q[u].z) | (c.q[s].w ^ c.q[u].w);
                        diff |= (y != 0u ? 1u : 0u) << p;
                        ++p;
                    }
                pdacc[x / PER] |= diff << (NPB * (x % PER));
                // HALF: file i's nibble, word (j0 >> 3) + x*RPI/8 (RPI is a
                // multiple of 8), shift (j0 & 7) * 4 in every sweep
                const int w8 = (j0 >> 3) + x * (RPI / 8), sh = (j0 & 7) * 4;
                const int q = HALF ? (int)(((uint32_t)ps[w8] >> sh) & 15u) : ps[i];
                const int s_sel = q & 7;
                uint4 w = c.q[0];
#pragma unroll
                for (int s = 1; s < R; ++s)
                    if (s_sel == s) w = c.q[s];
                if constexpr (HALF) {
                    if (q & 8) {
                        keys[x][0] = pack_high(to_key(w.x), to_key(w.y));
                        keys[x][1] = pack_high(to_key(w.z), to_key(w.w));
                    }
                } else {
                    keys[x][0] = to_key(w.x);
                    keys[x][1] = to_key(w.y);
                    keys[x][2] = to_key(w.z);
                    keys[x][3] = to_key(w.w);
                }
            }
        };
        // sweep 0 of the next tile, loaded early: before the barrier and the
        // hand-over, so that loads stay in flight meanwhile.  The 36-sweep
        // tile, the row-table reads and r = 5 (five chunks a sweep) have no
        // registers to spare for it and load it with their tile
        constexpr bool kEarly0 = SW <= 32 && !IND && R == 3;
        Chunks c0;
        // tile t from its sweep 0 (already in c0, or loaded first); the
        // other sweeps go in bursts of B, all loads of a burst issued first
        auto stream_rest = [&](int64_t t) __attribute__((always_inline)) {
            if constexpr (!kEarly0) c0 = load_sweep(t, 0);
            proc_sweep(0, c0);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int xb = 1; xb < SW; xb += B) {
                Chunks c[B];
#pragma unroll
                for (int b = 0; b < B; ++b)
                    if (xb + b < SW) c[b] = load_sweep(t, xb + b);
#pragma unroll
                for (int b = 0; b < B; ++b)
                    if (xb + b < SW) proc_sweep(xb + b, c[b]);
                // keep each burst's loads together: no scheduling across
                // bursts, which would hold more loads in registers than fit
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        auto put_tile = [&]() __attribute__((always_inline)) {
            if constexpr (HALF) {
                // pair-rows j0 + k*RPI of the sweep pairs holding a file
                int64_t fo = f;   // opaque: compared per tile, not held per pair
                asm volatile("" : "+s"(fo));
#pragma unroll
                for (int k = 0; k < SW / 2; ++k)
                    if (k * 2 * RPI < fo)
                        put_pairs<T, G>(tile, j0 + k * RPI, cq, keys[2 * k], keys[2 * k + 1]);
            } else {
#pragma unroll
                for (int x = 0; x < SW; ++x) {
                    const int i = j0 + x * RPI;
                    if (i < f) {
                        const int q = ps[i];
                        if (q >= 0) put_keys<T, G>(tile, q >> 3, cq, keys[x]);
                    }
                }
            }
        };
        int64_t t = blockIdx.x;
        if (t < ntiles) {
            if constexpr (kEarly0) c0 = load_sweep(t, 0);
            stream_rest(t);
        }
        if (kEarly0 && t + gridDim.x < ntiles) c0 = load_sweep(t + gridDim.x, 0);
        if (t < ntiles) put_tile();
        __syncthreads();
        for (; t < ntiles; t += gridDim.x) {
            const int64_t tn = t + gridDim.x;
            if (tn < ntiles) stream_rest(tn);
            if (kEarly0 && tn + gridDim.x < ntiles) c0 = load_sweep(tn + gridDim.x, 0);
            __syncthreads();
            if (tn < ntiles) put_tile();
            __syncthreads();
        }
        // the lane's pair-difference bits into the workgroup's words
#pragma unroll
        for (int x = 0; x < SW; ++x) {
            const int i = j0 + x * RPI;
            const uint32_t b = (pdacc[x / PER] >> (NPB * (x % PER))) & ((1u << NPB) - 1u);
            if (i < f && b) {
                if constexpr (PDN)
                    atomicOr(&pd[i >> 3], b << ((i & 7) * 4));
                else
                    atomicOr(&pd[i], b);
            }
        }
    } else {
        __syncthreads();
        for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
            if (n > 0) {
                if constexpr (HALF) {
                    // tile row j is file j: its guessed replica's row of g
                    auto row = [&](int j) __attribute__((always_inline)) -> int64_t {
                        const uint32_t q = j < f ? nib(j) : 0u;
                        if (!(q & 8u)) return -1;
                        return IND ? (int64_t)rt[j * R + (q & 7)] : (int64_t)j * R + (q & 7);
                    };
                    select_half_tile<T, G, RPI>(tile, hist, (int)half_pair_rows(f, T, FILL), n,
                                                t * T, d, out, tid - FILL, g, row);
                } else {
                    select_tile<T, G>(tile, hist, n, t * T, d, out, tid - FILL);
                }
            }
            __syncthreads();
            __syncthreads();
        }
    }
    __syncthreads();
    for (int64_t i = tid; i < f; i += kWsThreads) {
        const uint32_t b = PDN ? ((pd[i >> 3] >> ((i & 7) * 4)) & 15u) : pd[i];
        if (b) atomicOr(&pair_diff[i], b);
    }
}

// ---------------------------------------------------------------------------
// median of the kept rows, warp-specialised like fused_ws_kernel: waves 0-7
// stream the kept rows of tile t+1 (one row per kept file, through the row
// list of the selection) into registers while waves 8-15 select on tile t.
// Used by the two-pass path and after a wrong guess of the single pass.

template <int SW>
constexpr int mws_batch() { return SW >= 16 ? 4 : (SW < 6 ? SW : 6); }

template <int T, int SW, bool HALF, int FILL>
__global__ void __launch_bounds__(kWsThreads)
median_ws_kernel(const float *__restrict__ g, int64_t d, const int32_t *__restrict__ rows,
                 const int32_t *__restrict__ n_sel, int64_t ntiles, float *__restrict__ out,
                 TileMask mask) {
    extern __shared__ uint32_t smem[];
    constexpr int G = (kWsThreads - FILL) / T;   // selection lanes per column
    constexpr int CPR = T / 4;           // float4 chunks per row segment
    constexpr int RPI = FILL / CPR;      // rows per sweep of the streaming role
    constexpr int B = mws_batch<SW>();   // sweeps per burst of loads
    // key registers per sweep: 4 keys, or (HALF) 4 high halves packed in 2
    constexpr int KW = HALF ? 2 : 4;
    static_assert(!HALF || (SW % 2 == 0 && RPI == half_rpi(T, FILL)), "half-key sweeps");
    const int n = *n_sel;
    if (n <= 0) return;                  // uniform: no workgroup reaches a barrier
    const int64_t hwords = HALF ? half_hist_words(T) : hist_words(T);
    uint32_t *hist = smem;
    uint32_t *tile = smem + hwords;
    int32_t *rl = reinterpret_cast<int32_t *>(tile + (HALF ? half_tile_words(n, T, FILL)
                                                           : (int64_t)n * T));   // [n] kept rows
    const int tid = threadIdx.x;
    for (int i = tid; i < n; i += kWsThreads) rl[i] = rows[i];
    for (int i = tid; i < hwords; i += kWsThreads) hist[i] = 0u;
    __syncthreads();
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    if (wave < FILL / 64) {
        const int cq = tid % CPR, j0 = tid / CPR;
        uint32_t keys[SW][KW];
        // one 16-byte chunk of kept row j (a lane past the last kept row
        // re-reads row 0, which is never put; past the end of the rows it
        // re-reads the row's last chunk, whose median is never written)
        auto load_row = [&](int64_t t, int x) __attribute__((always_inline)) {
            const int64_t col = min(t * T + 4 * cq, d - 4);
            int j = j0 + x * RPI < n ? j0 + x * RPI : 0;
            asm volatile("" : "+v"(j));   // row address recomputed per tile
            return load_stream(g + (int64_t)rl[j] * d + col);
        };
        auto to_keys = [&](int x, uint4 q) __attribute__((always_inline)) {
            if constexpr (HALF) {
                // high key halves; 0xFFFF past the last kept row
                const bool keep = j0 + x * RPI < n;
                keys[x][0] = keep ? pack_high(to_key(q.x), to_key(q.y)) : 0xFFFFFFFFu;
                keys[x][1] = keep ? pack_high(to_key(q.z), to_key(q.w)) : 0xFFFFFFFFu;
            } else {
                keys[x][0] = to_key(q.x);
                keys[x][1] = to_key(q.y);
                keys[x][2] = to_key(q.z);
                keys[x][3] = to_key(q.w);
            }
        };
        uint4 c0;   // sweep 0 of the next tile, loaded early
        auto stream_rest = [&](int64_t t) __attribute__((always_inline)) {
            to_keys(0, c0);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int xb = 1; xb < SW; xb += B) {
                uint4 c[B];
#pragma unroll
                for (int b = 0; b < B; ++b)
                    if (xb + b < SW) c[b] = load_row(t, xb + b);
#pragma unroll
                for (int b = 0; b < B; ++b)
                    if (xb + b < SW) to_keys(xb + b, c[b]);
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        auto put_tile = [&]() __attribute__((always_inline)) {
            if constexpr (HALF) {
                int no = n;   // opaque: compared per tile, not held per pair
                asm volatile("" : "+s"(no));
#pragma unroll
                for (int k = 0; k < SW / 2; ++k) {
                    int p = j0 + k * RPI;
                    // opaque: the LDS addresses are recomputed per tile
                    // instead of being held in registers for every pair
                    asm volatile("" : "+v"(p));
                    if (k * 2 * RPI < no) put_pairs<T, G>(tile, p, cq, keys[2 * k], keys[2 * k + 1]);
                }
            } else {
#pragma unroll
                for (int x = 0; x < SW; ++x) {
                    int j = j0 + x * RPI;
                    asm volatile("" : "+v"(j));   // as above
                    if (j < n) put_keys<T, G>(tile, j, cq, keys[x]);
                }
            }
        };
        // the workgroup's tiles: t, then tn (whose sweep 0 is loaded early)
        const int64_t G0 = gridDim.x;
        int64_t t = mask.next(blockIdx.x, G0, ntiles);
        int64_t tn = mask.next(t + G0, G0, ntiles);
        if (t < ntiles) {
            c0 = load_row(t, 0);
            stream_rest(t);
        }
        if (tn < ntiles) c0 = load_row(tn, 0);
        if (t < ntiles) put_tile();
        __syncthreads();
        while (t < ntiles) {
            const int64_t tnn = mask.next(tn + G0, G0, ntiles);
            if (tn < ntiles) stream_rest(tn);
            if (tnn < ntiles) c0 = load_row(tnn, 0);
            __syncthreads();
            if (tn < ntiles) put_tile();
            __syncthreads();
            t = tn;
            tn = tnn;
        }
    } else {
        __syncthreads();
        for (int64_t t = mask.next(blockIdx.x, gridDim.x, ntiles); t < ntiles;
             t = mask.next(t + gridDim.x, gridDim.x, ntiles)) {
            if constexpr (HALF) {
                auto row = [&](int j) __attribute__((always_inline)) -> int64_t {
                    return j < n ? (int64_t)rl[j] : -1;
                };
                // FILL = 512: RPI = 4G, so every lane holds the same number of
                // words, at most 2 SW
                constexpr int REG = (FILL == kWsFill && RPI == 4 * G) ? 2 * SW : 0;
                select_half_tile<T, G, RPI, REG>(tile, hist, (int)half_pair_rows(n, T, FILL), n,
                                                 t * T, d, out, tid - FILL, g, row);
            } else {
                select_tile<T, G>(tile, hist, n, t * T, d, out, tid - FILL);
            }
            __syncthreads();
            __syncthreads();
        }
    }
}

// ---------------------------------------------------------------------------
// fused agreement + mean (one read of all r replicas): each thread owns four
// coordinates and walks every file in ascending order, comparing the r
// replicas and adding the guessed replica to an fp64 sum -- the file order
// of the sum is the mean kernel's and the oracle's.  A wave reads 1 KiB of
// one row per load.  The pair-difference bits of a wave are combined with
// ballots into per-workgroup LDS words, merged into pair_diff at the end.

// files per burst of loads (R rows each): 3 keeps the kernel at 62 VGPRs,
// 8 waves per SIMD (4 files: 74 VGPRs, 6 waves, 3.7 % slower at K=21, d=5M)
constexpr int kMeanFiles = 3;

template <int R, bool VEC>
__global__ void __launch_bounds__(kBlock)
fused_mean_kernel(const float *__restrict__ g, const int32_t *__restrict__ row_of, int64_t f,
                  int64_t d, const int32_t *__restrict__ sel, const int32_t *__restrict__ pos,
                  const int32_t *__restrict__ n_sel, uint32_t *__restrict__ pair_diff,
                  float *__restrict__ out) {
    extern __shared__ uint32_t pdw[];   // [f]
    const int tid = threadIdx.x;
    for (int64_t i = tid; i < f; i += kBlock) pdw[i] = 0u;
    __syncthreads();
    const int n = *n_sel;
    const int64_t nq = (d + 3) / 4;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    // every lane of a workgroup runs the same iterations (the ballots need
    // whole waves); lanes past the end of the rows read and write nothing
    for (int64_t q0 = (int64_t)blockIdx.x * kBlock; q0 < nq; q0 += stride) {
        const int64_t k = (q0 + tid) * 4;
        const int64_t kend = q0 + tid < nq ? d : 0;
        double acc[4] = {0.0, 0.0, 0.0, 0.0};
        for (int64_t ib = 0; ib < f; ib += kMeanFiles) {
            uint32_t v[kMeanFiles][R][4];
#pragma unroll
            for (int b = 0; b < kMeanFiles; ++b) {
                const int64_t i = ib + b;
                if (i < f) {
#pragma unroll
                    for (int s = 0; s < R; ++s)
                        load4<VEC>(g + replica_row(row_of, i, R, s) * d, k, kend, v[b][s]);
                }
            }
#pragma unroll
            for (int b = 0; b < kMeanFiles; ++b) {
                const int64_t i = ib + b;
                if (i >= f) break;
                uint32_t diff = 0u;
                int p = 0;
#pragma unroll
                for (int s = 0; s < R; ++s)
#pragma unroll
                    for (int u = s + 1; u < R; ++u) {
                        const uint32_t x = (v[b][s][0] ^ v[b][u][0]) | (v[b][s][1] ^ v[b][u][1]) |
                                           (v[b][s][2] ^ v[b][u][2]) | (v[b][s][3] ^ v[b][u][3]);
                        diff |= (x != 0u ? 1u : 0u) << p;
                        ++p;
                    }
                uint32_t wdiff = 0u;
#pragma unroll
                for (int q = 0; q < R * (R - 1) / 2; ++q)
                    if (__ballot((diff >> q) & 1u)) wdiff |= 1u << q;
                if ((tid & 63) == 0 && wdiff) atomicOr(&pdw[i], wdiff);
                if (pos[i] >= 0) {
                    const int s_sel = sel[i];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        uint32_t w = v[b][0][e];
#pragma unroll
                        for (int s = 1; s < R; ++s) w = (s_sel == s) ? v[b][s][e] : w;
                        acc[e] += (double)__uint_as_float(w);
                    }
                }
            }
        }
        if (kend != 0 && n > 0) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (k + e < d) out[k + e] = (float)(acc[e] / (double)n);
        }
    }
    __syncthreads();
    for (int64_t i = tid; i < f; i += kBlock)
        if (pdw[i]) atomicOr(&pair_diff[i], pdw[i]);
}

// ---------------------------------------------------------------------------
// mean of the kept rows (fp64, file order)

constexpr int kMeanRows = 8;
constexpr int64_t kMeanTileCols = kBlock * 4;   // coordinates per mean tile: four per thread

template <bool VEC>
__global__ void __launch_bounds__(kBlock)
mean_kernel(const float *__restrict__ g, int64_t d,
            const int32_t *__restrict__ rows, const int32_t *__restrict__ n_sel,
            float *__restrict__ out, TileMask mask) {
    const int n = *n_sel;
    if (n <= 0) return;
    // tiles of kMeanTileCols coordinates, four per thread
    const int64_t ntiles = (d + kMeanTileCols - 1) / kMeanTileCols;
    for (int64_t t = mask.next(blockIdx.x, gridDim.x, ntiles); t < ntiles;
         t = mask.next(t + gridDim.x, gridDim.x, ntiles)) {
        const int64_t k = t * kMeanTileCols + 4 * (int64_t)threadIdx.x;
        if (k >= d) continue;
        double acc[4] = {0.0, 0.0, 0.0, 0.0};
        // bursts of kMeanRows loads, then the additions in row order
        for (int j0 = 0; j0 < n; j0 += kMeanRows) {
            uint32_t v[kMeanRows][4];
#pragma unroll
            for (int b = 0; b < kMeanRows; ++b)
                if (j0 + b < n) load4<VEC>(g + (int64_t)rows[j0 + b] * d, k, d, v[b]);
#pragma unroll
            for (int b = 0; b < kMeanRows; ++b)
                if (j0 + b < n) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[e] += (double)__uint_as_float(v[b][e]);
                }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (k + e < d) out[k + e] = (float)(acc[e] / (double)n);
    }
}

// ---------------------------------------------------------------------------
// median of any number of kept rows: an MSB-first radix select over the
// 32-bit keys in four rounds of 8 bits, whose histograms live in LDS while
// the keys are read from HBM again in every round.  It takes over when not
// even a narrow tile of every kept row's keys fits in LDS (beyond about
// 10,000 kept files); it reads the kept rows four times, trading bandwidth
// for capacity.  Lane c of every wave owns column c of a 64-column tile and
// wave w reads rows w, w + 4, ... (256-byte row segments per wave load).

constexpr int kRadixCols = 64;
constexpr int kRadixThreads = 256;
constexpr int kRadixWaves = kRadixThreads / kRadixCols;
constexpr int kRadixBuckets = 256;
constexpr int kRadixStride = kRadixBuckets + 1;   // bucket b of column c at c*257 + b:
                                                  // bank (c + b) % 64
constexpr int kRadixBatch = 8;                    // row loads in flight per lane
constexpr int kRadixQuarter = kRadixBuckets / kRadixWaves;

__global__ void __launch_bounds__(kRadixThreads)
median_radix_kernel(const float *__restrict__ g, int64_t d, const int32_t *__restrict__ rows,
                    const int32_t *__restrict__ n_sel, int64_t ntiles, float *__restrict__ out,
                    TileMask mask) {
    __shared__ uint32_t hist[kRadixCols * kRadixStride];
    __shared__ uint32_t part[kRadixWaves][kRadixCols];   // bucket counts per quarter
    __shared__ uint32_t prefix[kRadixCols], rank[kRadixCols];
    const int n = *n_sel;
    if (n <= 0) return;   // uniform: no workgroup reaches a barrier
    const int tid = threadIdx.x, c = tid % kRadixCols, w = tid / kRadixCols;
    for (int64_t t = mask.next(blockIdx.x, gridDim.x, ntiles); t < ntiles;
         t = mask.next(t + gridDim.x, gridDim.x, ntiles)) {
        const int64_t k = t * kRadixCols + c;
        const bool valid = k < d;
        if (tid < kRadixCols) {
            prefix[tid] = 0u;
            rank[tid] = (uint32_t)(n - 1) / 2;
        }
        // round x settles key bits [24 - 8x, 32 - 8x) among the keys whose
        // higher bits equal the prefix settled so far
        for (int round = 0; round < 4; ++round) {
            for (int i = tid; i < kRadixCols * kRadixStride; i += kRadixThreads) hist[i] = 0u;
            __syncthreads();
            const int sh = 24 - 8 * round;
            const uint32_t pre = prefix[c];
            uint32_t *hc = hist + c * kRadixStride;
            auto count = [&](uint32_t v) __attribute__((always_inline)) {
                const uint32_t key = to_key(v);
                if (round == 0 || (key >> (sh + 8)) == pre) atomicAdd(&hc[(key >> sh) & 255u], 1u);
            };
            if (valid) {
                const float *col = g + k;
                int j = w;
                for (; j + (kRadixBatch - 1) * kRadixWaves < n; j += kRadixBatch * kRadixWaves) {
                    uint32_t v[kRadixBatch];
#pragma unroll
                    for (int u = 0; u < kRadixBatch; ++u)
                        v[u] = __float_as_uint(col[(int64_t)rows[j + u * kRadixWaves] * d]);
#pragma unroll
                    for (int u = 0; u < kRadixBatch; ++u) count(v[u]);
                }
                for (; j < n; j += kRadixWaves) count(__float_as_uint(col[(int64_t)rows[j] * d]));
            }
            __syncthreads();
            // the bucket holding the sought rank: wave w sums its quarter of
            // the column's buckets, then one lane per column walks the
            // quarters and the buckets of the quarter that holds it
            uint32_t sum = 0u;
#pragma unroll 8
            for (int b = 0; b < kRadixQuarter; ++b) sum += hc[w * kRadixQuarter + b];
            part[w][c] = sum;
            __syncthreads();
            if (tid < kRadixCols) {
                uint32_t m = rank[c], run = 0u;
                int qt = 0;
                for (; qt < kRadixWaves - 1; ++qt) {
                    if (run + part[qt][c] > m) break;
                    run += part[qt][c];
                }
                int b = qt * kRadixQuarter;
                for (; b < (qt + 1) * kRadixQuarter - 1; ++b) {
                    if (run + hc[b] > m) break;
                    run += hc[b];
                }
                rank[c] = m - run;
                prefix[c] = (prefix[c] << 8) | (uint32_t)b;
            }
            __syncthreads();
        }
        if (w == 0 && valid) out[k] = __uint_as_float(from_key(prefix[c]));
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// tie probe: how many values share the median's high 16 key bits.  The
// half-key tiles read back the low halves of every row tied with the
// median's high half, so heavily tied data (quantised gradients, values on
// a grid) is better served by full-key tiles.  For kTieCols coordinates
// spread over the probed prefix, one workgroup takes each file's value at
// that coordinate -- the value of its largest class of equal replicas, the
// file's vote on that coordinate alone, which is what the selection keeps
// in most files -- finds the high half H of their lower median (two
// 8-bit histogram rounds in LDS) and stores how many files have high half
// H.  It needs no selection, so it runs with the probe.

constexpr int kTieThreads = 256;

// Probed coordinate c (c < min(kTieCols, probe.coords())): the prefix
// split in kTieCols equal steps, or offsets spread over the blocks.
__device__ __forceinline__ int64_t tie_coord(const ProbeSet &probe, int c) {
    if (probe.seed == 0) {
        const int64_t kstep = probe.kend >= kTieCols ? probe.kend / kTieCols : 1;
        return (int64_t)c * kstep;
    }
    const int64_t per = (kTieCols + probe.nb - 1) / probe.nb;   // coordinates per block
    const int64_t step = kProbeBlockCols / per;
    return probe.block_start(c % probe.nb) + (c / probe.nb) * step;
}
constexpr int kTieMaxFiles = 4096;   // files looked at per coordinate (the first ones)
static_assert(kTieThreads == 256, "one histogram bucket per thread");

template <int R>
__global__ void __launch_bounds__(kTieThreads)
tie_probe_kernel(const float *__restrict__ g, const int32_t *__restrict__ row_of, int64_t f,
                 int64_t d, ProbeSet probe, uint32_t *__restrict__ out) {
    __shared__ uint16_t h[kTieMaxFiles];
    __shared__ uint32_t hist[256];
    __shared__ uint32_t wsum[kTieThreads / 64];
    __shared__ uint32_t pick[2];   // bucket, rank within it
    const int tid = threadIdx.x;
    const int64_t k = tie_coord(probe, blockIdx.x);
    const int n = (int)(f < kTieMaxFiles ? f : kTieMaxFiles);
    for (int i = tid; i < n; i += kTieThreads) {
        uint32_t v[R];
#pragma unroll
        for (int s = 0; s < R; ++s) v[s] = __float_as_uint(g[replica_row(row_of, i, R, s) * d + k]);
        // the value of the largest class of equal replicas, the lower slot
        // on a tie (Eq. (3) on this one coordinate)
        uint32_t val = v[0];
        int best = 0;
#pragma unroll
        for (int s = 0; s < R; ++s) {
            int c = 0;
#pragma unroll
            for (int t = 0; t < R; ++t) c += v[s] == v[t] ? 1 : 0;
            if (c > best) {
                best = c;
                val = v[s];
            }
        }
        h[i] = (uint16_t)(to_key(val) >> 16);
    }
    // round 0 counts the high bytes; round 1 the low bytes of the keys whose
    // high byte is the median's; the median's bucket count then is the number
    // of files tied with it
    uint32_t rank = (uint32_t)(n - 1) / 2, hi = 0u;
    for (int round = 0; round < 2; ++round) {
        hist[tid] = 0u;   // kTieThreads == 256 buckets
        __syncthreads();
        for (int i = tid; i < n; i += kTieThreads) {
            const uint32_t x = h[i];
            if (round == 0)
                atomicAdd(&hist[x >> 8], 1u);
            else if ((x >> 8) == hi)
                atomicAdd(&hist[x & 255u], 1u);
        }
        __syncthreads();
        // the bucket holding the rank: a prefix sum over the 256 buckets,
        // one per thread (wave scans, then the waves' totals)
        const uint32_t c = hist[tid];
        uint32_t incl = c;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t y = (uint32_t)__shfl_up((int)incl, o, 64);
            incl += (tid & 63) >= o ? y : 0u;
        }
        if ((tid & 63) == 63) wsum[tid >> 6] = incl;
        __syncthreads();
        for (int w = 0; w < (tid >> 6); ++w) incl += wsum[w];
        if (incl - c <= rank && rank < incl) {   // exactly one bucket
            pick[0] = (uint32_t)tid;
            pick[1] = rank - (incl - c);
        }
        __syncthreads();
        const uint32_t b = pick[0];
        if (round == 0) {
            hi = b;
            rank = pick[1];
        } else if (tid == 0) {
            out[blockIdx.x] = hist[b];
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// repair after a wrong guess (the guess kept the same files as the final
// selection and reduced them with the same median): the median computed with
// the guess already is the final one wherever each moved file's two
// replicas are equal, so only the tiles holding a coordinate where they
// differ are recomputed.

__global__ void save_sel_kernel(const int32_t *__restrict__ sel, int64_t f,
                                int8_t *__restrict__ sel_prev, int32_t *__restrict__ repair) {
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i < f) sel_prev[i] = (int8_t)sel[i];
    if (i < 4) repair[i] = 0;
}

constexpr int kDirtyMaxMoved = 2048;   // moved files a workgroup lists (LDS)
constexpr int kDirtyBatch = 4;         // moved files per burst of loads

// Every workgroup lists the moved files (replica rows of the guess and of the
// final selection, where the two differ somewhere in the vector), then sets
// the bits of its words: bit b of word w for the columns [b' << cshift,
// (b' + 1) << cshift), b' = 32w + b, when a listed pair differs there --
// every bit when the kept files differ or more files moved than the list
// holds.
template <int R, bool VEC>
__global__ void __launch_bounds__(kBlock)
dirty_tiles_kernel(const float *__restrict__ g, const int32_t *__restrict__ row_of, int64_t f,
                   int64_t d, int cshift, int64_t nbits,
                   const int8_t *__restrict__ sel_prev, const int32_t *__restrict__ sel,
                   const uint32_t *__restrict__ pair_diff, uint32_t *__restrict__ dirty,
                   int32_t *__restrict__ repair) {
    __shared__ int32_t moved[2 * kDirtyMaxMoved];
    __shared__ int32_t n_moved, every;
    __shared__ uint32_t word;
    const int tid = threadIdx.x;
    if (tid == 0) {
        n_moved = 0;
        every = 0;
        word = 0u;
    }
    __syncthreads();
    for (int64_t i = tid; i < f; i += kBlock) {
        const int a = sel_prev[i], b = sel[i];
        if ((a < 0) != (b < 0)) {
            atomicOr(&every, 1);
            continue;
        }
        if (a < 0 || a == b) continue;
        // bit of the slot pair (lo, hi) in the pair-difference word
        const int lo = a < b ? a : b, hi = a < b ? b : a;
        const int p = lo * (2 * R - lo - 1) / 2 + (hi - lo - 1);
        if (((pair_diff[i] >> p) & 1u) == 0u) continue;   // bitwise equal replicas
        const int x = atomicAdd(&n_moved, 1);
        if (x < kDirtyMaxMoved) {
            moved[2 * x] = (int32_t)replica_row(row_of, i, R, a);
            moved[2 * x + 1] = (int32_t)replica_row(row_of, i, R, b);
        } else {
            atomicOr(&every, 1);
        }
    }
    __syncthreads();
    const bool all = every != 0;
    const int n = n_moved < kDirtyMaxMoved ? n_moved : kDirtyMaxMoved;
    const int64_t nwords = (nbits + 31) / 32;
    for (int64_t w = blockIdx.x; w < nwords; w += gridDim.x) {
        const int64_t nb = nbits - 32 * w < 32 ? nbits - 32 * w : 32;
        const uint32_t full = nb == 32 ? 0xFFFFFFFFu : (1u << nb) - 1u;
        if (all) {
            if (tid == 0) {
                dirty[w] = full;
                atomicAdd(&repair[0], __popc(full));
            }
            continue;
        }
        const int64_t c0 = (w * 32) << cshift;
        const int64_t c1 = c0 + (nb << cshift) < d ? c0 + (nb << cshift) : d;
        uint32_t mine = 0u;
        for (int64_t k = c0 + 4 * tid; k < c1; k += 4 * kBlock) {
            const uint32_t bit = 1u << ((k - c0) >> cshift);
            if (mine & bit) continue;
            for (int x0 = 0; x0 < n; x0 += kDirtyBatch) {
                uint32_t va[kDirtyBatch][4], vb[kDirtyBatch][4];
#pragma unroll
                for (int u = 0; u < kDirtyBatch; ++u) {
                    if (x0 + u < n) {
                        load4<VEC>(g + (int64_t)moved[2 * (x0 + u)] * d, k, d, va[u]);
                        load4<VEC>(g + (int64_t)moved[2 * (x0 + u) + 1] * d, k, d, vb[u]);
                    }
                }
                uint32_t diff = 0u;
#pragma unroll
                for (int u = 0; u < kDirtyBatch; ++u)
                    if (x0 + u < n)
                        diff |= (va[u][0] ^ vb[u][0]) | (va[u][1] ^ vb[u][1]) |
                                (va[u][2] ^ vb[u][2]) | (va[u][3] ^ vb[u][3]);
                if (diff != 0u) {
                    mine |= bit;
                    break;
                }
            }
        }
        if (mine) atomicOr(&word, mine);
        __syncthreads();
        if (tid == 0) {
            dirty[w] = word;
            atomicAdd(&repair[0], __popc(word));
            word = 0u;
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// read-bandwidth probe

constexpr int kProbeBlocks = 2048;

__global__ void __launch_bounds__(kBlock)
read_probe_kernel(const uint4 *__restrict__ p, int64_t n16, uint32_t *sink) {
    uint32_t acc = 0u;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n16;
         i += (int64_t)gridDim.x * blockDim.x) {
        const uint4 v = load_stream(reinterpret_cast<const float *>(p + i));
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    sink[blockIdx.x * (int64_t)blockDim.x + threadIdx.x] = acc;
}

// Compute units of each device, looked up once per device (relaxed atomics:
// concurrent first calls store the same value).
constexpr int kMaxDevices = 64;
std::atomic<int> g_num_cus[kMaxDevices];

int num_cus() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
    int cus = g_num_cus[dev].load(std::memory_order_relaxed);
    if (cus == 0) {
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
        g_num_cus[dev].store(cus, std::memory_order_relaxed);
    }
    return cus;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int64_t grid_for(int64_t work, int64_t cap) { return work < cap ? (work < 1 ? 1 : work) : cap; }

// widest tile T whose [rows x T] key block (plus extra bytes) fits in LDS
int pick_tile(int64_t rows, int64_t extra_bytes) {
    for (int T : {64, 32, 16, 8, 4})
        if (rows * 4 * (int64_t)T + hist_words(T) * 4 + extra_bytes <= kLdsBytes) return T;
    return 0;
}

// workgroups per CU that the LDS allows, for the grid of a tile kernel
int64_t tile_grid(int64_t ntiles, size_t lds) {
    int per_cu = (int)(kLdsBytes / (int64_t)(lds ? lds : 1));
    per_cu = per_cu < 1 ? 1 : (per_cu > 2 ? 2 : per_cu);
    return grid_for(ntiles, (int64_t)num_cus() * per_cu);
}

}  // namespace

// ---------------------------------------------------------------------------
// launchers

// sel, pos, rows: int32 [f] each; 256 bytes of counters; 1,024 bytes of
// staged rows; the row table int32 [f*r].  Each part starts 256-aligned.
constexpr size_t kWsCounters = 256, kWsStage = 1024;

size_t workspace_bytes(int64_t f, int r) {
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    return up((size_t)f * 4) * 3 + kWsCounters + kWsStage + up((size_t)f * r * 4) + up((size_t)f) +
           (size_t)kDirtyWords * 4 + kWsCounters;
}

Workspace carve_workspace(void *base, int64_t f, int r) {
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    char *p = static_cast<char *>(base);
    Workspace w;
    w.sel = reinterpret_cast<int32_t *>(p);
    p += up((size_t)f * 4);
    w.pos = reinterpret_cast<int32_t *>(p);
    p += up((size_t)f * 4);
    w.rows = reinterpret_cast<int32_t *>(p);
    p += up((size_t)f * 4);
    w.n_sel = reinterpret_cast<int32_t *>(p);
    p += kWsCounters;
    w.stage = reinterpret_cast<uint64_t *>(p);
    p += kWsStage;
    w.row_of = reinterpret_cast<int32_t *>(p);
    p += up((size_t)f * r * 4);
    w.sel_prev = reinterpret_cast<int8_t *>(p);
    p += up((size_t)f);
    w.dirty = reinterpret_cast<uint32_t *>(p);
    p += (size_t)kDirtyWords * 4;
    w.repair = reinterpret_cast<int32_t *>(p);
    return w;
}

hipError_t launch_fill_u32(uint32_t *p, int64_t n, uint32_t v, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    fill_u32_kernel<<<(unsigned)grid_for((n + 255) / 256, 1024), 256, 0, s>>>(p, n, v);
    return hipGetLastError();
}
hipError_t launch_fill_u64(uint64_t *p, int64_t n, uint64_t v, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    fill_u64_kernel<<<(unsigned)grid_for((n + 255) / 256, 1024), 256, 0, s>>>(p, n, v);
    return hipGetLastError();
}

hipError_t launch_agree(const float *g, const int32_t *row_of, int64_t f, int r, int64_t d,
                        int64_t kend, uint32_t *pair_diff, hipStream_t s) {
    if (kend <= 0 || f <= 0) return hipSuccess;
    const int64_t nchunks = (kend + kAgreeChunk - 1) / kAgreeChunk;
    const unsigned grid = (unsigned)grid_for(f * nchunks, (int64_t)num_cus() * 16);
    const bool vec = (d % 4 == 0) && aligned16(g);
#define ASPIS_AGREE(RR)                                                              \
    if (vec)                                                                         \
        agree_kernel<RR, true><<<grid, kBlock, 0, s>>>(g, row_of, f, d, kend, nchunks, pair_diff); \
    else                                                                             \
        agree_kernel<RR, false><<<grid, kBlock, 0, s>>>(g, row_of, f, d, kend, nchunks, pair_diff);
    switch (r) {
    case 3: ASPIS_AGREE(3) break;
    case 5: ASPIS_AGREE(5) break;
    case 7: ASPIS_AGREE(7) break;
    default: return hipErrorInvalidValue;
    }
#undef ASPIS_AGREE
    return hipGetLastError();
}

hipError_t launch_vote(const uint32_t *pair_diff, const int32_t *subsets, int64_t f,
                       int r, int8_t *vote, uint8_t *has_majority, uint64_t *disagree,
                       hipStream_t s) {
    vote_kernel<<<(unsigned)grid_for((f + 255) / 256, 64), 256, 0, s>>>(
        pair_diff, subsets, f, r, vote, has_majority, disagree);
    return hipGetLastError();
}

hipError_t launch_vote_rows(const uint32_t *pair_diff, const int32_t *subsets, int64_t f,
                            int r, int K, int8_t *vote, uint8_t *has_majority,
                            uint64_t *disagree, uint64_t *stage, hipStream_t s) {
    if (f > kVoteRowsMaxFiles || K < 1 || K > 64) return hipErrorInvalidValue;
    vote_rows_kernel<<<1, 1024, 0, s>>>(pair_diff, subsets, f, r, K, vote, has_majority,
                                        disagree, stage);
    return hipGetLastError();
}

// Every probed coordinate inside [0, d), the blocks within their count.
bool probe_valid(const ProbeSet &p, int64_t d) {
    if (p.nb <= 0 || p.nb > kProbeMaxBlocks) return false;
    if (p.seed == 0) return p.kend > 0 && p.kend <= d && p.kend <= p.nb * kProbeBlockCols;
    for (int64_t j = 0; j < p.nb; ++j)
        if (p.start[j] < 0 || p.start[j] + kProbeBlockCols > d || p.start[j] % 4 != 0) return false;
    return true;
}

hipError_t launch_agree_file(const float *g, const int32_t *row_of, int64_t f, int r, int64_t d,
                             const ProbeSet &probe, uint32_t *pair_diff, hipStream_t s) {
    if (f <= 0) return hipSuccess;
    if (!probe_valid(probe, d)) return hipErrorInvalidValue;
    const unsigned grid = (unsigned)grid_for(f, (int64_t)num_cus() * 8);
    const bool vec = (d % 4 == 0) && aligned16(g);
#define ASPIS_AGREE_FILE(RR)                                                                    \
    if (vec)                                                                                    \
        agree_file_kernel<RR, true><<<grid, kBlock, 0, s>>>(g, row_of, f, d, probe, pair_diff); \
    else                                                                                        \
        agree_file_kernel<RR, false><<<grid, kBlock, 0, s>>>(g, row_of, f, d, probe, pair_diff);
    switch (r) {
    case 3: ASPIS_AGREE_FILE(3) break;
    case 5: ASPIS_AGREE_FILE(5) break;
    case 7: ASPIS_AGREE_FILE(7) break;
    default: return hipErrorInvalidValue;
    }
#undef ASPIS_AGREE_FILE
    return hipGetLastError();
}

hipError_t launch_select(const int32_t *subsets, const int8_t *vote, int64_t f, int r,
                         int success, uint64_t honest, const int32_t *row_of, const Workspace &ws,
                         int32_t *sel_out, uint32_t *zero, int64_t n_zero, hipStream_t s) {
    select_kernel<<<1, 1024, 0, s>>>(subsets, vote, f, r, success, honest, row_of, ws.sel,
                                     ws.pos, ws.rows, ws.n_sel, sel_out, zero, n_zero);
    return hipGetLastError();
}

namespace {

// Warp-specialised plans.  Full keys: the widest tile (8..64 columns) whose
// key block fits in LDS and whose rows fit the streaming role's registers
// (at most 16 sweeps of 4 key registers).  Half keys, for many rows: a wider
// tile (16..128 columns) with up to 32 sweeps of 2 key registers; taken
// only when it is wider than the full-key tile, since below kHalfMinRows
// rows a tile is streamed too quickly to hide the reads of the low halves.
// Half keys try the even split of streaming and selecting waves first, then
// 12 streaming waves and 4 selecting ones (kWsFillWide): 1.5x the rows per
// sweep, so that thousands of rows fit the registers of a 32- or 64-column
// tile.
struct WsPlan {
    int r = 3;
    int T = 0;
    int sweeps = 0;
    bool half = false;
    int fill = kWsFill;
    bool rtg = false;   // row table read from global memory (not in LDS)
};

constexpr int kWsFillWide = 768;
constexpr int64_t kHalfMinRows = 128;
constexpr int64_t kHalfMaxRows = 60000;   // row numbers (with padding) fit 16 bits

// Most sweeps a half-key plan may take: 32, and 36 for the 32-column tile
// with the even split.  There the streaming role spills 30 registers, and
// still the 8 selecting waves (16 lanes a column) beat the wide split's 4:
// 2,300 files, d = 2M, 9.14-9.58 against 11.36-11.40 ms (one process and
// allocation).  Not with a row table: reading it as well, the streaming
// role spills 88 registers (15.9 against 12.1 ms with the wide split).
constexpr int max_half_sweeps(int T, int fill) { return T == 32 && fill == kWsFill ? 36 : 32; }

// Sweep counts built for each plan (sweeps past the last row load nothing,
// so the count is rounded up only a little).  Half keys: an even count; 8
// only for 128 columns, where fewer than 128 rows never take a narrower
// half-key tile, and steps of 2 from 24 to 32 there; 36 for 32 columns
// (even split); 24 or 32 for the wide split.
int round_sweeps(int64_t sw, bool half, int T, int fill, int r = 3) {
    if (half && r != 3) {
        // r = 5: the sweep counts built for five replicas a file
        if (T == 128) return sw <= 16 ? 16 : sw <= 30 ? 30 : 32;
        return sw <= 16 ? 16 : sw <= 24 ? 24 : 32;
    }
    if (half) {
        if (fill == kWsFillWide) return sw <= 24 ? 24 : 32;
        if (T == 128 && sw > 24) return (int)((sw + 1) / 2 * 2);
        if (sw > 32) return 36;   // the 32-column even split only
        return sw <= 8 && T == 128 ? 8 : sw <= 16 ? 16 : sw <= 24 ? 24 : 32;
    }
    return sw <= 2 ? 2 : sw <= 4 ? 4 : sw <= 8 ? 8 : sw <= 12 ? 12 : 16;
}

// The half-key plan wider than `narrower` columns, or none; lds(T, fill)
// gives the kernel's LDS bytes.  The wide split is built for 64 and 32
// columns only.  With a row table (ind) the 128-column tile spills 15
// registers of the streaming role next to 30 sweeps of keys, and still
// beats the 64-column full-key tile (10.9 against 11.6 ms at 455 files,
// d = 11.2M, one process and allocation).  A row table staged in LDS rules
// out the wide split; one read from global memory (rtg) takes the wide
// split only: with the even split the streaming role would hold the
// table's addresses next to its keys (the kernels built for a global
// table are wide-split ones).
template <typename LdsFn>
WsPlan half_plan(int64_t f, int narrower, bool ind, bool rtg, LdsFn &&lds, int r = 3) {
    WsPlan p;
    if (f < kHalfMinRows || f > kHalfMaxRows) return p;
    for (int T : {128, 64, 32, 16}) {
        if (T <= narrower) break;
        for (int fill : {kWsFill, kWsFillWide}) {
            if (fill == kWsFillWide && ((ind && !rtg) || T == 128 || T == 16 || r != 3)) continue;
            if (rtg && fill != kWsFillWide) continue;
            const int64_t rpi = half_rpi(T, fill);
            const int64_t sw = (f + rpi - 1) / rpi;
            const int64_t max_sw = (ind || r != 3) ? 32 : max_half_sweeps(T, fill);
            if (sw > max_sw || lds(T, fill) > kLdsBytes) continue;
            p.T = T;
            p.sweeps = round_sweeps(sw, true, T, fill, r);
            p.half = true;
            p.fill = fill;
            p.rtg = rtg;
            return p;
        }
    }
    return p;
}

// LDS of the warp-specialised median: histograms, key tile, row list.
int64_t mws_lds_bytes(int64_t f, int T, bool half, int fill) {
    return half ? (half_hist_words(T) + half_tile_words(f, T, fill)) * 4 + f * 4
                : (hist_words(T) + f * (int64_t)T) * 4 + f * 4;
}

WsPlan mws_plan(int64_t f, bool vec, bool full_keys = false) {
    WsPlan p;
    if (!vec) return p;
    for (int T : {64, 32, 16, 8}) {
        if (mws_lds_bytes(f, T, false, kWsFill) > kLdsBytes) continue;
        const int64_t rpi = kWsFill / (T / 4);
        const int64_t sw = (f + rpi - 1) / rpi;
        // 16 sweeps fit the registers only next to the 64-column selection
        if (sw > (T == 64 ? 16 : 12)) continue;
        p.T = T;
        p.sweeps = sw <= 4 ? 4 : sw <= 8 ? 8 : sw <= 12 ? 12 : 16;
        break;
    }
    if (full_keys) return p;
    const WsPlan h = half_plan(f, p.T, false, false, [&](int T, int fill) {
        return mws_lds_bytes(f, T, true, fill);
    });
    return h.T != 0 ? h : p;
}

// LDS of the warp-specialised single pass: histograms, key tile, per-file
// words (half keys: two nibbles per file) and, with a row table in LDS, the
// table.
int64_t ws_lds_bytes(int64_t f, int r, int T, bool table_in_lds, bool half, int fill) {
    // half keys: slot nibbles, and pair-difference nibbles (r = 3) or words
    const int64_t words = half ? half_hist_words(T) + half_tile_words(f, T, fill) + (f + 7) / 8 +
                                     (r == 3 ? (f + 7) / 8 : f)
                               : hist_words(T) + f * (int64_t)T + 2 * f;
    return words * 4 + (table_in_lds ? f * r * 4 : 0);
}

// Warp-specialised single pass (16-byte aligned rows): plans as for the
// median above (the wide split without a row table in LDS).  r = 5: half-key
// tiles of the file-major tensor, even split (five 16-byte chunks a sweep
// leave the streaming role no registers for more).
WsPlan ws_plan(int64_t f, int r, bool vec, bool ind, bool full_keys = false) {
    WsPlan p;
    if (!vec) return p;
    if (r == 5 && !ind && !full_keys) {
        p.r = 5;
        WsPlan h = half_plan(f, 0, false, false, [&](int T, int fill) {
            return ws_lds_bytes(f, r, T, false, true, fill);
        }, 5);
        h.r = 5;
        return h.T != 0 ? h : WsPlan{};
    }
    if (r != 3) return p;
    for (int T : {64, 32, 16, 8}) {
        if (ws_lds_bytes(f, r, T, ind, false, kWsFill) > kLdsBytes) continue;
        const int64_t rpi = kWsFill / (T / 4);
        const int64_t sw = (f + rpi - 1) / rpi;
        if (sw > 16) continue;
        p.T = T;
        p.sweeps = round_sweeps(sw, false, T, kWsFill);
        break;
    }
    if (full_keys) return p;
    const WsPlan h = half_plan(f, p.T, ind, false, [&](int T, int fill) {
        return ws_lds_bytes(f, r, T, ind, true, fill);
    });
    WsPlan best = h.T != 0 ? h : p;
    if (ind) {
        // a wider tile when the row table, read from global memory (where it
        // stays cached), leaves LDS to the keys: 2,300 files take 32 columns
        // instead of 16
        const WsPlan wide = half_plan(f, best.T, true, true, [&](int T, int fill) {
            return ws_lds_bytes(f, r, T, false, true, fill);
        });
        if (wide.T != 0) best = wide;
    }
    return best;
}

// ---------------------------------------------------------------------------
// The kernels built for each plan.  A launcher looks its kernel up here; a
// plan with no entry is a planning error (reported by aspis_plan and the
// launchers alike, never launched).

using FusedWsFn = void (*)(const float *, const int32_t *, int64_t, int64_t, const int32_t *,
                           const int32_t *, const int32_t *, int64_t, uint32_t *, float *);
using MedianWsFn = void (*)(const float *, int64_t, const int32_t *, const int32_t *, int64_t,
                            float *, TileMask);

FusedWsFn fused_ws_fn(const WsPlan &p, bool ind) {
    const int key = p.T * 1000 + p.sweeps * 10 + (p.half ? 1 : 0);
#define ASPIS_KEY(TT, SWW, HH) TT * 1000 + SWW * 10 + (HH ? 1 : 0)
    if (p.r == 5) {
        // five replicas a file: half keys, file-major, even split
        if (ind || !p.half || p.fill != kWsFill || p.rtg) return nullptr;
        switch (key) {
#define ASPIS_FWS5(TT, SWW) \
    case ASPIS_KEY(TT, SWW, true): return &fused_ws_kernel<TT, 5, SWW, false, true, kWsFill, false>;
            ASPIS_FWS5(128, 16)
            ASPIS_FWS5(128, 30)
            ASPIS_FWS5(128, 32)
            ASPIS_FWS5(64, 16)
            ASPIS_FWS5(64, 24)
            ASPIS_FWS5(64, 32)
            ASPIS_FWS5(32, 16)
            ASPIS_FWS5(32, 24)
            ASPIS_FWS5(32, 32)
            ASPIS_FWS5(16, 16)
            ASPIS_FWS5(16, 24)
            ASPIS_FWS5(16, 32)
#undef ASPIS_FWS5
        default: return nullptr;
        }
    }
    if (p.r != 3) return nullptr;
    // file-major, or with the row table in LDS
#define ASPIS_FWS(TT, SWW, HH)                                                  \
    case ASPIS_KEY(TT, SWW, HH):                                                \
        return ind ? &fused_ws_kernel<TT, 3, SWW, true, HH, kWsFill, false>     \
                   : &fused_ws_kernel<TT, 3, SWW, false, HH, kWsFill, false>;
    if (p.rtg) {
        // row table read from global memory: wide split, half keys
        if (!ind || !p.half || p.fill != kWsFillWide) return nullptr;
        switch (key) {
#define ASPIS_FWS_RTG(TT, SWW)  \
    case ASPIS_KEY(TT, SWW, true): return &fused_ws_kernel<TT, 3, SWW, true, true, kWsFillWide, true>;
            ASPIS_FWS_RTG(64, 24)
            ASPIS_FWS_RTG(64, 32)
            ASPIS_FWS_RTG(32, 24)
            ASPIS_FWS_RTG(32, 32)
#undef ASPIS_FWS_RTG
        default: return nullptr;
        }
    }
    if (p.fill == kWsFillWide) {
        // wide split: half keys, file-major only
        if (ind || !p.half) return nullptr;
        switch (key) {
#define ASPIS_FWS_WIDE(TT, SWW) \
    case ASPIS_KEY(TT, SWW, true): return &fused_ws_kernel<TT, 3, SWW, false, true, kWsFillWide, false>;
            ASPIS_FWS_WIDE(64, 24)
            ASPIS_FWS_WIDE(64, 32)
            ASPIS_FWS_WIDE(32, 24)
            ASPIS_FWS_WIDE(32, 32)
#undef ASPIS_FWS_WIDE
        default: return nullptr;
        }
    }
    if (p.fill != kWsFill) return nullptr;
    if (p.half && p.T == 32 && p.sweeps == 36)   // no room for a row table in LDS
        return ind ? nullptr : &fused_ws_kernel<32, 3, 36, false, true, kWsFill, false>;
    switch (key) {
#define ASPIS_FWS_FULL(TT)    \
    ASPIS_FWS(TT, 2, false)   \
    ASPIS_FWS(TT, 4, false)   \
    ASPIS_FWS(TT, 8, false)   \
    ASPIS_FWS(TT, 12, false)  \
    ASPIS_FWS(TT, 16, false)
#define ASPIS_FWS_HALF(TT)    \
    ASPIS_FWS(TT, 16, true)   \
    ASPIS_FWS(TT, 24, true)   \
    ASPIS_FWS(TT, 32, true)
        ASPIS_FWS_FULL(64)
        ASPIS_FWS_FULL(32)
        ASPIS_FWS_FULL(16)
        ASPIS_FWS_FULL(8)
        ASPIS_FWS(128, 8, true)
        ASPIS_FWS(128, 16, true)
        ASPIS_FWS(128, 24, true)
        ASPIS_FWS(128, 26, true)
        ASPIS_FWS(128, 28, true)
        ASPIS_FWS(128, 30, true)
        ASPIS_FWS(128, 32, true)
        ASPIS_FWS_HALF(64)
        ASPIS_FWS_HALF(32)
        ASPIS_FWS_HALF(16)
#undef ASPIS_FWS_HALF
#undef ASPIS_FWS_FULL
    default: return nullptr;
    }
#undef ASPIS_FWS
}

MedianWsFn median_ws_fn(const WsPlan &p) {
    const int key = p.T * 1000 + p.sweeps * 10 + (p.half ? 1 : 0);
#define ASPIS_MWS(TT, SWW, HH, FF) \
    case ASPIS_KEY(TT, SWW, HH): return &median_ws_kernel<TT, SWW, HH, FF>;
    if (p.fill == kWsFillWide) {
        if (!p.half) return nullptr;
        switch (key) {
            ASPIS_MWS(64, 16, true, kWsFillWide)
            ASPIS_MWS(64, 24, true, kWsFillWide)
            ASPIS_MWS(64, 32, true, kWsFillWide)
            ASPIS_MWS(32, 16, true, kWsFillWide)
            ASPIS_MWS(32, 24, true, kWsFillWide)
            ASPIS_MWS(32, 32, true, kWsFillWide)
        default: return nullptr;
        }
    }
    if (p.fill != kWsFill) return nullptr;
    switch (key) {
#define ASPIS_MWS_FULL(TT)               \
    ASPIS_MWS(TT, 4, false, kWsFill)     \
    ASPIS_MWS(TT, 8, false, kWsFill)     \
    ASPIS_MWS(TT, 12, false, kWsFill)
#define ASPIS_MWS_HALF(TT)               \
    ASPIS_MWS(TT, 16, true, kWsFill)     \
    ASPIS_MWS(TT, 24, true, kWsFill)     \
    ASPIS_MWS(TT, 32, true, kWsFill)
        ASPIS_MWS_FULL(64)
        ASPIS_MWS(64, 16, false, kWsFill)
        ASPIS_MWS_FULL(32)
        ASPIS_MWS_FULL(16)
        ASPIS_MWS_FULL(8)
        ASPIS_MWS(128, 8, true, kWsFill)
        ASPIS_MWS(128, 16, true, kWsFill)
        ASPIS_MWS(128, 24, true, kWsFill)
        ASPIS_MWS(128, 26, true, kWsFill)
        ASPIS_MWS(128, 28, true, kWsFill)
        ASPIS_MWS(128, 30, true, kWsFill)
        ASPIS_MWS(128, 32, true, kWsFill)
        ASPIS_MWS_HALF(64)
        ASPIS_MWS_HALF(32)
        ASPIS_MWS(32, 36, true, kWsFill)
        ASPIS_MWS_HALF(16)
#undef ASPIS_MWS_HALF
#undef ASPIS_MWS_FULL
    default: return nullptr;
    }
#undef ASPIS_MWS
#undef ASPIS_KEY
}

KernelPlan ws_kernel_plan(int kind, const WsPlan &p, int64_t lds, int table) {
    KernelPlan k;
    k.kind = kind;
    k.tile_cols = p.T;
    k.sweeps = p.sweeps;
    k.half_keys = p.half ? 1 : 0;
    k.stream_threads = p.fill;
    k.row_table = table;
    k.lds_bytes = lds;
    k.block = kWsThreads;
    return k;
}

}  // namespace

bool plan_median(int64_t f, bool vec, KernelPlan *out, bool full_keys) {
    const WsPlan p = mws_plan(f, vec, full_keys);
    if (p.T != 0) {
        *out = ws_kernel_plan(median_ws_fn(p) ? kKernelMedianWs : kKernelUnbuilt, p,
                              mws_lds_bytes(f, p.T, p.half, p.fill), 0);
        return out->kind == kKernelMedianWs;
    }
    KernelPlan k;
    const int T = pick_tile(f, 0);
    if (T != 0) {
        k.kind = kKernelMedianTile;
        k.tile_cols = T;
        k.lds_bytes = f * 4 * T + hist_words(T) * 4;
        k.block = (T >= 16 ? 1024 : 64 * T);
    } else {
        k.kind = kKernelMedianRadix;
        k.tile_cols = kRadixCols;
        k.lds_bytes = 0;   // static
        k.block = kRadixThreads;
    }
    *out = k;
    return true;
}

bool plan_fused(int64_t f, int r, bool vec, bool ind, KernelPlan *out, bool full_keys) {
    *out = KernelPlan{};
    const WsPlan p = ws_plan(f, r, vec, ind, full_keys);
    if (p.T != 0) {
        const int table = ind ? (p.rtg ? 2 : 1) : 0;
        *out = ws_kernel_plan(fused_ws_fn(p, ind) ? kKernelFusedWs : kKernelUnbuilt, p,
                              ws_lds_bytes(f, r, p.T, ind && !p.rtg, p.half, p.fill), table);
        return out->kind == kKernelFusedWs;
    }
    if (r != 3 && r != 5 && r != 7) return false;
    const int T = pick_tile(f, f * 4);
    if (T == 0) return false;
    out->kind = kKernelFused;
    out->tile_cols = T;
    out->row_table = ind ? 2 : 0;
    out->lds_bytes = f * 4 * T + f * 4 + hist_words(T) * 4;
    out->block = (T >= 16 ? 1024 : 64 * T);
    return true;
}

bool fused_supported(int64_t f, int r) {
    KernelPlan k;
    return plan_fused(f, r, true, false, &k) || plan_fused(f, r, false, false, &k);
}

hipError_t launch_median(const float *g, int64_t d, const Workspace &ws, int64_t f,
                         float *out, hipStream_t s, TileUse *use, bool full_keys, bool repair) {
    const bool vec = (d % 4 == 0) && aligned16(g);
    KernelPlan k;
    if (!plan_median(f, vec, &k, full_keys)) return hipErrorInvalidValue;
    if (use) *use = TileUse{k.tile_cols, k.half_keys};
    const int T = k.tile_cols;
    const int64_t ntiles = (d + T - 1) / T;
    TileMask mask;
    if (repair) {
        mask.bits = ws.dirty;
        mask.count = ws.repair;
        mask.gshift = dirty_gran_shift(ntiles);
    }
    if (k.kind == kKernelMedianWs) {
        const unsigned grid = (unsigned)grid_for(ntiles, (int64_t)num_cus());
        const MedianWsFn fn = median_ws_fn(mws_plan(f, vec, full_keys));
        fn<<<grid, kWsThreads, (size_t)k.lds_bytes, s>>>(g, d, ws.rows, ws.n_sel, ntiles, out, mask);
        return hipGetLastError();
    }
    if (k.kind == kKernelMedianRadix) {
        // LDS: 66 KB of histograms, two workgroups per CU
        const unsigned grid = (unsigned)grid_for(ntiles, (int64_t)num_cus() * 2);
        median_radix_kernel<<<grid, kRadixThreads, 0, s>>>(g, d, ws.rows, ws.n_sel, ntiles, out,
                                                           mask);
        return hipGetLastError();
    }
    const size_t lds = (size_t)k.lds_bytes;
    const unsigned grid = (unsigned)tile_grid(ntiles, lds);
#define ASPIS_MED(TT)                                                                        \
    if (vec)                                                                                 \
        median_kernel<TT, true><<<grid, tile_block<TT>(), lds, s>>>(g, d, ws.rows, ws.n_sel, \
                                                                   ntiles, out, mask);       \
    else                                                                                     \
        median_kernel<TT, false><<<grid, tile_block<TT>(), lds, s>>>(g, d, ws.rows, ws.n_sel, \
                                                                    ntiles, out, mask);
    switch (T) {
    case 64: ASPIS_MED(64) break;
    case 32: ASPIS_MED(32) break;
    case 16: ASPIS_MED(16) break;
    case 8: ASPIS_MED(8) break;
    case 4: ASPIS_MED(4) break;
    default: return hipErrorInvalidValue;
    }
#undef ASPIS_MED
    return hipGetLastError();
}

hipError_t launch_save_sel(const Workspace &ws, int64_t f, hipStream_t s) {
    if (f <= 0) return hipErrorInvalidValue;
    save_sel_kernel<<<(unsigned)((f + kBlock - 1) / kBlock), kBlock, 0, s>>>(ws.sel, f, ws.sel_prev,
                                                                            ws.repair);
    return hipGetLastError();
}

hipError_t launch_dirty_tiles(const float *g, const int32_t *row_of, int64_t f, int r, int64_t d,
                              const Workspace &ws, const uint32_t *pair_diff, int tile_cols,
                              hipStream_t s) {
    const bool vec = (d % 4 == 0) && aligned16(g);
    if (f <= 0 || d <= 0 || tile_cols < 4 || (tile_cols & (tile_cols - 1)) != 0)
        return hipErrorInvalidValue;
    const int64_t ntiles = (d + tile_cols - 1) / tile_cols;
    const int gshift = dirty_gran_shift(ntiles);
    const int64_t nbits = (ntiles + (int64_t(1) << gshift) - 1) >> gshift;
    int cshift = gshift;   // columns per bit: tile_cols << gshift
    for (int c = tile_cols; c > 1; c >>= 1) ++cshift;
    const unsigned grid = (unsigned)grid_for((nbits + 31) / 32, (int64_t)num_cus() * 8);
#define ASPIS_DIRTY(RR)                                                                         \
    if (vec)                                                                                    \
        dirty_tiles_kernel<RR, true><<<grid, kBlock, 0, s>>>(g, row_of, f, d, cshift,          \
                                                             nbits, ws.sel_prev, ws.sel,       \
                                                             pair_diff, ws.dirty, ws.repair);  \
    else                                                                                        \
        dirty_tiles_kernel<RR, false><<<grid, kBlock, 0, s>>>(g, row_of, f, d, cshift,         \
                                                              nbits, ws.sel_prev, ws.sel,      \
                                                              pair_diff, ws.dirty, ws.repair);
    switch (r) {
    case 3: ASPIS_DIRTY(3) break;
    case 5: ASPIS_DIRTY(5) break;
    case 7: ASPIS_DIRTY(7) break;
    default: return hipErrorInvalidValue;
    }
#undef ASPIS_DIRTY
    return hipGetLastError();
}

hipError_t launch_fused(const float *g, const int32_t *row_of, int64_t f, int r, int64_t d,
                        const Workspace &ws, uint32_t *pair_diff, float *out, hipStream_t s,
                        TileUse *use, bool full_keys) {
    const bool vec = (d % 4 == 0) && aligned16(g);
    const bool ind = row_of != nullptr;
    KernelPlan k;
    if (!plan_fused(f, r, vec, ind, &k, full_keys)) return hipErrorInvalidValue;
    if (use) *use = TileUse{k.tile_cols, k.half_keys};
    const int T = k.tile_cols;
    const int64_t ntiles = (d + T - 1) / T;
    const size_t lds = (size_t)k.lds_bytes;
    if (k.kind == kKernelFusedWs) {
        const unsigned grid = (unsigned)grid_for(ntiles, (int64_t)num_cus());
        const FusedWsFn fn = fused_ws_fn(ws_plan(f, r, vec, ind, full_keys), ind);
        fn<<<grid, kWsThreads, lds, s>>>(g, ind ? row_of : nullptr, f, d, ws.sel, ws.pos, ws.n_sel,
                                         ntiles, pair_diff, out);
        return hipGetLastError();
    }
    const unsigned grid = (unsigned)tile_grid(ntiles, lds);
#define ASPIS_FUSED(TT, RR)                                                                  \
    if (vec)                                                                                 \
        fused_kernel<TT, RR, true><<<grid, tile_block<TT>(), lds, s>>>(                      \
            g, row_of, f, d, ws.sel, ws.pos, ws.n_sel, ntiles, pair_diff, out);              \
    else                                                                                     \
        fused_kernel<TT, RR, false><<<grid, tile_block<TT>(), lds, s>>>(                     \
            g, row_of, f, d, ws.sel, ws.pos, ws.n_sel, ntiles, pair_diff, out);
#define ASPIS_FUSED_R(TT)                     \
    switch (r) {                              \
    case 3: ASPIS_FUSED(TT, 3) break;         \
    case 5: ASPIS_FUSED(TT, 5) break;         \
    case 7: ASPIS_FUSED(TT, 7) break;         \
    default: return hipErrorInvalidValue;     \
    }
    switch (T) {
    case 64: ASPIS_FUSED_R(64) break;
    case 32: ASPIS_FUSED_R(32) break;
    case 16: ASPIS_FUSED_R(16) break;
    case 8: ASPIS_FUSED_R(8) break;
    case 4: ASPIS_FUSED_R(4) break;
    default: return hipErrorInvalidValue;
    }
#undef ASPIS_FUSED_R
#undef ASPIS_FUSED
    return hipGetLastError();
}

bool fused_mean_supported(int64_t f, int r) {
    return (r == 3 || r == 5 || r == 7) && f * 4 <= kFusedMeanLds;
}

hipError_t launch_fused_mean(const float *g, const int32_t *row_of, int64_t f, int r, int64_t d,
                             const Workspace &ws, uint32_t *pair_diff, float *out,
                             hipStream_t s) {
    if (!fused_mean_supported(f, r)) return hipErrorInvalidValue;
    const int64_t nq = (d + 3) / 4;
    // up to 8 workgroups per CU: each wave's loads follow one another file
    // after file, so more resident waves keep more rows in flight (4 per CU
    // left K=21, d=5M 7 % slower)
    const unsigned grid = (unsigned)grid_for((nq + kBlock - 1) / kBlock, (int64_t)num_cus() * 8);
    const size_t lds = (size_t)f * 4;
    const bool vec = (d % 4 == 0) && aligned16(g);
#define ASPIS_FMEAN(RR)                                                                      \
    if (vec)                                                                                 \
        fused_mean_kernel<RR, true><<<grid, kBlock, lds, s>>>(g, row_of, f, d, ws.sel,       \
                                                              ws.pos, ws.n_sel, pair_diff, out); \
    else                                                                                     \
        fused_mean_kernel<RR, false><<<grid, kBlock, lds, s>>>(g, row_of, f, d, ws.sel,      \
                                                               ws.pos, ws.n_sel, pair_diff, out);
    switch (r) {
    case 3: ASPIS_FMEAN(3) break;
    case 5: ASPIS_FMEAN(5) break;
    case 7: ASPIS_FMEAN(7) break;
    default: return hipErrorInvalidValue;
    }
#undef ASPIS_FMEAN
    return hipGetLastError();
}

hipError_t launch_mean(const float *g, int64_t d, const Workspace &ws, float *out,
                       hipStream_t s, bool repair) {
    const int64_t ntiles = (d + kMeanTileCols - 1) / kMeanTileCols;
    const unsigned grid = (unsigned)grid_for(ntiles, (int64_t)num_cus() * 8);
    TileMask mask;
    if (repair) {
        mask.bits = ws.dirty;
        mask.count = ws.repair;
        mask.gshift = dirty_gran_shift(ntiles);
    }
    if ((d % 4 == 0) && aligned16(g))
        mean_kernel<true><<<grid, kBlock, 0, s>>>(g, d, ws.rows, ws.n_sel, out, mask);
    else
        mean_kernel<false><<<grid, kBlock, 0, s>>>(g, d, ws.rows, ws.n_sel, out, mask);
    return hipGetLastError();
}

int reduce_tile_cols(const float *g, int64_t f, int64_t d, bool mean, bool full_keys) {
    if (mean) return (int)kMeanTileCols;
    KernelPlan k;
    const bool vec = (d % 4 == 0) && aligned16(g);
    return plan_median(f, vec, &k, full_keys) ? k.tile_cols : 0;
}

// The workspace of the allocation-free entry point: a static device array,
// one copy per device, whose device address is looked up once per device
// with that device current (in host code the array's name is a host-side
// stand-in, never a device address).
__device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
std::atomic<void *> g_scratch[kMaxDevices];
}  // namespace

hipError_t scratch_ptr(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    void *p = g_scratch[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_scratch[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return hipSuccess;
}

hipError_t launch_tie_probe(const float *g, const int32_t *row_of, int64_t f, int r, int64_t d,
                            const ProbeSet &probe, uint32_t *out, hipStream_t s) {
    const int64_t n = probe.coords();
    if (f <= 0 || n <= 0 || !probe_valid(probe, d)) return hipErrorInvalidValue;
    const unsigned grid = (unsigned)(n >= kTieCols ? kTieCols : n);
    switch (r) {
    case 3: tie_probe_kernel<3><<<grid, kTieThreads, 0, s>>>(g, row_of, f, d, probe, out); break;
    case 5: tie_probe_kernel<5><<<grid, kTieThreads, 0, s>>>(g, row_of, f, d, probe, out); break;
    case 7: tie_probe_kernel<7><<<grid, kTieThreads, 0, s>>>(g, row_of, f, d, probe, out); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

size_t read_probe_sink_words() { return (size_t)kProbeBlocks * kBlock; }

hipError_t launch_read_probe(const void *buf, size_t nbytes, uint32_t *sink, hipStream_t s) {
    read_probe_kernel<<<kProbeBlocks, kBlock, 0, s>>>(static_cast<const uint4 *>(buf),
                                                      (int64_t)(nbytes / 16), sink);
    return hipGetLastError();
}

}  // namespace aspis
