// aspis_internal.h -- launchers shared by the host library (aspis_host.cpp)
// and the HIP kernels (aspis_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace aspis {

// Median tile widths (coordinates per workgroup tile) the kernels support.
// The tile keeps every kept file's keys for T coordinates in LDS, so the
// widest tile whose [files x T] key block fits is chosen.
constexpr int kBlock = 256;                 // threads per workgroup
constexpr int64_t kLdsBytes = 160 * 1024;   // LDS per CU on gfx950

// The selection keeps a histogram block of kHistStride words per column
// (128 buckets, an overflow bucket, padding) next to the key tile.
constexpr int kHistBuckets = 128;
constexpr int kHistStride = 132;
constexpr int64_t hist_bytes(int T) { return (int64_t)T * kHistStride * 4; }

// Workspace layout (byte offsets) for f files.
struct Workspace {
    int32_t *sel;     // [f] kept slot or -1
    int32_t *pos;     // [f] row of the file in the kept-file list, or -1
    int32_t *rows;    // [f] kept replica rows (i*r + slot), file order
    int32_t *n_sel;   // [1] number of kept files
    uint64_t *stage;  // [104] staged for the host: [0,64) disagreement rows,
                      // [64] a vote-changed flag, [72,104) the tie probe's
                      // kTieCols uint32 counts (kStageTie)
    int32_t *row_of;  // [f*r] row of replica (i,s) in a worker-major upload
    int8_t *sel_prev; // [f] the guessed selection's slots (repair after a miss)
    uint32_t *dirty;  // [kDirtyWords] tile-group bits of the repair
    int32_t *repair;  // [4] repair counters: [0] dirty tile groups
};
// Tile-group bits of the repair after a wrong guess: bit b covers tiles
// [b << s, (b + 1) << s), s the least that fits every tile in these bits.
constexpr int64_t kDirtyWords = 4096;
constexpr int kStageTie = 72;      // first stage word of the tie counts
constexpr int kStageWords = 104;   // stage words the host reads back
size_t workspace_bytes(int64_t f, int r);
Workspace carve_workspace(void *base, int64_t f, int r);

hipError_t launch_fill_u32(uint32_t *p, int64_t n, uint32_t v, hipStream_t s);
hipError_t launch_fill_u64(uint64_t *p, int64_t n, uint64_t v, hipStream_t s);

// Replica (i,s) is row i*r+s of g (file-major, row_of == nullptr) or row
// row_of[i*r+s] (a device table, e.g. the worker-major upload order).

// Pairwise agreement over coordinates [0, k_end) of every file; ORs the
// per-file pair-difference bits into pair_diff (which the caller zeroes).
hipError_t launch_agree(const float *g, const int32_t *row_of, int64_t f, int r, int64_t d,
                        int64_t k_end, uint32_t *pair_diff, hipStream_t s);

// The coordinates the single pass guesses its selection from: nb blocks of
// kProbeBlockCols coordinates.  seed == 0: the prefix [0, kend), in
// consecutive blocks (the last one ends at kend).  Otherwise block j starts
// at start[j], a multiple of kProbeAlign in [0, d - kProbeBlockCols] that
// the host draws per call from a random seed (probe_block_start): a worker
// cannot know when it uploads which coordinates the guess reads.
constexpr int64_t kProbeBlockCols = 1024;
constexpr int64_t kProbeAlign = 64;
constexpr int kProbeMaxBlocks = 32;
struct ProbeSet {
    uint64_t seed = 0;   // 0: the prefix
    int64_t nb = 0;      // blocks (<= kProbeMaxBlocks)
    int64_t kend = 0;    // prefix: its end
    int64_t start[kProbeMaxBlocks] = {};
    int64_t coords() const { return seed ? nb * kProbeBlockCols : kend; }
    __host__ __device__ int64_t block_start(int64_t j) const {
        return seed ? start[j] : j * kProbeBlockCols;
    }
    __host__ __device__ int64_t block_end(int64_t b) const {
        if (seed != 0) return b + kProbeBlockCols;
        return b + kProbeBlockCols < kend ? b + kProbeBlockCols : kend;
    }
};
// SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): the output function of
// the generator, applied to the seed mixed with the block index.
inline uint64_t splitmix64(uint64_t x) {
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}
inline int64_t probe_block_start(uint64_t seed, int64_t j, int64_t d) {
    const uint64_t slots = (uint64_t)((d - kProbeBlockCols) / kProbeAlign) + 1u;
    return (int64_t)(splitmix64(seed ^ ((uint64_t)j << 32)) % slots) * kProbeAlign;
}

// Agreement over the probed coordinates with one workgroup per file; stores
// every file's word (no zero fill needed).
hipError_t launch_agree_file(const float *g, const int32_t *row_of, int64_t f, int r, int64_t d,
                             const ProbeSet &probe, uint32_t *pair_diff, hipStream_t s);

// Per-file vote / majority flag and the disagreement rows (caller zeroes
// disagree).
hipError_t launch_vote(const uint32_t *pair_diff, const int32_t *subsets,
                       int64_t f, int r, int8_t *vote, uint8_t *has_majority,
                       uint64_t *disagree, hipStream_t s);

// The same in one workgroup (f <= kVoteRowsMaxFiles): writes disagree[0..K)
// whole, copies the rows to stage[0..K) and sets stage[64] to 1 if a vote
// changed from the value vote[] held before.
constexpr int64_t kVoteRowsMaxFiles = 1 << 16;
hipError_t launch_vote_rows(const uint32_t *pair_diff, const int32_t *subsets, int64_t f,
                            int r, int K, int8_t *vote, uint8_t *has_majority,
                            uint64_t *disagree, uint64_t *stage, hipStream_t s);

// Selection of Algorithm 1 into the workspace (sel, pos, rows, n_sel), and
// into sel_out when it is not NULL.  ws.rows lists the kept rows of g
// (through row_of when it is not NULL).  zero, when not NULL, receives
// n_zero zero words in the same launch.
hipError_t launch_select(const int32_t *subsets, const int8_t *vote,
                         int64_t f, int r, int success, uint64_t honest,
                         const int32_t *row_of, const Workspace &ws,
                         int32_t *sel_out, uint32_t *zero, int64_t n_zero, hipStream_t s);

// Tile a median kernel ran with: columns per tile, and whether the tile
// kept only the high halves of the keys.
struct TileUse {
    int32_t cols = 0;
    int32_t half = 0;
};

// The kernel a launcher takes for a shape, decided without launching
// (the values of ASPIS_KERNEL_* in aspis.h).
constexpr int32_t kKernelNone = 0;          // no kernel of this kind for the shape
constexpr int32_t kKernelFusedWs = 1;       // fused_ws_kernel (warp-specialised single pass)
constexpr int32_t kKernelFused = 2;         // fused_kernel (single pass, load then select)
constexpr int32_t kKernelMedianWs = 3;      // median_ws_kernel
constexpr int32_t kKernelMedianTile = 4;    // median_kernel (LDS key tile)
constexpr int32_t kKernelMedianRadix = 5;   // median_radix_kernel (keys re-read from HBM)
constexpr int32_t kKernelUnbuilt = -1;      // planned, but no kernel is built for the plan
struct KernelPlan {
    int32_t kind = kKernelNone;
    int32_t tile_cols = 0;        // coordinates per tile
    int32_t sweeps = 0;           // streaming sweeps per tile (warp-specialised kernels)
    int32_t half_keys = 0;        // the tile keeps only the high 16 bits of each key
    int32_t stream_threads = 0;   // threads of the streaming role (warp-specialised)
    int32_t row_table = 0;        // 0 none, 1 staged in LDS, 2 read from global memory
    int32_t block = 0;            // threads per workgroup
    int64_t lds_bytes = 0;        // dynamic LDS per workgroup
};
// Median over up to f kept rows (always has a kernel); single pass for f
// files of r replicas (false: none, the step then takes two passes).  vec:
// d % 4 == 0 and a 16-byte aligned tensor; ind: rows through a row table;
// full_keys: tiles of 32-bit keys only (no half-key plan, no read-back).
bool plan_median(int64_t f, bool vec, KernelPlan *out, bool full_keys = false);
bool plan_fused(int64_t f, int r, bool vec, bool ind, KernelPlan *out, bool full_keys = false);

// Coordinate-wise lower median / fp64 mean of the kept rows.  With repair,
// only the tiles of the groups ws.dirty marks (launch_dirty_tiles with the
// launch's reduce_tile_cols) are computed; out keeps its values elsewhere.
hipError_t launch_median(const float *g, int64_t d, const Workspace &ws,
                         int64_t f, float *out, hipStream_t s, TileUse *use = nullptr,
                         bool full_keys = false, bool repair = false);
hipError_t launch_mean(const float *g, int64_t d, const Workspace &ws,
                       float *out, hipStream_t s, bool repair = false);

// Single pass: agreement bits of every file over [0, d) and the median of
// the rows selected by ws (a guess), in one read of the replica tensor.
hipError_t launch_fused(const float *g, const int32_t *row_of, int64_t f, int r, int64_t d,
                        const Workspace &ws, uint32_t *pair_diff, float *out,
                        hipStream_t s, TileUse *use = nullptr, bool full_keys = false);
bool fused_supported(int64_t f, int r);

// Single pass with the mean: agreement bits of every file over [0, d) and
// the fp64 mean of the rows selected by ws (a guess).
constexpr int64_t kFusedMeanLds = 64 * 1024;   // per-file words in LDS
hipError_t launch_fused_mean(const float *g, const int32_t *row_of, int64_t f, int r, int64_t d,
                             const Workspace &ws, uint32_t *pair_diff, float *out,
                             hipStream_t s);
bool fused_mean_supported(int64_t f, int r);

// Device address of this device's static scratch array (kScratchBytes,
// 256-aligned), the workspace of the allocation-free entry point.  Looked
// up on the first call per device (the calling thread's current device).
constexpr size_t kScratchBytes = (size_t)2 << 20;
hipError_t scratch_ptr(void **out);

// Tie probe over the probed coordinates: for min(kTieCols, probe.coords())
// coordinates spread over them, out[j] = the number of files whose value
// (the value of its largest class of equal replicas) shares the high 16-bit
// key half of those values' lower median.  The host reads that many words.
constexpr int kTieCols = 64;
hipError_t launch_tie_probe(const float *g, const int32_t *row_of, int64_t f, int r, int64_t d,
                            const ProbeSet &probe, uint32_t *out, hipStream_t s);

// Repair after a wrong guess whose selection kept the same files as the
// final one (only the kept replica of some files moved) and whose reduction
// was the same (the median, or the mean, summed in file order either way):
// the guessed result is already the final one on every coordinate where
// each moved file's two replicas are equal.
// launch_save_sel copies ws.sel (the guess) to ws.sel_prev before the final
// selection overwrites it, and zeroes the repair counters.
// launch_dirty_tiles, after the final selection, marks in ws.dirty the tile
// groups (tiles of tile_cols coordinates: reduce_tile_cols of the repairing
// launch) holding a coordinate where the replica of the guess and that of
// the final selection of a moved file differ -- every group when the kept
// files differ -- and counts them in ws.repair[0].  pair_diff: every file's
// pair-difference bits over the whole vector.
hipError_t launch_save_sel(const Workspace &ws, int64_t f, hipStream_t s);
hipError_t launch_dirty_tiles(const float *g, const int32_t *row_of, int64_t f, int r, int64_t d,
                              const Workspace &ws, const uint32_t *pair_diff, int tile_cols,
                              hipStream_t s);
// Coordinates per tile of launch_mean (mean) or launch_median (f kept rows,
// full_keys) on g: the tile width of their repair.
int reduce_tile_cols(const float *g, int64_t f, int64_t d, bool mean, bool full_keys);
// Tile groups: 2^shift tiles a bit, the least power of two that fits
// ntiles tiles in the bits.
inline int dirty_gran_shift(int64_t ntiles) {
    int sh = 0;
    while (((ntiles + (int64_t(1) << sh) - 1) >> sh) > kDirtyWords * 32) ++sh;
    return sh;
}

size_t read_probe_sink_words();
hipError_t launch_read_probe(const void *buf, size_t nbytes, uint32_t *sink,
                             hipStream_t s);

}  // namespace aspis
