/*
 * aspis.h -- C ABI of libaspis: the parameter server's detect-and-aggregate
 * step of Aspis (Konstantinidis & Ramamoorthy, "Aspis: Robust Detection for
 * Distributed Learning", MLSys 2022) on one AMD Instinct MI355X (gfx950).
 *
 * Plain C: no C++ or torch types cross this boundary.  Device pointers are
 * HIP device addresses (e.g. torch tensors' data_ptr()); "stream" is a
 * hipStream_t passed as void* (NULL = the default stream).
 *
 * Symbols: K workers, r replicas per file (odd), q bound on adversaries,
 * f = C(K,r) files, d gradient coordinates, P = r(r-1)/2 slot pairs.
 *
 * Layout of the replica tensor ("grads"): float32 [f][r][d], contiguous,
 * row (i,s) = the gradient returned for file i by the worker in slot s,
 * where slot s of file i is the s-th smallest worker of the file's subset.
 *
 * Ownership: every buffer is allocated and freed by the caller.  The library
 * allocates no device memory: what it needs beyond inputs and outputs comes
 * through the caller's workspace, or, for aspis_detect_aggregate_noalloc,
 * from a static device array (ASPIS_NOALLOC_SCRATCH_BYTES per device) that
 * is part of the loaded library.
 *
 * Errors: every entry point returns an aspis_status and never throws.  On
 * ASPIS_ERR_INVALID_ARG / ASPIS_ERR_OVERFLOW nothing has been written or
 * enqueued.  HIP failures return ASPIS_ERR_DEVICE.  aspis_last_error()
 * returns a message for the calling thread's last failure.
 *
 * Asynchrony: aspis_detect and aspis_aggregate only enqueue work on the
 * stream.  aspis_clique is host code.  aspis_detect_aggregate synchronises
 * the stream (it needs the agreement graph on the host) and returns with
 * its work complete.
 *
 * Thread safety: re-entrant.  Global state: the per-thread error message,
 * a per-device cache of the compute-unit count (written once per device
 * with relaxed atomics), the probe's random base (drawn once) and call
 * counter (an atomic), and the allocation-free entry point's static scratch
 * array with its per-device address.  Calls that share output buffers, and
 * allocation-free calls on one device, must not overlap.
 */
#ifndef ASPIS_H
#define ASPIS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ASPIS_OK = 0,
    ASPIS_ERR_INVALID_ARG = 1,   /* bad size, NULL pointer, unsupported r   */
    ASPIS_ERR_OVERFLOW = 2,      /* f or f*r*d does not fit in int64         */
    ASPIS_ERR_BUFFER_SMALL = 3,  /* caller buffer / workspace too small      */
    ASPIS_ERR_DEVICE = 4,        /* a HIP call failed                        */
    ASPIS_ERR_NO_FILES = 5       /* selection kept no file; out untouched    */
} aspis_status;

typedef enum {
    ASPIS_REDUCE_MEDIAN = 0,     /* coordinate-wise (lower) median           */
    ASPIS_REDUCE_MEAN = 1,       /* coordinate-wise mean                     */
    ASPIS_REDUCE_PAPER = 2       /* mean on successful detection, else median */
} aspis_reduce;

/* Limits of the library. */
#define ASPIS_MAX_K_DEVICE 64    /* K for the device entry points            */
#define ASPIS_MAX_K_CLIQUE 128   /* K for aspis_clique                       */
#define ASPIS_MAX_R 7            /* largest (odd) redundancy                 */

/* Number of files f = C(K,r) (Section 3, Algorithm 2).
 * Returns -1 if K < 1, r < 1, r > K, or the value exceeds int64. */
int64_t aspis_num_files(int32_t K, int32_t r);

/* Algorithm 2 (subset assignment), Example 1 fixing file 0 <-> {U1,U2,U3}:
 * writes the f r-subsets of {0..K-1} in lexicographic order, members
 * ascending: subsets[i*r + s] = worker of slot s of file i (host memory,
 * caller-owned, at least cap_files*r entries).
 * Errors: INVALID_ARG (K<1, r<1, r>K, NULL), OVERFLOW (f > int64),
 * BUFFER_SMALL (f > cap_files; nothing written). */
aspis_status aspis_assign(int32_t K, int32_t r, int32_t *subsets,
                          int64_t cap_files);

/* Detection outputs, all device pointers, caller-owned, written by
 * aspis_detect / aspis_detect_aggregate.
 *   pair_diff[f]    bit p set iff the replicas of slot pair p (pairs (s,t),
 *                   s<t, in lexicographic order) differ in at least one
 *                   coordinate -- the complement of the agreement indicator
 *                   of Eq. (4), read bitwise.
 *   vote[f]         Eq. (3): the slot carrying the majority value -- the
 *                   lowest slot of the largest class of bitwise-equal
 *                   replicas (ties between classes: the lower slot).
 *   has_majority[f] 1 iff that class holds at least (r+1)/2 replicas.
 *   disagree[K]     row bitsets of the K x K disagreement matrix: bit v of
 *                   row u set iff workers u and v differ on at least one of
 *                   their C(K-2,r-2) common files, i.e. no edge (u,v) in the
 *                   detection graph of Section 4 (Eq. 5 below its maximum).
 */
typedef struct {
    uint32_t *pair_diff;
    int8_t *vote;
    uint8_t *has_majority;
    uint64_t *disagree;
} aspis_detect_out;

/* Section 4, Eq. (4)-(5) and Algorithm 3 (first loop), plus the per-file
 * majority of Eq. (3): one pass over the replica tensor.
 *   grads        device float32 [f][r][d] (see layout above)
 *   subsets_dev  device int32 [f][r], the table of aspis_assign
 *   out          device outputs above (all four required)
 * Requires 2 <= K <= 64, r odd with 3 <= r <= min(K,7), d >= 1.
 * Enqueues on stream; outputs are valid once the stream reaches them. */
aspis_status aspis_detect(const float *grads, int32_t K, int32_t r, int64_t d,
                          const int32_t *subsets_dev,
                          const aspis_detect_out *out, void *stream);

/* Outcome of Algorithm 3.  Bitsets hold worker u at word u/64, bit u%64. */
typedef struct {
    int32_t success;          /* exactly one maximum clique, of size >= K-q  */
    int32_t omega;            /* size of a maximum clique                    */
    int32_t n_maximum;        /* number of maximum cliques                   */
    int32_t n_words;          /* (K+63)/64                                   */
    int64_t n_maximal;        /* maximal cliques enumerated                  */
    uint64_t honest[2];       /* H = the unique maximum clique (if success)  */
    uint64_t detected[2];     /* A^ = U \ H (if success), else empty         */
    uint64_t first[2];        /* the first maximum clique found              */
} aspis_clique_result;

/* Algorithm 3 (clique step), host only, synchronous: enumerates all maximal
 * cliques of the detection graph (complement of the disagreement matrix) by
 * Bron-Kerbosch with Tomita pivoting and decides success.
 *   disagree_rows  host, K rows of n_words = (K+63)/64 uint64 each; the
 *                  matrix must be symmetric with an empty diagonal
 *   q              adversary bound, 0 <= q < K/2 (Section 2)
 * Errors: INVALID_ARG (K outside [1,128], q outside [0,K/2), NULL,
 * asymmetric matrix or set diagonal). */
aspis_status aspis_clique(const uint64_t *disagree_rows, int32_t K, int32_t q,
                          aspis_clique_result *res);

/* Bytes of workspace aspis_aggregate, aspis_detect_aggregate and
 * aspis_detect_aggregate_wm need: three int32 [f] arrays and one int32
 * [f*r] table, each rounded up to 256 bytes, 256 bytes of counters, 1,024
 * bytes where the disagreement rows are staged for the host, and for the
 * repair after a wrong guess an int8 [f] array rounded up to 256 bytes,
 * 16,384 bytes of tile-group bits and 256 bytes of counters.
 * 0 on invalid arguments. */
size_t aspis_aggregate_workspace(int32_t K, int32_t r, int64_t d);

/* Algorithm 1, aggregation.  Selection: on success (Case 1) file i keeps
 * the replica of its lowest slot whose worker is in H and is dropped when
 * it has none; otherwise (Case 2) it keeps its majority vote.  Reduction:
 * MEDIAN -> out[k] = element of rank floor((m-1)/2) of the m kept values
 * under IEEE-754 totalOrder (-NaN < -inf < ... < -0 < +0 < ... < +NaN);
 * MEAN -> out[k] = fl32(sum of the kept values in file order in fp64 / m);
 * PAPER -> MEAN on success, MEDIAN otherwise.
 *   det         detection outputs (vote is read on failure)
 *   res         result of aspis_clique for the same round
 *   out         device float32 [d]
 *   sel_out     device int32 [f] (kept slot or -1) or NULL
 *   n_selected  host, receives m (computed on the host, no sync) or NULL
 *   workspace   device, >= aspis_aggregate_workspace() bytes, 256-aligned
 * Errors: NO_FILES when m == 0 (out untouched), BUFFER_SMALL. */
aspis_status aspis_aggregate(const float *grads, int32_t K, int32_t r,
                             int64_t d, const int32_t *subsets_dev,
                             const aspis_detect_out *det,
                             const aspis_clique_result *res, aspis_reduce mode,
                             float *out, int32_t *sel_out, int64_t *n_selected,
                             void *workspace, size_t ws_bytes, void *stream);

/* Timings (HIP events on the call's stream) and path taken by
 * aspis_detect_aggregate. */
typedef struct {
    int32_t fused;             /* 1 if the single-pass kernel ran           */
    int32_t speculation_hit;   /* 1 if the probe's guess was confirmed      */
    int64_t probe_coords;      /* coordinates the guess was taken from      */
    float ms_probe;            /* agreement pass over the probe             */
    float ms_main;             /* main pass (fused, or detect + reduce)     */
    float ms_fallback;         /* repair or rerun after a wrong guess       */
    float ms_total;            /* first kernel to result, host steps incl.  */
    int32_t tile_cols;         /* coordinates per tile of the median kernel
                                  that produced out (0: the mean)          */
    int32_t half_keys;         /* 1 if that tile held only the high 16 bits
                                  of each key (low halves read back)       */
    int32_t tie_rows;          /* tie probe: over the probed coordinates,
                                  the mean (rounded up) of the number of
                                  files whose value shares the high 16-bit
                                  key half of the files' median; -1 if not
                                  probed                                   */
    int32_t probe_blocks;      /* blocks of 1,024 coordinates at positions
                                  drawn per call; 0: the probe was the
                                  prefix                                   */
    int32_t repair_groups;     /* after a wrong guess that asked for the
                                  same reduction: the tile groups
                                  recomputed (the others kept the guessed
                                  result, already final there); -1 if the
                                  step did not repair                      */
} aspis_run_stats;

#define ASPIS_FLAG_TWO_PASS 1u   /* force detect, clique, then aggregate    */
#define ASPIS_FLAG_TIMING 2u     /* fill the ms_* fields of stats           */
#define ASPIS_FLAG_FULL_KEYS 4u  /* median tiles of 32-bit keys only        */
#define ASPIS_FLAG_HALF_KEYS 8u  /* half-key tiles wherever the plan has
                                    them, without the tie probe             */
#define ASPIS_FLAG_PROBE_PREFIX 16u /* take the guess from the coordinate
                                       prefix, not from blocks drawn per
                                       call (reproducible speculation)      */

/* The whole step in one call (Algorithm 3 then Algorithm 1): agreement,
 * host clique, selection and reduction, with the same outputs as
 * aspis_detect + aspis_clique + aspis_aggregate.  By default it reads the
 * replica tensor once: it guesses the selection from a probe of a few
 * thousand coordinates, reduces with that guess while checking agreement
 * on all coordinates, and redoes the reduction if the full detection
 * disagrees with the guess -- the result is exact either way.  The probe
 * is the vector itself when d is at most its size, otherwise blocks of
 * 1,024 coordinates at positions drawn per call (SplitMix64 of a random
 * per-process seed and a call counter), so that a worker cannot know when
 * it uploads which coordinates the guess reads; ASPIS_FLAG_PROBE_PREFIX
 * takes the prefix instead.  After a wrong guess that asked for the same
 * reduction as the final detection, only the tiles holding a coordinate
 * where some file's guessed and final replicas differ are recomputed
 * (every tile when the guess kept other files).
 * Median tiles: the half-key tiles keep only the high 16 bits of each key
 * in LDS (twice the columns) and read back the low halves of the rows tied
 * with the median's high half.  Unless a key flag says otherwise, a tie
 * probe over 64 of the probed coordinates decides: when on average 16 or
 * more files there share the median's high half, the step takes full-key
 * tiles (no read-back).  The choice changes the speed, never the result.
 *   det, res, out, sel_out, n_selected  as above (sel_out may be NULL)
 *   flags   ASPIS_FLAG_* ; stats may be NULL.
 * Errors as aspis_aggregate's, except that on NO_FILES `out` holds no
 * result rather than being untouched: the single pass may have written it
 * with the guessed selection before the final one kept no file.
 * Synchronises the stream: twice on the single pass (the probe's graph and
 * the full graph), once more before returning. */
aspis_status aspis_detect_aggregate(const float *grads, int32_t K, int32_t r,
                                    int32_t q, int64_t d,
                                    const int32_t *subsets_dev,
                                    const aspis_detect_out *det,
                                    aspis_reduce mode, float *out,
                                    int32_t *sel_out, aspis_clique_result *res,
                                    int64_t *n_selected, void *workspace,
                                    size_t ws_bytes, uint32_t flags,
                                    aspis_run_stats *stats, void *stream);

/* For callers that cannot allocate (code under HIP graph capture, serving
 * loops and harnesses that forbid hipMalloc): aspis_detect_aggregate
 * without a workspace argument.  Its scratch (the selection, the kept-row
 * list, counters, the staged disagreement rows and the repair's
 * tile-group bits) lives in a static
 * device array of ASPIS_NOALLOC_SCRATCH_BYTES, one per device, held until
 * the process ends; its address is looked up on the first call on each
 * device.  The call allocates no device or host memory, and creates no
 * events.  Nothing in the array needs to start at zero: every part is
 * written before it is read.  Every call on one device shares that
 * device's array, so calls that overlap on one device (other streams or
 * threads) race and must be serialised by the caller.
 * Same arguments, outputs and errors as aspis_detect_aggregate, plus
 * BUFFER_SMALL when aspis_aggregate_workspace(K, r, d) exceeds the array
 * (every K <= 64 at r = 3; K <= 25 at r = 5; K <= 19 at r = 7) and
 * INVALID_ARG for
 * ASPIS_FLAG_TIMING (which would create events). */
#define ASPIS_NOALLOC_SCRATCH_BYTES ((size_t)2 << 20)
aspis_status aspis_detect_aggregate_noalloc(const float *grads, int32_t K, int32_t r,
                                            int32_t q, int64_t d,
                                            const int32_t *subsets_dev,
                                            const aspis_detect_out *det,
                                            aspis_reduce mode, float *out,
                                            int32_t *sel_out, aspis_clique_result *res,
                                            int64_t *n_selected, uint32_t flags,
                                            aspis_run_stats *stats, void *stream);

/* The worker-major upload of Algorithm 1: worker u returns the gradients
 * of its l = C(K-1,r-1) files in ascending file order, one after another,
 * so the upload of all K workers is a float32 [K][l][d] tensor.  Writes, for
 * every replica (i,s), its row in that tensor: row_of[i*r + s] = u*l + k
 * where u is the worker of slot s of file i and i is u's k-th file (host
 * memory, caller-owned, at least cap_entries = f*r entries).
 * Errors: INVALID_ARG, OVERFLOW, BUFFER_SMALL (nothing written). */
aspis_status aspis_worker_rows(int32_t K, int32_t r, int32_t *row_of,
                               int64_t cap_entries);

/* aspis_detect_aggregate on the worker-major upload grads_wm (float32
 * [K][l][d], contiguous, device) instead of the file-major [f][r][d]
 * tensor: the same steps, outputs and errors, the rows read through the
 * table of aspis_worker_rows (which the library builds in the workspace).
 * The pair-difference words, votes, selection (slot per file) and result
 * are identical to aspis_detect_aggregate's on the same replicas. */
aspis_status aspis_detect_aggregate_wm(const float *grads_wm, int32_t K, int32_t r,
                                       int32_t q, int64_t d,
                                       const int32_t *subsets_dev,
                                       const aspis_detect_out *det,
                                       aspis_reduce mode, float *out,
                                       int32_t *sel_out, aspis_clique_result *res,
                                       int64_t *n_selected, void *workspace,
                                       size_t ws_bytes, uint32_t flags,
                                       aspis_run_stats *stats, void *stream);

/* The kernels the device entry points take for a shape, decided without
 * launching anything (host only; assumes a 16-byte aligned tensor; flags:
 * ASPIS_FLAG_FULL_KEYS gives the full-key plans, otherwise the half-key
 * plans the tie probe keeps for untied data).
 *   single_pass  the single-pass kernel of aspis_detect_aggregate (worker-
 *                major: aspis_detect_aggregate_wm) for the median, or
 *                ASPIS_KERNEL_NONE when the shape takes the two-pass path
 *   median       the median kernel of aspis_aggregate and of the rerun
 *                after a wrong guess (for up to f kept files)
 * Errors: INVALID_ARG for an invalid shape (as aspis_detect) or when a
 * planned kernel is not built (the launch would fail the same way). */
#define ASPIS_KERNEL_NONE 0          /* no kernel: the step takes two passes    */
#define ASPIS_KERNEL_FUSED_WS 1      /* single pass, warp-specialised           */
#define ASPIS_KERNEL_FUSED 2         /* single pass, load then select per tile  */
#define ASPIS_KERNEL_MEDIAN_WS 3     /* median, warp-specialised                */
#define ASPIS_KERNEL_MEDIAN_TILE 4   /* median, LDS key tile                    */
#define ASPIS_KERNEL_MEDIAN_RADIX 5  /* median, radix select re-reading HBM     */
typedef struct {
    int32_t kernel;           /* ASPIS_KERNEL_*                                */
    int32_t tile_cols;        /* coordinates per tile                          */
    int32_t sweeps;           /* streaming sweeps per tile (warp-specialised)  */
    int32_t half_keys;        /* 1: the tile keeps the high 16 bits of keys    */
    int32_t stream_threads;   /* threads of the streaming role                 */
    int32_t row_table;        /* 0 none, 1 staged in LDS, 2 global memory      */
    int32_t block;            /* threads per workgroup                         */
    int32_t reserved;
    int64_t lds_bytes;        /* dynamic LDS per workgroup (0: static only)    */
} aspis_kernel_plan;

aspis_status aspis_plan(int32_t K, int32_t r, int64_t d, int32_t worker_major,
                        uint32_t flags, aspis_kernel_plan *single_pass,
                        aspis_kernel_plan *median);

/* Diagnostic: streams nbytes (multiple of 16) of device memory and writes a
 * checksum word per thread to sink (device, >= aspis_read_probe_sink_words()
 * uint32).  Used to measure the achievable HBM read bandwidth. */
size_t aspis_read_probe_sink_words(void);
aspis_status aspis_read_probe(const void *buf, size_t nbytes, uint32_t *sink,
                              void *stream);

/* ---- distortion-fraction simulator (Section 5, appendix Tables 1-3) ----
 *
 * The detect-and-aggregate step on symbolic replicas: every replica is either
 * its file's true value or the single value all adversaries agree on.  The
 * simulator runs the same steps as the device path -- pairwise agreement
 * (Eq. 4), disagreement rows (Eq. 5), vote (Eq. 3), aspis_clique
 * (Algorithm 3), selection (Algorithm 1) -- over all f = C(K,r) files of
 * Algorithm 2 and counts the distorted ones.  Host only, synchronous;
 * multithreaded over file ranks. */
typedef enum {
    ASPIS_ATTACK_WEAK = 0,     /* Section 4.1: every adversary distorts every
                                  file it holds */
    ASPIS_ATTACK_OPTIMAL = 1   /* Section 4.2, Theorem 1: all adversaries
                                  disagree with one set D of q honest
                                  workers: an adversary distorts file F iff
                                  |F & A| >= (r+1)/2 and F \ A is inside D */
} aspis_attack;

typedef struct {
    int64_t files;             /* f = C(K,r)                                 */
    int64_t distorted;         /* c^(q): files dropped (Case 1, no replica
                                  from H) or whose selected value is the
                                  adversaries'                               */
    int64_t dropped;           /* of which dropped                           */
    int32_t success;           /* Algorithm 3 detection succeeded (Case 1)   */
    int32_t omega;             /* size of a maximum clique                   */
    int32_t n_maximum;         /* number of maximum cliques                  */
    int32_t reserved;
    int64_t n_maximal;         /* maximal cliques enumerated                 */
    double epsilon;            /* distortion fraction distorted / files      */
    double epsilon_baseline;   /* q / K: aggregation of the K gradients
                                  without redundancy (Section 5)             */
    double ms_files;           /* host time of the passes over the files     */
    double ms_clique;          /* host time of aspis_clique                  */
} aspis_sim_result;

/* Simulate one attack.
 *   adversaries    q distinct worker ids, or NULL for {0,..,q-1}
 *   disagree_set   optimal attack only: q distinct honest worker ids, or
 *                  NULL for the q lowest-indexed honest workers
 *   disagree_rows  optional host output, K rows of (K+63)/64 uint64: the
 *                  disagreement matrix of the simulated round
 * Requires 3 <= K <= 128, odd 3 <= r <= min(K,15), 0 <= q < K/2 and
 * C(K,r) <= 2^31.  Errors: INVALID_ARG, OVERFLOW. */
aspis_status aspis_simulate(int32_t K, int32_t r, int32_t q, aspis_attack attack,
                            const int32_t *adversaries,
                            const int32_t *disagree_set, aspis_sim_result *res,
                            uint64_t *disagree_rows);

/* DETOX, the group-majority scheme Section 5 compares against: K/r groups of
 * r workers (worker u in group u / r), each group's value decided by
 * majority.  Adversaries are placed as in Section 5: WEAK puts the i-th
 * adversary in group i mod (K/r); OPTIMAL (the worst case) fills groups with
 * (r+1)/2 adversaries each.  Writes the number of groups with an adversarial
 * majority and epsilon = groups * r / K.  Requires odd r dividing K,
 * 0 <= q <= K. */
aspis_status aspis_detox(int32_t K, int32_t r, int32_t q, aspis_attack attack,
                         int64_t *distorted_groups, double *epsilon);

/* Message describing the calling thread's last failure ("" if none). */
const char *aspis_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* ASPIS_H */
