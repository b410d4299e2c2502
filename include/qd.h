/*
 * qd.h -- C ABI of the MI355X (gfx950) MAP-Elites generation library, libqd.so.
 *
 * One call of qd_generation() runs one iteration of MAP-Elites after the first
 * (Algorithm 1 of "Accelerated Quality-Diversity through Massive Parallelism",
 * arXiv 2202.01258): uniform selection of parents from the filled cells
 * (Appendix A.2), Iso+LineDD variation (Algorithm 2, Appendix A.2), batched
 * evaluation of the N_B offspring (Appendix A.3 and B.2), descriptor to cell
 * (Appendix A.1) and per-cell insertion that keeps the better solution
 * (Algorithm 1, Appendix A.4).  All of it runs in HIP kernels on the caller's
 * stream; no call here returns control to the host between those steps.
 *
 * Conventions for every entry point:
 *   - Plain C types only.  `stream` is a hipStream_t passed as void* (NULL =
 *     the default stream).  Device pointers are plain void*.
 *   - Every call returns a qd_status; nothing throws across the ABI.
 *   - The caller owns all device memory: one workspace of
 *     qd_layout.workspace_bytes bytes, 256-byte aligned, sized by
 *     qd_layout_query().  The library never allocates or frees device memory.
 *     The library owns only the small host handle made by qd_archive_init().
 *   - A handle is not thread-safe; separate handles (with separate
 *     workspaces) are independent.  Calls on one handle must be ordered on one
 *     stream, or the caller orders the streams.
 *   - Numbers are fp32 except insertion keys (u64) and the statistics (fp64).
 */
#ifndef QD_H
#define QD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define QD_ABI_VERSION 6u

/* Candidate slots per fine bucket of a two-dimensional CVT (see QD_BUF_CAND_*). */
#define QD_CAND_SLOTS 16

/* Rows of the Gaussian sampler's table.  Algorithm 2 draws eps1 ~ N(0, I) and
 * eps2 ~ N(0, 1); each normal comes from one random word x by inversion:
 * k = (x & 0xffffff) + 1, p = k 2^-24, magnitude Phi^-1(1 - p/2), sign = bit
 * 31 of x.
 * Row 16 E + j (E = binary exponent of k, j = its next four bits) holds the
 * coefficients (c0, c1, c2, c3) of a cubic in the remaining 19 bits of k;
 * row 384 (k = 2^24) is zero. */
#define QD_NORMAL_ROWS 385

typedef enum {
  QD_OK = 0,
  QD_ERR_INVALID_ARG = 1,          /* bad config field, null pointer, bad g     */
  QD_ERR_WORKSPACE_TOO_SMALL = 2,  /* workspace shorter than the layout needs   */
  QD_ERR_EMPTY_ARCHIVE = 3,        /* selection found no filled cell            */
  QD_ERR_UNSUPPORTED = 4,          /* valid but not built (e.g. hidden width)   */
  QD_ERR_HIP = 5                   /* a HIP runtime or launch error             */
} qd_status;

/* Tasks (Appendix B.2 test functions; a synthetic policy rollout). */
enum { QD_TASK_RASTRIGIN = 0, QD_TASK_SPHERE = 1, QD_TASK_RASTRIGIN_PROJ = 2,
       QD_TASK_MLP_SYNTH = 3 };
/* Tessellations: regular grid, or nearest of num_cells centroids (CVT). */
enum { QD_TESS_GRID = 0, QD_TESS_CVT = 1 };

typedef struct {
  uint32_t abi_version;   /* QD_ABI_VERSION                                       */
  int32_t task;           /* QD_TASK_*                                            */
  int32_t tess;           /* QD_TESS_*                                            */
  int32_t genotype_dim;   /* n for the test functions; must be 0 for MLP          */
  int32_t batch_size;     /* N_B >= 1                                             */
  int32_t desc_dim;       /* D: 2 for the test functions, 4 for MLP               */
  int32_t grid_shape[4];  /* grid: bins per dimension; prod == num_cells          */
  int32_t num_cells;      /* C                                                    */
  float desc_lo[4];       /* descriptor box; the CVT maps it onto [0,1]^D and    */
  float desc_hi[4];       /*   the test-function descriptors are clipped to it    */
  float iso_sigma;        /* sigma_1 of Algorithm 2                               */
  float line_sigma;       /* sigma_2 of Algorithm 2                               */
  float init_lo, init_hi; /* first batch of the test functions: U[lo, hi)        */
  int32_t mlp_obs;        /* policy: observation size (27)                        */
  int32_t mlp_hidden;     /*         hidden width (64 or 128)                     */
  int32_t mlp_act;        /*         actions (8)                                  */
  int32_t episode_len;    /*         rollout steps T                              */
  int32_t keep_offspring; /* 1: also store every offspring genotype (tests)       */
  int32_t cvt_samples;    /* CVT: Lloyd iterations over this many uniform points  */
  int32_t cvt_iters;      /*   at set-up (0, 0: centroids stay uniform draws);    */
                          /*   0 <= cvt_samples <= 2^28, 0 <= cvt_iters <= 10^4,  */
                          /*   both 0 for the grid                                */
  int32_t death_mode;     /* policies (Appendix A.3, A.4 i): 0 full episodes;    */
                          /*   1 an episode ends at the first new state whose    */
                          /*   component 0 is below death_below, that step and   */
                          /*   the rest counting for nothing (return and         */
                          /*   descriptor over the states before it); 2 as 1,    */
                          /*   and every failed solution gets a NaN objective    */
                          /*   (never inserted).  In 1 and 2 an episode with no  */
                          /*   state before its failure gets a NaN objective and  */
                          /*   descriptor 0.  Must be 0 for the test functions.  */
  float death_below;      /*   the failure threshold (any non-NaN value)          */
  int32_t init_mode;      /* test functions' first batch: 0 every gene U[init_lo, */
                          /*   init_hi); 1 ("spread") individual j also draws one  */
                          /*   level per genotype half h (genes [0, n/2) and      */
                          /*   [n/2, n)), desc_lo[h] + U (desc_hi[h] - desc_lo[h]),*/
                          /*   added to every gene of that half, so the first     */
                          /*   batch covers the descriptor box even where a       */
                          /*   descriptor averages many genes.  Must be 0 for MLP. */
  uint64_t seed;          /* key of every Philox4x32-10 stream                    */
} qd_config;

/* Workspace buffers, in layout order.  Offsets/sizes are in bytes.  The
 * archive's state between generations is ARCHIVE_KEY .. ARCHIVE_GENO,
 * OCC_LIST and COUNTERS: copied out together with the next generation index
 * and written into the workspace of a fresh archive of the same
 * configuration (after its qd_archive_init), they let the run continue bit
 * for bit (checkpoint and resume). */
enum {
  QD_BUF_ARCHIVE_KEY = 0,  /* u64 [C]   0 = empty; else (order(f) << 32) | 0xFFFFFFFF */
  QD_BUF_ARCHIVE_FIT,      /* f32 [C]   objective of the elite (NaN when empty)       */
  QD_BUF_ARCHIVE_DESC,     /* f32 [C][D]                                              */
  QD_BUF_ARCHIVE_SLOT,     /* u32 [C]   which genotype bank (0/1) holds the elite     */
  QD_BUF_ARCHIVE_GENO,     /* f32 [2][C][row_stride] two genotype banks               */
  QD_BUF_CENTROIDS,        /* f32 [C][D] CVT centroids                                */
  QD_BUF_BUCKET_START,     /* i32 [num_buckets + 1] CVT bucket offsets                */
  QD_BUF_BUCKET_ITEMS,     /* f32x4 + i32: bucketed centroid copies and indices       */
  QD_BUF_CAND_COUNT,       /* i32 [cand_buckets] D = 2 CVT: how many centroids can be  */
                           /*   nearest to some point of each fine bucket             */
  QD_BUF_CAND_PTS,         /* f32x4 [cand_buckets][QD_CAND_SLOTS] those centroids, in  */
                           /*   ascending index: (x, y, index bits, 0); a bucket with  */
                           /*   more than QD_CAND_SLOTS uses the ring search instead   */
  QD_BUF_LLOYD_ACC,        /* u64 [C][D + 1] Lloyd point sums and counts (set-up)     */
  QD_BUF_ENV,              /* f32: A [obs][obs], B [obs][act], s0 [obs]               */
  QD_BUF_OCC_LIST,         /* i32 [C]   filled cells, ascending                       */
  QD_BUF_COUNTERS,         /* i32 [64]  [0] filled cells, [1] flags, [3] internal     */
  QD_BUF_OFF_PARENTS,      /* i32 [N_B][2] parent cells of the last batch            */
  QD_BUF_OFF_FIT,          /* f32 [N_B]                                               */
  QD_BUF_OFF_DESC,         /* f32 [N_B][D]                                            */
  QD_BUF_OFF_CELL,         /* i32 [N_B] cell, -1 = invalid (never inserted)          */
  QD_BUF_OFF_WON,          /* u8  [N_B] 1 = holds its cell after the batch           */
  QD_BUF_OFF_KEY,          /* u64 [N_B] insertion key (0 = not inserted)              */
  QD_BUF_OFF_BANK,         /* u8  [N_B] genotype banks of parent 1 (bit 0), 2 (bit 1) */
  QD_BUF_OFF_GENO,         /* f32 [N_B][row_stride] (keep_offspring only)            */
  QD_BUF_STATS,            /* f64 [8]   device-side statistics                        */
  QD_BUF_NORMAL_TAB,       /* f32x4 [QD_NORMAL_ROWS] Gaussian sampler table, written  */
                           /*   by qd_archive_init (see QD_NORMAL_ROWS)               */
  QD_NUM_BUFFERS
};

typedef struct {
  uint64_t workspace_bytes;
  uint64_t offset[QD_NUM_BUFFERS];
  uint64_t bytes[QD_NUM_BUFFERS];
  int32_t genotype_dim;    /* n (derived for MLP: h*obs + h + h*h + h + act*h + act) */
  int32_t row_stride;      /* floats between genotype rows (multiple of 64)          */
  int32_t bucket_res;      /* CVT buckets per dimension (0 for the grid)             */
  int32_t num_buckets;
  int32_t cand_res;        /* D = 2 CVT with C <= 65536: fine buckets per dimension,  */
  int32_t cand_buckets;    /*   largest R with R^2 <= 4 C (else both 0)               */
} qd_layout;

typedef struct {
  double qd_score;         /* sum over filled cells of (f + qd_offset), Eq. 1        */
  double coverage;         /* filled cells / C                                       */
  float best_fitness;      /* max f over filled cells (NaN when empty)               */
  int32_t num_occupied;
  uint32_t flags;          /* bit 0: a generation found the archive empty            */
  int32_t reserved;
} qd_stats;

typedef struct qd_archive qd_archive;

/* Kernels whose durations qd_kernel_times() reports. */
enum { QD_K_VARY_EVAL = 0, QD_K_ROLLOUT, QD_K_INSERT, QD_K_REGEN, QD_K_SETUP,
       QD_NUM_KERNELS };

/* Validates *cfg and fills *out with the workspace layout.  Host only; no GPU
 * work.  QD_ERR_INVALID_ARG for an inconsistent config (task/tessellation/D
 * mismatch, grid product != num_cells, n <= 0, N_B <= 0, genotype_dim != 0 for
 * MLP, sizes overflowing 64 bits), QD_ERR_UNSUPPORTED for a valid config this
 * build has no kernel for. */
qd_status qd_layout_query(const qd_config* cfg, qd_layout* out);

/* Creates an archive in the caller's workspace and enqueues its first
 * iteration on `stream` (Algorithm 1, random solutions): CVT centroids (uniform
 * draws, then cvt_iters Lloyd iterations over cvt_samples uniform points: each
 * point to its nearest centroid, each centroid that received points to their
 * mean) and the synthetic environment from their Philox streams, an empty
 * archive, N_B random genotypes evaluated and inserted.  The Gaussian sampler's
 * table (QD_BUF_NORMAL_TAB) is built on the host (once per process, about
 * 10 ms the first time) and written into the workspace on `stream`, ahead of
 * that work, by kernels that receive it as arguments.  Asynchronous: returns
 * once the work is enqueued.  *out receives a host handle owned by the library (free it
 * with qd_archive_destroy).  The workspace must stay valid until then. */
qd_status qd_archive_init(const qd_config* cfg, void* d_workspace, uint64_t workspace_bytes,
                          void* stream, qd_archive** out);

/* Enqueues generation gen_index (>= 1) on `stream`: select, vary, evaluate,
 * map to cells, insert.  gen_index keys every Philox stream of the generation,
 * so replaying a generation from the same archive state reproduces it exactly.
 * Asynchronous: no host synchronisation.  The per-offspring buffers
 * (QD_BUF_OFF_*) hold this batch until the next call.  An archive found empty
 * on the device sets flag bit 0 (reported by qd_archive_stats) and inserts
 * nothing. */
qd_status qd_generation(qd_archive* h, uint32_t gen_index, void* stream);

/* Enqueues generations first_gen, first_gen + 1, ..., first_gen + count - 1
 * on `stream`, in order: the same work as that many qd_generation() calls,
 * without a return to the caller between them (Algorithm 1's loop).  count 0
 * enqueues nothing.  QD_ERR_INVALID_ARG for a null handle, first_gen 0 or a
 * last index beyond 2^32 - 1, before any launch; a launch failure stops the
 * run and returns QD_ERR_HIP.  Asynchronous, like qd_generation(). */
qd_status qd_generations(qd_archive* h, uint32_t first_gen, uint32_t count, void* stream);

/* QD-score (Eq. 1) with each filled cell's objective shifted by qd_offset,
 * coverage and best objective (Appendix B.1), computed on the device and
 * copied into *out.  Synchronises `stream` (the only call that does). */
qd_status qd_archive_stats(qd_archive* h, double qd_offset, void* stream, qd_stats* out);

/* For callers that cannot allocate device memory or use workspace memory at
 * this point (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation): the same statistics as qd_archive_stats(), staged
 * on the device in the library's own scratch (a file-scope device array of
 * 256 bytes, one per GPU, held until the process ends) instead of the
 * workspace's statistics buffer.  Allocates nothing (no hipMalloc, hipFree or
 * allocating library call).  The scratch holds four results whatever the
 * archive's size, so no archive is too large for it.  The handle's device
 * (the one current at qd_archive_init) must be current: QD_ERR_INVALID_ARG
 * otherwise, and for a null handle or out.  Synchronises `stream`.  Every
 * call on one GPU shares that GPU's scratch, which keeps the last call's
 * results: calls that overlap on one GPU (several host threads, or streams
 * not ordered with one another) race. */
qd_status qd_archive_stats_noalloc(qd_archive* h, double qd_offset, void* stream, qd_stats* out);

/* The layout the handle was created with. */
qd_status qd_archive_layout(const qd_archive* h, qd_layout* out);

/* Host only, no GPU work: copies the Gaussian sampler's table, the one
 * qd_archive_init writes into QD_BUF_NORMAL_TAB, into out (QD_NORMAL_ROWS rows
 * of 4 floats, c0 .. c3, row-major; host memory owned by the caller).  The
 * table is built on the first call in the process (fp64 quantiles of the
 * half-normal law interpolated at Chebyshev points, rounded once to fp32).
 * QD_ERR_INVALID_ARG for a null pointer. */
qd_status qd_normal_table(float* out);

/* Standard normals from the archive's Gaussian sampler, the one Algorithm 2's
 * eps1 and eps2 come from in every generation (inversion through the table
 * described at QD_NORMAL_ROWS): d_out[i] = the normal of the 32-bit word
 * d_words[i] for i < count.  For checking the sampler on chosen words; the
 * generations do not call it.  d_words (u32) and d_out (f32) are device
 * memory owned by the caller, 4-byte aligned, each of count elements.
 * QD_ERR_INVALID_ARG for a null handle, a null or misaligned pointer with
 * count > 0, or count > 2^32; count 0 is a no-op.  Asynchronous on `stream`,
 * which must be ordered after the stream qd_archive_init used (the table is
 * written there). */
qd_status qd_sample_normals(const qd_archive* h, const void* d_words, void* d_out, uint64_t count,
                            void* stream);

/* Selects the kernels whose launches carry a pair of HIP events on the launch
 * stream (hipExtLaunchKernelGGL: the runtime stamps them when the dispatch
 * begins and ends): bit k of kernel_mask is kernel QD_K_k (0 = no timing, the
 * default).  The handle keeps every timed launch's events until
 * qd_kernel_times() collects them (two events per launch), so a caller that
 * times many launches collects periodically.  QD_ERR_INVALID_ARG for bits
 * beyond QD_NUM_KERNELS. */
qd_status qd_set_kernel_timing(qd_archive* h, uint32_t kernel_mask);

/* Waits for the recorded events and returns, per QD_K_* kernel, the summed
 * duration in ms and the number of launches since the last call; then clears
 * them.  ms and counts must hold QD_NUM_KERNELS entries. */
qd_status qd_kernel_times(qd_archive* h, double* ms, int32_t* counts);

/* Self-check of the short division sequences the kernels use in place of
 * IEEE division, over every input each can receive: mismatches[0] counts the
 * fp32 inputs of tanh (all 2^32) whose result differs from the IEEE-arithmetic
 * definition, mismatches[1] those of sigmoid in [-1, 1] (zeros mean
 * bit-identical results).  d_scratch: 16 bytes of device memory owned by the
 * caller, 8-byte aligned.  Synchronises `stream`. */
qd_status qd_check_fast_arith(void* d_scratch, void* stream, uint64_t* mismatches);

/* Frees the host handle (not the workspace).  NULL is accepted. */
qd_status qd_archive_destroy(qd_archive* h);

/* Static description of a status; for QD_ERR_HIP, of the last HIP error the
 * library saw on this thread. */
const char* qd_status_str(qd_status s);

#ifdef __cplusplus
}
#endif
#endif
