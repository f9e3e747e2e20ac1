/*
 * embx -- multi-table embedding-bag lookup with sum pooling for DLRM inference
 * on one AMD Instinct MI355X (gfx950).
 *
 * The operation (Ruggeri et al., "Deep Recommender Models Inference: Automatic
 * Asymmetric Data Flow Optimization", Sec. II-B; sum reduction per Sec. IV-A):
 * for every sample b of a batch and every table t (m_t rows of E elements),
 * look up the bag of rows the sample names in that table and reduce them to
 * one E-vector:
 *
 *     out[b, t, :] = sum over k in bag(t, b) of  W_t[indices[k], :]
 *
 * Sec. II-B also names averaging: a table may be mean-pooled (the bag's sum over
 * its length n_bt), and each lookup may carry a weight w_k that scales its row
 * (emb_lookup_weighted): out[b, t, :] = (1 or 1/n_bt) * sum of w_k W_t[indices[k], :].
 *
 * Planning follows Sec. III: a linear cost model (Eq. (2)) scores each table
 * under four per-core data flows and a greedy algorithm maps tables, row chunks
 * and batch slices asymmetrically onto the GPU's workers (Sec. III-B steps 1-4,
 * with the LIF fallback to symmetric partitioning of Sec. III-A).
 *
 * All functions return an emb_status_t (0 = EMB_OK); no C++ exception crosses
 * this interface.  Pointers documented as "device" must point to device memory
 * of the current HIP device; "host" pointers are read during the call only.
 * A "stream" argument is a hipStream_t passed as void* (NULL = null stream).
 */
#ifndef EMBX_H
#define EMBX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EMB_OK = 0,
  EMB_ERR_INVALID_ARGUMENT = 1,   /* bad pointer, size, shape, option or statistic   */
  EMB_ERR_UNSUPPORTED = 2,        /* E / dtype / size outside what the kernels handle */
  EMB_ERR_OUT_OF_MEMORY = 3,      /* device allocation at plan creation failed        */
  EMB_ERR_DEVICE = 4,             /* a HIP runtime call failed                        */
  EMB_ERR_NOT_BOUND = 5,          /* lookup before emb_plan_bind_weights              */
  EMB_ERR_INDEX_OUT_OF_RANGE = 6, /* emb_plan_check_errors found bad indices          */
  EMB_ERR_BUFFER_TOO_SMALL = 7    /* serialization buffer too small (len_out is set)  */
} emb_status_t;

typedef enum { EMB_DTYPE_F32 = 0, EMB_DTYPE_F16 = 1 } emb_dtype_t;

/* Reduction of a table's bags (Sec. II-B): the sum, or the sum over the bag length
 * (an empty bag gives +0.0 either way; an out-of-range index adds nothing but counts
 * in the length). */
typedef enum { EMB_POOL_SUM = 0, EMB_POOL_MEAN = 1 } emb_pooling_t;

/* Per-table data flows (Sec. II-B mapped onto a CU):
 *   LDS    -- the table, or a row chunk of it (Sec. III-B), staged into LDS and read from there
 *             (the paper's L1 / L1-UB flows; LDS does not persist across launches, so the
 *             staging is paid by every launch);
 *   HOT    -- the table's hottest rows staged into LDS behind an LDS hash of their ids; misses
 *             gather from HBM;
 *   DEDUP  -- each tile of indices is sorted, each distinct row fetched once into LDS, bags
 *             read their rows from there;
 *   GATHER -- one row per sub-wavefront straight from HBM with 16-byte loads (the GM flow);
 *   STREAM -- the whole table moves through LDS in chunks of floor(L / R) rows on one worker,
 *             each chunk serving the slice's lookups that fall in it (the GM-UB flow);
 *             partial sums are added onto the output in chunk order. */
typedef enum {
  EMB_STRAT_AUTO = -1,
  EMB_STRAT_LDS = 0,
  EMB_STRAT_HOT = 1,
  EMB_STRAT_DEDUP = 2,
  EMB_STRAT_GATHER = 3,
  EMB_STRAT_STREAM = 4
} emb_strategy_t;

/* Cost-model coefficients (Eq. (2) extended per strategy), picoseconds.  Layout of
 * emb_plan_options_t.beta: per-item (*0), per-lookup (*1, P, I), per staged byte (S; SH for
 * the hot rows, which are fetched by id rather than copied as a block).
 *   gather  = G0 + G1*lam
 *   lds     = L0 + S*(rows*R) + L1*lam
 *   chunk   = L0 + S*(rows*R) + I*lam + L1*lam/c
 *   hot     = H0 + SH*(C*R) + lam*(P + h*L1 + (1-h)*G1)
 *   dedup   = D0 + D1*lam + G1*u*lam
 *   stream  = L0 + S*(m*R) + I*lam*c + L1*lam   (c = ceil(m / floor(L / R)), m the table rows)
 * with lam the expected lookups of the slice, R the row bytes, c the chunk count,
 * C the hot rows staged, h the fraction of lookups they catch, u the unique fraction. */
enum {
  EMB_BETA_G0 = 0, EMB_BETA_G1, EMB_BETA_L0, EMB_BETA_L1, EMB_BETA_S, EMB_BETA_I,
  EMB_BETA_H0, EMB_BETA_P, EMB_BETA_D0, EMB_BETA_D1, EMB_BETA_SH, EMB_BETA_COUNT
};

#define EMB_MAX_HOT_STATS 4096   /* hot rows a table's statistics may list     */
#define EMB_MAX_HOT_SLOTS 2048   /* hot rows one HOT item stages at most        */
#define EMB_MAX_E 256

/* Per-table index statistics: the paper's S (sequence lengths) and I (query
 * distribution), Sec. III-A.  Measured on a representative batch. */
typedef struct {
  double mean_pooling;      /* s_t >= 0: mean lookups per bag                                   */
  int32_t max_pooling;      /* upper bound on lookups per bag; 0 = unknown.  Exactly 1 lets the
                               gather path store each bag's single row as its output (a bag that
                               holds more at run time is still summed, on a slower path); any
                               other value, 0 included, walks bags as sums                        */
  int32_t n_hot;            /* entries in hot_rows / hot_freq, 0..EMB_MAX_HOT_STATS             */
  const int64_t* hot_rows;  /* host, hottest first, distinct, each in [0, rows)                 */
  const double* hot_freq;   /* host, fraction of the table's lookups that hit each hot row       */
  double unique_frac;       /* distinct rows / lookups in a batch, in (0, 1]; <= 0 = unknown      */
} emb_table_stats_t;

typedef struct {
  int32_t wg_per_cu;        /* workers per CU; 0 -> 1.  K = CUs * wg_per_cu unless num_workers   */
  int32_t lds_budget_bytes; /* L, LDS bytes for staged rows per worker; 0 -> 131072 (capped by
                               the device's LDS per workgroup minus a 28 KiB metadata reserve)   */
  int32_t lif_milli;        /* LIF threshold x 1000 (Sec. III-B step 4); 0 -> 1500               */
  int32_t order_mode;       /* 0 = longest first with the paper's keys as tie-breaks;
                               1 = the paper's order (s desc, m asc)                             */
  int64_t chunk_max_bytes;  /* max row-chunk bytes (Sec. III-B); <= 0 -> lds_budget_bytes      */
  const double* beta;       /* host, EMB_BETA_COUNT finite non-negative coefficients (picoseconds);
                               NULL -> built-in MI355X fit (emb_default_beta); negative: invalid */
  const int32_t* force_strategy; /* host, T entries of emb_strategy_t, or NULL (all AUTO)        */
  int32_t num_workers;      /* > 0 overrides K (must not exceed 65535)                          */
  int32_t sym_max_gather;   /* 0: a GATHER table is split over all workers (symmetric partitioning,
                               Sec. III-A) when each slice would hold >= 64 expected lookups, else
                               placed by cost like the rest (Sec. III-B); > 0: also every GATHER
                               table while the plan has at most this many; < 0: never            */
  const int32_t* pooling;   /* host, T entries of emb_pooling_t, or NULL (all SUM); does not change
                               the placement, only each bag's final scaling                       */
  int32_t no_replication;   /* 1: no batch splits of any item (replication fixed to 1, as the
                               paper's solver does, Sec. III-B); with order_mode 1 the plan is
                               Sec. III-B steps 1-4 as printed; 0: splits allowed (default)       */
  const double* gather_lookup_ps; /* host, T entries or NULL: table t's cost of one lookup served
                               from memory in picoseconds (beta's G1 for that table: its gathers,
                               HOT misses and DEDUP's distinct rows), fitted on the device for the
                               table's size and query distribution (Sec. III-A fits the model per
                               configuration); 0 -> beta's G1; negative or non-finite: invalid   */
} emb_plan_options_t;

typedef struct emb_plan emb_plan_t;   /* opaque */

typedef struct {
  int32_t num_tables, embedding_dim, dtype, row_bytes;
  int32_t num_workers;      /* K = grid size of every lookup launch            */
  int32_t block_threads;    /* threads per worker                              */
  int32_t lds_bytes;        /* dynamic LDS per worker                          */
  int32_t num_items;        /* slices in the plan                              */
  int32_t max_batch;
  int32_t lds_budget_bytes;
  int64_t max_load_ps, sum_load_ps;
  int32_t lif_milli, r_symmetric;
  int32_t n_strategy[5];    /* slices per strategy (emb_strategy_t order)      */
  int32_t gather_runs[3];   /* gather slices over all workers' queues: a wavefront per bag
                               (long bags), single-lookup bags (max_pooling == 1), SW sums */
  int32_t kernel;           /* 0: the staged kernel (lookup_kernel, any plan); 1: the
                               wave-uniform gather kernel (gather_kernel; gather-only plans
                               with rows of 256, 512 or 1024 bytes)                        */
  int32_t debug_checks;     /* 1: made with EMBX_DEBUG_CHECKS set -- every launch first checks
                               its offsets (offsets[0] = 0, non-decreasing, within the indices'
                               and weights' allocations; else EMB_ERR_INVALID_ARGUMENT, nothing
                               launched) and reports out-of-range ids on stderr; synchronous  */
  int32_t gather_steps;     /* gather_kernel: row loads in flight per lane per step (12, 13 or
                               16: the fewest row rounds over the plan's multi-lookup chunks,
                               ties to the larger, 12 without such chunks; EMBX_GATHER_STEPS
                               overrides it); 0 for lookup_kernel                             */
} emb_plan_info_t;

/* Builds a plan for T tables of rows[t] x E elements of `dtype`, for batches of up to
 * max_batch samples, on the current HIP device (Sec. III-A problem statement: N, M, S, B,
 * K, I, L; the policy of Eq. (1) chosen with the cost model of Eq. (2) and mapped onto the
 * workers by Sec. III-B steps 1-4).  Host-side work plus one upload of the plan's metadata;
 * allocates the device workspace for row-chunk partial sums ([chunks, max_batch, E] fp32 per
 * row-chunked table).  No workspace grows with the number of indices: the kernels read
 * indices and offsets in place, and a DEDUP tile is sorted in LDS, so the plan needs no
 * index count.  rows[t] in [1, 2^31); E a multiple of 4 (fp32) or
 * 8 (fp16), E <= 256; opts may be NULL.  On success *plan_out owns everything it allocated.
 * EMB_ERR_UNSUPPORTED when a worker would hold more gather slices than its run queue in
 * LDS takes (48 B each, about 3,400 in 160 KiB): with every table split over all workers,
 * more than ~3,400 tables; such plans need sym_max_gather < 0 (tables placed whole).
 * Environment (debugging, read at each creation): EMBX_LOG (not "0") prints the plan in one
 * line on stderr -- strategies, LIF, predicted makespan, kernel; EMBX_FORCE_STRATEGY = lds,
 * hot, dedup, gather or stream forces every table to that strategy over opts (any other
 * non-empty value: EMB_ERR_INVALID_ARGUMENT; emb_plan_text honours it too);
 * EMBX_DEBUG_CHECKS (not "0") makes every launch check its input first
 * (emb_debug_check_input). */
emb_status_t emb_plan_create(emb_plan_t** plan_out, int32_t num_tables, const int64_t* rows,
                             int32_t embedding_dim, emb_dtype_t dtype,
                             const emb_table_stats_t* stats, int32_t max_batch,
                             const emb_plan_options_t* opts);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): emb_plan_create with the plan's device
 * data -- run queues, slice list, hot-row hashes, combine and error counters, row-chunk
 * partial sums -- placed in a fixed array of EMB_NOALLOC_SCRATCH_BYTES that the library
 * holds on every GPU it runs on until the process ends; no hipMalloc or hipFree is called
 * (the plan's metadata is copied into the array, synchronously).  The array is one per GPU
 * and shared by every such call: a later emb_plan_create_noalloc on the same device
 * replaces the plan in it, and the earlier handle then fails with EMB_ERR_INVALID_ARGUMENT
 * (emb_plan_destroy still frees its host part).  Lookups of such a plan must not overlap
 * another call that uses the array on that device.  EMB_ERR_UNSUPPORTED when the plan's
 * device data exceed the array; otherwise the same arguments, results and errors as
 * emb_plan_create. */
#define EMB_NOALLOC_SCRATCH_BYTES (64u << 20)
emb_status_t emb_plan_create_noalloc(emb_plan_t** plan_out, int32_t num_tables, const int64_t* rows,
                                     int32_t embedding_dim, emb_dtype_t dtype,
                                     const emb_table_stats_t* stats, int32_t max_batch,
                                     const emb_plan_options_t* opts);

/* Records the T device pointers of the tables: the paper's lookup tables of m_i rows of E
 * elements (Sec. II-B), weights[t] -> rows[t] x E contiguous, row-major, 16-byte aligned.
 * The caller keeps ownership and keeps them alive.  Copies the pointers into the plan's
 * device metadata (synchronous). */
emb_status_t emb_plan_bind_weights(emb_plan_t* plan, const void* const* weights);

/* One batch of the embedding-bag lookup of Sec. II-B (each sample's bag of rows per table,
 * reduced per Sec. IV-A by summation).  indices: device int64 [offsets[T*batch]], table-local row ids;
 * offsets: device int64 [T*batch + 1], table-major CSR (bag (t, b) is
 * indices[offsets[t*batch+b] .. offsets[t*batch+b+1]) ), offsets[0] = 0, non-decreasing;
 * out: device fp32 [batch, T, E].  Enqueues exactly one kernel on `stream`; never
 * allocates or synchronizes.  batch == 0 is a no-op.  An index outside [0, rows[t])
 * contributes nothing and is counted (see emb_plan_check_errors).  Empty bags give +0.0.
 * Calls on one plan must not overlap (the chunk workspace is per plan). */
emb_status_t emb_lookup(emb_plan_t* plan, const int64_t* indices, const int64_t* offsets,
                        int32_t batch, float* out, void* stream);

/* emb_lookup with per-lookup weights (per-sample weights): weights is device fp32
 * [offsets[T*batch]], 4-byte aligned, aligned element for element with indices; lookup k
 * adds weights[k] * W_t[indices[k], :] to its bag, computed as one fused multiply-add per
 * element in fp32 (before the division of a mean-pooled table).  A weight of an
 * out-of-range index is ignored.  NULL weights is an invalid argument.  Same launch, stream
 * and overlap rules as emb_lookup. */
emb_status_t emb_lookup_weighted(emb_plan_t* plan, const int64_t* indices, const int64_t* offsets,
                                 const float* weights, int32_t batch, float* out, void* stream);

/* Range errors.  Sec. III-B subtracts a chunk's first row from each index and clips the
 * result so that every address stays inside the chunk; an index outside the table itself
 * is never read here: it adds nothing and is counted on the device.  This call
 * synchronizes `stream`, returns the number of out-of-range indices seen since the last
 * call in *n_bad (may be NULL) and resets the counter; EMB_ERR_INDEX_OUT_OF_RANGE if any. */
emb_status_t emb_plan_check_errors(emb_plan_t* plan, void* stream, int64_t* n_bad);

/* Canonical text of the plan: the policy of Eq. (1) (a data flow per table) and its
 * mapping onto workers (Sec. III-B), one line per slice: worker, table, strategy, chunk,
 * chunks, first row, end row, split, slice, hot rows, cost in ps.  Writes at most cap bytes
 * (NUL-terminated when it fits); *len_out = text length without the NUL. */
emb_status_t emb_plan_serialize(const emb_plan_t* plan, char* buf, size_t cap, size_t* len_out);

/* Plan summary (the same plan as emb_plan_serialize): shapes, launch shape, slices per
 * strategy, the predicted makespan and the load imbalance factor of Sec. III-B step 4. */
emb_status_t emb_plan_get_info(const emb_plan_t* plan, emb_plan_info_t* info);

/* Per-slice timers for fitting the cost model (Sec. III-A: the coefficients of Eq. (2) are
 * fitted by least squares on hardware measurements).  With trace != NULL (device, at least
 * *needed uint64 entries, 8-byte aligned) every following emb_lookup on this plan records
 * 100 MHz real-time counter ticks:
 *   worker w (w < K):  trace[w*18 + 0] start, [w*18 + 1] end of its staged slices,
 *                      [w*18 + 2 + v] end of wavefront v (v < 16);
 *   slice i in emb_plan_serialize order:  trace[K*18 + 2i] begin, [K*18 + 2i + 1] end
 *                      (staged slices only; gather slices run merged per worker).
 * Timed lookups add one workgroup barrier per staged slice.  trace == NULL switches the
 * timers off; *needed (may be NULL) receives the required entry count either way. */
emb_status_t emb_plan_set_trace(emb_plan_t* plan, uint64_t* trace, size_t capacity, size_t* needed);

/* Frees the plan's device and host memory.  NULL is a no-op. */
emb_status_t emb_plan_destroy(emb_plan_t* plan);

/* Host-only planner: the same plan text emb_plan_create would produce for
 * num_workers workers (no device call; lds_budget_bytes 0 -> 131072). */
emb_status_t emb_plan_text(int32_t num_tables, const int64_t* rows, int32_t embedding_dim,
                           emb_dtype_t dtype, const emb_table_stats_t* stats, int32_t max_batch,
                           int32_t num_workers, const emb_plan_options_t* opts, char* buf,
                           size_t cap, size_t* len_out);

/* The built-in cost coefficients (the MI355X fit of Eq. (2), Sec. III-A) used when
 * emb_plan_options_t.beta is NULL, for rows of row_bytes bytes: writes EMB_BETA_COUNT
 * picosecond values to out (host, n >= EMB_BETA_COUNT entries).  Host only.
 * EMB_ERR_INVALID_ARGUMENT if out is NULL, n is too small or row_bytes < 1. */
emb_status_t emb_default_beta(int32_t row_bytes, double* out, int32_t n);

const char* emb_status_string(emb_status_t s);

/* ---- input checks (debugging) ----------------------------------------------------------
 * The checks every launch of a plan made with the environment variable EMBX_DEBUG_CHECKS
 * set (not "0") runs first (emb_plan_info_t.debug_checks = 1), callable on their own: the
 * launch's input as emb_lookup (weights NULL) or emb_lookup_weighted takes it.  Returns
 * EMB_ERR_INVALID_ARGUMENT, with the first fault on stderr, if offsets[0] != 0, offsets
 * decrease, or offsets[T*batch] indices (or weights) run past the device allocation that
 * holds them (the extent hipMemGetAddressRange reports: a caching allocator's whole
 * segment); ids outside their table are listed on stderr (first five) and not an error
 * (the kernels skip and count them).  Synchronises `stream`, copies offsets and indices to
 * the host, launches nothing.  EMB_ERR_INVALID_ARGUMENT also for a NULL plan, indices or
 * offsets, or batch outside [1, max_batch]. */
emb_status_t emb_debug_check_input(const emb_plan_t* plan, const int64_t* indices, const int64_t* offsets,
                                   const float* weights, int32_t batch, void* stream);

/* ---- index-handling probes (tests of the exact integer work) ---------------------------
 * Both run the same device functions as emb_lookup on one workgroup. */

/* Sorts and deduplicates one tile of n <= 2048 row ids (device int64, each in [0, 2^31)):
 * uniq (device int32 [n]) gets the distinct ids ascending, inv (device int32 [n]) the slot
 * of each input in uniq, *n_uniq (device int32) the count. */
emb_status_t emb_debug_dedup_tile(const int64_t* idx, int32_t n, int32_t* uniq, int32_t* inv,
                                  int32_t* n_uniq, void* stream);

/* Probes table t's LDS hot-row hash of a HOT plan for n ids (device int64): slot (device
 * int32 [n]) = position of the id among the table's first C hot rows, or -1.
 * EMB_ERR_INVALID_ARGUMENT if no HOT item of table t exists. */
emb_status_t emb_debug_hot_probe(const emb_plan_t* plan, int32_t table, const int64_t* idx,
                                 int32_t n, int32_t* slot, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* EMBX_H */
