/*
 * emb_cache.h -- C ABI of the MI355X library for the cached mixed-precision
 * EmbeddingBag training step of "Mixed-Precision Embedding Using a Cache".
 *
 * The method (Sec. 3 of the paper): each embedding table T is stored in a
 * precision lower than FP32 -- FP16 elements, or INT8, INT4 or INT2 codes with
 * one (scale, bias) pair per row ("Precision" knob, row-wise uniform min-max
 * quantization) --
 * and is augmented with an FP32 cache C of n sets x alpha ways ("Cache
 * Structure" knob).  fetch(T,C,i) returns the FP32 cache row when row i is
 * resident in set h(i), else the up-converted low-precision row;
 * update(T,C,i,x) writes an updated FP32 row back either into the cache or,
 * after down-conversion by round-to-nearest-even or stochastic rounding
 * ("Rounding" knob), into T, under the LRU/LFU admission rule of the "Cache
 * Replacement Policy" knob and Alg. 2.  Gradients of the rows of a mini-batch
 * are sorted by row and merged before the update (Sec. 5.1, "De-duplicate
 * gradients").
 *
 * Conventions for every call:
 *   - Every function returns an int status (EMB_OK or an EMB_E* code); no
 *     C++ exception crosses the ABI.  A handle is used by one thread at a time.
 *   - Device memory is owned by the caller.  The library never allocates
 *     device memory: the caller passes one state buffer and one workspace
 *     buffer (sizes from emb_cache_query_sizes) that must stay allocated until
 *     emb_cache_destroy.  The handle itself owns host metadata only.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Calls marked "enqueue-only" return after enqueueing kernels; their device
 *     inputs must stay unmodified until the stream has reached the call.
 *   - Errors found on the device (an index outside [0, rows[t])) do not abort
 *     the kernels: the lookup is skipped (contributes nothing, updates
 *     nothing) and a device flag is set; the next syncing call that checks it
 *     (emb_cache_check) returns EMB_EINDEX.
 */
#ifndef EMB_CACHE_H
#define EMB_CACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------------- */
#define EMB_OK 0
#define EMB_EINVAL 1 /* invalid argument or configuration */
#define EMB_ENOMEM 2 /* a caller buffer is smaller than required */
#define EMB_EINDEX 3 /* a kernel saw an index outside [0, rows[t]) or bad offsets */
#define EMB_EHIP 4   /* a HIP runtime call failed */

/* ---- knobs (Sec. 3) ---------------------------------------------------------- */
#define EMB_FP16 16 /* precision: IEEE binary16 elements, no scale/bias (sb_dtype is ignored) */
#define EMB_INT8 8  /* precision: codes in [0, 255], one byte per element */
#define EMB_INT4 4  /* precision: codes in [0, 15], two per byte, even column in the low nibble */
#define EMB_INT2 2  /* precision: codes in [0, 3], four per byte, column 4k+i in bits 2i..2i+1 of byte k */
#define EMB_SB_FP32 0 /* per-row (scale, bias) stored as FP32 (the paper's choice) */
#define EMB_SB_FP16 1 /* per-row (scale, bias) rounded to FP16 (nearest even) */
#define EMB_LRU 0 /* priority = step of last access, per cached row */
#define EMB_LFU 1 /* priority = access count, per embedding row */
#define EMB_ROUND_NEAREST 0
#define EMB_ROUND_STOCHASTIC 1
#define EMB_OPT_SGD 0             /* x <- x - lr*g (Sec. 3) */
#define EMB_OPT_ROWWISE_ADAGRAD 1 /* G += mean(g^2); x <- x - lr/(sqrt(G)+eps)*g */

/* ---- statistics, per table, as returned by emb_cache_get_stats ---------------- */
#define EMB_NSTAT 12
#define EMB_STAT_LOOKUPS 0       /* valid lookups seen by the last forward */
#define EMB_STAT_HIT_LOOKUPS 1   /* ... of which served from the FP32 cache */
#define EMB_STAT_BWD_LOOKUPS 2   /* valid lookups seen by the last backward_update */
#define EMB_STAT_UNIQUE 3        /* unique rows updated */
#define EMB_STAT_UNIQUE_HITS 4   /* ... of which resident before the step */
#define EMB_STAT_INSERTS 5       /* missed rows placed in the cache */
#define EMB_STAT_BYPASSES 6      /* missed rows written to the low-precision table */
#define EMB_STAT_EVICTIONS 7     /* valid residents displaced (includes hit evictions) */
#define EMB_STAT_EMPTY_FILLS 8   /* inserts into empty ways */
#define EMB_STAT_HIT_EVICTIONS 9 /* residents updated this step, then displaced (LFU) */
#define EMB_STAT_INVALID_FWD 10  /* out-of-range indices seen by the last forward */
#define EMB_STAT_INVALID_BWD 11  /* out-of-range indices seen by the last backward_update */

/* Configuration (host memory, read during the call only).  All tables share
 * dim, precision, cache fraction, associativity, policy, rounding and
 * optimizer.
 *   rows[t]           rows of table t, 1 <= rows[t] < 2^31.
 *   dim               row width d: 16, 32, 64, 128 or 256.
 *   precision         EMB_FP16, EMB_INT8, EMB_INT4 or EMB_INT2; sb_dtype
 *                     (EMB_SB_FP32 or EMB_SB_FP16) applies to integer codes.
 *   cache_fraction    FP32 cache rows per table = floor(cache_fraction*rows[t]),
 *                     grouped in n_sets = max(1, floor(that / assoc)) sets;
 *                     0 disables the cache (every row bypasses).
 *   assoc             ways per set alpha: a power of two, 1..64.  Row i maps to
 *                     set h(i) = i mod n_sets.
 *   lfu_decay_interval  LFU counts are halved at the start of every step
 *                     k > 0 with k % interval == 0 (0 = never).
 *   seed              key of the stochastic-rounding random stream.
 *   max_batch         bags per table in one call (B); max_indices: indices in
 *                     one call over all tables (1 .. 2^30 - 1).  They size the
 *                     workspace.
 */
typedef struct emb_cache_config {
  int32_t num_tables;
  int32_t dim;
  const int64_t* rows;
  int32_t precision;
  int32_t sb_dtype;
  double cache_fraction;
  int32_t assoc;
  int32_t policy;
  int32_t lfu_decay_interval;
  int32_t rounding;
  int32_t optimizer;
  float lr;
  float eps;
  uint64_t seed;
  int32_t max_batch;
  int64_t max_indices;
} emb_cache_config;

typedef struct emb_cache_sizes {
  size_t state_bytes;     /* persistent state: tables, caches, tags, policy and optimizer state */
  size_t workspace_bytes; /* per-call temporaries of forward/backward_update */
  int64_t total_rows;     /* sum of rows[t] */
  int64_t total_slots;    /* sum over tables of n_sets*assoc */
  int32_t row_bytes;      /* bytes of one low-precision row record: codes + scale + bias, then,
                             under row-wise Adagrad, the row's FP32 accumulator, padded to the
                             alignment of the first part (at most 16 bytes) -- unless the record
                             would then span one more 64-byte line (FP16 tables of dim >= 32),
                             whose accumulators are kept apart */
  int32_t pad;
  size_t table_bytes;     /* the low-precision table: the last table_bytes of state_bytes */
} emb_cache_sizes;

typedef struct emb_cache* emb_cache_t;

/* Validate `cfg` and report buffer sizes.  Pure host computation; no HIP call.
 * Returns EMB_EINVAL for an unsupported or inconsistent configuration. */
int emb_cache_query_sizes(const emb_cache_config* cfg, emb_cache_sizes* out);

/* Cache geometry of table `table`: n_sets (0 when the cache is disabled) and
 * slots = n_sets*assoc.  Pure host computation. */
int emb_cache_table_geometry(const emb_cache_config* cfg, int32_t table, int64_t* n_sets, int64_t* slots);

/* Create a handle over caller-owned device buffers (`state`, `workspace`, at
 * least the queried sizes, 256-byte aligned).  Enqueues the reset of the
 * state: empty cache (tags -1), LRU stamps -1, LFU counts 0, Adagrad state 0,
 * all codes/scale/bias 0; sets step = 0.  Synchronizes `stream`. */
int emb_cache_create(const emb_cache_config* cfg, void* state, size_t state_bytes, void* workspace,
                     size_t workspace_bytes, void* stream, emb_cache_t* out);

/* As emb_cache_create, with the low-precision table in a buffer of its own:
 * `table` (table_bytes >= the queried table_bytes, 256-byte aligned) is device
 * memory, or pinned host memory from hipHostMalloc, which the kernels then reach
 * over the host link -- the paper's table in unified memory with the FP32 cache
 * in device memory (Sec. 5.2 "Speed improvement", Fig. 9).  `state` then needs only state_bytes -
 * table_bytes.  Any other host memory is refused (EMB_EINVAL): a kernel could not
 * reach it.  Synchronizes `stream`. */
int emb_cache_create_with_table(const emb_cache_config* cfg, void* state, size_t state_bytes, void* table,
                                size_t table_bytes, void* workspace, size_t workspace_bytes, void* stream,
                                emb_cache_t* out);

/* Release host metadata.  Does not touch device memory. */
int emb_cache_destroy(emb_cache_t h);

/* Initial table.  The paper does not state how its tables are initialised; the
 * reading here: fill every row of every table with x_j = u*(hi-lo)+lo (fused
 * multiply-add), u a 24-bit uniform from Philox4x32-10 keyed on init_seed with
 * counter (j/4, row, table, 0xFFFFFFFF), then down-convert each row into T as
 * Sec. 3 "Precision" and Alg. 1 define it, with round-to-nearest-even ("Rounding"
 * knob).  Empties the cache, zeroes LFU counts and Adagrad state.  Enqueue-only. */
int emb_cache_init_uniform(emb_cache_t h, float lo, float hi, uint64_t init_seed, void* stream);

/* Forward: the fetch operator of Sec. 3 (the FP32 cache row of a row resident
 * in set h(i), else the row up-converted as in Alg. 1, q*s + b with one
 * rounding), pooled per bag (multi-hot lookups, Sec. 5.1; the paper does not
 * state the pooling mode, the reading is a sum):
 * pooled[b][t][:] = sum over positions p in [offsets[t*batch+b],
 * offsets[t*batch+b+1]) of fetch(T_t, C_t, indices[p]), summed left to right
 * in FP32 starting from the first term; an empty bag gives +0.
 *   indices   device int32 [num_indices], flat, table-major.
 *   offsets   device int32 [num_tables*batch + 1], non-decreasing, in [0, num_indices].
 *   out       device FP32 [batch][num_tables][dim].
 * Reads the state only.  Enqueue-only. */
int emb_cache_forward(emb_cache_t h, const int32_t* indices, int64_t num_indices, const int32_t* offsets,
                      int32_t batch, float* out, void* stream);

/* Forward for callers that cannot allocate device memory or pass a workspace:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  Same computation, results and statistics as emb_cache_forward,
 * but the per-call temporaries (one code per lookup and a few counter words)
 * live in a static device array owned by the library, EMB_NOALLOC_SCRATCH_BYTES
 * (64 MiB) per GPU, instead of the handle's workspace; the call allocates
 * nothing and calls no allocating routine.  num_indices may be at most
 * EMB_NOALLOC_MAX_INDICES; beyond it the call returns EMB_ENOMEM and enqueues
 * nothing (max_indices of the handle does not apply).  Each GPU the library
 * runs on holds its own copy of the array from the first handle created on it
 * until the process ends, and every call on that GPU shares it: calls that may
 * overlap on one GPU (on several streams, or from several handles) race on it
 * and must be serialised by the caller.  Enqueue-only. */
#define EMB_NOALLOC_SCRATCH_BYTES (64u << 20)
#define EMB_NOALLOC_MAX_INDICES ((int64_t)((EMB_NOALLOC_SCRATCH_BYTES - 256u) / 4u))
int emb_cache_forward_noalloc(emb_cache_t h, const int32_t* indices, int64_t num_indices, const int32_t* offsets,
                              int32_t batch, float* out, void* stream);

/* Backward + sparse update of one training step: the update operator of Sec. 3
 * under the "Cache Replacement Policy" knob and Alg. 2, applied once per unique
 * row after the gradients of the mini-batch are sorted by row and merged
 * (Sec. 5.1, "De-duplicate gradients"), for the same indices/offsets as the
 * forward and grad_out = dL/d(pooled), device FP32 [batch][num_tables][dim].
 * Per table:
 *   - sort the lookups by row and merge each row's gradient, its lookups taken
 *     in position order (the paper fixes no order; this one is fixed so that
 *     results are reproducible bit for bit): up to 64 lookups summed left to
 *     right from the first; 65..512 in chunks of 64 consecutive lookups, each
 *     summed left to right, then the chunk sums left to right; more than 512
 *     grouped by bag block (bags [k*NB, (k+1)*NB), NB = 32768/dim), each
 *     non-empty group summed left to right, then the group sums left to right
 *     in block order;
 *   - update priorities (LRU: hit ways stamped with the step; LFU: count +=
 *     occurrences, saturating; counts halved first on decay steps);
 *   - decide per set which missed rows enter the cache (victims by (priority
 *     asc, way asc), empty ways first; candidates by (priority desc, row asc);
 *     the k-th candidate takes the k-th victim while its priority is strictly
 *     higher; direct-mapped LRU always replaces);
 *   - apply SGD or row-wise Adagrad in FP32 to fetch(T,C,row); write each row
 *     to its cache way, or down-convert it into T (Alg. 1; nearest-even or
 *     stochastic rounding keyed on (seed, step, table, row, column));
 *     down-convert displaced residents into T.
 * Then step += 1.  Enqueue-only.
 * Malformed offsets (negative, decreasing, or past num_indices) reject the
 * call on the device: it changes no table, cache, count or accumulator (not
 * even the LFU decay of that step), its backward statistics read 0, and the
 * next emb_cache_check returns EMB_EINDEX.  A rejected call still counts as a
 * step (step += 1): the step counter lives on the host, which learns of the
 * rejection only at that check; a caller that retries the step with corrected
 * offsets gets LRU stamps and stochastic-rounding keys one step later, and a
 * decay that fell on the rejected step is skipped. */
int emb_cache_backward_update(emb_cache_t h, const int32_t* indices, int64_t num_indices, const int32_t* offsets,
                              int32_t batch, const float* grad_out, void* stream);

/* Copy the statistics of table `table` (EMB_NSTAT int64 values, layout
 * EMB_STAT_*) to host memory `out`.  Synchronizes `stream`. */
int emb_cache_get_stats(emb_cache_t h, int32_t table, int64_t* out, void* stream);

/* Synchronize `stream`, then return EMB_EINDEX (and clear the flag) if a
 * kernel has seen an out-of-range index or malformed offsets since the last
 * check, EMB_EHIP if a step's sort did not complete (its kernels gave up
 * waiting on each other; that step's results are unspecified), else EMB_OK. */
int emb_cache_check(emb_cache_t h, void* stream);

/* Copy rows [row0, row0+n) of table `table` to host buffers, in the canonical
 * layout: codes uint8 [n][dim] (one code per byte; for an FP16 table uint16
 * [n][dim], the binary16 bit patterns), scale and bias FP32 [n] (FP16 values
 * widened exactly when sb_dtype is FP16; 0 for an FP16 table), LFU counts int32
 * [n], Adagrad accumulators FP32 [n].  A NULL buffer is skipped; counts and
 * Adagrad state read as 0 when the configuration has none.  Synchronizes
 * `stream`. */
int emb_cache_export_rows(emb_cache_t h, int32_t table, int64_t row0, int64_t n, void* codes, float* scale,
                          float* bias, int32_t* lfu_count, float* adagrad, void* stream);

/* Inverse of emb_cache_export_rows (host buffers in the same layout; integer
 * codes must be <= 2^precision-1, FP16 scale/bias must be FP16-representable;
 * an FP16 table takes its codes alone, scale and bias may be NULL).
 * Synchronizes `stream`. */
int emb_cache_import_rows(emb_cache_t h, int32_t table, int64_t row0, int64_t n, const void* codes,
                          const float* scale, const float* bias, const int32_t* lfu_count, const float* adagrad,
                          void* stream);

/* Copy the whole cache of table `table` to host: rows FP32 [slots][dim],
 * tags int32 [slots] (-1 = empty way; slot = set*assoc + way), LRU stamps
 * int32 [slots] (-1 for empty ways, and everywhere under LFU).  NULL skips.
 * Synchronizes `stream`. */
int emb_cache_export_cache(emb_cache_t h, int32_t table, float* rows, int32_t* tags, int32_t* lru_stamp,
                           void* stream);

/* Inverse of emb_cache_export_cache.  Synchronizes `stream`. */
int emb_cache_import_cache(emb_cache_t h, int32_t table, const float* rows, const int32_t* tags,
                           const int32_t* lru_stamp, void* stream);

/* Step counter (LRU stamp of the next backward_update and the step word of
 * its stochastic-rounding counters). */
int emb_cache_get_step(emb_cache_t h, uint64_t* step);
int emb_cache_set_step(emb_cache_t h, uint64_t step);

/* Measurement support (not needed for training).  While enabled, every
 * backward_update records two HIP events on its stream, around its row-update
 * kernel (per unique row: merged gradient, fetch, optimizer, write-back to the
 * cache or T); the events of the last 64 calls are kept.  Host-only call. */
int emb_cache_set_update_timing(emb_cache_t h, int32_t enable);

/* Durations in milliseconds of that kernel in the last n timed backward_update
 * calls, oldest first, n = min(max, 64, calls timed since enabling) written to
 * *n.  Waits for those events to complete. */
int emb_cache_get_update_times(emb_cache_t h, float* ms, int32_t max, int32_t* n);

/* Static string for a status code. */
const char* emb_cache_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* EMB_CACHE_H */
