/*
 * mlkv.h - batched embedding-table get / put_grad on one AMD MI355X (gfx950).
 *
 * The calls follow the key-value interface of MLKV (He et al., "MLKV:
 * Efficiently Scaling up Large Embedding Model Training with Disk-based
 * Key-Value Storage", arXiv 2504.01506):
 *   Open(model_id, dim, staleness_bound)  Sec. III-A (Interfaces Summary)
 *   Get(keys) -> values                   Sec. III-A; workflow step 2, Sec. III-B
 *   Rmw at workflow step 8                Sec. III-B (Workflows); here the
 *                                         modify function is "sum the gradients
 *                                         of duplicate keys, then one row-wise
 *                                         Adagrad step"
 * Tables live in HBM (a tiered table keeps its rows in host memory with an HBM
 * cache, see mlkv_open_tiered). Calls on one table must be ordered on one HIP
 * stream. A table may carry a staleness bound (Sec. III-C1, see
 * mlkv_open_bounded); without one every get is served.
 *
 * Conventions for every call below
 *   - Pointers named d_* are DEVICE pointers (HBM), owned by the caller, that
 *     must stay valid until the stream work of the call has finished. The
 *     library never keeps them after the call's kernels complete.
 *   - `hip_stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   - Return codes cover host-side validation and launch failures only; calls
 *     are asynchronous. Conditions found on the device (capacity exceeded,
 *     a reserved key in the input) make the whole call a no-op on the table
 *     and are reported by the next mlkv_sync().
 *   - A failed call leaves the table unchanged; outputs are then unspecified.
 *   - mlkv_last_error() returns a thread-local message for the last failure.
 */
#ifndef MLKV_H
#define MLKV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct mlkv_table mlkv_table;

enum {
  MLKV_OK = 0,
  MLKV_EINVAL = -1,  /* bad argument, or a reserved key (all ones) in the input */
  MLKV_EFULL = -2,   /* the call would grow the table beyond its capacity */
  MLKV_ENOMEM = -3,  /* device allocation failed */
  MLKV_EDEVICE = -4  /* HIP runtime or launch error */
};

#define MLKV_DEFAULT_SEED 0x4D4C4B56ull /* seed of the initial rows for mlkv_open */
#define MLKV_RESERVED_KEY 0xFFFFFFFFFFFFFFFFull

/* Creates a table of `dim`-wide fp32 rows with room for `capacity` keys
 * (Open, Sec. III-A; model_id is not needed: one table per handle; no
 * staleness bound, see mlkv_open_bounded). Limits: 1 <= dim <= 1024, 1 <= capacity <= 2^32 - 2. The table
 * owns all of its device memory (hash index, rows, optimizer state,
 * scratch), allocated on the current HIP device. Returns NULL on failure
 * (see mlkv_last_error). Uses seed MLKV_DEFAULT_SEED and max load 0.75. */
mlkv_table *mlkv_open(int32_t dim, int64_t capacity);

/* As mlkv_open with an explicit initial-row seed and the largest fraction of
 * hash-index slots that may hold keys (0 < max_load <= 0.9). */
mlkv_table *mlkv_open_ex(int32_t dim, int64_t capacity, uint64_t seed, float max_load);

/* Open (Sec. III-A) with a staleness bound s (Sec. III-C1: bulk-synchronous
 * at s = 0, stale-synchronous above; a table without a bound is the
 * asynchronous end). The table keeps, per key, the number of gets served on
 * it that no put has completed yet (the count of the paper's per-record
 * vector clock, a word per row next to the Adagrad accumulator):
 *   - mlkv_get_bounded serves a key present before the call only while its
 *     count is at most s, then raises the count by one; otherwise the key is
 *     blocked. A key inserted by the call is served (count 1). The count
 *     moves once per call and key, however often the key occurs.
 *   - every put call (mlkv_put_grad, mlkv_put_grad_sgd, mlkv_put) lowers the
 *     count of each of its distinct keys by one, not below 0; a key a put
 *     inserts starts at 0.
 * The paper's "wait until below the bound" is left to the caller: it repeats
 * the blocked positions after the puts they wait for (the library never
 * waits on the device). Limits: 0 <= staleness_bound <= 2^24 - 2, at most
 * 2^40 get calls per table; otherwise as mlkv_open_ex. mlkv_get is refused
 * (MLKV_EINVAL) on such a table. Extra device memory: 8 bytes per row. */
mlkv_table *mlkv_open_bounded(int32_t dim, int64_t capacity, uint64_t seed, float max_load,
                              int64_t staleness_bound);

/* Get (Sec. III-A): d_out[i*dim + c] = row(d_keys[i])[c] for i < n, where a key
 * that is not yet in the table is first inserted. Within one call, the
 * distinct new keys take the rows size, size+1, ... in ascending key order,
 * and element c of a new key's row is
 *     t = (int32)(h >> 40) - 2^23,  h = mix64(mix64(key ^ seed) + c * 0x9E3779B97F4A7C15)
 *     value = (float)t * (0.01f * 2^-23)          (uniform on [-0.01, 0.01))
 * with mix64 the SplitMix64 output function. d_out may be NULL (insert only).
 * 0 <= n <= 2^31 - 1. d_keys: n uint64 keys. d_out: n*dim floats, row-major. */
int mlkv_get(mlkv_table *t, const uint64_t *d_keys, int64_t n, float *d_out, void *hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): mlkv_get
 * with the same results (rows, key -> row, size, errors), that allocates
 * nothing. Its per-call scratch (new-key lists and per-tile counts) lives in
 * a fixed device array of about 1.8 MiB per GPU, part of the library's code
 * object, which each GPU the library runs on holds until the process ends.
 *   - 0 <= n <= MLKV_NOALLOC_MAX_KEYS; larger n is refused with MLKV_EINVAL.
 *   - Every call on a GPU shares that GPU's array: calls of this function on
 *     one GPU (any tables, any streams) that may run at the same time race
 *     and give undefined results; order them on one stream or synchronize.
 *   - It does not record the rows it found for reuse by a later put_grad
 *     (that put probes the index itself where no earlier get recorded them).
 *   - Refused (MLKV_EINVAL) on a table with a staleness bound.
 * Calls no hipMalloc, hipFree or other allocating routine; launch timing
 * (mlkv_profile_enable) is not recorded for it. */
#define MLKV_NOALLOC_MAX_KEYS 65536
int mlkv_get_noalloc(mlkv_table *t, const uint64_t *d_keys, int64_t n, float *d_out, void *hip_stream);

/* Get on a table opened with mlkv_open_bounded (Sec. III-C1): as mlkv_get
 * for the served positions; d_blocked[i] = 1 where d_keys[i] is blocked (row
 * i of d_out is then left as it was), else 0. d_blocked: n bytes (device).
 * A failed call (see mlkv_sync) changes no count. MLKV_EINVAL on a table
 * without a bound. */
int mlkv_get_bounded(mlkv_table *t, const uint64_t *d_keys, int64_t n, float *d_out, uint8_t *d_blocked,
                     void *hip_stream);

/* Opens a tiered table (for tables larger than HBM; the paper's buffer over a
 * slower tier, Sec. III-C2): the rows live at home in pinned host memory
 * (capacity * dim * 4 bytes, allocated with hipHostMalloc), cache_rows of them
 * in an HBM cache; the index, the Adagrad accumulators and the staleness
 * counts stay in HBM. Every call works on it as on an ordinary table with the
 * same results: gets and puts read and write each row where it is (the cache
 * slot, else its home over the host link; a cached row written by a put is
 * written back when its slot is reused). mlkv_lookahead moves rows into the
 * cache. 1 <= cache_rows <= capacity; otherwise as mlkv_open_ex. */
mlkv_table *mlkv_open_tiered(int32_t dim, int64_t capacity, uint64_t seed, float max_load, int64_t cache_rows);

/* Lookahead (Sec. III-A; look-ahead prefetching, Sec. III-C2): makes d_keys
 * resident ahead of the gets that will read them. The missing keys are
 * inserted exactly as mlkv_get with d_out = NULL would (rows in ascending key
 * order, seeded initial rows); nothing is returned. On a tiered table the
 * keys' rows are then brought into the HBM cache: rows already cached stay;
 * each missing row takes the next cache slot, in FIFO order from a cursor,
 * whose row this call does not ask for (that row is evicted, and written back
 * home first if a put changed it); when the call asks for more rows than the
 * cache can give it, the rest stay at home (which ones may differ from run to
 * run; no result depends on it). It never blocks and changes no
 * staleness count (a new key starts at 0). 0 <= n <= 2^31 - 1; errors as for
 * mlkv_get. */
int mlkv_lookahead(mlkv_table *t, const uint64_t *d_keys, int64_t n, void *hip_stream);

/* Counters of a tiered table since it was opened (synchronizes the device):
 * out[0] rows copied into the cache, out[1] rows evicted from it, out[2]
 * evicted rows written back home, out[3] cache slots holding a row, out[4]
 * cache slots. out: 5 int64 (host). MLKV_EINVAL on a table that is not tiered. */
int mlkv_cache_stats(mlkv_table *t, int64_t *out);

/* Rmw (Sec. III-B, step 8) with row-wise Adagrad as the modify function:
 * missing keys are inserted as in mlkv_get; then for every distinct key k of
 * the batch, with positions i_1 < i_2 < ... holding k,
 *     g[c]  = fp32( sum_j fp64(d_grads[i_j*dim + c]) )
 *     m     = fp32( sum_c fp64(g[c])^2 / dim )
 *     G'    = G + m;   den = sqrtf(G') + eps
 *     w[c] -= lr * (g[c] / den)     (separate fp32 operations)
 *     G     = G'
 * G starts at 0 for every row. d_grads: n*dim floats, row-major.
 * 0 <= n <= 2^30 - 1; lr and eps must be finite, eps >= 0. */
int mlkv_put_grad(mlkv_table *t, const uint64_t *d_keys, const float *d_grads, int64_t n,
                  float lr, float eps, void *hip_stream);

/* Rmw (Sec. III-B, step 8) with plain SGD as the modify function, i.e. the
 * update form of Sec. II-A applied to the summed gradient: missing keys are
 * inserted as in mlkv_get; then for every distinct key k of the batch
 *     g[c] = fp32( sum_j fp64(d_grads[i_j*dim + c]) )   (positions ascending)
 *     w[c] -= lr * g[c]                                   (separate fp32 operations)
 * Adagrad accumulators are not touched. 0 <= n <= 2^30 - 1; lr finite. */
int mlkv_put_grad_sgd(mlkv_table *t, const uint64_t *d_keys, const float *d_grads, int64_t n, float lr,
                      void *hip_stream);

/* The Get of the next batch and the Rmw of the current one in the order of
 * asynchronous training (Sec. II: an embedding read at step t + 1 may predate
 * the update of step t, staleness s = t - k(t)), which a bounded table keeps
 * within its bound (Sec. III-C1). Same results (output rows, blocked flags,
 * key -> row, rows, accumulators, staleness counts, size, errors) as
 *     mlkv_get_bounded(t, d_get_keys, n_get, d_out, d_blocked, s)  (mlkv_get
 *                                                  on a table without a bound)
 *     mlkv_put_grad(t, d_put_keys, d_grads, n_put, lr, eps, s)
 * issued in that order, with one condition: every key of the put must be in
 * the table before this call (in a training loop the previous get inserted
 * it). A put key that is not, including one that this call's get inserts,
 * makes the put part a no-op and is reported by the next mlkv_sync as
 * MLKV_EINVAL; the get part is applied as if alone. Each part's other
 * device-side errors make that part alone a no-op (the first is reported).
 * The put's probe kernel runs first and takes the rows the last get recorded
 * by position, then the get's kernels, then the put's row updates, all on
 * hip_stream. get_done_event (a hipEvent_t, or NULL) is recorded on
 * hip_stream once the get's rows are in d_out, before the row updates: work
 * on another stream that waits for it (the model's step on the new batch)
 * runs beside the updates. At s = 0 every key of the get that the put
 * updates is blocked (its count is still 1); from s = 1 on, and on tables
 * without a bound, none is. Arguments as for the two calls; d_blocked may be
 * NULL on a table without a bound; d_out must not overlap d_get_keys,
 * d_put_keys or d_grads. n_get = 0 or n_put = 0 makes it the other call
 * alone (the event is then recorded after the get, or before the put). */
int mlkv_get_put_grad(mlkv_table *t, const uint64_t *d_get_keys, int64_t n_get, float *d_out, uint8_t *d_blocked,
                      const uint64_t *d_put_keys, const float *d_grads, int64_t n_put, float lr, float eps,
                      void *get_done_event, void *hip_stream);

/* Put (Sec. III-A), an upsert of a batch: for every distinct key of the batch
 * its row becomes d_values[i*dim ... i*dim + dim - 1] for the LAST position i
 * holding the key. Missing keys are inserted as in mlkv_get (rows in ascending
 * key order). The Adagrad accumulator of an existing key is kept; a new key's
 * is 0. d_values: n*dim floats, row-major. 0 <= n <= 2^30 - 1. */
int mlkv_put(mlkv_table *t, const uint64_t *d_keys, const float *d_values, int64_t n, void *hip_stream);

/* How the puts of a table (mlkv_put_grad, mlkv_put_grad_sgd, mlkv_put) find
 * the equal keys of a batch before summing their gradients (Rmw, Sec. III-B;
 * in-batch dedup of the sparse update):
 *   MLKV_DEDUP_HASH  (the default) items of keys repeated within a tile of
 *                    1024 positions are merged in LDS, then scattered by a
 *                    hash digit of the key's row into partitions, and each
 *                    partition is grouped by key with a hash table in LDS;
 *   MLKV_DEDUP_RADIX the same in-tile merge, then a stable LSD radix sort of
 *                    the items by the key's row (ceil(log2(capacity + index
 *                    slots)) bits, passes of at most 9 bits), then runs of
 *                    equal rows (run-length encoding) summed and applied.
 * Results are identical either way. With MLKV_DEDUP_RADIX a put call takes at
 * most 2^20 keys (MLKV_EINVAL above), and the table needs capacity + index
 * slots < 2^32 (else this call fails with MLKV_EINVAL). Takes effect for the
 * puts issued after it; returns MLKV_OK or MLKV_EINVAL. */
#define MLKV_DEDUP_HASH 0
#define MLKV_DEDUP_RADIX 1
int mlkv_set_dedup(mlkv_table *t, int mode);

/* Waits for all work on `hip_stream`, then returns and clears the first error
 * latched on the device since the previous mlkv_sync (MLKV_EFULL or
 * MLKV_EINVAL), or MLKV_OK. */
int mlkv_sync(mlkv_table *t, void *hip_stream);

/* Number of rows in use (synchronizes the device). -1 on error. */
int64_t mlkv_size(mlkv_table *t);

/* Number of hash-index slots (8 per bucket). */
int64_t mlkv_num_slots(mlkv_table *t);

/* Sizes the table's per-call scratch for calls of up to n keys (0 <= n <=
 * 2^31 - 1), so that later calls of at most n keys allocate nothing. A call
 * larger than any reserved or seen before grows the scratch itself: it
 * allocates device memory (hipMalloc) but does not wait for the device; the
 * replaced buffers are freed by the next mlkv_sync, mlkv_reserve or
 * mlkv_close once the work queued before the replacement has finished. This
 * call synchronizes the device. Not part of the paper's interface: a setup
 * call for callers that want no allocation on the path of their steps. */
int mlkv_reserve(mlkv_table *t, int64_t n);

/* Releases the table and all of its device memory (synchronizes the device). */
void mlkv_close(mlkv_table *t);

/* Thread-local text of the last error reported by this library. */
const char *mlkv_last_error(void);

/* ---- inspection (tests and debugging; asynchronous on hip_stream) ---- */

/* d_rows_out[i] = row of d_keys[i] or -1 if absent; never inserts.
 * 0 <= n <= 2^31 - 1. */
int mlkv_lookup_rows(mlkv_table *t, const uint64_t *d_keys, int64_t n, int64_t *d_rows_out,
                     void *hip_stream);

/* Copies table contents into caller buffers (any may be NULL):
 * d_rows_out [nrows*dim] rows 0..nrows-1, d_state_out [nrows] their Adagrad
 * accumulators, d_slot_keys_out [num_slots] / d_slot_rows_out [num_slots] the
 * raw index slots (empty slots hold MLKV_RESERVED_KEY / 0xFFFFFFFF).
 * nrows must be <= the current size. */
int mlkv_export(mlkv_table *t, int64_t nrows, float *d_rows_out, float *d_state_out,
                uint64_t *d_slot_keys_out, uint32_t *d_slot_rows_out, void *hip_stream);

/* d_rows_out[i*dim + c] = element c of row d_rows[i], d_state_out[i] = its
 * Adagrad accumulator (either output may be NULL), for 0 <= n <= 2^31 - 1 row
 * ids. A row id outside [0, size) gives a NaN row and accumulator and makes
 * the next mlkv_sync return MLKV_EINVAL. */
int mlkv_read_rows(mlkv_table *t, const int64_t *d_rows, int64_t n, float *d_rows_out,
                   float *d_state_out, void *hip_stream);

/* d_out[i] = staleness count of row d_rows[i] (table opened with
 * mlkv_open_bounded, else MLKV_EINVAL). A row id outside [0, size) gives
 * 0xFFFFFFFF and makes the next mlkv_sync return MLKV_EINVAL. */
int mlkv_read_staleness(mlkv_table *t, const int64_t *d_rows, int64_t n, uint32_t *d_out, void *hip_stream);

/* ---- per-kernel timing (benchmarks) ----
 * The library runs MLKV_NUM_KERNELS kernels: 0 get_probe_gather and
 * 1 assign_new for mlkv_get, mlkv_get_bounded and mlkv_lookahead;
 * 2 put_probe and 3 put_reduce for mlkv_put_grad, mlkv_put_grad_sgd and
 * mlkv_put; 4 tier_mark, 5 tier_plan and 6 tier_copy for mlkv_lookahead on a
 * tiered table; with radix dedup (mlkv_set_dedup) a put runs 2 put_probe,
 * then 7 rsort_count and 8 rsort_scatter once per radix pass, then
 * 9 rsort_reduce. While enabled, HIP events are recorded on
 * the call's stream before and after every launch. mlkv_profile_read waits
 * for the recorded launches, writes per-kernel sums of their durations (ms)
 * and launch counts into the host arrays total_ms[MLKV_NUM_KERNELS] and
 * launches[MLKV_NUM_KERNELS], and forgets them. */
#define MLKV_NUM_KERNELS 10
int mlkv_profile_enable(mlkv_table *t, int enable);
int mlkv_profile_read(mlkv_table *t, double *total_ms, int64_t *launches);
/* Name of kernel `kernel` (0 <= kernel < MLKV_NUM_KERNELS), else NULL. */
const char *mlkv_kernel_name(int kernel);

#ifdef __cplusplus
}
#endif

#endif /* MLKV_H */
