/*
 * recis_mi355x.h — C ABI of the MI355X (gfx950) sparse embedding step.
 *
 * The library implements the sparse component's per-step hot path described
 * by RecIS (arXiv 2509.20883): the two-tier dynamic embedding store (an IDMap
 * from feature id to an offset, and Blocks holding embedding rows together
 * with their optimizer state; "Optimization for Memory Bound", "Moving to
 * GPU"), its forward workflow (dedup, one IDMap lookup per id, read the row,
 * pool it: sum / mean / padded copy — "Reduction Operations", "Gather"), and
 * its backward workflow (per-id gradient aggregation using the offsets kept
 * from the forward pass, then a row-sparse Adagrad / Adam update of the rows
 * and their state in place — "Backward Update", "Optimizer", "Scatter").
 * Beside the step: the sequence tile (a bag's rows concatenated, keeping its
 * first or last ids), row-wise optimizer state, eviction of stale keys, the
 * ids partition (dedup + split by owner shard) and the bucketize / mod
 * feature transforms fused over columns.
 *
 * Conventions shared by every entry point
 *  - All array arguments are DEVICE pointers owned by the caller, unless a
 *    comment says "host".  The table object (IDMap + Blocks) is owned by the
 *    library.
 *  - Every call that takes an `rs_stream` only enqueues work on that HIP
 *    stream (a hipStream_t; NULL = the null stream) and returns without
 *    waiting, except where a comment says it synchronizes.  Calls on one
 *    table must be issued in stream order from one host thread: the table's
 *    counters are shared by its calls.
 *  - Sizes and counts that depend on the data (the number of unique ids U,
 *    the number of inserted ids) stay on the device; buffers are sized by
 *    the upper bound n.
 *  - Every call returns an rs_status; no C++ exception crosses the ABI.  A
 *    message for the last non-OK status of the calling thread is returned by
 *    rs_last_error().  Errors the kernels detect (a reserved key, a full
 *    table) are latched in the table and returned by the next synchronizing
 *    call (ht_size, ht_reserve, ht_evict, ht_destroy, rs_table_check).
 *  - Keys are opaque int64.  INT64_MIN (empty) and INT64_MIN+1 (tombstone)
 *    are reserved; a key equal to either is rejected with RS_EKEY and does
 *    not take part in the step.
 */
#ifndef RECIS_MI355X_H
#define RECIS_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RS_VERSION 10

typedef enum {
  RS_OK = 0,
  RS_EINVAL = 1, /* an argument the host can check is invalid              */
  RS_ENOMEM = 2, /* the allocator returned NULL                            */
  RS_EFULL = 3,  /* auto_grow is off and an insert found no room; the keys
                    that did not fit get row -1 and are skipped downstream  */
  RS_EKEY = 4,   /* a reserved key was in the input                        */
  RS_EHIP = 5    /* a HIP runtime call failed                               */
} rs_status;

/* Pooling of a bag ("Reduction Operations": sum, mean, tile).  The two
 * padded copies are the sequence tile: viewed as [bags, pad_len * D], a
 * bag's row is the concatenation of its rows.  RS_POOL_NONE keeps the first
 * pad_len ids of a longer bag, RS_POOL_TILE_TAIL its last pad_len (the most
 * recent behaviours), both in their order from slot 0, zero after. */
typedef enum { RS_POOL_SUM = 0, RS_POOL_MEAN = 1, RS_POOL_NONE = 2, RS_POOL_TILE_TAIL = 3 } rs_pool;
typedef enum { RS_F32 = 0, RS_BF16 = 1 } rs_dtype;
/* Row-sparse optimizers (every one keeps fp32 state beside the row: Adagrad
 * one accumulator per element, the Adam family two moments per element; the
 * row-wise forms one scalar per row in place of a per-element vector).
 *  RS_ADAGRAD: Duchi et al. 2011.
 *  RS_ADAM:    Kingma & Ba 2015, Algorithm 1 (the paper's SparseAdam).
 *  RS_ADAMW:   Adam with decoupled weight decay (Loshchilov & Hutter 2019;
 *              the paper's SparseAdamW): the touched row first decays by
 *              lr * weight_decay * w, then takes the Adam step.
 *  RS_ADAM_TF: Adam in the reordered form with epsilon-hat (Kingma & Ba
 *              2015, end of section 2; the form TensorFlow implements, which
 *              the paper's TF-compatible optimizers follow).
 *  RS_ADAGRAD_ROWWISE: one accumulator per row, fed the row mean of g^2
 *              (the memory-saving form of embedding-table Adagrad).
 *  RS_ADAM_ROWWISE: m per element, v per row from the row mean of g^2. */
typedef enum {
  RS_ADAGRAD = 0,
  RS_ADAM = 1,
  RS_ADAMW = 2,
  RS_ADAM_TF = 3,
  RS_ADAGRAD_ROWWISE = 4,
  RS_ADAM_ROWWISE = 5
} rs_optim;

typedef struct rs_table rs_table; /* opaque, library-owned */
typedef void* rs_stream;          /* hipStream_t */

/* Device-memory allocator for everything a table owns: the IDMap, the
 * Blocks (rows + optimizer state) and internal workspace, so that a
 * framework's caching allocator (PyTorch's) can back the table.  With an
 * allocator the Blocks are separate allocations of block_rows rows each,
 * found through a device table of their addresses; rows never move.  NULL
 * as the allocator argument means hipMalloc / hipFree for the IDMap and
 * workspace, and Blocks made of physical chunks (hipMemCreate) mapped back
 * to back into one reserved virtual range (no address table).  alloc returns
 * NULL on failure (the call then returns RS_ENOMEM).  A free callback is
 * only invoked after the table's work has completed. */
typedef struct {
  void* (*alloc)(size_t bytes, void* ctx);
  void (*free)(void* ptr, void* ctx);
  void* ctx;
} rs_allocator;

/* Table descriptor (the Embedding Engine's KV table; all ids in one table
 * share one dim, the "merge same-dim tables" layout of Load Balancing). */
typedef struct {
  int32_t dim;            /* D: 8, 16, 32, 64, 128 or 256                         */
  int32_t row_dtype;      /* rs_dtype of stored rows; optimizer state is fp32      */
  int32_t optimizer;      /* rs_optim: fixes the state held beside each row        */
  float init_lo, init_hi; /* new rows draw uniform values in [lo, hi]              */
  uint64_t seed;          /* row-init seed: a new key's row is a pure function
                             of (seed, key)                                      */
  int64_t capacity_slots; /* IDMap slots, a power of two >= 16                     */
  float max_load;         /* IDMap load limit, in (0, 0.9]                          */
  int64_t block_rows;     /* rows per Blocks chunk (the unit of growth), a power
                             of two >= 64                                        */
  int32_t auto_grow;      /* 1: rehash the IDMap (x2) and add Blocks on demand;
                             0: inserts beyond max_load*capacity fail (RS_EFULL) */
  int32_t evictable;      /* 1: keep each row's key and the lookup clock of its
                             last lookup (16 more bytes per row at most), so
                             that ht_evict can drop stale keys; 0: no eviction */
} rs_table_desc;

/* Optimizer hyper-parameters.  Adagrad uses lr, eps; the Adam family lr,
 * eps (epsilon-hat for RS_ADAM_TF), beta1, beta2; RS_ADAMW also
 * weight_decay.  Given in double: the kernels take fp32 constants that the
 * library derives in double (lr, eps, beta, 1 - beta, bias corrections,
 * lr * weight_decay), so 1 - beta2 does not inherit the fp32 rounding error
 * of beta2. */
typedef struct {
  double lr, eps, beta1, beta2;
  double weight_decay;
} rs_opt_params;

/* Forward context: the caller provides the workspace; lookup_pool_fwd fills
 * the rest.  It holds the forward offsets the backward needs ("retained
 * forward-pass offsets"), so the workspace, the offsets array and this struct
 * must stay alive and unmodified until the matching lookup_pool_bwd /
 * sparse_opt_step / lookup_pool_bwd_opt has been enqueued. */
typedef struct {
  /* in */
  void* workspace;        /* device, >= lookup_workspace_bytes(n, bags, pad_len, t) bytes */
  size_t workspace_bytes;
  /* out: device pointers into the workspace, valid after lookup_pool_fwd */
  int64_t* unique;   /* [n] unique keys, first-occurrence order; first U valid          */
  int32_t* inverse;  /* [n] occurrence -> index into unique (-1 for a rejected key)     */
  int64_t* rows;     /* [n] Blocks row of unique[u] (-1 if it could not be inserted)    */
  int64_t* scalars;  /* [4] U, inserted this call, occurrences kept, live rows before   */
  /* library-private (retained forward state) */
  const int64_t* offsets;
  const rs_table* table;
  int64_t n, bags, pad_len;
  int32_t mode, dim;
  int64_t priv[16];
} rs_ctx;

/* Library version (RS_VERSION). */
int rs_version(void);

/* Message describing the calling thread's last non-OK status ("" if none). */
const char* rs_last_error(void);

/* Create a table (IDMap with desc->capacity_slots empty slots, no rows yet)
 * on the current HIP device.  `alloc` may be NULL.  The stream is used for
 * the initial clears, which are complete when the call returns.
 * Errors: RS_EINVAL for a bad descriptor, RS_ENOMEM, RS_EHIP. */
rs_status ht_create(const rs_table_desc* desc, const rs_allocator* alloc, rs_stream stream,
                    rs_table** out);

/* Synchronize the device, free everything the table owns, and return any
 * latched device error.  NULL is accepted (RS_OK). */
rs_status ht_destroy(rs_table* t);

/* IDMap find-or-insert (the KV store inserts a feature the first time it is
 * seen).  keys: [n] int64 (n <= 2^28), duplicates allowed.  rows_out: [n] int64, the row
 * of each key (equal keys get equal rows; -1 for a key that did not fit).
 * A missing key gets the next free row — new rows are numbered live, live+1,
 * ... in the first-occurrence order of the new keys — and its row is
 * initialised: element j = fma(u_j, hi - lo, lo) in fp32 (bf16 rows: rounded
 * to nearest even) with u_j = (splitmix64 output j+1 from state
 * mix(key ^ mix(seed))) >> 40 times 2^-24; optimizer state = 0.
 * n_inserted_dev: device int64 scalar receiving the number inserted (may be NULL).
 * May synchronize the stream when the table has to grow. */
rs_status ht_find_or_insert(rs_table* t, const int64_t* keys, int64_t n, int64_t* rows_out,
                            int64_t* n_inserted_dev, rs_stream stream);

/* IDMap find only: rows_out[i] = row of keys[i], or -1 if absent.  Inserts nothing. */
rs_status ht_find(rs_table* t, const int64_t* keys, int64_t n, int64_t* rows_out, rs_stream stream);

/* Synchronize the stream and return the number of live keys (host pointer);
 * returns (and clears) any latched device error. */
rs_status ht_size(rs_table* t, int64_t* live_host, rs_stream stream);

/* Feature eviction (Embedding Engine, Framework Components: the KV table
 * drops features that went stale while training goes on).  Every lookup
 * call (ht_find_or_insert,
 * lookup_prepare / lookup_pool_fwd) advances the table's lookup clock by
 * one, and each key it looks up (found or inserted) records that clock.
 * ht_evict removes every key whose age -- the current clock minus its
 * recorded clock, modulo 2^32 -- exceeds max_age (max_age = 0 keeps only the
 * keys of the latest lookup call): its IDMap slot becomes a tombstone (a
 * later rehash drops it) and its row is pushed on a stack of free rows, in
 * ascending row order.  New keys take free rows from the top of that stack
 * (re-initialised exactly like a new row) before new rows are added.
 * Only for tables created with evictable = 1 and fewer than 2^31 rows
 * provisioned (else RS_EINVAL).  Synchronizes the stream (only that one):
 * the caller orders ht_evict after every outstanding pool, backward and
 * optimizer call of the table on any stream, since a freed row may be handed
 * to a new key by the next lookup.  *n_evicted_host (may be NULL) receives
 * the count. */
rs_status ht_evict(rs_table* t, uint32_t max_age, int64_t* n_evicted_host, rs_stream stream);

/* Compaction of the Blocks after eviction (the Blocks grow by appending
 * chunks of rows; this gives memory back once keys have been evicted).  With
 * L live keys, every row at or above row L that holds a key moves -- values,
 * optimizer state, key and last-lookup clock -- into a free row below L: the
 * k-th such row in ascending row order into the k-th free row below L in
 * ascending order; the IDMap follows the moved keys.  Afterwards rows 0 ..
 * L-1 hold every live key, no row is free (new keys take rows L, L+1, ...),
 * and the Blocks chunks wholly past row L are released (unmapped, or handed
 * back to the table's allocator).  Row ids returned before the call
 * (rows_out, ctx->rows) are no longer valid; the call must be ordered after
 * all outstanding work of the table, and synchronizes the stream.
 * *moved_host / *bytes_released_host (either may be NULL) receive the rows
 * moved and the bytes of Blocks memory released.  Only for tables created
 * with evictable = 1 (else RS_EINVAL).  Errors: RS_ENOMEM, RS_EHIP. */
rs_status ht_compact(rs_table* t, int64_t* moved_host, int64_t* bytes_released_host, rs_stream stream);

/* Synchronize the stream and return (and clear) any latched device error. */
rs_status rs_table_check(rs_table* t, rs_stream stream);

/* Current IDMap capacity in slots (host pointer).  No synchronization. */
rs_status ht_capacity(const rs_table* t, int64_t* slots_host);

/* Copy every (key, row) pair out of the IDMap, in slot order, into keys[cap]
 * and rows[cap]; n_dev (device int64) receives the live count, which may
 * exceed cap (then only cap pairs are written). */
rs_status ht_export(rs_table* t, int64_t* keys, int64_t* rows, int64_t cap, int64_t* n_dev,
                    rs_stream stream);

/* Read rows by row id: w_out [n, D] fp32 (bf16 rows widened exactly),
 * state_out [n, SE] fp32, the row's state in storage order: Adagrad [acc (D)]
 * (SE = D), the Adam family [m (D) | v (D)] (SE = 2D), row-wise Adagrad
 * [acc] (SE = 1), row-wise Adam [m (D) | v] (SE = D + 1); either may be NULL.
 * Rows outside [0, live) give NaN. */
rs_status ht_read_rows(rs_table* t, const int64_t* rows, int64_t n, float* w_out, float* state_out,
                       rs_stream stream);

/* Grow the IDMap (rehash into the smallest power-of-two capacity with
 * live_upper_bound <= max_load * capacity) and the Blocks (to hold
 * live_upper_bound rows).  Key -> row pairs and row contents are unchanged.
 * Synchronizes; returns (and clears) any latched device error. */
rs_status ht_reserve(rs_table* t, int64_t live_upper_bound, rs_stream stream);

/* Workspace bytes lookup_pool_fwd needs for n ids on table t.  Every
 * workspace array is sized by the ids (and the table's dim); bags and
 * pad_len do not change the size in this version (per-bag data lives in the
 * caller's offsets and output), and are taken so that a later version may
 * size per-bag arrays without changing the call. */
size_t lookup_workspace_bytes(int64_t n, int64_t bags, int64_t pad_len, const rs_table* t);

/* Forward: dedup + find-or-insert + fused gather/pool.
 * values [n] int64 (n <= 2^28), offsets [bags+1] int64 (CSR: offsets[0] = 0,
 * nondecreasing, offsets[bags] = n; bag g = feature-major f*B + b).
 *  RS_POOL_SUM : out fp32 [bags, D], out[g] = sum of the rows of bag g
 *  RS_POOL_MEAN: out fp32 [bags, D], the sum divided by the bag length; an
 *                empty bag gives 0
 *  RS_POOL_NONE: out [bags, pad_len, D] in the row dtype, out[g][t] = row of
 *                the t-th id of bag g for t < min(len, pad_len), else 0;
 *                mask uint8 [bags, pad_len] = (t < len).  Ids past pad_len
 *                are looked up (and inserted) but not copied.
 *  RS_POOL_TILE_TAIL: the same with the bag's last min(len, pad_len) ids:
 *                out[g][t] = row of id skip + t, skip = max(len - pad_len, 0);
 *                the skipped ids are looked up (and inserted) but not copied.
 * New keys are inserted (and initialised) before the gather.
 * validate != 0 also checks the CSR offsets on the host (copies them back:
 * slow, synchronizing).  Errors: RS_EINVAL (sizes, workspace, mode),
 * RS_ENOMEM / RS_EHIP; device-detected errors are latched. */
rs_status lookup_pool_fwd(rs_table* t, const int64_t* values, const int64_t* offsets, int64_t n,
                          int64_t bags, int32_t mode, int64_t pad_len, void* out, uint8_t* mask,
                          rs_ctx* ctx, int32_t validate, rs_stream stream);

/* The forward in two halves, for callers that overlap the next batch's id
 * processing with the current batch's pool and backward on a second stream.
 *
 * lookup_prepare: everything of lookup_pool_fwd except the gather + pool:
 * dedup, IDMap find-or-insert, row init of new keys, and the per-occurrence
 * bookkeeping, into ctx (same arguments and errors as lookup_pool_fwd
 * minus out / mask).  It writes the IDMap, the rows of the keys it inserts
 * and ctx; on a table with eviction it also records the lookup clock in the
 * key record of every row it finds (bytes no pool, backward or optimizer
 * touches).  New keys take new rows, or rows that ht_evict freed; so a
 * prepare may run while an earlier batch's lookup_pool_prepared / backward /
 * optimizer are still running on another stream, provided no ht_evict was
 * issued after that batch's forward (its freed rows could still be in use).
 * Prepares of one table must be issued in order on one stream.
 *
 * lookup_pool_prepared: the gather + pool of a prepared ctx.  The caller
 * orders it after the prepare (same stream, or an event) and after the
 * optimizer of every earlier batch (whose updates it must read).
 * lookup_pool_fwd = lookup_prepare + lookup_pool_prepared on one stream. */
rs_status lookup_prepare(rs_table* t, const int64_t* values, const int64_t* offsets, int64_t n, int64_t bags,
                         int32_t mode, int64_t pad_len, rs_ctx* ctx, int32_t validate, rs_stream stream);
rs_status lookup_pool_prepared(rs_table* t, rs_ctx* ctx, void* out, uint8_t* mask, rs_stream stream);

/* Backward: per-unique gradient sums.  grad_out has the forward output's
 * shape: fp32 [bags, D] (sum, mean) or [bags, pad_len, D] in the row dtype
 * (none; positions with mask 0 are never read).
 * grad_unique [n, D] fp32: row u (< U) receives
 *   sum over occurrences i of unique u of scale(bag(i)) * grad_out[bag(i)]
 * (scale 1 for sum, 1/len for mean; padded: grad_out[g][t] for the id copied
 * to slot t; ids that were not copied contribute nothing).  Its first launch
 * lays out the per-key occurrence list from the gradient row of each id that
 * the ctx's pool wrote, so the pool precedes it; ids outside
 * [offsets[0], offsets[bags]) contribute nothing.  The order of a key's
 * occurrences in that list (so the fp32 summation order) is not fixed from
 * run to run: sums may differ in their last bits between runs. */
rs_status lookup_pool_bwd(rs_table* t, const rs_ctx* ctx, const void* grad_out, float* grad_unique,
                          rs_stream stream);

/* Row-sparse optimizer on the U rows touched by ctx's forward (every unique
 * key of the step, even one whose gradient is zero); untouched rows and their
 * state are not read or written.
 *   Adagrad: acc += g*g;  w -= lr * g / (sqrt(acc) + eps)
 *   Adam:    t += 1 (once per call, table-global);  m = b1*m + (1-b1)*g;
 *            v = b2*v + (1-b2)*g*g;  w -= lr * (m/(1-b1^t)) / (sqrt(v/(1-b2^t)) + eps)
 *   AdamW:   w -= lr * weight_decay * w, then the Adam step
 *   Adam (epsilon-hat): the same moments;  w -= lr_t * m / (sqrt(v) + eps)
 *            with lr_t = lr * sqrt(1-b2^t) / (1-b1^t)
 *   Row-wise, with ms = (sum over the row of g*g) / dim:
 *     Adagrad: acc += ms;  w -= lr * g / (sqrt(acc) + eps)
 *     Adam:    t += 1;  m = b1*m + (1-b1)*g;  v = b2*v + (1-b2)*ms (per row);
 *              w -= lr * (m/(1-b1^t)) / (sqrt(v/(1-b2^t)) + eps)
 * Arithmetic in fp32; bf16 rows are widened, updated, and rounded to nearest
 * even.  grad_unique [n, D] fp32 as written by lookup_pool_bwd. */
rs_status sparse_opt_step(rs_table* t, const rs_ctx* ctx, const float* grad_unique,
                          const rs_opt_params* p, rs_stream stream);

/* lookup_pool_bwd followed by sparse_opt_step in one pass: the per-unique
 * gradient is applied to its row as soon as it is complete and never written
 * out.  Same results as the two calls (up to fp32 summation order). */
rs_status lookup_pool_bwd_opt(rs_table* t, const rs_ctx* ctx, const void* grad_out,
                              const rs_opt_params* p, rs_stream stream);

/* Ids partition ("Ids Partition" among the benchmarked operators; "Request
 * Merging & Sharding" under Load Balancing): the batch's ids deduplicated and
 * split by the shard that owns them, in one call, before the exchange of
 * each shard's ids.  No table is involved.
 *   owner(k) = mix64((uint64_t)k ^ owner_seed) mod nshards, with mix64 the
 *   splitmix64 output function (Steele, Lea & Flood 2014).
 * Outputs (device, caller-owned):
 *   keys_out [n] int64: the U distinct keys, shard 0's first, each shard's
 *                keys in the order of their first occurrence in values;
 *                entries past U are unspecified
 *   shard_offsets [nshards+1] int64: shard s holds
 *                keys_out[shard_offsets[s] .. shard_offsets[s+1]);
 *                shard_offsets[nshards] = U
 *   inverse [n] int32: keys_out[inverse[i]] == values[i]; -1 for a reserved
 *                key (INT64_MIN, INT64_MIN+1), which takes no part
 *   info [2] int64: {U, error bits}: bit 0 (1) a reserved key was skipped;
 *                bit 3 (8) an internal dedup pass overflowed (outputs
 *                invalid; not expected for any input)
 * values [n] int64, n <= 2^28; 1 <= nshards <= 1024.  workspace: device,
 * 256-byte aligned, >= ids_partition_workspace_bytes(n, nshards) bytes,
 * reusable by the next call once this one has completed in stream order.
 * Enqueues on `stream` and returns without waiting.  Errors: RS_EINVAL
 * (sizes, null pointers, workspace), RS_EHIP. */
size_t ids_partition_workspace_bytes(int64_t n, int32_t nshards);
rs_status ids_partition(const int64_t* values, int64_t n, int32_t nshards, uint64_t owner_seed, int64_t* keys_out,
                        int64_t* shard_offsets, int32_t* inverse, int64_t* info, void* workspace,
                        size_t workspace_bytes, rs_stream stream);

/* ids_partition without allocation, for callers that cannot allocate device
 * memory (code under HIP graph capture, serving loops, harnesses that forbid
 * hipMalloc): the same computation and outputs as ids_partition, but the
 * workspace is a fixed 54 MiB array inside this library (one per GPU, held
 * until the process ends) instead of a caller's buffer, so the call itself
 * allocates nothing.  n <= RS_IDS_STATIC_MAX_IDS (2^20; else RS_EINVAL).
 * Every call on one GPU uses that GPU's array: calls that overlap on one GPU
 * (other streams, other host threads) race and must be ordered by the
 * caller.  Nothing needs clearing between calls.  Errors: RS_EINVAL (as
 * ids_partition, and n above the limit), RS_EHIP. */
#define RS_IDS_STATIC_MAX_IDS (1 << 20)
rs_status ids_partition_static(const int64_t* values, int64_t n, int32_t nshards, uint64_t owner_seed,
                               int64_t* keys_out, int64_t* shard_offsets, int32_t* inverse, int64_t* info,
                               rs_stream stream);

/* Feature transforms fused over many columns, one launch for all of them
 * ("Bucketize and Mod" among the benchmarked operators: models hold dozens
 * to hundreds of such columns).  The columns are one flat array of n
 * elements; column c holds [col_offsets[c], col_offsets[c+1]) (int64
 * [ncols+1], col_offsets[0] = 0, nondecreasing, col_offsets[ncols] = n).
 *
 * fused_bucketize: values fp32 [n] -> out int64 [n], out[i] = the number of
 *   boundaries b of i's column with b <= values[i] (TensorFlow's Bucketize:
 *   boundaries[k-1] <= x < boundaries[k] gives k; a NaN, below no boundary,
 *   gives the number of boundaries).  Column c's
 *   boundaries are boundaries[bnd_offsets[c] .. bnd_offsets[c+1]), fp32,
 *   nondecreasing and not NaN (int64 [ncols+1] offsets, bnd_offsets[0] = 0).
 * fused_mod: values int64 [n] -> out int64 [n], out[i] = values[i] mod m in
 *   [0, m) (floor modulus) with m = moduli[column of i] (int64 [ncols],
 *   m > 0; a modulus <= 0 gives -1).
 * All arrays are device arrays.  The offsets are read by the kernels; the
 * caller guarantees the layout above (validate != 0 checks it, and the
 * moduli, on the host: it copies them back, so it synchronizes).  Errors:
 * RS_EINVAL (sizes, null pointers, a layout validate rejects), RS_EHIP. */
rs_status fused_bucketize(const float* values, int64_t n, const int64_t* col_offsets, int32_t ncols,
                          const float* boundaries, const int64_t* bnd_offsets, int64_t* out, int32_t validate,
                          rs_stream stream);
rs_status fused_mod(const int64_t* values, int64_t n, const int64_t* col_offsets, int32_t ncols,
                    const int64_t* moduli, int64_t* out, int32_t validate, rs_stream stream);

/* Kernel timing hook: from now on, hipEvent_t `start` / `stop` time every
 * launch of the named kernel (NULL, NULL clears it).  For RS_K_POOL,
 * RS_K_BWD_SHORT and RS_K_BWD_LONG the events are handed to the launch and
 * timestamped by the dispatch (the kernel's own execution; for RS_K_BWD_LONG
 * from the unit sums' start to the finish's end); for the other kernels they
 * are recorded on the call's stream immediately before / after the launch.
 * The events must exist (created, e.g. recorded once) before the call that
 * uses them.  For measurement only. */
typedef enum {
  RS_K_TILE_DEDUP = 0,     /* tile dedup in LDS, records per hash partition     */
  RS_K_PARTITION = 1,      /* per-partition dedup + IDMap probe, then the
                              first-occurrence tile sums and their scan
                              (several kernels)                                 */
  RS_K_COMPACT_INSERT = 2, /* unique ids, segments, rows, IDMap inserts         */
  RS_K_INIT_ROWS = 3,      /* same launch as RS_K_OCC (it writes the new rows)  */
  RS_K_POOL = 4,           /* gather + pool (and each id's gradient row)        */
  RS_K_BWD_SHORT = 5,      /* per-key gradient sum (+ optimizer), short keys    */
  RS_K_BWD_LONG = 6,       /* hot keys: unit partial sums + finish (two kernels) */
  RS_K_OPT = 7,            /* optimizer from grad_unique (two-call path)        */
  RS_K_OCC = 8,            /* per-occurrence rows, list positions, inverse; the
                              same launch writes the rows of inserted keys      */
  RS_K_OCC_LIST = 9,       /* the backward's first launch: the occurrence list
                              (each position's gradient row)                    */
  RS_K_COUNT = 10
} rs_kernel_id;
rs_status rs_set_kernel_events(rs_table* t, int32_t kernel, void* start_event, void* stop_event);

/* Bandwidth probes, for measurement only: plain device operations with the
 * access widths and launch shapes of the step's kernels, so the step's
 * bandwidth can be set against what this GPU delivers for each access
 * pattern.  Enqueued on `stream`; the caller times them (events).
 *  RS_PROBE_READ:   read n bytes of a (n a multiple of 16); b >= 4 bytes
 *                   receives nothing unless the data hash to one value
 *  RS_PROBE_WRITE:  write n bytes of a (a multiple of 16), streaming stores
 *  RS_PROBE_COPY:   copy n bytes from a to b (a multiple of 16)
 *  RS_PROBE_GATHER: b[i] = row idx[i] of a, for i < n, rows of row_bytes
 *                   (16 * 2^k * c bytes with 2^k <= 64 lanes and c <= 4 words
 *                   per lane: 16 ... 4096); indices outside
 *                   [0, a_bytes / row_bytes) are skipped
 *  RS_PROBE_RMW:    row idx[i] of a += 1.0f (every fp32 word), for i < n
 * a_bytes / b_bytes: the buffers' sizes in bytes.  idx: device int64 [n].
 * Errors: RS_EINVAL (kinds, sizes, null pointers), RS_EHIP. */
typedef enum { RS_PROBE_READ = 0, RS_PROBE_WRITE = 1, RS_PROBE_COPY = 2, RS_PROBE_GATHER = 3, RS_PROBE_RMW = 4 } rs_probe_kind;
rs_status rs_bandwidth_probe(int32_t kind, void* a, int64_t a_bytes, void* b, int64_t b_bytes, const int64_t* idx,
                             int64_t n, int32_t row_bytes, rs_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* RECIS_MI355X_H */
