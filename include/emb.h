/*
 * emb.h -- C ABI of one GPU's shard of a pooled sparse embedding layer
 * (MI355X / gfx950, HIP).
 *
 * The layer: a recommendation model's large sparse embedding lookup layer,
 * which turns massive high-dimensional sparse ids into dense features and is
 * the part of the model with a high data-access cost (paper: Introduction;
 * Section "Multi-mode Execution", heterogeneous pipeline paragraph, where it
 * forms the embedding stage that pulls rows forward and pushes sparse
 * updates back).  The paper states the layer only in words; the operations
 * below are the plain definitions of a bag-pooled embedding lookup and its
 * training step:
 *
 *   key(j)   = row_offset[t(j)] + indices[j]                 (global row)
 *   out[m]   = scale_m * sum_{j in bag m} W[key(j)]           (forward)
 *   grad W_r = sum_{j : key(j) = r} scale_{m(j)} * G[m(j)]    (backward)
 *   W_r     <- opt(W_r, grad W_r) for every touched row r     (update)
 *
 * with scale_m = 1 (sum pooling) or 1/L_m (mean pooling), L_m the length of
 * bag m, and an empty bag pooling to zero.
 *
 * Conventions shared by every entry point:
 *  - Pointers are DEVICE pointers unless marked "host".  The caller
 *    allocates and frees every buffer, including the workspace; the library
 *    allocates no memory (emb_route_ids_noalloc's scratch array is part of
 *    its loaded code) and keeps no pointer after returning.  The state
 *    carried from call to call lives in the caller's dedup workspace: its
 *    header (call generation, per-call error word) must be zeroed once by
 *    emb_workspace_init, and its coordination words are tagged by call, so
 *    they never need clearing again.  The regions of a workspace are placed
 *    by its size and the tables' dim, not by the batch, so every call on a
 *    workspace must pass the same ws_bytes and tables of the same dim (after
 *    a change of either, run emb_workspace_init again); batches of any size
 *    up to the one it was sized for may then follow each other in any order.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Every call only enqueues work on it; nothing synchronises.  Buffers must
 *    stay alive until the stream has reached the enqueued work.
 *  - Host-checkable problems return an error before anything is enqueued.
 *    Device-content errors (an id >= rows of its table, decreasing offsets,
 *    offsets[M] != num_indices) are undefined behaviour on the fast path:
 *    emb_validate_batch detects them.
 *  - For identical inputs every output is bitwise identical from run to run
 *    (no floating-point atomics).
 *  - Calls that share a workspace must be ordered (same stream or events);
 *    calls with disjoint buffers may run concurrently on different streams.
 */
#ifndef EMB_H
#define EMB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EMB_OK = 0,
  EMB_EINVAL = 1,       /* null pointer, negative size, bad enum, bad table layout */
  EMB_EWORKSPACE = 2,   /* ws_bytes < emb_workspace_size(...) or misaligned workspace */
  EMB_EUNSUPPORTED = 3, /* dim*sizeof(dtype) not a multiple of 16, total rows >= 2^32,
                           num_indices >= 2^30, more than EMB_MAX_TABLES tables */
  EMB_EHIP = 4          /* a kernel launch failed (hipGetLastError) */
} emb_status;

typedef enum { EMB_FP32 = 0, EMB_BF16 = 1 } emb_dtype;
typedef enum { EMB_POOL_SUM = 0, EMB_POOL_MEAN = 1 } emb_pool;
typedef enum { EMB_OPT_SGD = 0, EMB_OPT_ADAGRAD_ROWWISE = 1, EMB_OPT_ADAGRAD_ELEMENTWISE = 2 } emb_opt;

#define EMB_MAX_TABLES 256
#define EMB_MAX_RANKS 256

/* All tables of one call share dim and dtype and are stacked row-wise in one
 * buffer: the rows of table t are global rows row_offset[t] .. row_offset[t+1]-1. */
typedef struct {
  int32_t num_tables;        /* T, 1 <= T <= EMB_MAX_TABLES */
  const int64_t* row_offset; /* host [T+1]; row_offset[0] = 0, nondecreasing, row_offset[T] = R < 2^32 */
  int32_t dim;               /* D >= 1 with D * sizeof(dtype) a multiple of 16 bytes */
  int32_t dtype;             /* emb_dtype */
  void* weights;             /* device [R][D] row-major, 16-byte aligned */
} emb_tables;

/* One batch: M = T * bags_per_table bags, table-major (bag m belongs to table
 * m / bags_per_table), given in CSR form. */
typedef struct {
  int32_t bags_per_table;    /* B >= 0 */
  const int32_t* offsets;    /* device [M+1]; offsets[0] = 0, nondecreasing, offsets[M] = num_indices */
  const void* indices;       /* device [N] int32 or int64 (index_bytes); table-local ids,
                                0 <= id < rows of the bag's table */
  int64_t num_indices;       /* N, host value, 0 <= N < 2^30 */
  int32_t index_bytes;       /* 4 (int32; 0 means 4) or 8 (int64) */
} emb_batch;

typedef enum { EMB_ROUND_NEAREST_EVEN = 0, EMB_ROUND_STOCHASTIC = 1 } emb_rounding;

/* Optimizer of one sparse step (the paper's push step applies the sparse
 * gradient to the touched rows; it does not fix the optimizer).
 *   SGD:                   W_r <- W_r - lr * g_r
 *   row-wise Adagrad:      h_r <- h_r + (1/D) sum_d g_r[d]^2
 *                          W_r <- W_r - lr * g_r / (sqrt(h_r) + eps)
 *   element-wise Adagrad:  h_r[d] <- h_r[d] + g_r[d]^2
 *   (Duchi et al. 2011)    W_r[d] <- W_r[d] - lr * g_r[d] / (sqrt(h_r[d]) + eps)
 * The new h is used in the same step.  Arithmetic is fp32; bf16 tables store
 * the fp32 result rounded to nearest even. */
typedef struct {
  int32_t opt;    /* emb_opt */
  float lr;
  float eps;      /* Adagrad only */
  float* state;   /* device fp32 accumulators h: [R] (row-wise), [R][D] row-major
                     (element-wise); NULL for SGD */
  int32_t rounding; /* emb_rounding of bf16 table stores (fp32 tables ignore it).
                       Stochastic: the 16 bits below the bf16 mantissa are added to
                       16 random bits and cut off (unbiased); the bits of element
                       (row r, column d) are the top 16 of
                       splitmix64(seed ^ splitmix64(r * D + d)) (Steele, Lea and
                       Flood 2014), so a caller passes a fresh seed every step */
  uint64_t seed;
} emb_update;

/* Forward (the pull of the embedding stage): out[m][d] = scale_m * sum over
 * bag m of W[key(j)][d], fp32 accumulation (bf16 rows are widened exactly).
 * out: device fp32 [M][D], fully overwritten (empty bags get zeros).  The
 * layer's forward as defined above (paper: Introduction, the layer that turns
 * sparse ids into dense features at a high data-access cost; Section
 * "Multi-mode Execution", heterogeneous pipeline paragraph). */
emb_status emb_pool_fwd(const emb_tables* tables, const emb_batch* batch, int32_t pool, float* out,
                        void* stream);

/* Bytes of workspace that emb_unique_ids / emb_grad_reduce need for batches
 * of up to num_indices ids (N < 2^30: published counts and offsets keep 30
 * bits) and num_bags bags, rows of dim floats.  The size does not depend on
 * the tables' row count.  Returns 0 for invalid sizes. */
size_t emb_workspace_size(int64_t num_indices, int64_t num_bags, int32_t dim);

/* Zero-fill a freshly allocated workspace (enqueued on stream).  Must run once
 * before the workspace's first use: it zeroes the header that carries each
 * call's generation and error record; later calls need no clearing (their
 * coordination words are tagged by call, and the counters they use are
 * cleared by the kernel that uses them). */
emb_status emb_workspace_init(void* ws, size_t ws_bytes, void* stream);

/* Dedup of the batch's ids, the step that makes the sparse update (the push
 * of the embedding stage, paper: Section "Multi-mode Execution",
 * heterogeneous pipeline paragraph) race-free: every touched row gets
 * exactly one owner.
 *   key[j]          = row_offset[t(j)] + indices[j]   (uint32)
 *   sort_perm       = the stable ascending sort of positions 0..N-1 by key
 *                     (equal keys keep position order), device int32 [N]
 *   num_unique[0]   = U, the number of distinct keys, device int32 [1]
 *   unique_keys[u]  = the u-th smallest distinct key, device uint32 [>= N]
 *   seg_offsets[u]  = first sorted position of unique_keys[u];
 *                     seg_offsets[U] = N, device int32 [>= N+1]
 *   counts[u]       = seg_offsets[u+1] - seg_offsets[u], device int32 [>= N]
 * Only the first U entries (U+1 of seg_offsets) are written.  ws (device,
 * 256-byte aligned, ws_bytes >= emb_workspace_size(N, M, D)) also receives
 * the per-position bag ids and sorted keys that emb_grad_reduce reads. */
emb_status emb_unique_ids(const emb_tables* tables, const emb_batch* batch, uint32_t* unique_keys, int32_t* counts,
                          int32_t* seg_offsets, int32_t* sort_perm, int32_t* num_unique, void* ws, size_t ws_bytes,
                          void* stream);

/* emb_unique_ids with the same outputs, bit for bit, from kernels in which no
 * workgroup ever waits for another (the sort's passes each preceded by their
 * tile counts and a column scan, the unique scan preceded by its tile counts
 * and their scan).  emb_unique_ids may make the workgroups of a pass wait for
 * one another when they all fit the device at once, so at most one such call
 * may be in flight on a device; any number of these may run concurrently, on
 * any streams, beside any other work (each with its own outputs and
 * workspace).  Slower alone; used to run the dedups of several upcoming
 * batches at once beside the forward and update of the current ones. */
emb_status emb_unique_ids_concurrent(const emb_tables* tables, const emb_batch* batch, uint32_t* unique_keys,
                                     int32_t* counts, int32_t* seg_offsets, int32_t* sort_perm, int32_t* num_unique,
                                     void* ws, size_t ws_bytes, void* stream);

/* The buffers of one dedup: emb_unique_ids outputs and workspace (device
 * pointers; ws_bytes >= emb_workspace_size of the largest batch, the
 * workspace initialised by emb_workspace_init). */
typedef struct {
  uint32_t* unique_keys; /* [>= N] */
  int32_t* counts;       /* [>= N] */
  int32_t* seg_offsets;  /* [>= N + 1] */
  int32_t* sort_perm;    /* [>= N] */
  int32_t* num_unique;   /* [1] */
  void* ws;
  size_t ws_bytes;
} emb_dedup_set;

/* The dedups of n_batches batches (1..16) as one sort: each batch's key gets
 * the batch's index above the key bits, so the sorted keys hold each batch's
 * keys in turn, each in exactly the stable order of its own sort; each
 * batch's share is then split off and its unique scan runs on it.  sets[i]
 * receives, bit for bit, what emb_unique_ids(tables, &batches[i], sets[i]'s
 * buffers) would leave there -- outputs, and in sets[i].ws the bag ids,
 * chunk map and call record that emb_grad_reduce reads -- so each batch's
 * gradient reduce follows as usual.  Same dedup as above (paper: Section
 * "Multi-mode Execution", heterogeneous pipeline paragraph), one sort for a
 * group of upcoming batches instead of one per batch: fewer, wider kernels.
 * No workgroup waits for another (as emb_unique_ids_concurrent).
 *   ws:  device, 256-byte aligned, ws_bytes >= emb_workspace_size(sum of
 *        the batches' num_indices, sum of their bags, dim), initialised by
 *        emb_workspace_init; used for this call only (its own state: pass
 *        the same ws_bytes every call), distinct from every sets[i].ws.
 *   sets[i].ws: as for emb_unique_ids, one per batch, all distinct.
 * EMB_EUNSUPPORTED: more than 16 batches, a total of 2^30 ids or more, or
 * key bits plus batch-index bits above 32 (tables of more than 2^(32 - b)
 * rows for 2^b batches). */
emb_status emb_unique_ids_batched(const emb_tables* tables, int32_t n_batches, const emb_batch* batches,
                                  const emb_dedup_set* sets, void* ws, size_t ws_bytes, void* stream);

/* n_steps training steps of the layer enqueued with the pipelined schedule:
 * step k pools batches[k] into outs[k] (device fp32 [M][D]) and applies the
 * fused backward and optimizer step with grads[k] (device fp32 [M][D]), in
 * order, on main_stream, exactly as emb_pool_fwd, emb_unique_ids and
 * emb_grad_reduce one after another would, bit for bit.  The dedups of each
 * next group of `group` batches run early on the n_side side streams (dealt
 * round-robin), since the dedup never reads the table: the dedup of step k
 * overlaps the forward and update of the steps before it -- the paper's
 * embedding stage run ahead within its pipeline (Section "Multi-mode
 * Execution", heterogeneous pipeline paragraph), here with no staleness.
 * With n_side = 1 the dedups are emb_unique_ids, one at a time; with
 * n_side > 1 they are emb_unique_ids_concurrent (no workgroup waits for
 * another), several at a time.  With group_ws non-NULL (n_side must be 1,
 * group at most 16) the dedups of a group are one emb_unique_ids_batched
 * call with group_ws as its workspace (device, group_ws_bytes >=
 * emb_workspace_size of a whole group's ids and bags, initialised by
 * emb_workspace_init); NULL otherwise.
 *   depth:   buffer set parities P (2..8): groups of steps whose dedup
 *            buffers are in use at once (a group's dedups wait for the main
 *            stream's group P earlier, whose buffers they reuse)
 *   sets:    host [depth * group] buffer sets, group g of the call using
 *            those of parity (group_base + g) % depth
 *   events:  host [1 + depth + depth * n_side] hipEvent_t created by the
 *            caller (no timing needed); the library only records and waits
 *            on them
 *   update:  the optimizer; step k uses update->seed + k for bf16
 *            stochastic rounding
 * Chained calls (a training loop's look-ahead): with ahead = A (0..depth-1),
 * batches holds n_steps + A * group entries and the call also dedups the
 * last A * group of them (the next call's first A groups) on the side
 * streams, overlapping its own last groups' forwards and updates; the next
 * call, given primed = A and those same batches (unchanged) as its first A
 * groups' (n_steps >= A * group), does not dedup them again.  group_base
 * numbers groups across chained calls: a call's group_base is the previous
 * call's plus its number of groups, ceil(n_steps / group); 0 and
 * primed = ahead = 0 for a call on its own.
 * All of the side streams' work precedes the end of the work enqueued on
 * main_stream (the look-ahead dedups too), so one synchronisation of
 * main_stream completes every step.
 * The side streams must differ from main_stream; calls that share sets,
 * events or side streams must be ordered.  With more than one group, each
 * side stream's work is enqueued by a host thread of its own, started and
 * joined within the call, while the calling thread enqueues main_stream's
 * (the device order is the same as from one thread).  Every step's
 * arguments are checked before anything is enqueued (EMB_EINVAL,
 * EMB_EWORKSPACE, EMB_EUNSUPPORTED as the per-step calls would return, and
 * EMB_EUNSUPPORTED for n_side > 16 or depth > 8; EMB_EINVAL for ahead with
 * n_steps = 0, depth < 2, primed or ahead outside 0..depth-1, or primed
 * groups beyond the steps); EMB_EHIP (a failed launch or event call)
 * returns with part of the schedule enqueued. */
emb_status emb_pipeline_steps(const emb_tables* tables, int32_t pool, const emb_update* update, int32_t n_steps,
                              const emb_batch* batches, float* const* outs, const float* const* grads,
                              int32_t group, const emb_dedup_set* sets, void* main_stream, int32_t n_side,
                              void* const* side_streams, void* const* events, void* group_ws,
                              size_t group_ws_bytes,
                              int32_t group_base, int32_t primed, int32_t ahead, int32_t depth);

/* Backward segment-reduce (the gradient the embedding stage pushes back,
 * paper: Section "Multi-mode Execution", heterogeneous pipeline paragraph),
 * optionally fused with the optimizer step:
 *   g_u[d] = sum over sorted positions k in segment u of scale_{m(k)} * grad_out[m(k)][d],
 * m(k) the bag holding position sort_perm[k], in a fixed order per segment
 * (deterministic, no float atomics).  grad_out: device fp32 [M][D].
 * grad_rows: device fp32 [>= N][D] receiving g_u for u < U, or NULL.
 * fuse: NULL = reduce only (grad_rows required); otherwise the optimizer step
 * is applied to tables->weights (and fuse->state) on rows unique_keys[u],
 * each row by exactly one owner, so the update is race-free.
 * sort_perm, seg_offsets, unique_keys, num_unique and ws must be those that
 * emb_unique_ids produced for this same batch, unmodified. */
emb_status emb_grad_reduce(const emb_tables* tables, const emb_batch* batch, int32_t pool, const float* grad_out,
                           const int32_t* sort_perm, const int32_t* seg_offsets, const uint32_t* unique_keys,
                           const int32_t* num_unique, float* grad_rows, const emb_update* fuse, void* ws,
                           size_t ws_bytes, void* stream);

/* Unfused optimizer step (the push of the sparse update to the touched rows,
 * paper: Section "Multi-mode Execution", heterogeneous pipeline paragraph):
 * for u < num_unique[0], row r = unique_keys[u] gets
 * opt(W_r, grad_rows[u]) as defined for emb_update.  max_unique (host) bounds
 * num_unique[0] (the batch's N is a valid bound).  unique_keys must be
 * distinct (one owner per row). */
emb_status emb_sparse_update(const emb_tables* tables, const emb_update* update, const uint32_t* unique_keys,
                             const int32_t* num_unique, int64_t max_unique, const float* grad_rows, void* stream);

/* Bytes of workspace emb_route_ids needs for batches of up to num_indices
 * ids and num_bags bags over world_size ranks (0 for invalid sizes). */
size_t emb_route_workspace_size(int64_t num_indices, int64_t num_bags, int32_t world_size);

/* Routing of the batch's ids to the owners of a row-range sharding of the
 * stacked tables: the step before the forward when the layer is spread over
 * world_size devices (the paper's distributed sparse lookup layer, its
 * Introduction), rank r owning global rows [shard_start[r], shard_start[r+1]).
 * Table-wise placement is the case of bounds at table starts.
 *   key[j]          = row_offset[t(j)] + indices[j]
 *   owner(j)        = the r with shard_start[r] <= key[j] < shard_start[r+1]
 * The send order lists the positions rank by rank, and in position order
 * within a rank.  Outputs (device, caller-owned):
 *   send_counts[r]  positions owned by rank r, int32 [world_size]
 *   send_ids[k]     key - shard_start[owner] of the k-th sent position, int32 [N]
 *   send_pos[k]     its position j, int32 [N]
 *   send_bag[k]     the bag holding it, int32 [N]
 * Rank r's range of the send order starts at the sum of send_counts[< r].
 * Within it the positions of one bag are consecutive (a bag's positions are),
 * so the runs of equal send_bag are the bag fragments the owner pools from its
 * rows (sum pooling); adding the fragments' pooled rows by bag (then scaling
 * by 1 / bag length for mean pooling) reassembles the forward.
 * shard_start: host [world_size + 1], shard_start[0] = 0, nondecreasing,
 * shard_start[world_size] = R; 1 <= world_size <= EMB_MAX_RANKS, else
 * EMB_EINVAL.  ws: device, ws_bytes >= emb_route_workspace_size(N, M, W).
 * Device contents are not validated (emb_validate_batch). */
emb_status emb_route_ids(const emb_tables* tables, const emb_batch* batch, int32_t world_size,
                         const int64_t* shard_start, int32_t* send_counts, int32_t* send_ids, int32_t* send_pos,
                         int32_t* send_bag, void* ws, size_t ws_bytes, void* stream);

/* emb_route_ids for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same outputs, bit for bit, with the per-block owner counts kept in a
 * scratch array inside the library instead of a workspace argument.  The
 * array holds EMB_ROUTE_SCRATCH_BYTES (4 MiB) on every GPU the library runs
 * on, for the life of the process; a batch for which
 * emb_route_workspace_size(N, M, world_size) exceeds it is rejected with
 * EMB_EUNSUPPORTED before anything is enqueued.  The call allocates nothing;
 * all calls on one GPU share that GPU's array, so calls that overlap in time
 * on one GPU (different streams without ordering) race on it.  Nothing in the
 * array needs clearing: every call writes each entry it reads. */
#define EMB_ROUTE_SCRATCH_BYTES (4u << 20)
emb_status emb_route_ids_noalloc(const emb_tables* tables, const emb_batch* batch, int32_t world_size,
                                 const int64_t* shard_start, int32_t* send_counts, int32_t* send_ids,
                                 int32_t* send_pos, int32_t* send_bag, void* stream);

/* Debug check of device contents (never on the timed path): flag[0] (device
 * int32) is set to 0 if the batch is well formed, else to a bitwise OR of
 * 1 (offsets[0] != 0), 2 (decreasing offsets), 4 (offsets[M] != N),
 * 8 (an id out of range of its table). */
emb_status emb_validate_batch(const emb_tables* tables, const emb_batch* batch, int32_t* flag, void* stream);

/* Failures a kernel finds on the device are recorded per call in the
 * workspace.  Every wait of a workgroup for a word another workgroup
 * publishes is bounded to 20 ms, far beyond any wait of a healthy call.  A
 * wait that runs out makes the call fail: its waits all give up within
 * microseconds, every write stays inside the caller's buffers, its
 * emb_unique_ids outputs are undefined except num_unique[0] = 0 when the sort
 * failed, and the emb_grad_reduce that follows it writes no table or state
 * row (unfused, it writes zero gradient rows, so an emb_sparse_update of
 * them leaves every row as it is for SGD and for Adagrad with eps > 0).  The
 * next emb_unique_ids on the workspace starts afresh.
 *
 * emb_workspace_status enqueues on stream a kernel that writes the status of
 * the last emb_unique_ids call on ws, and of the emb_grad_reduce that
 * followed it, to status (device int32 [4]):
 *   status[0]  error bits of that call, 0 if it completed normally:
 *              1 a wait of the dedup ran out, 2 a sort pass found digit
 *              totals inconsistent with its keys (a workspace that was not
 *              initialised), 4 a wait of the gradient combine ran out
 *   status[1]  site code of the first wait that ran out since the workspace
 *              was initialised (0: none): 0x1p0 / 0x1p2-0x1p5 a sort pass
 *              (pass p), 0x200 the unique scan, 0x300 the gradient combine
 *   status[2]  the workgroup of that wait
 *   status[3]  number of waits that ran out since the workspace was
 *              initialised
 * emb_workspace_init clears everything.  Returns EMB_EWORKSPACE if ws is
 * misaligned or ws_bytes is smaller than a workspace header (256 bytes). */
emb_status emb_workspace_status(const void* ws, size_t ws_bytes, int32_t* status, void* stream);

/* Layout of the workspace header, for callers that read or set it directly:
 * the uint32 at offset 0 is the generation g of the last dedup call (the
 * next call has generation g + 1, or 1 after 0xffffffff), and the uint64 at
 * the offset returned here holds (generation << 32) | error bits of the last
 * call that set any; its bits belong to a call only while its generation is
 * that call's. */
size_t emb_workspace_error_offset(void);

const char* emb_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* EMB_H */
