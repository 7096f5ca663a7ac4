/*
 * gear.h - C ABI of the MI355X (gfx950) experience-replay library.
 *
 * The library keeps a fixed-capacity store of trajectories as column tables
 * and runs the data-parallel hot path of GPU-centric experience replay
 * (GEAR, Wang et al., arXiv 2310.05205) on one GPU:
 *   selection  - FIFO / LIFO / uniform / prioritized (prefix scan over the
 *                priorities, then one search per uniform draw),
 *                importance-sampling weights, priority-update scatter;
 *   collection - gather of fixed-length windows of selected trajectories
 *                into contiguous per-column batches, from a table held in
 *                HBM or in pinned host memory read zero-copy by the kernel.
 *
 * Conventions for every call:
 *   - Return value: GEAR_OK (0) or a negative GEAR_E_* code, with a message
 *     for the calling thread in gear_last_error().  A call that returns
 *     GEAR_E_INVAL, GEAR_E_EMPTY or GEAR_E_INSUFFICIENT has enqueued nothing
 *     and left the table unchanged.  After GEAR_E_HIP or GEAR_E_NOMEM from a
 *     call that enqueues work, part of that work may have been enqueued or
 *     recorded (an insertion may have written some columns, an allocation
 *     released some victims); the table should then be closed.
 *   - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *     Every device-side effect is enqueued on `stream` and is asynchronous
 *     to the host.  Calls do not wait for the device, except:
 *     gear_table_sync(), which exists to; gear_table_create,
 *     gear_table_use_allocator and gear_table_destroy, which synchronise the
 *     device at set-up and tear-down; calls that pass an index list through
 *     the table's four pinned staging slots (gear_allocate, gear_commit,
 *     gear_write_rows, and gear_insert with an index manager), which wait
 *     only when every slot is still being read by earlier work; and copies
 *     from pageable host memory, which HIP performs synchronously.
 *   - Pointers named d_* are device memory (hipMalloc, or a torch CUDA
 *     tensor's data pointer) on the table's device.  They are owned by the
 *     caller and must stay valid until the enqueued work has completed.
 *   - A table is not thread-safe.  All calls on one table must be ordered:
 *     issue them from one host thread, on one stream, or order the streams
 *     with events.  Separate tables are independent.  One exception on the
 *     device side: gear_collect reads only the columns and the caller's index
 *     and start buffers, which selection and priority updates never write,
 *     so its kernels may run on another stream concurrently with selection
 *     (gear_select, the shard calls) and gear_update_priorities of the same
 *     table, as long as the host calls still come from one thread and the
 *     index buffers it reads are not rewritten meanwhile.  Never concurrently
 *     with insertion, allocation or row writes, which change the columns.
 *   - HIP graph capture: a captured call replays the kernels and arguments
 *     it chose when it was captured.  These calls choose them from nothing
 *     that their replays change, so captures of them replay correctly:
 *       gear_collect and gear_select_prioritized_noalloc;
 *       gear_select_collect;
 *       gear_select with GEAR_FIFO, GEAR_LIFO, GEAR_UNIFORM or GEAR_TOPK,
 *         and with GEAR_PRIORITIZED on a table of at most
 *         GEAR_SMALL_SELECT_MAX_N slots, for batches of at most
 *         GEAR_SMALL_SELECT_MAX_B and without GEAR_OPT_INCREMENTAL_TREE
 *         (one launch, no sum tree);
 *       gear_update_priorities without GEAR_OPT_INCREMENTAL_TREE.
 *     They read the table's ring position, live count and options when
 *     captured, so no insertion, allocation, commit or option change may
 *     come between a capture and its replays.  Prioritized selection on
 *     larger tables decides at each call whether to rebuild the sum tree,
 *     and insertion, allocation and commits change host-side queues and
 *     counters, so a replay would repeat stale decisions: call those
 *     directly.
 *   - A HIP error left pending by an earlier call outside the library (a
 *     failed allocation, say) is cleared when a library call starts, so a
 *     return code describes only that call's own work.
 *   - Conditions only the device can see (all priorities zero, an index or
 *     window start out of range) are recorded in the table's device status
 *     word, returned and cleared by gear_table_sync().
 */
#ifndef GEAR_H
#define GEAR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define GEAR_OK              0
#define GEAR_E_INVAL        -1   /* invalid argument (null pointer, size out of range, ...) */
#define GEAR_E_NOMEM        -2   /* device or pinned host allocation failed */
#define GEAR_E_EMPTY        -3   /* selection from a table with nothing inserted */
#define GEAR_E_INSUFFICIENT -4   /* FIFO/LIFO asked for more trajectories than are live */
#define GEAR_E_HIP          -5   /* a HIP runtime call or kernel launch failed */

/* Bits of the device status word (gear_table_sync). */
#define GEAR_STATUS_NO_WEIGHT  1u  /* prioritized select saw a priority total of 0 */
#define GEAR_STATUS_BAD_INDEX  2u  /* collect/update saw an index or start out of range */
#define GEAR_STATUS_INTERNAL   4u  /* a TopK selection found its own counts inconsistent (priorities
                                       changed while it ran, against the ordering rule, or a
                                       library defect); its output is incomplete */

/* Where the column tables live. */
#define GEAR_DEVICE       0  /* HBM of the table's GPU */
#define GEAR_HOST_PINNED  1  /* page-locked host memory, mapped and read zero-copy by kernels */

/* Selection strategies (GEAR Sec. 1 list of strategies; Sec. 3.3). */
#define GEAR_FIFO         0
#define GEAR_LIFO         1
#define GEAR_UNIFORM      2
#define GEAR_PRIORITIZED  3
#define GEAR_TOPK         4  /* deterministic: the highest priorities (Sec. 3.3, decentralized selection) */

/* Table options (gear_table_set_options). */
#define GEAR_OPT_INCREMENTAL_TREE 1u  /* updates maintain the selection sum tree in place */
#define GEAR_OPT_IS_GLOBAL_MIN    2u  /* IS weights (p_min / p_b)^beta with p_min the smallest
                                         non-zero priority of the whole table, not of the
                                         batch (every select after a change rescans; updates
                                         then do not maintain the tree) */
#define GEAR_OPT_GATHER_SHARE_CU  4u  /* long gathers from an HBM table hold at most 2
                                         workgroups per CU instead of 4, so that kernels
                                         on other streams start sooner beside them; the
                                         gather itself runs about 1% slower.  Results
                                         are unchanged. */

/* Limits. */
#define GEAR_MAX_CAPACITY  (1ll << 30)  /* keeps every priority total below 2^62 */
#define GEAR_MAX_COLUMNS   64
#define GEAR_MAX_BATCH     (1 << 24)
#define GEAR_MAX_TOPK      16384        /* B limit of GEAR_TOPK */
#define GEAR_NOALLOC_MAX_N (1 << 24)    /* N limit of gear_select_prioritized_noalloc */
#define GEAR_NOALLOC_SCRATCH_BYTES 536832  /* its fixed device scratch per GPU */
#define GEAR_SMALL_SELECT_MAX_N 16384  /* prioritized selection over at most this many slots, */
#define GEAR_SMALL_SELECT_MAX_B 2048   /* for batches up to this size and without the incremental
                                          tree, runs in one launch and keeps no sum tree */

typedef struct gear_table gear_table;

/* Element types of typed columns (gear_column.dtype).  The library moves
 * bytes and never interprets them; the type fixes the element size and
 * lets a binding hand out typed views of gathered batches. */
#define GEAR_DTYPE_U8    0   /* 1 byte */
#define GEAR_DTYPE_I8    1   /* 1 */
#define GEAR_DTYPE_U16   2   /* 2 */
#define GEAR_DTYPE_I16   3   /* 2 */
#define GEAR_DTYPE_F16   4   /* 2, IEEE binary16 */
#define GEAR_DTYPE_BF16  5   /* 2, bfloat16 */
#define GEAR_DTYPE_U32   6   /* 4 */
#define GEAR_DTYPE_I32   7   /* 4 */
#define GEAR_DTYPE_F32   8   /* 4 */
#define GEAR_DTYPE_U64   9   /* 8 */
#define GEAR_DTYPE_I64  10   /* 8 */
#define GEAR_DTYPE_F64  11   /* 8 */
#define GEAR_MAX_NAME   63   /* longest column name, bytes */

/* A typed column (Sec. 3.2, shard storage format: each field has a name and
 * a fixed per-step shape, set when the store is created).  One step holds
 * elems_per_step elements of dtype, i.e. elem_bytes = size(dtype) *
 * elems_per_step; the per-step shape itself (for example 8 x 64) is the
 * caller's, the library keeps only the element count. */
typedef struct {
    const char *name;        /* 1 .. GEAR_MAX_NAME bytes, unique in the table; copied */
    int32_t dtype;           /* GEAR_DTYPE_* */
    int32_t elems_per_step;  /* >= 1 */
} gear_column;

/*
 * gear_table_create - allocate an empty store (Sec. 3.2, shard storage
 * format: one column table per field type, each a contiguous array of
 * `capacity` equal blocks; a block holds one field of one trajectory as T
 * steps of elem_bytes[c] bytes; all tables share the capacity).
 *
 *   elem_bytes  host array of ncols sizes, bytes per step of each column (>= 1)
 *   ncols       0 .. GEAR_MAX_COLUMNS (0 gives a selection-only store)
 *   capacity    number of trajectory slots N, 1 .. GEAR_MAX_CAPACITY
 *   T           steps per trajectory, >= 1
 *   residency   GEAR_DEVICE or GEAR_HOST_PINNED
 *   device      HIP device ordinal that runs the kernels
 *   out         receives the table handle
 *
 * Column c is laid out as [capacity][T][elem_bytes[c]] bytes, all zero
 * at creation (pinned columns are cleared through their mapped address, at
 * host-link speed).  The store
 * also owns the uint32 priority array [capacity] (zero = not selectable,
 * Sec. 3.2 index manager) in HBM, and the scan, search and scatter scratch,
 * all sized by `capacity` at creation; no later call allocates except
 * gear_table_use_allocator.
 * Errors: GEAR_E_INVAL, GEAR_E_NOMEM, GEAR_E_HIP.
 */
int gear_table_create(const int64_t *elem_bytes, int32_t ncols, int64_t capacity, int32_t T,
                      int32_t residency, int32_t device, gear_table **out);

/*
 * gear_table_create_columns - gear_table_create with typed, named columns
 * (Sec. 3.2: the storage format is defined by the fields and their shapes).
 * Column c has elem_bytes = size(cols[c].dtype) * cols[c].elems_per_step and
 * the same layout, residency and ownership as above; names and types are
 * kept with the table (gear_table_column_info, gear_table_find_column).
 *
 *   cols   host array of ncols descriptors (0 .. GEAR_MAX_COLUMNS; the
 *          strings are copied, so they need not outlive the call)
 *
 * Errors: GEAR_E_INVAL (NULL or repeated name, name too long, unknown dtype,
 * elems_per_step < 1, and as gear_table_create), GEAR_E_NOMEM, GEAR_E_HIP.
 */
int gear_table_create_columns(const gear_column *cols, int32_t ncols, int64_t capacity, int32_t T,
                              int32_t residency, int32_t device, gear_table **out);

/* gear_table_column_info - name, dtype and elements per step of column c.
 * A table made by gear_table_create has byte columns: name "c<index>",
 * GEAR_DTYPE_U8, elems_per_step = elem_bytes.  *name stays valid while the
 * table exists.  Any output may be NULL.  Errors: GEAR_E_INVAL. */
int gear_table_column_info(const gear_table *t, int32_t c, const char **name, int32_t *dtype,
                           int32_t *elems_per_step);

/* gear_table_find_column - index of the column called `name` (for the
 * col_ids of gear_collect).  Errors: GEAR_E_INVAL (NULL argument, no such
 * column; *c is then -1). */
int gear_table_find_column(const gear_table *t, const char *name, int32_t *c);

/* gear_table_destroy - synchronize the table's device and free all its
 * memory.  NULL is accepted.  Errors: GEAR_E_HIP. */
int gear_table_destroy(gear_table *t);

/*
 * gear_insert - append n trajectories with FIFO removal (Sec. 3.2, insertion
 * and deletion: once the store is full the oldest trajectory is the
 * victim).  Insertion number k (counted from 0 over the table's life) is
 * written to slot k mod capacity; when n > capacity only the last
 * `capacity` rows are kept, as if written one after another.
 *
 *   n           number of rows, >= 0
 *   col_src     host array of ncols pointers; col_src[c] holds n*T*elem_bytes[c]
 *               bytes ([n][T][elem_bytes[c]]), host or device memory
 *               (may be NULL when ncols == 0)
 *   priorities  n uint32 values, host or device memory; 0 inserts an
 *               unselectable trajectory
 *
 * Copies are enqueued on `stream`; sources must stay valid until they
 * complete.  Updates the host-side insertion count at once.
 * Errors: GEAR_E_INVAL, GEAR_E_HIP.
 */
int gear_insert(gear_table *t, int64_t n, const void *const *col_src, const uint32_t *priorities,
                void *stream);
/* On a table with an index manager, gear_insert is one gear_allocate of n,
 * gear_write_rows into the allocated slots, and one gear_commit of the n
 * indices with `priorities` (GEAR_E_INSUFFICIENT if pending + n would exceed
 * the maximum). */

/*
 * Index manager (Sec. 3.2): a block allocator with one queue of free indices,
 * and a status table in which the priority of an index that is free or still
 * being written is zero.  A table with an index manager inserts by
 * gear_allocate -> in-place writes -> gear_commit (Sec. 3.2, trajectory
 * insertion and deletion) instead of the ring above; FIFO, LIFO and uniform
 * selection then follow the commit order, and the live count is the number
 * of committed indices.
 */

/*
 * gear_table_use_allocator - give the table an index manager.  Must be
 * called before anything is inserted.
 *
 *   removal         GEAR_FIFO (release the oldest commit) or GEAR_LIFO (the
 *                   newest) when an index is requested and none is free, or
 *                   when committed + pending indices have reached the maximum
 *   max_selectable  the preset maximum, in [1, capacity]
 *
 * Allocates the manager's arrays: 4 + 1 bytes per slot in HBM and 9 bytes per
 * slot of host memory, plus fixed staging buffers.  Every index starts free,
 * in index order.  Errors: GEAR_E_INVAL, GEAR_E_NOMEM, GEAR_E_HIP.
 */
int gear_table_use_allocator(gear_table *t, int32_t removal, int64_t max_selectable);

/*
 * gear_allocate - request n indices for new trajectories (Sec. 3.2: the
 * client asks the block allocator for free indices).  Indices come from the
 * front of the free queue; whenever none is free, or committed + pending
 * indices have reached the maximum, a victim is released first (its index
 * joins the back of the free queue).
 *
 *   n        >= 0; pending + n must not exceed max_selectable
 *   idx_out  host int64[n] receives the indices, in dequeue order
 *
 * The victims' priorities are zeroed by work enqueued on `stream`, before
 * anything the caller enqueues later.  The blocks of index i in column c are
 * base_c + i*T*elem_bytes[c] (gear_table_column); the caller fills them in
 * place, ordered after this call's stream work, then commits.
 * Errors: GEAR_E_INVAL (no index manager, n < 0, NULL idx_out),
 * GEAR_E_INSUFFICIENT (pending would exceed the maximum; nothing changes),
 * GEAR_E_HIP.
 */
int gear_allocate(gear_table *t, int64_t n, int64_t *idx_out, void *stream);

/*
 * gear_commit - make pending indices selectable (Sec. 3.2: commit updates
 * the status table).  Sets their priorities and appends them to the commit
 * order in the order given.
 *
 *   idx         host int64[n]; each must be pending (allocated, not yet
 *               committed) and appear once
 *   priorities  n uint32 values, host or device memory, valid until the
 *               enqueued copies complete; 0 commits an unselectable index
 *
 * Errors: GEAR_E_INVAL (no index manager, an index not pending or repeated;
 * nothing changes), GEAR_E_HIP.
 */
int gear_commit(gear_table *t, int64_t n, const int64_t *idx, const uint32_t *priorities, void *stream);

/*
 * gear_write_rows - write n trajectories into given slots in place (the
 * client's write of Sec. 3.2, for data already on a device): row r of every
 * column source goes to slot idx[r].  Any table; with an index manager the
 * slots are normally ones just allocated, committed afterwards.
 *
 *   idx      host int64[n], slots in [0, capacity)
 *   col_src  host array of ncols pointers, col_src[c] holding n*T*elem_bytes[c]
 *            bytes ([n][T][elem_bytes[c]]); device or pinned host memory is
 *            read by one scatter kernel per column, pageable host memory by
 *            one copy per run of consecutive slots
 *
 * Enqueued on `stream`; sources must stay valid until it completes.  The
 * rows of a slot listed twice are written in unspecified order.
 * Errors: GEAR_E_INVAL, GEAR_E_HIP.
 */
int gear_write_rows(gear_table *t, int64_t n, const int64_t *idx, const void *const *col_src, void *stream);

/* gear_allocator_info - committed, pending and free index counts of a table
 * with an index manager.  Any output may be NULL.  Errors: GEAR_E_INVAL. */
int gear_allocator_info(const gear_table *t, int64_t *committed, int64_t *pending, int64_t *free_count);

/*
 * gear_select - choose B trajectories and an L-step window in each (Sec. 1
 * strategies; Sec. 3.3 centralized selection: weighted sampling is a prefix
 * sum over the weights followed by a binary search for each uniformly drawn
 * number; Sec. 3.2: items with priority zero are never selected).
 *
 *   strategy  GEAR_FIFO: the B oldest live trajectories, oldest first.
 *             GEAR_LIFO: the B newest, newest first.
 *             GEAR_UNIFORM: B draws with replacement, uniform over live slots.
 *             GEAR_PRIORITIZED: B draws with replacement, slot i with
 *             probability p_i / S, S the sum of all priorities.
 *             GEAR_TOPK: the B slots with the highest non-zero priorities,
 *             higher priority first and the lower slot first among equal
 *             priorities; if fewer than B slots have non-zero priority the
 *             remaining draws get idx = -1, start = 0, weight 0 and
 *             GEAR_STATUS_NO_WEIGHT is set.
 *   B         1 .. GEAR_MAX_BATCH (FIFO/LIFO: at most the live count;
 *             TOPK: at most GEAR_MAX_TOPK)
 *   L         window length in steps, 1 .. T
 *   seed      draw b uses splitmix64 outputs 2b (index) and 2b+1 (start) of
 *             the stream seeded with `seed`; a draw is floor(u * n / 2^64)
 *   beta      importance-sampling exponent (used only when d_weights != NULL)
 *   d_idx     out, int64[B]: selected slot per draw
 *   d_start   out, int32[B]: window start, uniform on [0, T-L]
 *   d_weights out, float[B] or NULL: prioritized: (n*P(i))^-beta normalised
 *             by the batch maximum (n = live count); other strategies: 1
 *
 * A prioritized select rescans the priorities only if an insert or update
 * changed them since the last scan.  If all priorities are zero the device
 * writes idx = -1, start = 0, weight = 0 and sets GEAR_STATUS_NO_WEIGHT.
 * Errors: GEAR_E_INVAL, GEAR_E_EMPTY (nothing inserted), GEAR_E_INSUFFICIENT,
 * GEAR_E_HIP.
 */
int gear_select(gear_table *t, int32_t strategy, int32_t B, int32_t L, uint64_t seed, float beta,
                int64_t *d_idx, int32_t *d_start, float *d_weights, void *stream);

/*
 * gear_collect - gather L consecutive steps of the requested columns of each
 * selected trajectory into contiguous batches (Sec. 3.2: a client reads a
 * range of timesteps of a subset of fields; Sec. 3.4: one collection kernel
 * reads the selected blocks of each requested table, from pinned host memory
 * without a CPU copy).  For draw b, step t < L and requested column j:
 *     out[j][b][t][:] = column col_ids[j], slot d_idx[b], step d_start[b] + t
 *
 *   d_idx, d_start  device int64[B], int32[B] (as written by gear_select)
 *   B, L            1 .. GEAR_MAX_BATCH, 1 .. T
 *   col_ids         host int32[ncols] column numbers, or NULL for all columns
 *   ncols           number of requested columns (table's ncols when col_ids is NULL)
 *   d_out           host array of ncols device pointers; d_out[j] receives
 *                   B*L*elem_bytes[col_ids[j]] bytes laid out [B][L][elem_bytes]
 *
 * Index -1 marks a draw with no trajectory (a missing TopK entry, a draw
 * another shard owns): its window is zero bytes.  A draw whose index is
 * otherwise outside [0, capacity), or whose start lies outside [0, T-L],
 * also gets zero bytes and sets GEAR_STATUS_BAD_INDEX.
 * Errors: GEAR_E_INVAL, GEAR_E_HIP.
 */
int gear_collect(gear_table *t, const int64_t *d_idx, const int32_t *d_start, int32_t B, int32_t L,
                 const int32_t *col_ids, int32_t ncols, void *const *d_out, void *stream);

/*
 * gear_select_collect - gear_select followed by gear_collect, in one launch,
 * for the strategies whose draws are index arithmetic and counter-based
 * random numbers (Sec. 3.3: FIFO and LIFO are deterministic, uniform
 * sampling needs no weights), so the gather computes each window's slot and
 * start itself instead of reading them from memory.  The results are those
 * of gear_select(strategy, B, L, seed) with weights, then gear_collect over
 * its d_idx and d_start: the same slots, starts, weights (all 1) and bytes.
 *
 *   strategy        GEAR_FIFO, GEAR_LIFO or GEAR_UNIFORM
 *   B, L, seed      as for gear_select
 *   d_idx, d_start  device int64[B], int32[B]: receive the draws
 *   d_weights       device float[B] receiving 1 per draw, or NULL
 *   col_ids, ncols, d_out  as for gear_collect
 *
 * Errors: GEAR_E_INVAL (NULL argument, another strategy, B, L or a column
 * out of range; nothing enqueued), GEAR_E_EMPTY (nothing inserted),
 * GEAR_E_INSUFFICIENT (FIFO/LIFO with B above the live count), GEAR_E_HIP.
 */
int gear_select_collect(gear_table *t, int32_t strategy, int32_t B, int32_t L, uint64_t seed, int64_t *d_idx,
                        int32_t *d_start, float *d_weights, const int32_t *col_ids, int32_t ncols,
                        void *const *d_out, void *stream);

/*
 * Selection over G shards, one GPU's share (Sec. 3.3 centralized and
 * decentralized selection; Sec. 3.4: global index = shard * capacity +
 * local index).  Each shard is a table on its own GPU; the exchanges between
 * the calls (an all-gather of G totals, an all-reduce of B values, a gather
 * of G*K candidates) are the caller's collectives.
 */

/*
 * gear_shard_total - the sum of the table's priorities (uint64), written to
 * device memory d_total (rescanning first if needed): this shard's entry of
 * the totals that every shard needs.  Errors: GEAR_E_INVAL, GEAR_E_HIP.
 */
int gear_shard_total(gear_table *t, uint64_t *d_total, void *stream);

/*
 * gear_select_shard - shard g's part of prioritized selection over G shards.
 * Every shard draws the same numbers r_b in [0, S) with S the sum of
 * d_totals (device uint64[G], identical on every shard; the sum must fit in
 * 64 bits) and resolves the draws in [P_g, P_g + S_g), P_g the sum of the
 * totals before g, exactly as gear_select(GEAR_PRIORITIZED) over the
 * concatenated shards.
 *
 *   base        added to the slot of an owned draw (g * capacity gives global
 *               indices, 0 local ones)
 *   d_idx       device int64[B]: slot + base for owned draws, -1 otherwise
 *   d_start     device int32[B]: window starts of all B draws (the same on
 *               every shard)
 *   d_sel_prio  device uint32[B] or NULL: the priority of each owned draw,
 *               0 otherwise (an all-reduce-max over shards gives every
 *               shard the full list for gear_is_weights)
 *
 * When S is 0 every draw gets -1 and GEAR_STATUS_NO_WEIGHT is set.
 * Errors: GEAR_E_INVAL, GEAR_E_HIP.
 */
int gear_select_shard(gear_table *t, int32_t G, int32_t g, const uint64_t *d_totals, int64_t base, int32_t B,
                      int32_t L, uint64_t seed, int64_t *d_idx, int32_t *d_start, uint32_t *d_sel_prio,
                      void *stream);

/*
 * gear_is_weights - importance-sampling weights (p_min / p_b)^beta of B
 * selected priorities d_sel_prio (device uint32[B]), p_min the smallest
 * non-zero one, computed in double and rounded once; 0 where p_b is 0.  The
 * same weights gear_select returns.  Uses the table's scratch and stream
 * order.  Errors: GEAR_E_INVAL, GEAR_E_HIP.
 */
int gear_is_weights(gear_table *t, const uint32_t *d_sel_prio, int32_t B, float beta, float *d_weights,
                    void *stream);

/*
 * gear_topk_merge - the global top-K of G local top-K lists (Sec. 3.3,
 * decentralized selection: the central GPU computes the global top-K of the
 * shards' partial results).  Runs on the current HIP device.
 *
 *   d_prio, d_gidx  device uint32[G][K] and int64[G][K]: list g is shard g's
 *                   gear_select(GEAR_TOPK) result as global indices, with
 *                   the priorities; sorted (priority descending, index
 *                   ascending), entries with index -1 last
 *   T, L, seed      as for gear_select: output position b gets the window
 *                   start drawn for draw b
 *   d_idx, d_start  device int64[K], int32[K]; positions past the candidates
 *                   get -1 and 0
 *   d_weights       device float[K] or NULL: 1, or 0 past the candidates
 *   d_out_prio      device uint32[K] or NULL: the merged priorities
 *
 * Equals gear_select(GEAR_TOPK) over the concatenated shards when the lists
 * are sorted as stated.  Errors: GEAR_E_INVAL, GEAR_E_HIP.
 */
int gear_topk_merge(const uint32_t *d_prio, const int64_t *d_gidx, int32_t G, int32_t K, int32_t T, int32_t L,
                    uint64_t seed, int64_t *d_idx, int32_t *d_start, float *d_weights, uint32_t *d_out_prio,
                    void *stream);

/*
 * gear_select_prioritized_noalloc - gear_select(GEAR_PRIORITIZED) over a
 * caller's priority array, allocating nothing.  For callers that cannot
 * allocate device memory: code being captured into a HIP graph, serving
 * loops that forbid allocation.  It keeps no host-side state besides the
 * scratch address, so a captured call replays correctly with the array's
 * contents at replay time.  Runs on the current HIP device.
 *
 *   d_priority  device uint32[N]: slot i is drawn with probability p_i / S,
 *               S the sum; zero is never drawn
 *   N           1 .. GEAR_NOALLOC_MAX_N (all N slots are live)
 *   T, L, B, seed, beta, d_idx, d_start, d_weights
 *               as for gear_select: the same draws, windows and weights a
 *               table holding these priorities returns
 *
 * Scratch: the sum tree (GEAR_NOALLOC_SCRATCH_BYTES in all, sized for
 * GEAR_NOALLOC_MAX_N) lives in a fixed device array of the library, one per
 * GPU, held until the process ends.  Every call on a GPU shares it, so calls
 * that overlap on one GPU (different streams, or different host threads,
 * without ordering) race and give wrong draws; order them.  When every
 * priority is zero, each draw gets idx = -1, start = 0, weight 0 (there is
 * no status word to read).
 * Errors: GEAR_E_INVAL (NULL pointer, N above GEAR_NOALLOC_MAX_N, B, L or T
 * out of range, NaN beta; nothing enqueued), GEAR_E_HIP.
 */
int gear_select_prioritized_noalloc(const uint32_t *d_priority, int64_t N, int32_t T, int32_t B, int32_t L,
                                    uint64_t seed, float beta, int64_t *d_idx, int32_t *d_start,
                                    float *d_weights, void *stream);

/*
 * gear_update_priorities - write new priorities for selected slots (Sec. 3.2:
 * the status table holds the priorities; changes to it are gathered, then
 * applied).  Applied as if in batch order: when a slot appears more than
 * once, the last occurrence's value wins.
 *
 *   d_idx            device int64[B], slots in [0, live count) (a table
 *                    with an index manager: [0, capacity))
 *   d_new_priorities device uint32[B]
 *   B                0 .. GEAR_MAX_BATCH
 *
 * An index outside that range is skipped and sets GEAR_STATUS_BAD_INDEX.  With
 * an index manager, the update of an index that is not committed (released,
 * or being written again) is dropped, so it never becomes selectable.
 * Errors: GEAR_E_INVAL, GEAR_E_HIP.
 */
int gear_update_priorities(gear_table *t, const int64_t *d_idx, const uint32_t *d_new_priorities,
                           int32_t B, void *stream);

/*
 * gear_table_set_options - set the table's GEAR_OPT_* bits (replacing the
 * previous set).  Takes effect for the next calls; switching
 * GEAR_OPT_IS_GLOBAL_MIN on makes the next prioritized select rescan.
 * Errors: GEAR_E_INVAL (NULL table, unknown bits).
 */
int gear_table_set_options(gear_table *t, uint32_t options);

/*
 * gear_table_sync - wait for `stream`, then read and clear the device status
 * word.  *device_status (may be NULL) receives the GEAR_STATUS_* bits set
 * since the previous sync.  The only blocking call.
 * Errors: GEAR_E_INVAL, GEAR_E_HIP.
 */
int gear_table_sync(gear_table *t, void *stream, int32_t *device_status);

/* gear_table_info - live count (min(next_seq, capacity) for a ring table,
 * the committed count with an index manager) and the number of insertions
 * (commits) so far.  Either output may be NULL. */
int gear_table_info(const gear_table *t, int64_t *count, uint64_t *next_seq);

/*
 * gear_table_column - base address of column c ([capacity][T][elem_bytes]):
 * a device pointer for GEAR_DEVICE tables, a device-accessible mapped
 * pointer for GEAR_HOST_PINNED ones; *host_ptr receives the host-side
 * address of a pinned table (NULL for device tables).  Writing through it
 * is the in-place insertion path (Sec. 3.2, allocate/commit); the caller
 * orders such writes with the table's stream.  Any output may be NULL.
 */
int gear_table_column(const gear_table *t, int32_t c, void **base, void **host_ptr,
                      int64_t *elem_bytes);

/* gear_table_priorities - device pointer of the uint32 priority array
 * [capacity].  Reading it is safe after the stream work that wrote it. */
int gear_table_priorities(const gear_table *t, uint32_t **d_priority);

/* gear_last_error - message describing the last failed call on this
 * thread ("" if none).  Valid until the next call on the same thread. */
const char *gear_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GEAR_H */
