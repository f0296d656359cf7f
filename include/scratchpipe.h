/*
 * scratchpipe.h - C ABI of an MI355X embedding-training scratchpad.
 *
 * The library trains embedding tables that live in host memory through a
 * GPU-resident cache (the "scratchpad": Storage plus Hit-Map, Sec. IV-D).
 * Because the sparse IDs of upcoming mini-batches are already known from the
 * training data (Sec. IV-A), every batch is planned before it is trained: its
 * missing rows are brought in and victims are chosen only among slots that no
 * batch of the look-forward window uses (Sec. IV-C), so forward and backward
 * always hit in HBM.  One training step is
 *
 *     sp_plan(window)  ->  sp_forward(ticket)  ->  sp_backward_update(ticket)
 *
 * and sp_flush() makes the host tables authoritative again.
 *
 * Conventions shared by every call:
 *  - Batches are table-major CSR: ids[] holds table 0's row IDs, then table
 *    1's, ...; bag g = t*B + b spans ids[bag_off[g] .. bag_off[g+1]); row IDs
 *    are local to their table; bag_off has T*B+1 entries, bag_off[0] = 0 and
 *    bag_off[T*B] = nnz.
 *  - Pooled outputs and their gradients are fp32 [T][B][D] in device memory
 *    owned by the caller (row g = t*B + b).
 *  - Return value: SP_OK (0) or a negative sp_status.  After SP_ERR_HIP the
 *    context is unusable and only sp_destroy is valid.  sp_last_error()
 *    describes the last failure.
 *  - One context is used from one host thread at a time.
 */
#ifndef SCRATCHPIPE_H
#define SCRATCHPIPE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t sp_status;
#define SP_OK 0
#define SP_ERR_INVALID_ARG (-1) /* bad config, bad IDs or offsets, bad pointer        */
#define SP_ERR_OOM (-2)         /* device or pinned allocation failed                  */
#define SP_ERR_CAPACITY (-3)    /* some table has more misses than unheld slots        */
#define SP_ERR_SEQUENCE (-4)    /* call out of plan -> forward -> backward order       */
#define SP_ERR_HIP (-5)         /* a HIP runtime call failed (sticky)                  */
#define SP_ERR_STATE (-6)       /* context unusable (after SP_ERR_HIP) or null handle  */

/* sp_config.policy: how victims are chosen among unheld slots (Sec. VI-E
 * names LRU as the default and random eviction and LFU as alternatives).
 * Every policy takes the slots with the smallest (priority, slot):
 *   LRU     priority = last plan that used the slot (never used: first)
 *   LFU     priority = plans that used the slot since its current row was
 *           placed there, the placing plan included (never used: 0, first)
 *   RANDOM  priority = 0 for a never-used slot, else 1 + the top 24 bits of
 *           output number u * 2^31 + g + 1 of a SplitMix64 stream started at
 *           sp_config.seed (u = plan index, g = global slot): a fresh uniform
 *           draw per slot and plan */
#define SP_POLICY_LRU 0
#define SP_POLICY_LFU 1
#define SP_POLICY_RANDOM 2

/* sp_config.hold_past at most: earlier batches a plan may hold as well */
#define SP_MAX_HOLD_PAST 4

/* sp_config.prefetch at most: successor batches a plan may fill ahead */
#define SP_MAX_PREFETCH 4

/* sp_config.flags */
#define SP_FLAG_DEBUG_SYNC 0x1u /* synchronise the device at the end of every call     */
#define SP_FLAG_TIMING 0x2u     /* time forward/backward/plan/fill kernels with events */
#define SP_FLAG_EVENT_WAITS 0x4u /* wait on events where the library otherwise waits on
                                    stream values (hipStreamWaitValue64); for tools
                                    that run one dispatch at a time, under which a
                                    value wait would wait for a dispatch held back */
#define SP_FLAG_POISON 0x8u     /* debugging aid, read by sp_create: Storage starts as
                                    NaN instead of zeros, and with the staged fill the
                                    device staging of filled rows is set to NaN once
                                    the fill has used it, so a read of a slot before
                                    its fill landed, or of stale staging, shows up as
                                    NaN in outputs and tables                        */
#define SP_FLAG_DEFER_SORTS 0x10u /* debugging aid, staged fill: batches prepared ahead
                                    are always sorted behind the update of the plan
                                    that received them (sp_backward_update enqueues
                                    them; the allocation-free variant leaves them to
                                    the next sp_plan), as they are by default only
                                    behind a write-back copy above 256 MiB           */

/* sp_config.fill: how missing rows reach the scratchpad (Sec. IV-B) */
#define SP_FILL_MAPPED 0 /* the move kernel reads them straight from pinned,
                            device-mapped host tables over the host link          */
#define SP_FILL_STAGED 1 /* host threads gather them from the tables into pinned
                            staging ([Collect]), copies take them to the device in
                            pieces as they are gathered ([Exchange]) and the move
                            kernel writes them into their slots ([Insert]); the
                            tables may then be any host memory                    */

typedef struct sp_ctx *sp_handle;

typedef struct {
    int32_t num_tables;         /* T, 1..64                                            */
    const int64_t *rows;        /* [T] rows per table, 1 .. 2^25                       */
    int32_t dim;                /* D, fp32 elements per row; multiple of 4, <= 256     */
    const int64_t *slots;       /* [T] scratchpad slots per table, 1 .. rows[t]         */
    int32_t lookahead;          /* L >= 0: successor batches a plan may hold           */
    float *const *host_tables;  /* [T] row-major [rows][D] fp32 host tables, caller-owned,
                                   must outlive the context, each 16-byte aligned; read
                                   on misses, written on evictions and flush.
                                   SP_FILL_MAPPED: pinned,
                                   device-mapped memory from sp_host_alloc (or
                                   hipHostMalloc with the mapped flag); SP_FILL_STAGED:
                                   any host memory                                   */
    int32_t max_batch;          /* largest B any batch will have; T * max_batch * dim * 4
                                   (the bytes of one [T*B][D] gradient) must stay
                                   below 4 GiB                                         */
    int64_t max_ids;            /* largest nnz any batch will have (all tables)        */
    uint32_t flags;             /* SP_FLAG_*                                           */
    int32_t device;             /* HIP device ordinal                                  */
    int32_t policy;             /* SP_POLICY_* (0 = LRU)                               */
    int32_t hold_past;          /* 0..SP_MAX_HOLD_PAST, and lookahead + 1 + hold_past
                                   <= 16: a plan also holds the rows of this many
                                   batches planned before it (the past window of
                                   Sec. IV-C), so no row a recent batch used is
                                   evicted; 0 = look-forward window only          */
    uint64_t seed;              /* SP_POLICY_RANDOM's stream                           */
    int64_t max_table_ids;      /* 0, or the most IDs one table has in any batch: a
                                   batch with a table above it is rejected
                                   (SP_ERR_INVALID_ARG).  With max_table_ids and
                                   max_batch both <= 8192 each table of a batch is
                                   sorted and deduplicated by one workgroup in LDS,
                                   the whole batch in one launch                    */
    int32_t prefetch;           /* depth d in 0 .. SP_MAX_PREFETCH (above lookahead it
                                   acts as lookahead): each plan also fills the rows
                                   of its next d window batches (window[1..d], those
                                   given) that are
                                   neither cached nor in an earlier window batch: the
                                   earlier fill of future misses that the multi-stage
                                   overlap of Sec. IV-C allows.  Per table the planned
                                   batch's misses come first, then window[1]'s rows,
                                   then window[2]'s, ..., each ascending; the capacity
                                   check counts them all, so SP_ERR_CAPACITY can come
                                   earlier than without prefetch.  0 = none        */
    int32_t fill;               /* SP_FILL_MAPPED (0) or SP_FILL_STAGED               */
} sp_config;

typedef struct {
    int32_t batch;              /* B, 0 .. max_batch                                   */
    int64_t nnz;                /* number of IDs, 0 .. max_ids                          */
    const int32_t *ids;         /* [nnz] row IDs, table-major                          */
    const int32_t *bag_off;     /* [T*B+1] bag offsets                                 */
    int32_t on_device;          /* 0: ids/bag_off are host memory, copied before sp_plan
                                   returns; 1: device memory, which must hold the batch
                                   when sp_plan is called (the library reads it on its
                                   own stream, with no order against the caller's
                                   streams: synchronise the stream that wrote it first)
                                   and stay unchanged until an sp_plan call that holds
                                   the batch (window index <= lookahead) has returned */
} sp_batch;

typedef struct {
    int64_t plans;              /* plans committed                                     */
    int64_t updates;            /* backward updates issued                              */
    int64_t lookups;            /* IDs planned (sum of nnz)                             */
    int64_t unique;             /* unique (table,row) keys planned                      */
    int64_t hits, misses;       /* unique keys found / not found in the Hit-Map         */
    int64_t evictions;          /* misses placed in a slot that held a row              */
    int64_t bytes_fill;         /* host -> HBM bytes of miss fills                      */
    int64_t bytes_writeback;    /* HBM -> host bytes of evicted rows                    */
    int64_t hash_rebuilds;
    int64_t chunks;             /* backward work chunks processed                       */
    int64_t min_capacity_margin;/* min over plans and tables of unheld slots - misses  */
    int64_t device_bytes;       /* device memory held by the context                    */
    int64_t pinned_bytes;       /* pinned staging held by the context                   */
    /* SP_FLAG_TIMING only: summed time in ms and number of timed launches.
     * forward, backward (per-chunk kernel) and combine (runs split over several
     * chunks, launched only when there are any) and fill (evicted-row
     * staging and miss fill, plans with misses only) are kernel execution
     * times; plan (the commit sequence: victims, Hit-Map, slot metadata)
     * spans its launch sequence. */
    double ms_forward, ms_backward, ms_combine, ms_plan, ms_fill;
    int64_t timed_forward, timed_backward, timed_combine, timed_plan, timed_fill;
    /* host time spent inside sp_plan, in ms: enqueueing ingest, enqueueing the
     * query, waiting for its counts, enqueueing the commit, and the mover
     * (including waits for the write-back thread) */
    double host_ms_ingest, host_ms_query, host_ms_wait, host_ms_commit, host_ms_mover;
    /* SP_FLAG_TIMING only: ingest of a batch (keys, sort, dedup, backward
     * chunks) and the query of a plan (hold marks and probe, from the moment
     * its stream reaches it, waits for ingests included) */
    double ms_ingest, ms_query;
    int64_t timed_ingest, timed_query;
    /* host time, in ms, that sp_plan spends before returning waiting until its
     * ingests have read the caller's window arrays */
    double host_ms_inputs;
    /* prefetch mode: rows filled for the next batch (included in misses,
     * evictions and bytes_fill, not in hits: hits count the planned batch's
     * keys found cached, prefetched ones included) */
    int64_t prefetched;
    /* SP_FILL_STAGED: host time of the fill thread gathering missing rows into
     * pinned staging, and host time the calling thread spent waiting for the
     * fill thread to enqueue a plan's fill (ms); SP_FLAG_TIMING: the span of a
     * plan's host-to-device copies of gathered rows, first start to last end */
    double host_ms_gather, host_ms_fill_join, ms_h2d;
    int64_t timed_h2d;
} sp_stats;

/* Per-plan decisions copied to the host for checking.  The caller allocates
 * every array with room for the planned batch's nnz entries.  Slots are global
 * (table t's slots follow tables 0..t-1).  Filled fields:
 *   u_table,u_row,hit,slot_u [n_unique]  the batch's unique keys, ascending
 *                                        (table,row); hit=1 if it was cached;
 *                                        slot_u = its slot after the plan
 *   inv,slot_of [nnz]                    index into u_*, slot of ids[j]
 *   m_table,m_row,v_slot,v_old_row,v_old_use [n_miss]
 *                                        misses in ascending (table,row), the
 *                                        slot each one gets, the row evicted
 *                                        from it (-1 if none) and that slot's
 *                                        previous last-use plan index (-1 if
 *                                        never used).  In prefetch mode these
 *                                        hold, per table, the planned batch's
 *                                        misses then the prefetched rows, and
 *                                        need room for the nnz of the planned
 *                                        batch and its d successors together */
typedef struct {
    int32_t *u_table, *u_row, *inv, *m_table, *m_row, *v_slot, *v_old_row, *v_old_use;
    int32_t *slot_u, *slot_of;
    uint8_t *hit;
    int64_t n_unique, n_miss, n_evict, nnz;
} sp_plan_dump;

/*
 * Create a context: allocates Storage (sum(slots) x D fp32), the Hit-Map hash,
 * per-slot metadata and holds, two int32 per row of every table (sum(rows) x 8
 * bytes: the row index behind the holds of filled rows), the window ring and
 * staging buffers on config->device, and four library streams at default
 * priority (plan, ingest, move and copy).
 * Nothing is cached initially.
 * Errors: SP_ERR_INVALID_ARG (config out of range; with SP_FILL_MAPPED a host
 * table that is not pinned and mapped), SP_ERR_OOM, SP_ERR_HIP.  *out is set
 * only on success; on failure everything allocated so far is freed.  For
 * testing that path, the environment variable SP_FAIL_ALLOC_AFTER=n makes the
 * allocation after the first n of this call fail with SP_ERR_OOM.
 * (Sec. IV-D "GPU scratchpad design": Storage and Hit-Map.)
 */
sp_status sp_create(const sp_config *config, sp_handle *out);

/* Batches after the hold window that sp_plan accepts for early sorting. */
#define SP_MAX_AHEAD 2

/*
 * Plan the next mini-batch.  window[0] is the batch to plan (ticket k = number
 * of plans so far) and window[1..] are the batches that follow it, n of them
 * in all, 1 <= n <= lookahead + 1 + SP_MAX_AHEAD.  The first
 * min(n, lookahead+1) batches form the hold window; any after them are only
 * sorted and deduplicated ahead of time (not held), which takes that work off
 * later plans' paths.  Handing over at least one such batch also lets this
 * plan issue the next plan's query right behind its own commit.  Batches
 * enter the device window
 * ring once, when first seen, and are not read again: the same batch must be
 * passed with the same content every time it appears (after a failed plan
 * all of that call's batches are read again on the next call).  Host window
 * buffers may be reused when the call returns; device ones once a call that
 * holds their batch has returned (a batch prepared ahead in device memory is
 * read asynchronously, before the query of the first plan that holds it).
 * The plan queries the Hit-Map
 * for window[0]'s unique keys, holds
 * every cached slot used by any window batch (and by the hold_past batches
 * planned before this one), takes for each table's misses the unheld slots
 * that come first under the policy (smallest priority first, ties by slot;
 * the ascending misses take them in that order), updates Hit-Map, slot keys,
 * last-use and use counts, and enqueues the evicted rows' write-back and the
 * misses' fill (Sec. IV-C "Putting everything together", Sec. IV-D
 * Algorithm 1; policies from Sec. VI-E).  With sp_config.prefetch = d the
 * misses also include the rows of window[1..d] that are neither cached nor in
 * an earlier window batch (after window[0]'s own misses, per table).  The host waits once for
 * per-table counts.
 * Requires the previous ticket's sp_backward_update to have been issued.
 * Transactional: on SP_ERR_INVALID_ARG (ID out of range, bad offsets, sizes
 * above the config) or SP_ERR_CAPACITY (misses > unheld slots in some table)
 * the scratchpad state is unchanged and the same ticket can be planned again.
 */
sp_status sp_plan(sp_handle h, const sp_batch *window, int32_t n, int64_t *ticket);

/*
 * Pooled forward of a planned batch: d_out[t*B+b][:] = sum of the Storage rows
 * of bag (t,b) (Sec. II-B "Forward propagation", sum reduction; empty bag ->
 * zeros).  Enqueued on `stream` (a hipStream_t; NULL = default stream) after
 * the ticket's fill, or, when the batch had no misses of its own (all its
 * rows cached before this plan, as with prefetch), after the ticket's commit
 * and the previous ticket's fill: this plan's fill touches none of its rows.
 * `ticket` must be the latest plan, not yet forwarded.
 * d_out: caller-owned device fp32 [T][B][D].  Errors: SP_ERR_SEQUENCE,
 * SP_ERR_INVALID_ARG (null d_out with B*T > 0).
 */
sp_status sp_forward(sp_handle h, int64_t ticket, float *d_out, void *stream);

/*
 * Backward and update of a forwarded batch: every unique row gets the sum of
 * the gradients of the bags that gathered it, positions in ascending order,
 * and Storage[row] -= lr * sum in place (Sec. II-B "Backpropagation"; plain
 * SGD).  d_grad: device fp32 [T][B][D].  Enqueued on `stream`.
 * Errors: SP_ERR_SEQUENCE, SP_ERR_INVALID_ARG.
 */
sp_status sp_backward_update(sp_handle h, int64_t ticket, const float *d_grad, float lr,
                             void *stream);

/*
 * For callers that cannot allocate device memory at call time or at all
 * outside set-up (code under graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): sp_backward_update with the partial sums of runs
 * split over several backward chunks kept in a fixed device array of 32 MiB
 * instead of the context's buffer.  The array exists once per GPU for the
 * life of the process; its address is taken in sp_create.  It holds the
 * partials of at most 32 MiB / (4 * dim) backward chunks, one chunk per run
 * of up to 16 positions of one key, so a batch with nnz * dim * 4 <= 32 MiB
 * always fits; a ticket above that (with a split run) is rejected with
 * SP_ERR_INVALID_ARG and nothing changes, and sp_backward_update can then be
 * called for it.  Every call on one GPU uses the same array: calls that
 * overlap on one GPU (contexts on different streams) race and must be
 * ordered by the caller.  Otherwise as sp_backward_update; it allocates
 * nothing.
 */
sp_status sp_backward_update_static(sp_handle h, int64_t ticket, const float *d_grad, float lr,
                                    void *stream);

/*
 * Synchronise everything and write every cached row back to its host table;
 * afterwards the host tables hold the trained model.  The scratchpad keeps
 * its contents, so training may continue.  (Evicted entries are dirty and must
 * be written back, Sec. IV-B; flush applies that to all entries.)
 */
sp_status sp_flush(sp_handle h);

/*
 * Wait until every effect of the calls so far is complete: all device work
 * (on the library's streams and the rest of the device) has finished and
 * every row evicted so far has been written back to its host table.  Unlike
 * sp_flush it writes no cached row back.  Training may continue afterwards.
 */
sp_status sp_sync(sp_handle h);

/* Counters since sp_create (synchronises pending timing events). */
sp_status sp_get_stats(sp_handle h, sp_stats *out);

/* Replace the context's SP_FLAG_* bits for the calls that follow, e.g. to
 * time only a sample of the steps.  SP_ERR_INVALID_ARG for unknown bits. */
sp_status sp_set_flags(sp_handle h, uint32_t flags);

/* Copy the decisions of the most recent plan (ticket must equal it) to host
 * arrays; for checking against a reference.  Synchronises the library stream. */
sp_status sp_debug_plan(sp_handle h, int64_t ticket, sp_plan_dump *out);

/* Wait for all work, join the write-back thread, free everything.  NULL is ok. */
void sp_destroy(sp_handle h);

/* Text of the last error on this context (or of the last failed sp_create
 * when h is NULL).  Valid until the next call on the context. */
const char *sp_last_error(sp_handle h);

/* Pinned, device-mapped host memory for host tables (hipHostMalloc with the
 * mapped and portable flags; exact size).  *ptr is set on SP_OK. */
sp_status sp_host_alloc(size_t bytes, void **ptr);
void sp_host_free(void *ptr);

#ifdef __cplusplus
}
#endif
#endif /* SCRATCHPIPE_H */
