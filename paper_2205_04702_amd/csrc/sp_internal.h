// Host-side declarations shared by the scratchpad library's translation units.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sp {

constexpr int MAX_TABLES = 64;
constexpr int MAX_PF = 4;        // successor batches a plan may prefetch
constexpr int MAX_WINDOW = 16;   // batches one plan may look at (lookahead <= 15)
constexpr int QUERY_TILE = 256;  // unique keys per block of the query (one per thread)
constexpr int SEL_BITS = 11;     // digit width of the LRU radix select
constexpr int SEL_BINS = 1 << SEL_BITS;

// Holds.  hold_to[slot] is the last plan whose hold set contains the slot: a
// slot is held at plan k when hold_to >= k.  A batch q's cached slots get
// q + hold_past when q enters the hold window, a filled row gets the last
// window batch holding its key plus hold_past, so every value lies within
// k .. k + lookahead + hold_past (< HOLD_SPAN) at plan k.  hcnt[t][v %
// HOLD_RING] counts table t's slots whose hold_to is v, for the live v.
constexpr int HOLD_SPAN = 16;
constexpr int HOLD_RING = 32;
static_assert(MAX_WINDOW <= HOLD_SPAN, "lookahead + hold_past < MAX_WINDOW <= HOLD_SPAN");
static_assert(HOLD_RING >= HOLD_SPAN + 2, "an expired count is cleared before its reuse");

// Single-pass scan: indices per tile, published words per tile (sum and
// inclusive prefix, two 32-bit halves each), tiles of nseg segments.
constexpr int LB_TILE = 2048;
constexpr int LB_WORDS = 4;
inline int64_t scan_tiles(int nseg, int64_t max_len)
{
    return (int64_t)nseg * ((max_len + LB_TILE - 1) / LB_TILE);
}

// Workspace of the single-pass scan; each stream that runs scans owns one.
struct ScanWs {
    uint64_t *status = nullptr;   // [4 * max_tiles] tile sums published by the scan, epoch-tagged
    uint32_t *counter = nullptr;  // tiles handed out so far (wraps)
    int32_t *err = nullptr;       // gets ERR_PLAN when a look-back stops waiting
    int64_t max_tiles = 0;
    uint32_t issued = 0;          // value *counter holds once every launch so far has run
    uint32_t epoch = 0;           // tag of the last launch
    bool overflow = false;        // a scan needed more than max_tiles tiles and was skipped
};

// Per-table constants passed by value to kernels.
struct Tables {
    int32_t T;
    int32_t row_bits;            // key = table << row_bits | row
    int64_t rows[MAX_TABLES];
    int64_t slot_base[MAX_TABLES + 1];
};

// Counters written by the planning kernels and copied to the host once per plan.
// Everything before err_sticky is cleared right after each copy, ready for
// the next query; err_sticky collects errors of later plan stages and of the
// scans and is never cleared.
struct DevCounters {
    int32_t err;                 // ERR_* bits of this plan's window (ids, offsets)
    int32_t n_unique;            // unique keys of the planned batch
    int32_t n_chunks;            // backward work chunks of the planned batch
    int32_t n_multi;             // its runs longer than one chunk
    int32_t miss[MAX_TABLES];
    int32_t held[MAX_TABLES];
    int32_t pf[MAX_PF][MAX_TABLES];  // rows of successor w + 1 to prefetch (prefetch mode)
    int32_t err_sticky;          // ERR_HASH_FULL / ERR_PLAN from any earlier commit
    int32_t pad2[3];
};
constexpr int COUNTERS_CLEARED = (int)(offsetof(DevCounters, err_sticky) / sizeof(int32_t));
constexpr int PART_COPIES = 64;  // copies of the per-table counters the probe adds into
// one copy: miss, held and the prefetch counts of each successor
constexpr int PART_WORDS = (2 + MAX_PF) * MAX_TABLES;
constexpr int COUNTER_WORDS = (int)(sizeof(DevCounters) / sizeof(int32_t));
constexpr int32_t ERR_ID_RANGE = 1, ERR_OFFSETS = 2, ERR_HASH_FULL = 4, ERR_PLAN = 8;
constexpr int32_t ERR_TABLE_IDS = 16;  // a table has more IDs than the configured bound

// Entries of a batch's list of runs longer than one chunk: such a run has at
// least chunk + 1 positions.
__host__ __device__ inline int64_t multi_capacity(int64_t max_ids, int chunk) { return max_ids / (chunk + 1) + 2; }

// Batches whose tables each have at most IG_MAX IDs (and at most IG_MAX bags)
// are ingested by one launch entirely in LDS, ingest_splits(T) workgroups per
// table, each owning a range of the table's rows (T * splits stays within the
// 256 compute units).
constexpr int IG_MAX = 8192;
constexpr int IG_SPLIT_MAX = 16;
inline bool ingest_in_lds(int64_t max_table_ids, int64_t B)
{
    return max_table_ids > 0 && max_table_ids <= IG_MAX && B <= IG_MAX;
}
inline int ingest_splits(int T) { return T <= 16 ? 16 : (T <= 32 ? 8 : 4); }

// One window-ring entry: a batch as it arrived plus its sort/dedup products.
struct BatchDev {
    int32_t *ids, *bag_off, *bag_of;  // raw CSR, bag of each position
    uint32_t *skeys, *perm;          // keys sorted ascending, position of each sorted key
    int32_t *sbag;                   // bag of each sorted position
    uint32_t *ukeys;                 // unique keys ascending
    int32_t *inv;                    // [nnz] index of each position's key in ukeys
    int32_t *seg_off;                // [n_unique+1] start of each key's run in skeys
    int32_t *seg_chunk0;             // [n_unique] first backward chunk of each run
    int4 *chunk_desc;                // [n_chunks] first pos, end pos, run, chunks of the run
    int32_t *multi;                  // [n_multi] runs longer than one chunk (any order)
    int32_t *scal;                   // [0] n_unique, [1] n_chunks, [2] ERR_* bits, [3] n_multi
    int32_t *eslot;                  // [n_unique] slot of each unique key when the batch
                                     // entered the hold window (-1: not cached)
};

// Per-plan device buffers.
struct TicketDev {
    int32_t *hit, *slot_u;           // [n_unique]
    int32_t *slot_of;                // [nnz]
    uint32_t *m_key;                 // [n_miss] missing keys ascending
    int32_t *m_uidx;                 // [n_miss] their index in ukeys
    int32_t *v_slot;                 // [n_miss] slot given to each miss
    int32_t *v_old_key, *v_old_lu;   // [n_miss] previous occupant / last use of that slot
};

// Replacement policies (Sec. VI-E): the values of SP_POLICY_*.
constexpr int POLICY_LRU = 0, POLICY_LFU = 1, POLICY_RANDOM = 2;

// Eviction priority of a slot: smaller goes first, ties by slot.  src[g] is
// the slot's last use (LRU, random) or use count (LFU).
//   LRU     last use + 1 (a never-used slot: 0)
//   LFU     uses of the slot's current row (never used: 0)
//   random  0 for a never-used slot, else 1 + the top 24 bits of SplitMix64
//           output number u * 2^31 + g + 1 of the stream started at `seed`
//           (Steele, Lea and Flood, OOPSLA 2014): a fresh draw per plan.
struct Prio {
    const int32_t *src;
    int32_t policy;
    uint32_t u;
    uint64_t seed;
    // Written without branches, so that loops over slots keep their loads in
    // flight together: every case is computed and the policy's is selected.
    __host__ __device__ uint32_t key(int32_t v, int64_t g) const
    {
        uint64_t z = seed + (((uint64_t)u << 31) + (uint64_t)g + 1) * 0x9E3779B97F4A7C15ull;
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        z ^= z >> 31;
        const uint32_t rnd = v < 0 ? 0u : 1u + (uint32_t)(z >> 40);
        const uint32_t other = policy == POLICY_LFU ? (uint32_t)v : (uint32_t)(v + 1);
        return policy == POLICY_RANDOM ? rnd : other;
    }
    __device__ uint32_t operator()(int64_t g) const { return key(src[g], g); }
};

// The rows of a plan's query.  Probe arrays: window batches 0 .. nhold-1,
// then the past batches.  Row 0 is the planned batch (array index 0), rows
// for the successors to prefetch (1 .. depth) and for the batches entering
// the hold window (their cached keys are marked held by the commit sequence,
// after the plan has been accepted) follow.  With `rebuild` every hold is
// dropped and every window and past batch enters again.
struct QueryRows {
    int32_t n;                       // rows
    int32_t idx[MAX_WINDOW];         // probe-array index of each row
    int32_t qoff[MAX_WINDOW];        // per probe-array index: its batch less the planned one
    uint32_t entrant;                // bit per probe-array index
    int32_t rebuild;
    int32_t span;                    // lookahead + hold_past
    int32_t *eslot[MAX_WINDOW];      // per probe-array index: where an entrant's slots go
};

// The batches entering the hold window, as their slots are marked held:
// row r's keys are covered by threads start[r] .. start[r+1] - 1.
struct HoldRows {
    int32_t n;
    const uint32_t *uk[MAX_WINDOW];
    const int32_t *nu[MAX_WINDOW];
    const int32_t *es[MAX_WINDOW];
    int32_t nv_off[MAX_WINDOW];      // batch + hold_past - plan
    int32_t q_off[MAX_WINDOW];       // batch - plan
    int64_t start[MAX_WINDOW + 1];
};

// Rows of all tables, one index each: table t's row r is rbase[t] + r.
// lastq[row]: the last batch that entered the hold window with the row not
// cached (-1: none), written once its plan is accepted; pend[row]: the stamp
// of the last query whose entering batch has the row not cached.  A row
// missing at plan k is in no earlier window batch's cached set, so these
// two give the last window batch that has it without a search.
struct RowIndex {
    const int64_t *rbase;
    int32_t *lastq, *pend;
};

// Victim selection arguments (active tables = those with misses).
struct SelArgs {
    int32_t nact;
    int32_t prio_bits;               // bits of the priority values
    int32_t act_bits;                // bits of the active-table index in sort keys
    int32_t plan;                    // slots with hold_to >= plan are held,
    int32_t stamp;                   // and those the plan's query stamped
    Prio prio;
    int32_t t[MAX_TABLES];
    int32_t k[MAX_TABLES];           // misses
    int64_t base[MAX_TABLES];        // first global slot of the table
    int64_t S[MAX_TABLES];           // slots of the table
    int32_t vbase[MAX_TABLES];       // first victim index of the table
};

// Victims taken straight from the tables' never-used slots (fresh path):
// table y's k[y] victims are global slots first[y] .. first[y] + k[y] - 1,
// written from victim index vbase[y] on.
struct FreshArgs {
    int32_t n;
    int32_t vbase[MAX_TABLES];
    int32_t k[MAX_TABLES];
    int64_t first[MAX_TABLES];
};

// Positions per backward chunk: one lane group sums at most this many
// gradient rows before a run is split across groups.
constexpr int BWD_CHUNK = 16;
inline int chunk_positions(int /*dim*/) { return BWD_CHUNK; }

// ---------------------------------------------------------------- launchers
// k_ingest.hip
void launch_zero_i32(int32_t *p, int64_t n, hipStream_t s);
void launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s);
// How an ingest in LDS reports that it has read its inputs: blocks count
// themselves in *counter (it only grows); the one that reaches target writes
// seq to the host-coherent *word.
struct IngestCons {
    uint32_t *counter;
    uint32_t target;
    uint64_t *word;
    uint32_t seq;
};
// Ingest one batch.  In LDS (ingest_in_lds and nnz > 0) the inputs are known
// read when *ic.word reads ic.seq; otherwise when `consumed` (if not null)
// completes.
void launch_ingest(const Tables &tb, const BatchDev &b, const int32_t *ids, const int32_t *bag_off,
                   int32_t B, int64_t nnz, int key_bits, int chunk, int64_t max_table_ids,
                   int64_t cap_u, int64_t cap_c, uint32_t *tmp_k, uint32_t *tmp_v,
                   uint32_t *hist, ScanWs &ws, hipEvent_t consumed, const IngestCons &ic,
                   hipStream_t s);

void launch_radix_sort(uint32_t *k0, uint32_t *v0, uint32_t *k1, uint32_t *v1, int64_t n,
                       int bits, uint32_t *hist, ScanWs &ws, bool *in_k1, hipStream_t s,
                       bool prehist);
int64_t radix_hist_entries(int64_t n);
int radix_passes(int64_t n, int bits);  // passes launch_radix_sort makes (result in k1 if odd)
// Layout of a sort of n keys of `bits` bits: passes of dbits-wide digits over
// tiles of BLOCK * items keys; one-launch passes (fused) when the per-pass
// table of (1 << dbits) x tiles counters has at most 16384 entries.
struct RadixPlan {
    int passes, dbits, items;
    int64_t tiles, table;
    bool fused;
};
RadixPlan radix_plan(int64_t n, int bits);

// k_plan.hip
// The query: hold marks, hits, the misses in ascending key order (tk.m_key,
// tk.m_uidx) and per-table counts of one plan, published to host_mapped
// (word i = seq << 32 | counter word i) by the last block.  Without prefetch,
// host_keys (device-visible pinned memory, or null) also gets the first
// host_cap missing keys, complete once the kernel is.
// Prefetch mode (depth d >= 1): the query compacts the planned batch's own
// misses into own_key / own_uidx and flags (flag[(w-1) * stride + j] = 1) the
// unique keys j of successor w = 1..d to prefetch; the arrangement then
// writes both into the ticket's miss list.
struct PrefetchDev {
    int32_t depth;
    uint32_t *own_key;
    int32_t *own_uidx;
    int32_t *flag;
    int64_t stride;
};
void launch_query(const Tables &tb, const uint64_t *hash, uint32_t mask,
                  const uint32_t *const *ukeys, const int32_t *const *nuniq, int nwin,
                  int64_t max_unique, const int32_t *hold_to, int32_t *held, int32_t stamp,
                  int32_t *hcnt, int32_t plan, const QueryRows &qr, const RowIndex &ri,
                  TicketDev tk, PrefetchDev pf,
                  DevCounters *cnt, int32_t *part, int32_t *arrived, const int32_t *scal0,
                  uint64_t *host_mapped, uint32_t seq, uint32_t *host_keys, int64_t host_cap,
                  ScanWs &ws, hipStream_t s);
// Every hold dropped, then the cached keys of hr's batches marked held:
// hold_to = max(hold_to, batch + hold_past), with the counts moved (a plan
// that rebuilds the holds, before its victims are chosen; otherwise the
// commit marks them).
void launch_hold_rebuild(const Tables &tb, const HoldRows &hr, const RowIndex &ri,
                         int32_t *hold_to, int32_t *hcnt, int32_t plan, hipStream_t s);

void launch_hash_rebuild(uint64_t *hash, uint32_t mask, const int32_t *key_of_slot, int64_t nslots,
                         DevCounters *cnt, hipStream_t s);
void launch_fresh_victims(const FreshArgs &f, int64_t max_k, int32_t *v_slot, hipStream_t s);
void launch_select_victims(const SelArgs &a, int levels, int64_t maxS, const int32_t *hold_to,
                           const int32_t *held, int32_t *sel_state, int32_t *sel_hist,
                           uint32_t *vk0, uint32_t *vv0, uint32_t *vk1, uint32_t *vv1,
                           int64_t n_victims, uint32_t *hist, ScanWs &ws, int32_t *v_slot,
                           int32_t *err, hipStream_t s);
// The window batches' sorted unique keys (0 = the planned batch), for the
// hold of filled rows.  fast: at most one batch enters (at window index ent,
// 0 if none) and the holds were not rebuilt, so lastq / pend (with this
// plan's query stamp) answer; otherwise binary searches do.
struct WindowKeys {
    int32_t n;                       // nhold
    int32_t hold_past;
    int32_t fast, ent, stamp;
    const uint32_t *uk[MAX_WINDOW];
    const int32_t *nu[MAX_WINDOW];
};
// Misses into their victim slots, Hit-Map and slot metadata updated, every
// slot the batch uses touched (last_use = u), slot_of filled.  A filled row is
// held through the last window batch that has its key (plus hold_past), and
// the cached keys of the entering batches hr (none after a rebuild) are
// marked held.
// uses: per-slot use counts (LFU), or null when the policy does not keep them
void launch_commit(const Tables &tb, uint64_t *hash, uint32_t mask, TicketDev tk,
                   const BatchDev &b, int64_t n_miss, int64_t n_unique, int64_t nnz,
                   int32_t *key_of_slot, int32_t *last_use, int32_t *uses, int32_t u,
                   bool prefetch, const WindowKeys &wk, const HoldRows &hr, const RowIndex &ri,
                   int32_t *hold_to, int32_t *hcnt, DevCounters *cnt, hipStream_t s);
// Prefetch mode: the ticket's miss list, per table the planned batch's own
// misses (ascending) then, successor by successor, its flagged keys
// (ascending), from vbase[t] = first victim of table t; prefetched entries get
// m_uidx = -1.  Successor w (1..pf.depth): n_next[w-1] points at its count of
// unique keys (at most max_next[w-1]), next_ukeys[w-1] at the keys.
void launch_pf_arrange(const Tables &tb, PrefetchDev pf, int64_t n_own,
                       const int32_t *const *n_next, const int64_t *max_next,
                       const uint32_t *const *next_ukeys, const int32_t *own,
                       const int32_t (*pf_count)[MAX_TABLES], TicketDev tk, int64_t n_miss,
                       int32_t *err, ScanWs &ws, hipStream_t s);

// k_train.hip
// Victim i: stage its slot's old row (if any) in stage row i, then write the
// missing row m_key[i] into the slot: from `staged` row i when given (the
// staged fill), else straight from the mapped host table.
void launch_move(float *storage, int dim, const Tables &tb, float *const *host_dev, TicketDev tk,
                 int64_t n_miss, int32_t u, float *stage, const float *staged, hipStream_t s);
void launch_forward(const float *storage, int dim, int64_t nslots, const int32_t *slot_of,
                    const int32_t *bag_off, int64_t nbags, float *out, hipStream_t s,
                    hipEvent_t e0, hipEvent_t e1);
// The fixed partial-sum array of sp_backward_update_static: its bytes, and
// its device address on the current device.
constexpr int64_t STATIC_PARTIAL_BYTES = 32ll << 20;
hipError_t static_partial_address(void **ptr);
void launch_backward(float *storage, int dim, int64_t nslots, const BatchDev &b,
                     const int32_t *slot_u, int64_t n_chunks, int64_t n_multi, int chunk,
                     const float *grad, int64_t nbags, float lr, float *partial, hipStream_t s,
                     hipEvent_t ev[4]);

}  // namespace sp
