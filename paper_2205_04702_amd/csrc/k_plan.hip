// Planner kernels: Hit-Map query, holds over the hold window, victim
// choice among unheld slots by the replacement policy, and the Hit-Map /
// slot-metadata commit (Sec. IV-C "Putting everything together", Sec. IV-D
// Algorithm 1; LRU is the default replacement policy of Sec. VI-E, LFU and
// random eviction its alternatives).
#include "sp_device.h"
#include "sp_internal.h"

namespace sp {

// ---------------------------------------------------------------- query + hold

static_assert(QUERY_TILE == BLOCK, "one unique key per query thread");

struct ProbeArgs {
    const uint32_t *uk[MAX_WINDOW];
    const int32_t *nu[MAX_WINDOW];
};

// a[w] for a block-uniform w, chosen among the kernel-argument words without
// indexing them by a register (which makes the compiler fetch them through
// memory, one dependent round trip before the real loads can start)
template <typename P>
__device__ __forceinline__ P pick_uniform(const P (&a)[MAX_WINDOW], int w)
{
    P r = a[0];
#pragma unroll
    for (int q = 1; q < MAX_WINDOW; ++q)
        if (w == q) r = a[q];
    return r;
}

// The query of one plan, one launch.  blockIdx.y = row (QueryRows).  Batch 0
// (the planned one) records hit / slot, counts misses and compacts them in
// ascending key order into m_key / m_uidx with a single-pass scan (its blocks
// take their tiles of keys from an atomic counter, so a tile only looks back
// at tiles whose blocks have started).  A batch entering the hold window
// records the slot of each of its keys (eslot) and stamps each cached slot
// with this query's stamp (held[slot] = stamp, which the victim choice of
// this plan treats as held); the first stamp of a slot counts it, per table,
// when hold_to < plan: the slots the plan newly holds.  An uncached key of
// such a batch writes the stamp to its row's pend entry, which tells this
// plan's commit that the key is in the entering batch.  hold_to is not
// written here, so a rejected plan changes nothing (its stamp is never
// matched again); the commit raises it.  Held slots at this plan are those
// newly held plus those whose hold_to lies in plan .. plan + span - 1,
// counted in hcnt.  Per-table counts are summed
// across the wave (keys are sorted, so a wave nearly always covers one table),
// then across the block in LDS, then added to one of PART_COPIES copies of the
// counters so that few blocks contend for an address.
//
// Every add a block makes returns its old value, and each thread tests the
// values before the block's barrier, so all of a block's adds have been
// performed when the block arrives.  The last block to arrive then publishes:
// it sums the copies (device-scope atomic loads) and writes every counter word
// to pinned, device-mapped, host-coherent memory as one 64-bit store tagged
// with the query's sequence number.  The host polls until every word carries
// it; no copy command, fence or stream synchronisation is involved, and each
// word is whole when seen.  It then clears the copies, the per-plan counters
// and the arrival count for the next query, and the hold count of value
// plan + span: no slot has that value yet (this plan's commit is the first
// that may give it), and its entry last counted an expired value.
//
// Prefetch mode (depth d): batch 0's misses go to pf.own_key / pf.own_uidx
// instead, and each successor w = 1..d flags every unique key that is not
// cached and not a key of an earlier batch 0..w-1 (binary searches of their
// sorted keys) and counts them per table, so the plan can fill them too.
// Whether key is among the n sorted keys a[0..n).
__device__ __forceinline__ bool in_sorted(const uint32_t *__restrict__ a, int32_t n, uint32_t key)
{
    int32_t lo = 0, hi = n;
    while (lo < hi) {
        const int32_t mid = lo + (hi - lo) / 2;
        if (a[mid] < key) lo = mid + 1;
        else hi = mid;
    }
    return lo < n && a[lo] == key;
}

__global__ void __launch_bounds__(BLOCK) k_query(int32_t row_bits, int32_t T,
                                                 const uint64_t *__restrict__ hash, uint32_t mask,
                                                 ProbeArgs pa, PrefetchDev pf,
                                                 const int32_t *__restrict__ hold_to,
                                                 int32_t *held, int32_t stamp,
                                                 int32_t *hcnt, int32_t plan, QueryRows qr,
                                                 RowIndex ri,
                                                 int32_t *hit, int32_t *slot_u, DevCounters *cnt,
                                                 int32_t *part, int32_t *arrived,
                                                 const int32_t *scal0, uint64_t *host_mapped,
                                                 uint32_t seq, uint32_t *m_key, int32_t *m_uidx,
                                                 uint32_t *host_keys, int64_t host_cap, ScanDev d)
{
    __shared__ int32_t c_miss[MAX_TABLES], c_held[MAX_TABLES], c_pf[MAX_TABLES];  // c_pf: row w's
    __shared__ int32_t last_s;
    __shared__ uint32_t tile_s, pref_s;
    __shared__ uint32_t lds_scan[BLOCK / WAVE];
    const int w = pick_uniform(qr.idx, (int)blockIdx.y);
    const bool entrant = (qr.entrant >> w) & 1u;
    for (int t = threadIdx.x; t < T; t += BLOCK) c_miss[t] = c_held[t] = c_pf[t] = 0;
    if (w == 0 && threadIdx.x == 0) tile_s = atomicAdd(d.counter, 1u) - d.base;
    __syncthreads();
    const int64_t xb = w == 0 ? (int64_t)tile_s : (int64_t)blockIdx.x;
    if (xb >= (int64_t)gridDim.x) {  // the counter and the host disagree: give up loudly
        if (threadIdx.x == 0) atomicOr(d.err, ERR_PLAN);
        return;
    }
    const int64_t i = xb * BLOCK + threadIdx.x;
    int32_t seen = 0;  // returned old values; tested below so the adds complete first
    if (w == 0 && i == 0) {
        seen |= atomicExch(&cnt->n_unique, scal0[0]) == INT32_MIN;
        seen |= atomicExch(&cnt->n_chunks, scal0[1]) == INT32_MIN;
        seen |= atomicExch(&cnt->n_multi, scal0[3]) == INT32_MIN;
    }
    const uint32_t *const ukw = pick_uniform(pa.uk, w);
    const int32_t *const nuw = pick_uniform(pa.nu, w);
    if (i == 0 && nuw[2]) seen |= atomicOr(&cnt->err, nuw[2]) == INT32_MIN;
    const bool valid = i < *nuw;
    int t = 0;
    bool miss = false, fresh = false, fetch = false;
    uint32_t key = 0;
    if (valid) {
        key = ukw[i];
        t = (int)(key >> row_bits);
        const int32_t slot = hash_find_ro(hash, mask, key);  // the map is not written here
        if (w == 0) {
            hit[i] = slot >= 0;
            slot_u[i] = slot;
            miss = slot < 0;
        }
        if (entrant) {
            if (slot >= 0)
                fresh = atomicExch(&held[slot], stamp) != stamp &&
                        (qr.rebuild || hold_to[slot] < plan);
            else if (t < T)
                ri.pend[ri.rbase[t] + (key & ((1u << row_bits) - 1u))] = stamp;
            pick_uniform(qr.eslot, w)[i] = slot;
        }
        if (w >= 1 && w <= pf.depth) {
            fetch = slot < 0;
#pragma unroll
            for (int e = 0; e < MAX_PF; ++e)  // the earlier batches 0 .. w-1
                if (e < w && fetch) fetch = !in_sorted(pa.uk[e], *pa.nu[e], key);
            pf.flag[(int64_t)(w - 1) * pf.stride + i] = fetch;
        }
    }
    if (w == 0 && xb * BLOCK < (int64_t)*pa.nu[0]) {  // uniform per block
        uint32_t tot;
        const uint32_t ex = block_excl_scan((uint32_t)miss, lds_scan, tot);
        if (threadIdx.x < WAVE) {
            const uint32_t pre = lb_lookback<uint32_t>(d, (uint32_t)xb, (int)xb, tot);
            if (threadIdx.x == 0) pref_s = pre;
        }
        __syncthreads();
        if (miss) {
            uint32_t *const mk = pf.depth > 0 ? pf.own_key : m_key;
            int32_t *const mu = pf.depth > 0 ? pf.own_uidx : m_uidx;
            mk[pref_s + ex] = key;
            mu[pref_s + ex] = (int32_t)i;
            // the staged fill's host threads read the misses from pinned memory
            if (host_keys && pref_s + ex < (uint64_t)host_cap) host_keys[pref_s + ex] = key;
        }
    }
    uint64_t todo = __ballot(valid);
    while (todo) {
        const int leader = __ffsll((unsigned long long)todo) - 1;
        const int tl = __shfl(t, leader, WAVE);
        const bool mine = valid && t == tl;
        const uint64_t same = __ballot(mine);
        const int nm = __popcll(__ballot(mine && miss));
        const int nh = __popcll(__ballot(mine && fresh));
        const int nf = __popcll(__ballot(mine && fetch));
        if (lane_id() == leader) {
            if (nm) atomicAdd(&c_miss[tl], nm);
            if (nh) atomicAdd(&c_held[tl], nh);
            if (nf) atomicAdd(&c_pf[tl], nf);
        }
        todo &= ~same;
    }
    __syncthreads();
    int32_t *p = part + (int64_t)((blockIdx.y * gridDim.x + blockIdx.x) % PART_COPIES) * PART_WORDS;
    const int pfw = w >= 1 && w <= MAX_PF ? w - 1 : 0;  // this row's prefetch counts
    for (int tt = threadIdx.x; tt < T; tt += BLOCK) {
        if (c_miss[tt]) seen |= atomicAdd(&p[tt], c_miss[tt]);
        if (c_held[tt]) seen |= atomicAdd(&p[MAX_TABLES + tt], c_held[tt]);
        if (c_pf[tt]) seen |= atomicAdd(&p[(2 + pfw) * MAX_TABLES + tt], c_pf[tt]);
    }
    if (seen < 0) cnt->pad2[0] = seen;  // never taken (counts are not negative)
    __syncthreads();
    if (threadIdx.x == 0)
        last_s = atomicAdd(arrived, 1) == (int32_t)(gridDim.x * gridDim.y) - 1;
    __syncthreads();
    if (!last_s) return;  // uniform per block

    // ---- last block: publish
    __shared__ int32_t sums[PART_WORDS];
    for (int j = threadIdx.x; j < PART_WORDS; j += BLOCK) sums[j] = 0;
    __syncthreads();
    const int na = 2 + pf.depth;  // live arrays per copy: miss, held, one per successor
    const int n_rel = PART_COPIES * na * T;
    auto word = [T, na](int r) {  // the r-th live word: copy c, array a, table
        const int c = r / (na * T), jj = r % (na * T), a = jj / T;
        return c * PART_WORDS + a * MAX_TABLES + (jj - a * T);
    };
    for (int r = threadIdx.x; r < n_rel; r += BLOCK) {
        const int idx = word(r);
        const int32_t v = __hip_atomic_load(&part[idx], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (v) atomicAdd(&sums[idx % PART_WORDS], v);
    }
    __syncthreads();
    int32_t *src = reinterpret_cast<int32_t *>(cnt);
    constexpr int MISS0 = (int)(offsetof(DevCounters, miss) / sizeof(int32_t));
    constexpr int HELD0 = (int)(offsetof(DevCounters, held) / sizeof(int32_t));
    constexpr int PF0 = (int)(offsetof(DevCounters, pf) / sizeof(int32_t));
    for (int k = threadIdx.x; k < COUNTER_WORDS; k += BLOCK) {
        int32_t v;
        if (k >= MISS0 && k < MISS0 + MAX_TABLES) v = k - MISS0 < T ? sums[k - MISS0] : 0;
        else if (k >= HELD0 && k < HELD0 + MAX_TABLES) {
            const int t = k - HELD0;
            v = 0;
            if (t < T) {
                v = sums[MAX_TABLES + t];
                for (int j = 0; j < qr.span && !qr.rebuild; ++j)
                    v += __hip_atomic_load(&hcnt[t * HOLD_RING + ((plan + j) & (HOLD_RING - 1))],
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        else if (k >= PF0 && k < PF0 + MAX_PF * MAX_TABLES)  // successor a, table tt
            v = (k - PF0) % MAX_TABLES < T ? sums[2 * MAX_TABLES + (k - PF0)] : 0;
        else v = __hip_atomic_load(&src[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        host_mapped[k] = ((uint64_t)seq << 32) | (uint32_t)v;
        if (k < COUNTERS_CLEARED)
            __hip_atomic_store(&src[k], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    for (int r = threadIdx.x; r < n_rel; r += BLOCK)
        __hip_atomic_store(&part[word(r)], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (int t = threadIdx.x; t < T; t += BLOCK)
        __hip_atomic_store(&hcnt[t * HOLD_RING + ((plan + qr.span) & (HOLD_RING - 1))], 0,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (threadIdx.x == 0) __hip_atomic_store(arrived, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

void launch_query(const Tables &tb, const uint64_t *hash, uint32_t mask,
                  const uint32_t *const *ukeys, const int32_t *const *nuniq, int nwin,
                  int64_t max_unique, const int32_t *hold_to, int32_t *held, int32_t stamp,
                  int32_t *hcnt, int32_t plan, const QueryRows &qr, const RowIndex &ri,
                  TicketDev tk, PrefetchDev pf,
                  DevCounters *cnt, int32_t *part, int32_t *arrived, const int32_t *scal0,
                  uint64_t *host_mapped, uint32_t seq, uint32_t *host_keys, int64_t host_cap,
                  ScanWs &ws, hipStream_t s)
{
    if (pf.depth > nwin - 1 || pf.depth > MAX_PF || qr.n < 1 || qr.n > nwin || qr.idx[0] != 0 ||
        qr.span < 0 || qr.span >= HOLD_SPAN) {  // the caller keeps to these
        ws.overflow = true;
        return;
    }
    for (int r = 0; r < qr.n; ++r)
        if (qr.idx[r] < 0 || qr.idx[r] >= nwin) {
            ws.overflow = true;
            return;
        }
    ProbeArgs pa{};
    for (int w = 0; w < nwin; ++w) pa.uk[w] = ukeys[w], pa.nu[w] = nuniq[w];
    // at least one block per batch so that every batch's error word is read
    const int64_t n = max_unique > 0 ? max_unique : 1;
    const int64_t gx = (n + BLOCK - 1) / BLOCK;
    if (gx > ws.max_tiles) {
        ws.overflow = true;
        return;
    }
    if (ws.epoch == 0xFFFFFFFFu) {  // epochs wrapped: forget every published word
        (void)hipMemsetAsync(ws.status, 0, sizeof(uint64_t) * LB_WORDS * ws.max_tiles, s);
        ws.epoch = 0;
    }
    ScanDev d{ws.status, ws.counter, ws.err, ws.issued, ++ws.epoch, (uint32_t)gx, (int32_t)gx};
    ws.issued += (uint32_t)gx;  // the planned batch's row of blocks takes tiles
    hipLaunchKernelGGL(k_query, dim3((unsigned)gx, (unsigned)qr.n), dim3(BLOCK), 0, s, tb.row_bits,
                       tb.T, hash, mask, pa, pf, hold_to, held, stamp, hcnt, plan, qr, ri, tk.hit,
                       tk.slot_u, cnt,
                       part, arrived, scal0, host_mapped, seq, tk.m_key, tk.m_uidx, host_keys,
                       host_cap, d);
}

// ---------------------------------------------------------------- holds

// Adds per (table, value - plan) gathered in LDS, then into hcnt.
__device__ __forceinline__ void hold_counts_flush(const int32_t *c, int32_t *hcnt, int32_t plan)
{
    for (int x = threadIdx.x; x < MAX_TABLES * HOLD_SPAN; x += BLOCK)
        if (c[x])
            atomicAdd(&hcnt[(x / HOLD_SPAN) * HOLD_RING + ((plan + x % HOLD_SPAN) & (HOLD_RING - 1))],
                      c[x]);
}

// Thread j of a HoldRows section: its row's arrays and its key index.
struct HoldRef {
    const uint32_t *uk;
    const int32_t *nu, *es;
    int32_t off, qo;
    int64_t i;
};
__device__ __forceinline__ HoldRef hold_ref(const HoldRows &hr, int64_t j)
{
    HoldRef h{hr.uk[0], hr.nu[0], hr.es[0], hr.nv_off[0], hr.q_off[0], j};
#pragma unroll
    for (int r = 1; r < MAX_WINDOW; ++r)  // selects, no indexing by a register
        if (r < hr.n && j >= hr.start[r]) {
            h.uk = hr.uk[r];
            h.nu = hr.nu[r];
            h.es = hr.es[r];
            h.off = hr.nv_off[r];
            h.qo = hr.q_off[r];
            h.i = j - hr.start[r];
        }
    return h;
}

// One key of an entering batch: its slot (if cached) is held through the
// batch (+ hold_past): hold_to rises to that value and, if it rose, the count
// moves from the old value (if still live) to the new one.  Keys of two
// entering batches may share a slot: atomicMax orders the raises, and each
// raise moves the count exactly once.  A key not cached records the batch in
// lastq.
__device__ __forceinline__ void hold_key(const HoldRef &h, int32_t row_bits, int32_t T,
                                         const RowIndex &ri, int32_t *hold_to, int32_t plan,
                                         int32_t *c)
{
    if (h.i >= *h.nu) return;
    const int32_t slot = h.es[h.i];
    const uint32_t key = h.uk[h.i];
    const int t = (int)(key >> row_bits);
    if (t >= T) return;
    if (slot < 0) {
        atomicMax(&ri.lastq[ri.rbase[t] + (key & ((1u << row_bits) - 1u))], plan + h.qo);
        return;
    }
    if (h.off < 0 || h.off >= HOLD_SPAN) return;
    const int32_t old = atomicMax(&hold_to[slot], plan + h.off);
    if (old < plan + h.off) {
        if (old >= plan) atomicSub(&c[t * HOLD_SPAN + (old - plan)], 1);
        atomicAdd(&c[t * HOLD_SPAN + h.off], 1);
    }
}

__global__ void __launch_bounds__(BLOCK) k_hold(HoldRows hr, int32_t row_bits, int32_t T,
                                                RowIndex ri, int32_t *hold_to, int32_t *hcnt,
                                                int32_t plan)
{
    __shared__ int32_t c[MAX_TABLES * HOLD_SPAN];
    for (int x = threadIdx.x; x < MAX_TABLES * HOLD_SPAN; x += BLOCK) c[x] = 0;
    __syncthreads();
    const int64_t j = (int64_t)blockIdx.x * BLOCK + threadIdx.x;
    if (j < hr.start[hr.n]) hold_key(hold_ref(hr, j), row_bits, T, ri, hold_to, plan, c);
    __syncthreads();
    hold_counts_flush(c, hcnt, plan);
}

__global__ void k_hold_clear(int32_t *hold_to, int64_t nslots, int32_t *hcnt)
{
    const int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x;
    if (i < nslots) hold_to[i] = -1;
    if (i < MAX_TABLES * HOLD_RING) hcnt[i] = 0;
}

void launch_hold_rebuild(const Tables &tb, const HoldRows &hr, const RowIndex &ri,
                         int32_t *hold_to, int32_t *hcnt, int32_t plan, hipStream_t s)
{
    const int64_t ns = tb.slot_base[tb.T];
    const int64_t n = ns > MAX_TABLES * HOLD_RING ? ns : MAX_TABLES * HOLD_RING;
    hipLaunchKernelGGL(k_hold_clear, dim3((unsigned)((n + BLOCK - 1) / BLOCK)), dim3(BLOCK), 0, s,
                       hold_to, ns, hcnt);
    const int64_t m = hr.start[hr.n];
    if (hr.n > 0 && m > 0)
        hipLaunchKernelGGL(k_hold, dim3((unsigned)((m + BLOCK - 1) / BLOCK)), dim3(BLOCK), 0, s,
                           hr, tb.row_bits, tb.T, ri, hold_to, hcnt, plan);
}

// ---------------------------------------------------------------- hash rebuild

__global__ void k_hash_clear(uint64_t *hash, int64_t n)
{
    int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x;
    if (i < n) hash[i] = ENTRY_EMPTY;
}

__global__ void k_hash_reinsert(uint64_t *hash, uint32_t mask, const int32_t *key_of_slot,
                                int64_t nslots, int32_t *err)
{
    int64_t s = (int64_t)blockIdx.x * BLOCK + threadIdx.x;
    if (s >= nslots) return;
    int32_t k = key_of_slot[s];
    if (k >= 0 && !hash_insert(hash, mask, (uint32_t)k, (int32_t)s)) atomicOr(err, ERR_HASH_FULL);
}

void launch_hash_rebuild(uint64_t *hash, uint32_t mask, const int32_t *key_of_slot, int64_t nslots,
                         DevCounters *cnt, hipStream_t s)
{
    int64_t cap = (int64_t)mask + 1;
    hipLaunchKernelGGL(k_hash_clear, dim3((unsigned)((cap + BLOCK - 1) / BLOCK)), dim3(BLOCK), 0, s,
                       hash, cap);
    if (nslots > 0)
        hipLaunchKernelGGL(k_hash_reinsert, dim3((unsigned)((nslots + BLOCK - 1) / BLOCK)),
                           dim3(BLOCK), 0, s, hash, mask, key_of_slot, nslots, &cnt->err_sticky);
}

// ---------------------------------------------------------------- victims
//
// For each table with k misses: the k smallest (priority, slot) among its
// unheld slots, the priority being the policy's (Prio: last use + 1 for LRU,
// so never-used slots go first; use count for LFU; a fresh random draw for
// random eviction).  A radix select on the priority (SEL_BITS per level, most
// significant first) finds the threshold value v* and how many slots equal to
// v* to take (r); a segmented scan then compacts, in slot order, every unheld
// slot below v* and the first r equal to it; a stable radix sort on (table,
// priority) puts them in priority order with ties in slot order.
// sel_state[2a] = v* prefix,
// sel_state[2a+1] = slots still to take at the current level,
// sel_state[2 * MAX_TABLES + a] = blocks of the current level done with table a.

constexpr int SEL_ITEMS = 16;
constexpr int SEL_CHUNK = BLOCK * SEL_ITEMS;

// One level of the select, one launch.  Every block counts its chunk of one
// active table's unheld slots by the current SEL_BITS of the priority (among
// slots matching the prefix found so far) and adds the counts to the table's
// histogram.  The last block of a table to arrive then fixes the next SEL_BITS
// of v* and the slots still to take, and leaves the histogram and its arrival
// counter cleared.  The adds return their old values and each thread tests
// them before the block's barrier, so every add of a block has been performed
// before the block arrives; the last block reads the histogram with
// device-scope atomic loads.  The first level starts from k misses still to
// place and an empty prefix; its last blocks also mark the table's victim
// entries invalid (-1) before the compaction fills them, and clear (all
// tables together) the n_zero counters the global victim sort accumulates into.
__global__ void __launch_bounds__(BLOCK) k_sel_level(SelArgs a, int shift, int first,
                                                     const int32_t *hold_to, const int32_t *held,
                                                     int32_t *st, int32_t *hist, int32_t *arrived,
                                                     int32_t *victims, uint32_t *zero,
                                                     int64_t n_zero)
{
    __shared__ int32_t h[SEL_BINS];
    __shared__ int32_t lds[BLOCK / WAVE];
    __shared__ int32_t last_s;
    for (int b = threadIdx.x; b < SEL_BINS; b += BLOCK) h[b] = 0;
    __syncthreads();
    const int ai = blockIdx.y;
    const int64_t S = a.S[ai];
    const int64_t s0 = (int64_t)blockIdx.x * SEL_CHUNK;
    const int32_t prefix = first ? 0 : st[2 * ai];
    if (s0 < S) {
        const uint64_t want = (uint64_t)(uint32_t)prefix >> (shift + SEL_BITS);
        const int64_t base = a.base[ai];
        int32_t hv[SEL_ITEMS], sv[SEL_ITEMS], lv[SEL_ITEMS];
#pragma unroll
        for (int r = 0; r < SEL_ITEMS; ++r) {  // all loads in flight together
            const int64_t s = s0 + (int64_t)r * BLOCK + threadIdx.x;
            hv[r] = s < S ? hold_to[base + s] : a.plan;
            sv[r] = s < S ? held[base + s] : a.stamp;
            lv[r] = s < S ? a.prio.src[base + s] : 0;
        }
#pragma unroll
        for (int r = 0; r < SEL_ITEMS; ++r) {
            if (hv[r] < a.plan && sv[r] != a.stamp) {  // unheld
                const uint32_t key = a.prio.key(lv[r], base + s0 + (int64_t)r * BLOCK + threadIdx.x);
                if (((uint64_t)key >> (shift + SEL_BITS)) == want)
                    atomicAdd(&h[(key >> shift) & (SEL_BINS - 1)], 1);
            }
        }
    }
    __syncthreads();
    int32_t *out = hist + (int64_t)ai * SEL_BINS;
    int32_t seen = 0;
    for (int b = threadIdx.x; b < SEL_BINS; b += BLOCK)
        if (h[b]) seen |= atomicAdd(&out[b], h[b]);
    if (seen < 0) victims[0] = -1;  // never (counts are not negative); waits for the adds
    __syncthreads();
    if (threadIdx.x == 0) last_s = atomicAdd(&arrived[ai], 1) == (int32_t)gridDim.x - 1;
    __syncthreads();
    if (!last_s) return;  // uniform per block

    constexpr int PER = SEL_BINS / BLOCK;
    const int32_t krem = first ? a.k[ai] : st[2 * ai + 1];
    int32_t c[PER], sum = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        c[q] = __hip_atomic_load(&out[threadIdx.x * PER + q], __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
        sum += c[q];
    }
    int32_t total;
    int32_t excl = block_excl_scan(sum, lds, total);
    if (excl < krem && krem <= excl + sum) {
        int32_t cum = excl;
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            if (cum + c[q] >= krem) {
                st[2 * ai] = prefix | ((threadIdx.x * PER + q) << shift);
                st[2 * ai + 1] = krem - cum;
                break;
            }
            cum += c[q];
        }
    }
#pragma unroll
    for (int q = 0; q < PER; ++q)
        __hip_atomic_store(&out[threadIdx.x * PER + q], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (threadIdx.x == 0) __hip_atomic_store(&arrived[ai], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (first) {
        for (int i = threadIdx.x; i < a.k[ai]; i += BLOCK) victims[a.vbase[ai] + i] = -1;
        for (int64_t i = (int64_t)ai * BLOCK + threadIdx.x; i < n_zero; i += (int64_t)a.nact * BLOCK)
            zero[i] = 0;
    }
}

struct SegAct {
    int64_t base[MAX_TABLES], S[MAX_TABLES];
    __device__ int64_t beg(int y) const { return base[y]; }
    __device__ int64_t end(int y) const { return base[y] + S[y]; }
};

// (below v*) << 32 | (equal to v*) for an unheld slot, 0 for a held one.
struct VictimFlag {
    const int32_t *hold_to, *held, *st;
    Prio prio;
    int32_t plan, stamp;
    __device__ uint64_t operator()(int64_t g, int y) const
    {
        // every load unconditional (the scan batches them across items)
        const int32_t h = hold_to[g], hs = held[g], src = prio.src[g];
        const uint32_t key = prio.key(src, g), vstar = (uint32_t)st[2 * y];
        const uint64_t f = key < vstar ? (1ull << 32) : (key == vstar ? 1ull : 0ull);
        return h >= plan || hs == stamp ? 0ull : f;
    }
};

struct VictimOut {
    const int32_t *st;
    Prio prio;
    int32_t vbase[MAX_TABLES], k[MAX_TABLES];
    int32_t prio_bits;
    uint32_t *vk, *vv;
    uint32_t *hist0;                 // first sort pass's counters (digit-major), or null
    uint32_t digit_mask, tile_len, tiles;
    int64_t last[MAX_TABLES];        // last slot of each active table
    int32_t *err;
    __device__ void operator()(int64_t g, uint64_t e, uint64_t v, int y) const
    {
        if (g == last[y]) {  // every victim entry of the table must get a slot
            const uint64_t tot = e + v;
            const uint32_t below = (uint32_t)(tot >> 32), eq = (uint32_t)tot;
            const uint32_t r = (uint32_t)st[2 * y + 1];
            if (below + (eq < r ? eq : r) < (uint32_t)k[y]) atomicOr(err, ERR_PLAN);
        }
        if (!v) return;
        const uint32_t below = (uint32_t)(e >> 32), eq = (uint32_t)e, r = (uint32_t)st[2 * y + 1];
        uint32_t pos;
        if (v >> 32) pos = below + (eq < r ? eq : r);
        else if (eq < r) pos = below + eq;
        else return;
        if (pos >= (uint32_t)k[y]) return;  // never write past the table's victims
        const int64_t idx = vbase[y] + pos;
        const uint32_t key = ((uint32_t)y << prio_bits) | prio(g);
        vk[idx] = key;
        vv[idx] = (uint32_t)g;
        if (hist0) atomicAdd(&hist0[(key & digit_mask) * tiles + (uint32_t)idx / tile_len], 1u);
    }
};

// ---------------------------------------------------------------- victim order in LDS
//
// When every active table has at most VS_MAX victims, one block per table puts
// its compacted victims (slot order) into priority order: the stable LDS radix
// sort on entries (priority << 32 | slot), keyed on the priority bits only.
constexpr int VS_THREADS = 1024;
constexpr int VS_WAVES = VS_THREADS / WAVE;
constexpr int VS_MAX = 2048;

__global__ void __launch_bounds__(VS_THREADS) k_victim_sort(SelArgs a, const uint32_t *vk,
                                                          const uint32_t *vv, int32_t *v_slot)
{
    __shared__ uint64_t eb[2][VS_MAX];
    __shared__ uint32_t wc[VS_WAVES][256];
    __shared__ uint32_t lds[VS_WAVES];
    const int y = blockIdx.x;
    const int n = a.k[y] < VS_MAX ? a.k[y] : VS_MAX;
    const int64_t off = a.vbase[y];
    const int tid = threadIdx.x;
    const uint32_t kmask = a.prio_bits >= 32 ? ~0u : ((1u << a.prio_bits) - 1u);
    for (int i = tid; i < n; i += VS_THREADS)
        eb[0][i] = (uint64_t)(vk[off + i] & kmask) << 32 | vv[off + i];
    __syncthreads();
    const uint64_t *srt = lds_radix_sort<VS_THREADS, VS_MAX / VS_THREADS>(
        eb[0], eb[1], n, 32, a.prio_bits, wc, lds);
    for (int i = tid; i < n; i += VS_THREADS) v_slot[off + i] = (int32_t)(uint32_t)srt[i];
}

// Victims when every table's misses fit in its never-used slots.  Those slots
// have priority 0 under every policy and come before every used slot (LFU
// with prefetch excepted: a prefetched row not yet used also has 0 uses, and
// the host then always selects), they are never held, and each plan takes
// them in slot order; so they are always the last slots of each table, and
// the k smallest (priority, slot) among unheld slots are simply the next k
// of them.  This is the select's own result without the select.
__global__ void __launch_bounds__(BLOCK) k_fresh_victims(FreshArgs f, int32_t *v_slot)
{
    const int y = blockIdx.y;
    const int64_t k = f.k[y];
    for (int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x; i < k;
         i += (int64_t)gridDim.x * BLOCK)
        v_slot[f.vbase[y] + i] = (int32_t)(f.first[y] + i);
}

void launch_fresh_victims(const FreshArgs &f, int64_t max_k, int32_t *v_slot, hipStream_t s)
{
    if (f.n <= 0 || max_k <= 0) return;
    const int64_t gx = (max_k + BLOCK - 1) / BLOCK;
    hipLaunchKernelGGL(k_fresh_victims, dim3((unsigned)(gx < 1024 ? gx : 1024), (unsigned)f.n),
                       dim3(BLOCK), 0, s, f, v_slot);
}

void launch_select_victims(const SelArgs &a, int levels, int64_t maxS, const int32_t *hold_to,
                           const int32_t *held, int32_t *sel_state, int32_t *sel_hist,
                           uint32_t *vk0, uint32_t *vv0, uint32_t *vk1, uint32_t *vv1,
                           int64_t n_victims, uint32_t *hist, ScanWs &ws, int32_t *v_slot,
                           int32_t *err, hipStream_t s)
{
    if (a.nact <= 0 || n_victims <= 0) return;
    // small victim sets are ordered per table in LDS; otherwise one global
    // sort on (table, priority), whose compaction lands where the sort's last
    // pass will end in v_slot
    bool small = true;
    for (int y = 0; y < a.nact; ++y) small = small && a.k[y] <= VS_MAX;
    const int bits = a.act_bits + a.prio_bits;
    const int passes = small ? 1 : radix_passes(n_victims, bits);
    uint32_t *ck = (passes & 1) ? vk0 : vk1;
    uint32_t *cv = (passes & 1) ? vv0 : (uint32_t *)v_slot;
    uint32_t *ok = (passes & 1) ? vk1 : vk0;
    uint32_t *ov = (passes & 1) ? (uint32_t *)v_slot : vv0;
    // the compaction counts the global sort's first digits when its passes
    // are one launch each; their counters are cleared by the first pick
    const RadixPlan rp = radix_plan(n_victims, bits);
    const bool prehist = !small && rp.passes > 0 && rp.fused;
    const unsigned chunks = (unsigned)((maxS + SEL_CHUNK - 1) / SEL_CHUNK);
    for (int l = 0; l < levels; ++l) {
        int shift = (levels - 1 - l) * SEL_BITS;
        hipLaunchKernelGGL(k_sel_level, dim3(chunks, a.nact), dim3(BLOCK), 0, s, a, shift,
                           (int)(l == 0), hold_to, held, sel_state, sel_hist,
                           sel_state + 2 * MAX_TABLES, (int32_t *)cv, hist,
                           prehist ? rp.table * rp.passes : (int64_t)0);
    }
    SegAct seg;
    VictimOut out;
    for (int y = 0; y < a.nact; ++y) {
        seg.base[y] = a.base[y];
        seg.S[y] = a.S[y];
        out.vbase[y] = a.vbase[y];
        out.k[y] = a.k[y];
        out.last[y] = a.base[y] + a.S[y] - 1;
    }
    out.err = err;
    out.prio = a.prio;
    out.st = sel_state;
    out.prio_bits = a.prio_bits;
    out.vk = ck;
    out.vv = cv;
    out.hist0 = prehist ? hist : nullptr;
    out.digit_mask = prehist ? (1u << rp.dbits) - 1u : 0u;
    out.tile_len = prehist ? (uint32_t)(BLOCK * rp.items) : 1u;
    out.tiles = prehist ? (uint32_t)rp.tiles : 0u;
    seg_scan<uint64_t>(seg, a.nact, maxS, VictimFlag{hold_to, held, sel_state, a.prio, a.plan, a.stamp}, out, ws,
                       s);
    if (small) {
        hipLaunchKernelGGL(k_victim_sort, dim3(a.nact), dim3(VS_THREADS), 0, s, a,
                           (const uint32_t *)ck, (const uint32_t *)cv, v_slot);
        return;
    }
    bool in_k1 = false;
    launch_radix_sort(ck, cv, ok, ov, n_victims, bits, hist, ws, &in_k1, s, prehist);
}

// ---------------------------------------------------------------- commit

// Threads [0, n_miss): miss i goes to victim slot v = v_slot[i]: record the
// slot's previous occupant and its last use, erase that key from the Hit-Map,
// enter the new key, then touch the slot (last_use = u; with use counts, the
// new row's count starts at this plan's use) and point every position of the
// key at it.  Erases and inserts may interleave across
// threads: inserts only claim EMPTY or erased entries, so they never disturb
// a live key another thread is erasing, and the keys inserted are known to be
// absent.  Threads [n_miss, n_miss + max(n_unique, nnz)): touch the slots of
// hits and point the positions of hit keys at them.  Victims are unheld and
// hits are held, so the two groups never share a slot.  A placed row is held
// through the last window batch that has its key (binary searches of the
// later batches' sorted keys), plus hold_past; its slot was unheld, so only
// the new value is counted.
__device__ __forceinline__ bool commit_fill(int64_t i, uint64_t *hash, uint32_t mask,
                                            const TicketDev &tk, const int32_t *seg_off,
                                            const uint32_t *perm, int64_t n_unique, int64_t nnz,
                                            int64_t nslots, int32_t *key_of_slot,
                                            int32_t *last_use, int32_t *uses, int32_t u,
                                            int32_t prefetch, int32_t *err)
{
    // independent loads first: later stores could alias them, so the
    // compiler would otherwise keep each behind the stores before it
    const int32_t v = tk.v_slot[i];
    const int32_t ui = tk.m_uidx[i];
    const uint32_t key = tk.m_key[i];
    // a prefetched row (prefetch mode, m_uidx = -1) is placed but not used
    const bool fetched = prefetch && ui == -1;
    if ((uint32_t)v >= (uint64_t)nslots || (!fetched && (uint32_t)ui >= (uint64_t)n_unique)) {
        atomicOr(err, ERR_PLAN);
        tk.v_old_key[i] = -1;
        tk.v_old_lu[i] = -1;
        return false;
    }
    const int32_t old = key_of_slot[v];
    const int32_t old_lu = last_use[v];
    const int32_t p0 = fetched ? 0 : seg_off[ui], p1 = fetched ? 0 : seg_off[ui + 1];
    tk.v_old_key[i] = old;
    tk.v_old_lu[i] = old_lu;
    if (old >= 0) hash_erase(hash, mask, (uint32_t)old);
    key_of_slot[v] = (int32_t)key;
    if (!hash_insert(hash, mask, key, v)) atomicOr(err, ERR_HASH_FULL);
    last_use[v] = u;
    if (uses) uses[v] = fetched ? 0 : 1;
    if (fetched) return true;
    tk.slot_u[ui] = v;
    for (int32_t p = p0; p < p1; ++p) {
        const uint32_t j = perm[p];
        if (j < (uint64_t)nnz) tk.slot_of[j] = v;
    }
    return true;
}

// The last window batch 1 .. n-1 whose sorted unique keys hold key (0 if
// none).  The binary searches of all batches advance together, so their
// loads are in flight at once and a miss waits for one search, not n - 1.
__device__ __forceinline__ int32_t last_batch_with(const WindowKeys &wk, uint32_t key)
{
    int32_t lo[MAX_WINDOW], hi[MAX_WINDOW];
#pragma unroll
    for (int w = 0; w < MAX_WINDOW; ++w) {
        lo[w] = 0;
        hi[w] = w >= 1 && w < wk.n ? *wk.nu[w] : 0;
    }
    bool active = true;
    while (active) {
        active = false;
#pragma unroll
        for (int w = 1; w < MAX_WINDOW; ++w)
            if (lo[w] < hi[w]) {
                const int32_t mid = lo[w] + (hi[w] - lo[w]) / 2;
                if (wk.uk[w][mid] < key) lo[w] = mid + 1;
                else hi[w] = mid;
                active = true;
            }
    }
    int32_t q = 0;
#pragma unroll
    for (int w = 1; w < MAX_WINDOW; ++w)
        if (w < wk.n && lo[w] < *wk.nu[w] && wk.uk[w][lo[w]] == key) q = w;
    return q;
}

__global__ void __launch_bounds__(BLOCK) k_commit(uint64_t *hash, uint32_t mask, TicketDev tk,
                                                  const int32_t *inv, const int32_t *seg_off,
                                                  const uint32_t *perm, int64_t n_miss,
                                                  int64_t n_unique, int64_t nnz, int64_t nslots,
                                                  int32_t *key_of_slot, int32_t *last_use,
                                                  int32_t *uses, int32_t u, int32_t prefetch,
                                                  WindowKeys wk, HoldRows hr, RowIndex ri,
                                                  int64_t ent0, int32_t row_bits, int32_t T,
                                                  int32_t *hold_to, int32_t *hcnt, int32_t plan,
                                                  int32_t *err)
{
    __shared__ int32_t c[MAX_TABLES * HOLD_SPAN];
    // blocks that move hold counts (uniform per block): fills, entering keys
    const int64_t b0 = (int64_t)blockIdx.x * BLOCK;
    const bool fills = b0 < n_miss || b0 + BLOCK > ent0;
    if (fills) {
        for (int x = threadIdx.x; x < MAX_TABLES * HOLD_SPAN; x += BLOCK) c[x] = 0;
        __syncthreads();
    }
    const int64_t t = (int64_t)blockIdx.x * BLOCK + threadIdx.x;
    if (t < n_miss) {
        if (commit_fill(t, hash, mask, tk, seg_off, perm, n_unique, nnz, nslots, key_of_slot,
                        last_use, uses, u, prefetch, err)) {
            const uint32_t key = tk.m_key[t];
            const int32_t v = tk.v_slot[t];
            const int tt = (int)(key >> row_bits);
            int32_t q = 0;  // the last window batch with the key
            if (wk.fast && tt < T) {
                const int64_t row = ri.rbase[tt] + (key & ((1u << row_bits) - 1u));
                const int32_t lq = ri.lastq[row], pd = ri.pend[row];
                if (lq > plan + wk.n - 1) {  // from a window since shortened
                    q = last_batch_with(wk, key);
                } else {
                    q = lq >= plan ? lq - plan : 0;
                    if (pd == wk.stamp && wk.ent > q) q = wk.ent;
                }
            } else {
                q = last_batch_with(wk, key);
            }
            const int32_t off = q + wk.hold_past;
            hold_to[v] = plan + off;
            if (tt < T && off < HOLD_SPAN) atomicAdd(&c[tt * HOLD_SPAN + off], 1);
        }
    } else if (t >= ent0) {
        if (t - ent0 < hr.start[hr.n])
            hold_key(hold_ref(hr, t - ent0), row_bits, T, ri, hold_to, plan, c);
    } else {
        const int64_t j = t - n_miss;
        if (j < n_unique && tk.hit[j]) {
            const int32_t v = tk.slot_u[j];
            if ((uint32_t)v < (uint64_t)nslots) {
                last_use[v] = u;
                if (uses) uses[v] += 1;  // one thread per unique key, so one per slot
            }
        }
        if (j < nnz) {
            const int32_t i = inv[j];
            if ((uint32_t)i >= (uint64_t)n_unique) tk.slot_of[j] = -1;
            else if (tk.hit[i]) tk.slot_of[j] = tk.slot_u[i];
        }
    }
    if (fills) {
        __syncthreads();
        hold_counts_flush(c, hcnt, plan);
    }
}

void launch_commit(const Tables &tb, uint64_t *hash, uint32_t mask, TicketDev tk,
                   const BatchDev &b, int64_t n_miss, int64_t n_unique, int64_t nnz,
                   int32_t *key_of_slot, int32_t *last_use, int32_t *uses, int32_t u,
                   bool prefetch, const WindowKeys &wk, const HoldRows &hr, const RowIndex &ri,
                   int32_t *hold_to, int32_t *hcnt, DevCounters *cnt, hipStream_t s)
{
    // threads: misses, then the planned batch's keys and positions, then the
    // entering batches' keys
    const int64_t ent0 = n_miss + (nnz > n_unique ? nnz : n_unique);
    const int64_t n = ent0 + (hr.n > 0 ? hr.start[hr.n] : 0);
    if (n <= 0) return;
    const int64_t nslots = tb.slot_base[tb.T];
    hipLaunchKernelGGL(k_commit, dim3((unsigned)((n + BLOCK - 1) / BLOCK)), dim3(BLOCK), 0, s,
                       hash, mask, tk, (const int32_t *)b.inv, (const int32_t *)b.seg_off,
                       (const uint32_t *)b.perm, n_miss, n_unique, nnz, nslots, key_of_slot,
                       last_use, uses, u, (int32_t)prefetch, wk, hr, ri, ent0, tb.row_bits, tb.T,
                       hold_to, hcnt, u, &cnt->err_sticky);
}

// ---------------------------------------------------------------- prefetch arrangement
//
// One single-pass scan over a virtual range: indices [0, n_own) are the
// planned batch's own misses (ascending, all tables); then successor w's
// segment of len[w] indices (a bound on its unique keys), index j valued 1
// when its key j is flagged for prefetch.  The scan's prefix at a flagged key
// counts the flagged keys before it: all of the earlier successors', then
// those of the same successor in tables before t (keys are ascending by
// table), then its rank in table t.  The host folds the first two and the
// table's place into off[w][t], so the key goes to off[w][t] + prefix.

struct PfSeg {
    int64_t total;
    __device__ int64_t beg(int) const { return 0; }
    __device__ int64_t end(int) const { return total; }
};

struct PfVal {
    int64_t n_own;
    int32_t depth;
    int64_t start[MAX_PF + 1];     // first index of each successor's segment, then the end
    const int32_t *n_next[MAX_PF];  // unique keys of each successor
    const int32_t *flag;
    int64_t stride;
    __device__ uint32_t operator()(int64_t i, int) const
    {
        if (i < n_own) return 0u;
        uint32_t f = 0;
#pragma unroll
        for (int w = 0; w < MAX_PF; ++w) {  // the segment holding i, without indexing by w
            const int64_t j = i - start[w];
            if (w < depth && j >= 0 && i < start[w + 1] && j < *n_next[w])
                f = flag[(int64_t)w * stride + j] ? 1u : 0u;
        }
        return f;
    }
};

struct PfOut {
    int64_t n_own, n_miss;
    int32_t row_bits, T, depth;
    const uint32_t *own_key;
    const int32_t *own_uidx;
    const uint32_t *next_keys[MAX_PF];
    int64_t start[MAX_PF + 1];
    uint32_t *m_key;
    int32_t *m_uidx, *err;
    int32_t pf_before[MAX_TABLES];      // prefetched keys of the tables before t (all successors)
    int32_t off[MAX_PF][MAX_TABLES];    // successor w, table t: destination less the prefix
    __device__ void operator()(int64_t i, uint32_t e, uint32_t v, int) const
    {
        uint32_t key = 0;
        int32_t uidx;
        int64_t dst = -1;
        if (i < n_own) {
            key = own_key[i];
            uidx = own_uidx[i];
            const int t = (int)(key >> row_bits);
            if (t >= T) {
                atomicOr(err, ERR_PLAN);
                return;
            }
            dst = i + pf_before[t];
        } else {
            if (!v) return;
            uidx = -1;
#pragma unroll
            for (int w = 0; w < MAX_PF; ++w) {
                const int64_t j = i - start[w];
                if (w < depth && j >= 0 && i < start[w + 1]) {
                    key = next_keys[w][j];
                    const int t = (int)(key >> row_bits);
                    dst = t < T ? (int64_t)off[w][t] + e : -1;
                }
            }
        }
        if (dst < 0 || dst >= n_miss) {  // the counts and the lists disagree
            atomicOr(err, ERR_PLAN);
            return;
        }
        m_key[dst] = key;
        m_uidx[dst] = uidx;
    }
};

void launch_pf_arrange(const Tables &tb, PrefetchDev pf, int64_t n_own,
                       const int32_t *const *n_next, const int64_t *max_next,
                       const uint32_t *const *next_ukeys, const int32_t *own,
                       const int32_t (*pf_count)[MAX_TABLES], TicketDev tk, int64_t n_miss,
                       int32_t *err, ScanWs &ws, hipStream_t s)
{
    const int d = pf.depth;
    if (d < 1 || d > MAX_PF) {
        ws.overflow = true;
        return;
    }
    PfOut o{};
    PfVal val{};
    o.n_own = n_own;
    o.n_miss = n_miss;
    o.row_bits = tb.row_bits;
    o.T = tb.T;
    o.depth = d;
    o.own_key = pf.own_key;
    o.own_uidx = pf.own_uidx;
    o.m_key = tk.m_key;
    o.m_uidx = tk.m_uidx;
    o.err = err;
    val.n_own = n_own;
    val.depth = d;
    val.flag = pf.flag;
    val.stride = pf.stride;
    int64_t at = n_own;
    for (int w = 0; w < MAX_PF; ++w) {
        o.start[w] = val.start[w] = at;
        if (w < d) {
            o.next_keys[w] = next_ukeys[w];
            val.n_next[w] = n_next[w];
            at += max_next[w];
        }
    }
    o.start[MAX_PF] = val.start[MAX_PF] = at;
    // destinations: table t's victims start at vbase[t]; its own misses come
    // first, then successor 0's flagged keys, then successor 1's, ...
    int32_t tot[MAX_PF] = {};
    for (int w = 0; w < d; ++w)
        for (int t = 0; t < tb.T; ++t) tot[w] += pf_count[w][t];
    int32_t vb = 0, pfb = 0;
    for (int t = 0; t < tb.T; ++t) {
        o.pf_before[t] = pfb;
        int32_t before_w = 0;     // table t's flagged keys of the successors before w
        for (int w = 0; w < d; ++w) {
            int32_t first = 0;    // flagged keys before (successor w, table t) in the scan
            for (int w2 = 0; w2 < w; ++w2) first += tot[w2];
            for (int t2 = 0; t2 < t; ++t2) first += pf_count[w][t2];
            o.off[w][t] = vb + own[t] + before_w - first;
            before_w += pf_count[w][t];
        }
        pfb += before_w;
        vb += own[t] + before_w;
    }
    seg_scan<uint32_t>(PfSeg{at}, 1, at, val, o, ws, s);
}

}  // namespace sp
