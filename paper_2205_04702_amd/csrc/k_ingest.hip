// Window ingest: a batch that becomes visible to the planner is turned into
// sorted (table,row) keys, its unique keys, the inverse map and the runs of
// equal keys that the backward pass coalesces (gradient duplication and
// coalescing, Sec. II-B).  Everything here runs once per batch, when the batch
// enters the look-forward window.
#include "sp_device.h"
#include "sp_internal.h"

namespace sp {

// ---------------------------------------------------------------- small fills

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

void launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s)
{
    if (n <= 0) return;
    hipLaunchKernelGGL(k_fill_i32, dim3((unsigned)((n + BLOCK - 1) / BLOCK)), dim3(BLOCK), 0, s,
                       p, n, v);
}

void launch_zero_i32(int32_t *p, int64_t n, hipStream_t s) { launch_fill_i32(p, n, 0, s); }

// ---------------------------------------------------------------- keys and bags

// One launch over max(nnz, nbags) threads, two independent jobs:
//  * position j < nnz: key = table << row_bits | row, where the table is the
//    one whose span [bag_off[t*B], bag_off[(t+1)*B]) contains j; rows out of
//    range raise ERR_ID_RANGE and are clamped so nothing downstream leaves
//    its array;
//  * bag g < nbags: validate the offsets (non-decreasing, from 0 to nnz;
//    ERR_OFFSETS otherwise, ranges clamped into [0, nnz)), write bag_of[j] = g
//    for the bag's positions and copy the offsets into the window ring (when
//    they are read from the caller's device memory); the first bag of each
//    table also checks the table's ID count against max_table_ids (when set,
//    ERR_TABLE_IDS).
__global__ void __launch_bounds__(BLOCK) k_prepare(Tables tb, const int32_t *ids,
                                                   const int32_t *bag_off, int32_t *bag_off_copy,
                                                   int32_t B, int64_t nnz, int64_t nbags,
                                                   int64_t max_table_ids, uint32_t *keys,
                                                   uint32_t *pos, int32_t *bag_of, int32_t *err)
{
    const int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x;
    if (i < nnz) {
        int lo = 0, hi = tb.T - 1;  // largest t with bag_off[t*B] <= i
        while (lo < hi) {
            int mid = (lo + hi + 1) >> 1;
            if ((int64_t)bag_off[(int64_t)mid * B] <= i) lo = mid; else hi = mid - 1;
        }
        int32_t row = ids[i];
        if (row < 0 || (int64_t)row >= tb.rows[lo]) {
            atomicOr(err, ERR_ID_RANGE);
            row = 0;
        }
        keys[i] = ((uint32_t)lo << tb.row_bits) | (uint32_t)row;
        pos[i] = (uint32_t)i;
    }
    if (i < nbags) {
        int64_t lo = bag_off[i], hi = bag_off[i + 1];
        if (bag_off_copy != bag_off) {
            bag_off_copy[i] = (int32_t)lo;
            if (i == nbags - 1) bag_off_copy[i + 1] = (int32_t)hi;
        }
        bool bad = lo > hi || lo < 0 || hi > nnz || (i == 0 && lo != 0) ||
                   (i == nbags - 1 && hi != nnz);
        if (bad) {
            atomicOr(err, ERR_OFFSETS);
            lo = lo < 0 ? 0 : (lo > nnz ? nnz : lo);
            hi = hi < lo ? lo : (hi > nnz ? nnz : hi);
        }
        for (int64_t j = lo; j < hi; ++j) bag_of[j] = (int32_t)i;
        if (max_table_ids > 0 && i % B == 0 &&
            (int64_t)bag_off[i + B] - bag_off[i] > max_table_ids)
            atomicOr(err, ERR_TABLE_IDS);
    }
}

// ---------------------------------------------------------------- LSD radix sort
//
// Stable.  Per pass: tile histograms (digit-major), one scan of the histogram
// table, then a scatter in which every tile ranks its keys per digit with wave
// ballots, round by round (BLOCK keys per round), so equal digits keep input
// order.  Digits are up to RS_MAXBITS wide; a key of b bits takes
// ceil(b / 11) passes of ceil(b / passes) bits each.  A tile is `items`
// rounds: small inputs get short tiles so that more blocks share the work.
constexpr int RS_ITEMS = 8;                 // most rounds per tile
constexpr int RS_TILE = BLOCK * RS_ITEMS;   // longest tile
constexpr int RS_MAXBITS = 11;
constexpr int RS_MAXBINS = 1 << RS_MAXBITS;
// One-launch passes when every block can afford to read the whole
// (bins x tiles) histogram table.
constexpr int64_t RS_FUSED_TABLE = 16384;

int radix_passes(int64_t n, int bits)
{
    return (n <= 1 || bits <= 0) ? 0 : (bits + RS_MAXBITS - 1) / RS_MAXBITS;
}

RadixPlan radix_plan(int64_t n, int bits)
{
    RadixPlan p{};
    p.passes = radix_passes(n, bits);
    if (p.passes == 0) return p;
    p.dbits = (bits + p.passes - 1) / p.passes;
    const int64_t bins = (int64_t)1 << p.dbits;
    auto tiles_for = [n](int r) { return (n + (int64_t)BLOCK * r - 1) / ((int64_t)BLOCK * r); };
    p.items = RS_ITEMS;
    while (p.items > 1 && tiles_for(p.items) < 128 && bins * tiles_for(p.items / 2) <= RS_FUSED_TABLE)
        p.items /= 2;
    p.tiles = tiles_for(p.items);
    p.table = bins * p.tiles;
    p.fused = p.table <= RS_FUSED_TABLE;
    return p;
}

int64_t radix_hist_entries(int64_t n)
{
    const int64_t tiles = (n + RS_TILE - 1) / RS_TILE + 1;
    const int64_t big = (int64_t)RS_MAXBINS * tiles;
    return big > 4 * RS_FUSED_TABLE ? big : 4 * RS_FUSED_TABLE;
}

// hist[d * tiles + tile] = keys of the tile with digit d.  With zero_from /
// zero_n, also clears a range (the histograms later passes accumulate into).
__global__ void __launch_bounds__(BLOCK) k_radix_hist(const uint32_t *keys, int64_t n, int shift,
                                                      int dbits, int items, uint32_t *hist,
                                                      int tiles, uint32_t *zero_from,
                                                      int64_t zero_n)
{
    __shared__ uint32_t h[RS_MAXBINS];
    const int bins = 1 << dbits;
    const uint32_t mask = (uint32_t)bins - 1u;
    for (int d = threadIdx.x; d < bins; d += BLOCK) h[d] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * BLOCK * items;
    for (int r = 0; r < items; ++r) {
        const int64_t i = base + (int64_t)r * BLOCK + threadIdx.x;
        if (i < n) atomicAdd(&h[(keys[i] >> shift) & mask], 1u);
    }
    __syncthreads();
    for (int d = threadIdx.x; d < bins; d += BLOCK) hist[(int64_t)d * tiles + blockIdx.x] = h[d];
    for (int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x; i < zero_n;
         i += (int64_t)gridDim.x * BLOCK)
        zero_from[i] = 0;
}

// Stable scatter of one tile by one digit.  Keys are ranked round by round
// (256 keys per round, in input order): lanes of a wave with the same digit
// find each other with one ballot per digit bit; the lowest of them records
// the wave's count for that digit, stamped with the round, so stale counts of
// earlier rounds read as zero and nothing has to be cleared between rounds.
// base[d] is where the tile's next key of digit d goes.
//  FUSED: base comes from the raw per-tile histogram table (this block sums
//  its column prefix and the digit totals), and the scatter adds each key to
//  the next pass's histogram at its output tile, so a pass is one launch.
//  Otherwise base comes from a scanned (exclusive, digit-major) table.
template <bool FUSED>
__global__ void __launch_bounds__(BLOCK) k_radix_scatter(const uint32_t *kin, const uint32_t *vin,
                                                         int64_t n, int shift, int dbits,
                                                         int items, const uint32_t *table,
                                                         int tiles, uint32_t *kout,
                                                         uint32_t *vout, uint32_t *hist_next,
                                                         int shift_next, int dbits_next)
{
    __shared__ uint32_t base[RS_MAXBINS];
    __shared__ uint32_t wc[BLOCK / WAVE][RS_MAXBINS];
    __shared__ uint32_t lds[BLOCK / WAVE];
    const int tid = threadIdx.x, w = wave_id(), lane = lane_id();
    const int bins = 1 << dbits;
    const uint32_t mask = (uint32_t)bins - 1u;
    const int tile = blockIdx.x;
    const int tile_len = BLOCK * items;
    const int64_t tbase = (int64_t)tile * tile_len;
    // the tile's keys and values, all loads in flight at once
    uint32_t kr[RS_ITEMS], vr[RS_ITEMS];
#pragma unroll
    for (int r = 0; r < RS_ITEMS; ++r) {
        const int64_t i = tbase + (int64_t)r * BLOCK + tid;
        const bool in = r < items && i < n;
        kr[r] = in ? kin[i] : 0u;
        vr[r] = in ? vin[i] : 0u;
    }
    if (FUSED) {
        // digit totals into wc[0], this tile's column prefix into base
        for (int d = tid; d < bins; d += BLOCK) {
            const uint32_t *row = table + (int64_t)d * tiles;
            uint32_t before = 0, total = 0;
#pragma unroll 8
            for (int t = 0; t < tiles; ++t) {
                const uint32_t x = row[t];
                before += t < tile ? x : 0u;
                total += x;
            }
            base[d] = before;
            wc[0][d] = total;
        }
        __syncthreads();
        // exclusive scan of the digit totals: thread tid owns bins/BLOCK
        // consecutive digits (or one digit when bins < BLOCK)
        const int per = bins >= BLOCK ? bins / BLOCK : 1;
        const int d0 = tid * per;
        uint32_t mine = 0;
        for (int q = 0; q < per; ++q)
            if (d0 + q < bins) mine += wc[0][d0 + q];
        uint32_t total;
        uint32_t run = block_excl_scan(mine, lds, total);
        for (int q = 0; q < per; ++q)
            if (d0 + q < bins) {
                const uint32_t x = wc[0][d0 + q];
                base[d0 + q] += run;
                run += x;
            }
    } else {
        for (int d = tid; d < bins; d += BLOCK) base[d] = table[(int64_t)d * tiles + tile];
    }
    __syncthreads();
    for (int q = 0; q < BLOCK / WAVE; ++q)
        for (int d = tid; d < bins; d += BLOCK) wc[q][d] = 0;
    __syncthreads();

    const uint64_t lt = lanemask_lt();
    const uint32_t mask_next = (1u << dbits_next) - 1u;
#pragma unroll
    for (int r = 0; r < RS_ITEMS; ++r) {
        if (r >= items) break;  // uniform
        const uint32_t stamp = (uint32_t)(r + 1) << 16;
        const int64_t i = tbase + (int64_t)r * BLOCK + tid;
        const bool valid = i < n;
        const uint32_t k = kr[r];
        const uint32_t v = vr[r];
        const uint32_t d = (k >> shift) & mask;
        uint64_t peers = __ballot(valid);
        for (int b = 0; b < dbits; ++b) {
            const uint32_t bit = (d >> b) & 1u;
            const uint64_t bb = __ballot(bit);
            peers &= bit ? bb : ~bb;
        }
        const int leader = valid ? __ffsll((unsigned long long)peers) - 1 : lane;
        const bool is_leader = valid && leader == lane;
        if (is_leader) wc[w][d] = stamp | (uint32_t)__popcll(peers);
        __syncthreads();
        uint32_t start = 0;
        bool last_wave = false;
        uint32_t total = 0;
        if (is_leader) {
            uint32_t before = 0;
            last_wave = true;
            for (int q = 0; q < BLOCK / WAVE; ++q) {
                const uint32_t e = wc[q][d];
                const uint32_t c = (e & 0xFFFF0000u) == stamp ? (e & 0xFFFFu) : 0u;
                if (q < w) before += c;
                if (q > w && c) last_wave = false;
                total += c;
            }
            start = base[d] + before;
        }
        start = __shfl(start, leader, WAVE);
        __syncthreads();  // every leader has read base[d]
        if (is_leader && last_wave) base[d] += total;
        if (valid) {
            uint32_t p = start + (uint32_t)__popcll(peers & lt);
            p = p < (uint64_t)n ? p : (uint32_t)(n - 1);  // never write past the output
            kout[p] = k;
            vout[p] = v;
            if (FUSED && hist_next)
                atomicAdd(&hist_next[(int64_t)((k >> shift_next) & mask_next) * tiles +
                                     p / (uint32_t)tile_len],
                          1u);
        }
        __syncthreads();
    }
}

struct ValU32 {
    const uint32_t *p;
    __device__ uint32_t operator()(int64_t i, int) const { return p[i]; }
};
struct OutU32 {
    uint32_t *p;
    __device__ void operator()(int64_t i, uint32_t e, uint32_t, int) const { p[i] = e; }
};

// Sorts (k0, v0) by key (LSD, stable); k1/v1 are scratch of the same size.
// The result is in k1/v1 when radix_passes(n, bits) is odd (*in_k1).  With
// prehist (one-launch passes only), the caller has already filled the first
// pass's table (tile t = keys [t * BLOCK * items, ...)) and zeroed the other
// passes' tables (radix_plan gives the layout).
void launch_radix_sort(uint32_t *k0, uint32_t *v0, uint32_t *k1, uint32_t *v1, int64_t n,
                       int bits, uint32_t *hist, ScanWs &ws, bool *in_k1, hipStream_t s,
                       bool prehist)
{
    *in_k1 = false;
    const RadixPlan rp = radix_plan(n, bits);
    const int passes = rp.passes;
    if (passes == 0) return;
    const int dbits = rp.dbits, items = rp.items;
    const int tiles = (int)rp.tiles;
    const int64_t table = rp.table;
    uint32_t *ki = k0, *vi = v0, *ko = k1, *vo = v1;
    if (rp.fused) {
        // hist + P one-launch passes; pass p reads table p and fills table p+1
        if (!prehist)
            hipLaunchKernelGGL(k_radix_hist, dim3(tiles), dim3(BLOCK), 0, s, ki, n, 0, dbits, items,
                               hist, tiles, hist + table, table * (passes - 1));
        for (int p = 0; p < passes; ++p) {
            uint32_t *next = p + 1 < passes ? hist + table * (p + 1) : nullptr;
            hipLaunchKernelGGL(k_radix_scatter<true>, dim3(tiles), dim3(BLOCK), 0, s, ki, vi, n,
                               dbits * p, dbits, items, hist + table * p, tiles, ko, vo, next,
                               dbits * (p + 1), dbits);
            uint32_t *t;
            t = ki, ki = ko, ko = t;
            t = vi, vi = vo, vo = t;
        }
    } else {
        for (int p = 0; p < passes; ++p) {
            const int shift = dbits * p;
            hipLaunchKernelGGL(k_radix_hist, dim3(tiles), dim3(BLOCK), 0, s, ki, n, shift, dbits,
                               items, hist, tiles, (uint32_t *)nullptr, (int64_t)0);
            seg_scan<uint32_t>(SegN{table}, 1, table, ValU32{hist}, OutU32{hist}, ws, s);
            hipLaunchKernelGGL(k_radix_scatter<false>, dim3(tiles), dim3(BLOCK), 0, s, ki, vi, n,
                               shift, dbits, items, hist, tiles, ko, vo, (uint32_t *)nullptr, 0,
                               dbits);
            uint32_t *t;
            t = ki, ki = ko, ko = t;
            t = vi, vi = vo, vo = t;
        }
    }
    *in_k1 = (ki == k1);
}

// ---------------------------------------------------------------- unique keys

struct HeadFlag {
    const uint32_t *k;
    __device__ uint32_t operator()(int64_t i, int) const
    {
        const uint32_t a = k[i], b = k[i > 0 ? i - 1 : i];  // both loads, no branch
        return i == 0 || a != b;
    }
};

// Segment (run of equal keys) bookkeeping for sorted position i.
struct UniqueOut {
    const uint32_t *skeys, *perm;
    const int32_t *bag_of;
    uint32_t *ukeys;
    int32_t *inv, *seg_off, *sbag, *scal;
    int64_t n;
    __device__ void operator()(int64_t i, uint32_t e, uint32_t f, int) const
    {
        uint32_t seg = e + f - 1;
        uint32_t p = perm[i];
        if (f) {
            ukeys[seg] = skeys[i];
            seg_off[seg] = (int32_t)i;
        }
        inv[p] = (int32_t)seg;
        sbag[i] = bag_of[p];
        if (i == n - 1) {
            scal[0] = (int32_t)(seg + 1);
            seg_off[seg + 1] = (int32_t)n;
        }
    }
};

// Backward work split: a run of len positions becomes ceil(len / chunk) chunks.
struct ChunkCount {
    const int32_t *seg_off;
    int32_t chunk;
    __device__ uint32_t operator()(int64_t s, int) const
    {
        int32_t len = seg_off[s + 1] - seg_off[s];
        return (uint32_t)((len + chunk - 1) / chunk);
    }
};
// Chunk c of run s gets the descriptor {first position, end position, s,
// chunks of s}; runs with more than one chunk are also listed in `multi`.
struct ChunkOut {
    const int32_t *seg_off;
    int32_t chunk;
    int32_t *seg_chunk0;
    int4 *chunk_desc;
    int32_t *multi, *scal;
    __device__ void operator()(int64_t s, uint32_t e, uint32_t v, int) const
    {
        seg_chunk0[s] = (int32_t)e;
        const int32_t s0 = seg_off[s], s1 = seg_off[s + 1];
        for (uint32_t c = 0; c < v; ++c) {
            const int32_t p0 = s0 + (int32_t)c * chunk;
            chunk_desc[e + c] = make_int4(p0, p0 + chunk < s1 ? p0 + chunk : s1, (int32_t)s,
                                          (int32_t)v);
        }
        if (v > 1) multi[atomicAdd(scal + 3, 1)] = (int32_t)s;  // list order is irrelevant
        if (s == scal[0] - 1) scal[1] = (int32_t)(e + v);
    }
};

// ---------------------------------------------------------------- tables in LDS, split by rows
//
// When every table of a batch has at most IG_MAX IDs and the batch at most
// IG_MAX bags per table, one launch does all of the above.  Each table is
// handled by S workgroups, each owning one contiguous range of its rows
// (workgroups take (table, range) pairs in the order they start, from an
// atomic counter).  A workgroup reads the table's offsets and IDs, keeps the
// entries whose row falls in its range in position order (entry = row offset
// << 26 | bag << 13 | position, positions and bags local to the table), sorts
// them by row in LDS, finds the runs of equal rows and their backward chunks,
// then publishes its entry, unique-key, chunk and long-run counts and its
// error bits (epoch-tagged, as the single-pass scan does).  It adds up the
// counts of every workgroup that started before it to place its outputs.
// Keys are table-major and the ranges ascend, so this is the order of the
// general path: a workgroup's sorted entries follow those of the ranges
// before it within the table's span of the batch.  Once a workgroup has read
// all of its inputs it counts itself in *cons; the one that completes the
// count (cons_target) writes cons_seq to the host-coherent word cons_word,
// which tells the host that the caller's arrays are no longer needed, long
// before the kernel ends.  A workgroup can hold a whole table, so any
// distribution of rows over the ranges is handled; an even one spreads the
// sort over S compute units.
constexpr int IG_THREADS = 1024;
constexpr int IG_WAVES = IG_THREADS / WAVE;
constexpr int IG_ITEMS = 8;
constexpr int IG_SHIFT_BAG = 13, IG_SHIFT_ROW = 26;
constexpr uint32_t IG_LOW = (1u << IG_SHIFT_BAG) - 1u;
static_assert(IG_THREADS * IG_ITEMS == IG_MAX, "one item per thread per round");
static_assert(MAX_TABLES * IG_SPLIT_MAX <= IG_THREADS, "one earlier workgroup per thread");

__global__ void __launch_bounds__(IG_THREADS) k_ingest_table(Tables tb, const int32_t *ids,
                                                             const int32_t *bag_off,
                                                             int32_t *bag_off_copy, int32_t B,
                                                             int64_t nnz, int32_t chunk,
                                                             int64_t max_table_ids, BatchDev b,
                                                             int64_t cap_u, int64_t cap_c,
                                                             ScanDev d, int32_t S, uint32_t *cons,
                                                             uint32_t cons_target,
                                                             uint64_t *cons_word, uint32_t cons_seq)
{
    __shared__ uint64_t buf[2][IG_MAX];
    __shared__ uint32_t wc[IG_WAVES][256];
    __shared__ uint32_t lds[IG_WAVES];
    __shared__ uint32_t id_s, multi_s, m_s;
    __shared__ int32_t err_s;
    __shared__ uint32_t before_s[5];
    const int tid = threadIdx.x, w = wave_id(), lane = lane_id();
    if (tid == 0) {
        id_s = atomicAdd(d.counter, 1u) - d.base;
        multi_s = 0;
        err_s = 0;
    }
    __syncthreads();
    const uint32_t id = id_s;
    const int t = (int)(id / (uint32_t)S), sub = (int)(id % (uint32_t)S);
    auto inputs_read = [&]() {  // thread 0, after every read of ids and bag_off
        if (atomicAdd(cons, 1u) + 1u == cons_target)
            __hip_atomic_store(cons_word, (uint64_t)cons_seq, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_SYSTEM);
    };
    if (t >= tb.T) {  // the counter and the host disagree: give up loudly
        if (tid == 0) {
            atomicOr(d.err, ERR_PLAN);
            inputs_read();
        }
        return;
    }
    const int64_t nbags = (int64_t)tb.T * B;
    // ---- the table's span of the batch, then its IDs and offsets, all loads
    // in flight together
    int64_t j0 = bag_off[(int64_t)t * B], j1 = bag_off[(int64_t)(t + 1) * B];
    j0 = j0 < 0 ? 0 : (j0 > nnz ? nnz : j0);
    j1 = j1 < j0 ? j0 : (j1 > nnz ? nnz : j1);
    const int n = (int)(j1 - j0 < IG_MAX ? j1 - j0 : IG_MAX);
    // a table past the configured bound: the rest is left out and the plan fails
    int32_t err = j1 - j0 > max_table_ids ? ERR_TABLE_IDS : 0;
    int32_t rv[IG_ITEMS];
#pragma unroll
    for (int r = 0; r < IG_ITEMS; ++r) {
        const int i = r * IG_THREADS + tid;
        rv[r] = n > 0 ? ids[j0 + (i < n ? i : n - 1)] : 0;
    }
    // offsets: validate, mark the bag of every position; the first range's
    // workgroup copies them into the ring
    uint32_t *bag_at = reinterpret_cast<uint32_t *>(buf[1]);
    for (int lb = tid; lb < B; lb += IG_THREADS) {
        const int64_t g = (int64_t)t * B + lb;
        const int64_t lo = bag_off[g], hi = bag_off[g + 1];
        if (sub == 0 && bag_off_copy != bag_off) {
            bag_off_copy[g] = (int32_t)lo;
            if (g == nbags - 1) bag_off_copy[g + 1] = (int32_t)hi;
        }
        if (lo > hi || lo < 0 || hi > nnz || (g == 0 && lo != 0) || (g == nbags - 1 && hi != nnz))
            err |= ERR_OFFSETS;
        const int64_t a = lo - j0 < 0 ? 0 : lo - j0, e = hi - j0 > n ? n : hi - j0;
        for (int64_t i = a; i < e; ++i) bag_at[i] = (uint32_t)lb;
    }
    // this workgroup's rows
    const int64_t rows_t = tb.rows[t];
    const int64_t span = (rows_t + S - 1) / S;
    const int64_t r0 = (int64_t)sub * span;
    const int64_t r1 = r0 + span < rows_t ? r0 + span : rows_t;
    int rbits = 0;
    while ((int64_t)1 << rbits < span) ++rbits;
    __syncthreads();
    // ---- keep the entries of this range, in position order: per round r the
    // waves' counts are laid out (r, wave) and scanned by wave 0
    const uint64_t lt = lanemask_lt();
    uint32_t kept = 0, rank[IG_ITEMS];
    uint32_t *cnt = &wc[0][0];
#pragma unroll
    for (int r = 0; r < IG_ITEMS; ++r) {
        const int i = r * IG_THREADS + tid;
        int32_t row = rv[r];
        if (i < n && (row < 0 || (int64_t)row >= rows_t)) {
            err |= ERR_ID_RANGE;
            row = 0;
        }
        rv[r] = row;
        const bool keep = i < n && row >= r0 && row < r1;
        const uint64_t bal = __ballot(keep);
        kept |= (uint32_t)keep << r;
        rank[r] = (uint32_t)__popcll(bal & lt);
        if (lane == 0) cnt[r * IG_WAVES + w] = (uint32_t)__popcll(bal);
    }
    if (err) atomicOr(&err_s, err);
    __syncthreads();
    if (tid == 0) inputs_read();
    if (w == 0) {
        static_assert(IG_ITEMS * IG_WAVES == 2 * WAVE, "two counts per lane");
        const uint32_t c0 = cnt[2 * lane], c1 = cnt[2 * lane + 1];
        const uint32_t incl = wave_incl_scan(c0 + c1);
        cnt[2 * lane] = incl - c0 - c1;
        cnt[2 * lane + 1] = incl - c1;
        if (lane == WAVE - 1) m_s = incl;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < IG_ITEMS; ++r) {
        if ((kept >> r) & 1u) {
            const int i = r * IG_THREADS + tid;
            uint32_t bag = bag_at[i];
            bag = bag < (uint32_t)B ? bag : 0u;  // positions no bag covers: flagged above
            buf[0][cnt[r * IG_WAVES + w] + rank[r]] =
                ((uint64_t)(rv[r] - r0) << IG_SHIFT_ROW) | ((uint64_t)bag << IG_SHIFT_BAG) |
                (uint64_t)i;
        }
    }
    const int m = (int)m_s;
    __syncthreads();
    uint64_t *srt = lds_radix_sort<IG_THREADS, IG_ITEMS>(buf[0], buf[1], m, IG_SHIFT_ROW, rbits,
                                                         wc, lds);
    // the other buffer holds each run's first sorted index and its first chunk
    uint32_t *run0 = reinterpret_cast<uint32_t *>(srt == buf[0] ? buf[1] : buf[0]);
    uint32_t *chunk0 = run0 + IG_MAX;

    // ---- runs of equal rows (blocked: thread tid owns items tid*K .. tid*K+K-1)
    const int K = (m + IG_THREADS - 1) / IG_THREADS;
    const int i0 = tid * K;
    uint32_t heads = 0;
    uint64_t e[IG_ITEMS];
#pragma unroll
    for (int q = 0; q < IG_ITEMS; ++q) {
        const int i = i0 + q;
        const bool in = q < K && i < m;
        e[q] = in ? srt[i] : 0ull;
        const bool h = in && (i == 0 || (srt[i - 1] >> IG_SHIFT_ROW) != (e[q] >> IG_SHIFT_ROW));
        heads |= (uint32_t)h << q;
    }
    uint32_t nU;
    const uint32_t seg_first = block_excl_scan_n<IG_THREADS>((uint32_t)__popc(heads), lds, nU);
    {
        uint32_t sg = seg_first;
#pragma unroll
        for (int q = 0; q < IG_ITEMS; ++q)
            if ((heads >> q) & 1u) run0[sg++] = (uint32_t)(i0 + q);
    }
    __syncthreads();
    // chunks per run (blocked over runs the same way)
    uint32_t nch[IG_ITEMS], csum = 0, msum = 0;
#pragma unroll
    for (int q = 0; q < IG_ITEMS; ++q) {
        const uint32_t sr = (uint32_t)(i0 + q);
        nch[q] = 0;
        if (q < K && sr < nU) {
            const uint32_t len = (sr + 1 < nU ? run0[sr + 1] : (uint32_t)m) - run0[sr];
            nch[q] = (len + (uint32_t)chunk - 1) / (uint32_t)chunk;
            csum += nch[q];
            msum += nch[q] > 1;
        }
    }
    uint32_t nC;
    uint32_t cb = block_excl_scan_n<IG_THREADS>(csum, lds, nC);
    uint32_t nM;
    (void)block_excl_scan_n<IG_THREADS>(msum, lds, nM);
#pragma unroll
    for (int q = 0; q < IG_ITEMS; ++q) {
        const uint32_t sr = (uint32_t)(i0 + q);
        if (q < K && sr < nU) chunk0[sr] = cb;
        cb += nch[q];
    }

    // ---- publish this workgroup's counts, add up those of every earlier one
    uint64_t *st = d.status + (int64_t)id * LB_WORDS;
    if (tid == 0) {
        const uint32_t mine[4] = {nU, nC, nM, (uint32_t)err_s << 16 | (uint32_t)m};
#pragma unroll
        for (int c = 0; c < 4; ++c) lb_publish<uint32_t>(st + c, d.epoch, mine[c]);
    }
    uint32_t v[4] = {0, 0, 0, 0};
    if (tid < (int)id) {  // one thread per earlier workgroup
        const uint64_t *wd = d.status + (int64_t)tid * LB_WORDS;
        int spins = 0;
        bool ok = false;
        while (!ok) {
            ok = true;
#pragma unroll
            for (int c = 0; c < 4; ++c) ok = lb_read<uint32_t>(wd + c, d.epoch, v[c]) && ok;
            if (!ok && ++spins > LB_SPIN) {  // counted as zero; result flagged wrong
                atomicOr(d.err, ERR_PLAN);
                v[0] = v[1] = v[2] = v[3] = 0;
                break;
            }
            if (!ok) __builtin_amdgcn_s_sleep(1);
        }
    }
    {
        // entries before this range within the table; error bits of them all
        const uint32_t ent = tid >= t * S ? (v[3] & 0xFFFFu) : 0u;
        uint32_t eo = v[3] >> 16;
#pragma unroll
        for (int o = WAVE / 2; o > 0; o >>= 1) eo |= __shfl_xor(eo, o, WAVE);
        const uint32_t part[5] = {wave_sum(v[0]), wave_sum(v[1]), wave_sum(v[2]), eo,
                                  wave_sum(ent)};
        if (lane == 0)
#pragma unroll
            for (int c = 0; c < 5; ++c) wc[c][w] = part[c];
        __syncthreads();
        if (tid < 5) {
            uint32_t acc = 0;
            for (int q = 0; q < IG_WAVES; ++q) acc = tid == 3 ? (acc | wc[tid][q]) : acc + wc[tid][q];
            before_s[tid] = acc;
        }
        __syncthreads();
    }
    const uint32_t U0 = before_s[0], C0 = before_s[1], M0 = before_s[2];
    const int64_t jb = j0 + (int64_t)before_s[4];  // this range's first sorted position
    const int rb = tb.row_bits;
    const int64_t n_multi = multi_capacity(cap_u, chunk);

    // ---- outputs: positions
    uint32_t sg = seg_first;
#pragma unroll
    for (int q = 0; q < IG_ITEMS; ++q) {
        const int i = i0 + q;
        if (q >= K || i >= m) break;
        const uint32_t row = (uint32_t)((e[q] >> IG_SHIFT_ROW) + (uint64_t)r0);
        const int32_t bag = (int32_t)((e[q] >> IG_SHIFT_BAG) & IG_LOW);
        const int64_t pos = j0 + (int64_t)(e[q] & IG_LOW);
        const int64_t gi = jb + i;
        if ((heads >> q) & 1u) {
            if ((int64_t)U0 + sg < cap_u) {
                b.ukeys[U0 + sg] = ((uint32_t)t << rb) | row;
                b.seg_off[U0 + sg] = (int32_t)gi;
            }
            ++sg;
        }
        b.perm[gi] = (uint32_t)pos;
        b.sbag[gi] = (int32_t)((int64_t)t * B + bag);
        b.inv[pos] = (int32_t)(U0 + sg - 1);
    }
    // ---- outputs: runs and their backward chunks
#pragma unroll
    for (int q = 0; q < IG_ITEMS; ++q) {
        const uint32_t sr = (uint32_t)(i0 + q);
        if (q >= K || sr >= nU) break;
        const int64_t gs = (int64_t)U0 + sr;
        const int64_t c0 = (int64_t)C0 + chunk0[sr];
        if (gs >= cap_u) break;
        b.seg_chunk0[gs] = (int32_t)c0;
        const int32_t s0 = (int32_t)(jb + run0[sr]);
        const int32_t s1 = (int32_t)(jb + (sr + 1 < nU ? run0[sr + 1] : (uint32_t)m));
        for (uint32_t c = 0; c < nch[q] && c0 + c < cap_c; ++c) {
            const int32_t p0 = s0 + (int32_t)c * chunk;
            b.chunk_desc[c0 + c] = make_int4(p0, p0 + chunk < s1 ? p0 + chunk : s1, (int32_t)gs,
                                             (int32_t)nch[q]);
        }
        if (nch[q] > 1) {
            const uint32_t mi = M0 + atomicAdd(&multi_s, 1u);  // list order is irrelevant
            if ((int64_t)mi < n_multi) b.multi[mi] = (int32_t)gs;
        }
    }
    if (id == (uint32_t)(tb.T * S - 1) && tid == 0) {  // the batch totals
        const uint32_t U = U0 + nU;
        if ((int64_t)U < cap_u + 1) b.seg_off[U] = (int32_t)nnz;
        b.scal[0] = (int32_t)U;
        b.scal[1] = (int32_t)(C0 + nC);
        b.scal[2] = (int32_t)(before_s[3] | (uint32_t)err_s);
        b.scal[3] = (int32_t)(M0 + nM);
    }
}

// Sort, deduplicate and split into backward chunks one batch of the window.
// ids / bag_off may be the caller's device arrays (read once, here) or the
// ring's own copies; the ring always ends up with the offsets.  Input errors
// are recorded in the batch's own scal[2].
void launch_ingest(const Tables &tb, const BatchDev &b, const int32_t *ids, const int32_t *bag_off,
                   int32_t B, int64_t nnz, int key_bits, int chunk, int64_t max_table_ids,
                   int64_t cap_u, int64_t cap_c, uint32_t *tmp_k, uint32_t *tmp_v,
                   uint32_t *hist, ScanWs &ws, hipEvent_t consumed, const IngestCons &ic,
                   hipStream_t s)
{
    const int64_t nbags = (int64_t)tb.T * B;
    if (nnz > 0 && ingest_in_lds(max_table_ids, B)) {
        const int S = ingest_splits(tb.T);
        const int64_t grid = (int64_t)tb.T * S;
        if (grid > ws.max_tiles) {
            ws.overflow = true;
            return;
        }
        if (ws.epoch == 0xFFFFFFFFu) {  // epochs wrapped: forget every published word
            (void)hipMemsetAsync(ws.status, 0, sizeof(uint64_t) * LB_WORDS * ws.max_tiles, s);
            ws.epoch = 0;
        }
        ScanDev d{ws.status, ws.counter, ws.err, ws.issued, ++ws.epoch, (uint32_t)grid, 1};
        ws.issued += (uint32_t)grid;
        hipLaunchKernelGGL(k_ingest_table, dim3((unsigned)grid), dim3(IG_THREADS), 0, s, tb, ids,
                           bag_off, b.bag_off, B, nnz, chunk, max_table_ids, b, cap_u, cap_c, d,
                           S, ic.counter, ic.target, ic.word, ic.seq);
        return;
    }
    launch_zero_i32(b.scal, 4, s);
    // place the keys so that the final sort pass lands in skeys/perm
    const int passes = radix_passes(nnz, key_bits);
    uint32_t *k0 = (passes & 1) ? tmp_k : b.skeys, *v0 = (passes & 1) ? tmp_v : b.perm;
    uint32_t *k1 = (passes & 1) ? b.skeys : tmp_k, *v1 = (passes & 1) ? b.perm : tmp_v;
    const int64_t nthr = nnz > nbags ? nnz : nbags;
    if (nthr > 0)
        hipLaunchKernelGGL(k_prepare, dim3((unsigned)((nthr + BLOCK - 1) / BLOCK)), dim3(BLOCK), 0,
                           s, tb, ids, bag_off, b.bag_off, B, nnz, nbags, max_table_ids, k0, v0,
                           b.bag_of, b.scal + 2);
    else if (bag_off != b.bag_off)
        (void)hipMemcpyAsync(b.bag_off, bag_off, sizeof(int32_t), hipMemcpyDeviceToDevice, s);
    if (consumed) (void)hipEventRecord(consumed, s);  // the inputs are not read after this point
    if (nnz > 0) {
        bool in_k1 = false;
        launch_radix_sort(k0, v0, k1, v1, nnz, key_bits, hist, ws, &in_k1, s, false);
        seg_scan<uint32_t>(SegN{nnz}, 1, nnz, HeadFlag{b.skeys},
                           UniqueOut{b.skeys, b.perm, b.bag_of, b.ukeys, b.inv, b.seg_off, b.sbag,
                                     b.scal, nnz},
                           ws, s);
        seg_scan<uint32_t>(SegDevN{b.scal}, 1, nnz, ChunkCount{b.seg_off, chunk},
                           ChunkOut{b.seg_off, chunk, b.seg_chunk0, b.chunk_desc, b.multi, b.scal},
                           ws, s);
    }
}

}  // namespace sp
