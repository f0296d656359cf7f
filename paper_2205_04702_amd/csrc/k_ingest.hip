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
//    they are read from the caller's device memory).
__global__ void __launch_bounds__(BLOCK) k_prepare(Tables tb, const int32_t *ids,
                                                   const int32_t *bag_off, int32_t *bag_off_copy,
                                                   int32_t B, int64_t nnz, int64_t nbags,
                                                   uint32_t *keys, uint32_t *pos, int32_t *bag_of,
                                                   int32_t *err)
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
    __device__ uint32_t operator()(int64_t i, int) const { return i == 0 || k[i] != k[i - 1]; }
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

// Sort, deduplicate and split into backward chunks one batch of the window.
// ids / bag_off may be the caller's device arrays (read once, here) or the
// ring's own copies; the ring always ends up with the offsets.  Input errors
// are recorded in the batch's own scal[2].
void launch_ingest(const Tables &tb, const BatchDev &b, const int32_t *ids, const int32_t *bag_off,
                   int32_t B, int64_t nnz, int key_bits, int chunk, uint32_t *tmp_k,
                   uint32_t *tmp_v, uint32_t *hist, ScanWs &ws, hipEvent_t consumed,
                   hipStream_t s)
{
    const int64_t nbags = (int64_t)tb.T * B;
    launch_zero_i32(b.scal, 4, s);
    // place the keys so that the final sort pass lands in skeys/perm
    const int passes = radix_passes(nnz, key_bits);
    uint32_t *k0 = (passes & 1) ? tmp_k : b.skeys, *v0 = (passes & 1) ? tmp_v : b.perm;
    uint32_t *k1 = (passes & 1) ? b.skeys : tmp_k, *v1 = (passes & 1) ? b.perm : tmp_v;
    const int64_t nthr = nnz > nbags ? nnz : nbags;
    if (nthr > 0)
        hipLaunchKernelGGL(k_prepare, dim3((unsigned)((nthr + BLOCK - 1) / BLOCK)), dim3(BLOCK), 0,
                           s, tb, ids, bag_off, b.bag_off, B, nnz, nbags, k0, v0, b.bag_of,
                           b.scal + 2);
    else if (bag_off != b.bag_off)
        hipMemcpyAsync(b.bag_off, bag_off, sizeof(int32_t), hipMemcpyDeviceToDevice, s);
    hipEventRecord(consumed, s);  // the caller's arrays are not read after this point
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
