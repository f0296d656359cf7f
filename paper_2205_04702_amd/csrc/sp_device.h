// Device-side building blocks shared by the scratchpad kernels (CDNA4, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sp_internal.h"

namespace sp {

constexpr int WAVE = 64;
constexpr int BLOCK = 256;                 // 4 waves

__device__ __forceinline__ int lane_id() { return threadIdx.x & (WAVE - 1); }
__device__ __forceinline__ int wave_id() { return threadIdx.x / WAVE; }
__device__ __forceinline__ uint64_t lanemask_lt() { return (1ull << lane_id()) - 1ull; }

// The hardware hands the blocks of a launch to the 8 XCDs in turn (block b to
// XCD b % 8), and each XCD has its own L2.  This maps block b to a logical
// block so that XCD x works through the x-th eighth of the logical blocks: work
// that is contiguous in logical order (one table's bags, chunks or rows) then
// shares one L2.  A bijection on [0, n).
constexpr int XCDS = 8;
__device__ __forceinline__ int64_t xcd_block(int64_t b, int64_t n)
{
    const int64_t x = b % XCDS, i = b / XCDS, q = n / XCDS, rem = n % XCDS;
    return x * q + (x < rem ? x : rem) + i;
}

template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v)
{
    const int lane = lane_id();
#pragma unroll
    for (int o = 1; o < WAVE; o <<= 1) {
        T n = __shfl_up(v, o, WAVE);
        if (lane >= o) v += n;
    }
    return v;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v)
{
#pragma unroll
    for (int o = WAVE / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
    return v;
}

// Exclusive scan over a 256-thread block.  `lds` holds 4 entries; `total`
// receives the block sum.  Contains two barriers; every thread must call it.
template <typename T>
__device__ __forceinline__ T block_excl_scan(T v, T *lds, T &total)
{
    T incl = wave_incl_scan(v);
    if (lane_id() == WAVE - 1) lds[wave_id()] = incl;
    __syncthreads();
    T base = 0, sum = 0;
#pragma unroll
    for (int w = 0; w < BLOCK / WAVE; ++w) {
        T x = lds[w];
        if (w < wave_id()) base += x;
        sum += x;
    }
    __syncthreads();
    total = sum;
    return base + incl - v;
}

// Exclusive scan over a block of NT threads (every thread calls it; `lds`
// holds NT / WAVE entries; two barriers).
template <int NT, typename T>
__device__ __forceinline__ T block_excl_scan_n(T v, T *lds, T &total)
{
    T incl = wave_incl_scan(v);
    if (lane_id() == WAVE - 1) lds[wave_id()] = incl;
    __syncthreads();
    T base = 0, sum = 0;
#pragma unroll
    for (int w = 0; w < NT / WAVE; ++w) {
        T x = lds[w];
        if (w < wave_id()) base += x;
        sum += x;
    }
    __syncthreads();
    total = sum;
    return base + incl - v;
}

template <typename T>
__device__ __forceinline__ T block_sum(T v, T *lds)
{
    T total;
    (void)block_excl_scan(v, lds, total);
    return total;
}

// ---------------------------------------------------------------- segmented scan
//
// Segmented exclusive scan over index ranges in one launch (single pass with
// decoupled look-back).  Segment y covers [seg.beg(y), seg.end(y)); values
// come from val(i, y) and every index receives out(i, prefix, value, y).
// Tiles of LB_TILE indices are handed out in launch order through an atomic
// counter, so every tile a block looks back at belongs to a block that has
// already started.  A tile publishes its own sum, then its inclusive prefix
// once known; a successor adds published sums walking backwards until it
// meets an inclusive prefix.  Published words carry the launch's epoch in
// their upper half, so nothing is cleared between launches.  Values are one
// 32-bit counter (uint32_t) or two independent 32-bit counters packed in a
// uint64_t (low and high half, each sum below 2^32).

struct SegDevN {  // one contiguous range [0, *n) whose length lives on the device
    const int32_t *n;
    __device__ int64_t beg(int) const { return 0; }
    __device__ int64_t end(int) const { return *n; }
};
struct SegN {  // one contiguous range [0, n)
    int64_t n;
    __device__ int64_t beg(int) const { return 0; }
    __device__ int64_t end(int) const { return n; }
};

constexpr int LB_ITEMS = LB_TILE / BLOCK;
static_assert(LB_ITEMS * BLOCK == LB_TILE, "scan tile must be a multiple of the block");
constexpr int LB_SPIN = 1 << 16;     // polls before a look-back stops waiting

struct ScanDev {
    uint64_t *status;
    uint32_t *counter;
    int32_t *err;
    uint32_t base, epoch, grid;
    int32_t tiles;                   // per segment
};

template <typename T> struct LbHalves;
template <> struct LbHalves<uint32_t> { static constexpr int N = 1; };
template <> struct LbHalves<uint64_t> { static constexpr int N = 2; };

template <typename T>
__device__ __forceinline__ void lb_publish(uint64_t *w, uint32_t epoch, T v)
{
#pragma unroll
    for (int c = 0; c < LbHalves<T>::N; ++c)
        __hip_atomic_store(w + c, ((uint64_t)epoch << 32) | (uint32_t)((uint64_t)v >> (32 * c)),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Reads one half-set of words: true when every half carries this epoch.
template <typename T>
__device__ __forceinline__ bool lb_read(const uint64_t *w, uint32_t epoch, T &v)
{
    bool ok = true;
    uint64_t acc = 0;
#pragma unroll
    for (int c = 0; c < LbHalves<T>::N; ++c) {
        const uint64_t x = __hip_atomic_load(w + c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = ok && (uint32_t)(x >> 32) == epoch;
        acc |= (uint64_t)(uint32_t)x << (32 * c);
    }
    v = (T)acc;
    return ok;
}

// The look-back of tile `id`, the x-th tile of its segment, whose own sum is
// `total`: publishes the sum, adds the sums published by earlier tiles of the
// segment until it meets an inclusive prefix, then publishes its own inclusive
// prefix.  Returns the exclusive prefix.  Called by the 64 lanes of one wave.
template <typename T>
__device__ T lb_lookback(const ScanDev &d, uint32_t id, int x, T total)
{
    const int lane = lane_id();
    uint64_t *st = d.status + (int64_t)id * LB_WORDS;
    T prefix = 0;
    if (x == 0) {
        if (lane == 0) lb_publish(st + 2, d.epoch, total);
        return prefix;
    }
    if (lane == 0) lb_publish(st, d.epoch, total);
    const int64_t first = (int64_t)id - x;  // the segment's first tile
    int64_t t = (int64_t)id - 1 - lane;
    int spins = 0;
    while (true) {
        T pv = 0;
        int state = 2;  // lanes before the segment act as a zero inclusive prefix
        if (t >= first) {
            const uint64_t *w = d.status + t * LB_WORDS;
            state = lb_read(w + 2, d.epoch, pv) ? 2 : (lb_read(w, d.epoch, pv) ? 1 : 0);
        }
        const uint64_t incl = __ballot(state == 2);
        const int stop = incl ? __ffsll((unsigned long long)incl) - 1 : WAVE;
        const uint64_t need = stop >= WAVE - 1 ? ~0ull : ((2ull << stop) - 1ull);
        if (__ballot(state == 0) & need) {
            if (++spins <= LB_SPIN) {
                __builtin_amdgcn_s_sleep(1);
                continue;
            }
            if (lane == 0) atomicOr(d.err, ERR_PLAN);  // counted as zero; result flagged wrong
        }
        prefix += wave_sum(lane <= stop && state != 0 ? pv : T(0));
        if (stop < WAVE) break;
        t -= WAVE;
    }
    if (lane == 0) lb_publish(st + 2, d.epoch, prefix + total);
    return prefix;
}

template <class Seg, class Val, class Out, typename T>
__global__ void __launch_bounds__(BLOCK) k_scan_lookback(Seg seg, Val val, Out out, ScanDev d)
{
    __shared__ T lds[BLOCK / WAVE];
    __shared__ T prefix_s;
    __shared__ uint32_t id_s;
    if (threadIdx.x == 0) id_s = atomicAdd(d.counter, 1u) - d.base;
    __syncthreads();
    const uint32_t id = id_s;
    if (id >= d.grid) {  // the counter and the host disagree: give up loudly
        if (threadIdx.x == 0) atomicOr(d.err, ERR_PLAN);
        return;
    }
    const int y = (int)(id / (uint32_t)d.tiles), x = (int)(id % (uint32_t)d.tiles);
    const int64_t beg = seg.beg(y), end = seg.end(y);
    const int64_t tbase = beg + (int64_t)x * LB_TILE;
    if (tbase >= end) return;  // whole tile past the segment: no later tile of it needs us
    const int64_t i0 = tbase + (int64_t)threadIdx.x * LB_ITEMS;
    T v[LB_ITEMS];
    T sum = 0;
    // values are read at an index clamped into the segment and masked after:
    // with no branch around them, every item's loads are in flight together
    // (val must be branch-free and have no side effects)
#pragma unroll
    for (int q = 0; q < LB_ITEMS; ++q) {
        const int64_t i = i0 + q;
        const T x = val(i < end ? i : end - 1, y);
        v[q] = i < end ? x : T(0);
        sum += v[q];
    }
    T total;
    const T excl = block_excl_scan(sum, lds, total);
    if (threadIdx.x < WAVE) {
        const T prefix = lb_lookback(d, id, x, total);
        if (threadIdx.x == 0) prefix_s = prefix;
    }
    __syncthreads();
    T run = prefix_s + excl;
#pragma unroll
    for (int q = 0; q < LB_ITEMS; ++q) {
        if (i0 + q < end) out(i0 + q, run, v[q], y);
        run += v[q];
    }
}

// Launch the scan on stream s, which must be the only stream using ws.
template <typename T, class Seg, class Val, class Out>
inline void seg_scan(Seg seg, int nseg, int64_t max_len, Val val, Out out, ScanWs &ws,
                     hipStream_t s)
{
    if (nseg <= 0 || max_len <= 0) return;
    const int64_t tiles = (max_len + LB_TILE - 1) / LB_TILE;
    const int64_t grid = tiles * nseg;
    if (grid > ws.max_tiles) {
        ws.overflow = true;
        return;
    }
    if (ws.epoch == 0xFFFFFFFFu) {  // epochs wrapped: forget every published word
        (void)hipMemsetAsync(ws.status, 0, sizeof(uint64_t) * LB_WORDS * ws.max_tiles, s);
        ws.epoch = 0;
    }
    ScanDev d{ws.status, ws.counter, ws.err, ws.issued, ++ws.epoch, (uint32_t)grid, (int32_t)tiles};
    ws.issued += (uint32_t)grid;
    hipLaunchKernelGGL((k_scan_lookback<Seg, Val, Out, T>), dim3((unsigned)grid), dim3(BLOCK), 0,
                       s, seg, val, out, d);
}

// ---------------------------------------------------------------- radix sort in LDS
//
// Stable LSD radix sort of n entries (n <= NT * ITEMS) held in LDS, by bits
// [lo, lo + bits) of the entry, 8-bit digits, by a block of NT threads.  a
// holds the input and b is scratch of the same size; the return value is the
// buffer that holds the result.  Wave w ranks its own contiguous share of the
// entries, 64 at a time in input order: lanes with the same digit find each
// other with one ballot per digit bit, and the lowest of them advances the
// wave's running count of that digit, wc[w][d].  One block scan over the digit
// totals then gives every (wave, digit) its first output index, so a digit's
// entries land in wave order and, within a wave, in input order: the pass is
// stable with five barriers whatever n is.  wc is [NT / WAVE][256] and lds
// [NT / WAVE]; every thread must call it.
template <int NT, int ITEMS, typename E>
__device__ E *lds_radix_sort(E *a, E *b, int n, int lo, int bits, uint32_t (*wc)[256],
                             uint32_t *lds)
{
    constexpr int NW = NT / WAVE;
    static_assert(ITEMS * WAVE <= 65536, "ranks within a wave take 16 bits");
    const int tid = threadIdx.x, w = wave_id(), lane = lane_id();
    const uint64_t lt = lanemask_lt();
    const int per = ((n + NW - 1) / NW + WAVE - 1) / WAVE * WAVE;  // entries per wave
    const int i0 = w * per;
    for (int shift = lo; shift < lo + bits; shift += 8) {
        const int dbits = lo + bits - shift < 8 ? lo + bits - shift : 8;
        const uint32_t dmask = (1u << dbits) - 1u;
        for (int i = tid; i < NW * 256; i += NT) (&wc[0][0])[i] = 0;
        __syncthreads();
        uint32_t rk[ITEMS];  // digit << 16 | rank of the entry among the wave's entries
#pragma unroll
        for (int g = 0; g < ITEMS; ++g) {
            rk[g] = 0;
            if (g * WAVE >= per) break;  // uniform over the wave
            const int i = i0 + g * WAVE + lane;
            const bool valid = i < n;
            const uint32_t d = valid ? (uint32_t)(a[i] >> shift) & dmask : 0u;
            uint64_t peers = __ballot(valid);
            for (int q = 0; q < dbits; ++q) {
                const uint32_t bit = (d >> q) & 1u;
                const uint64_t bb = __ballot(bit);
                peers &= bit ? bb : ~bb;
            }
            const int leader = valid ? __ffsll((unsigned long long)peers) - 1 : lane;
            uint32_t before = 0;
            if (valid && leader == lane) {
                before = wc[w][d];
                wc[w][d] = before + (uint32_t)__popcll(peers);
            }
            before = __shfl(before, leader, WAVE);
            rk[g] = d << 16 | (before + (uint32_t)__popcll(peers & lt));
        }
        __syncthreads();
        uint32_t cnt = 0;
        if (tid < 256)
            for (int q = 0; q < NW; ++q) cnt += wc[q][tid];
        uint32_t tot;
        const uint32_t ex = block_excl_scan_n<NT>(cnt, lds, tot);
        if (tid < 256) {
            uint32_t run = ex;
            for (int q = 0; q < NW; ++q) {
                const uint32_t c = wc[q][tid];
                wc[q][tid] = run;
                run += c;
            }
        }
        __syncthreads();
#pragma unroll
        for (int g = 0; g < ITEMS; ++g) {
            if (g * WAVE >= per) break;
            const int i = i0 + g * WAVE + lane;
            if (i < n) {
                uint32_t p = wc[w][rk[g] >> 16] + (rk[g] & 0xFFFFu);
                p = p < (uint32_t)n ? p : (uint32_t)(n - 1);  // never write past the buffer
                b[p] = a[i];
            }
        }
        __syncthreads();
        E *t = a;
        a = b;
        b = t;
    }
    return a;
}

// ---------------------------------------------------------------- Hit-Map hash
//
// Open addressing with linear probing over 64-bit entries (key << 32 | slot).
// Keys are (table << row_bits | row) < 2^31.  EMPTY ends a probe; TOMB marks an
// erased entry that probes skip and inserts may reuse.

constexpr uint32_t KEY_EMPTY = 0xFFFFFFFFu;
constexpr uint32_t KEY_TOMB = 0xFFFFFFFEu;
constexpr uint64_t ENTRY_EMPTY = ~0ull;

__device__ __forceinline__ uint32_t hash_key(uint32_t k)
{
    // murmur3 32-bit finaliser
    k ^= k >> 16;
    k *= 0x85ebca6bu;
    k ^= k >> 13;
    k *= 0xc2b2ae35u;
    k ^= k >> 16;
    return k;
}

__device__ __forceinline__ uint64_t load_entry(const uint64_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Returns the slot of key, or -1, in a kernel during which nothing modifies
// the map (plain loads, served by the caches).
__device__ __forceinline__ int32_t hash_find_ro(const uint64_t *__restrict__ tab, uint32_t mask,
                                                uint32_t key)
{
    uint32_t pos = hash_key(key) & mask;
    for (uint32_t n = 0; n <= mask; ++n) {
        const uint64_t e = tab[pos];
        const uint32_t k = (uint32_t)(e >> 32);
        if (k == key) return (int32_t)(uint32_t)e;
        if (k == KEY_EMPTY) return -1;
        pos = (pos + 1) & mask;
    }
    return -1;
}

// Marks key's entry erased.  Returns false if the key was absent.
__device__ __forceinline__ bool hash_erase(uint64_t *tab, uint32_t mask, uint32_t key)
{
    uint32_t pos = hash_key(key) & mask;
    for (uint32_t n = 0; n <= mask; ++n) {
        uint64_t e = load_entry(tab + pos);
        uint32_t k = (uint32_t)(e >> 32);
        if (k == key) {
            atomicExch((unsigned long long *)(tab + pos),
                       (unsigned long long)(((uint64_t)KEY_TOMB << 32) | 0xFFFFFFFFull));
            return true;
        }
        if (k == KEY_EMPTY) return false;
        pos = (pos + 1) & mask;
    }
    return false;
}

// Inserts a key known to be absent.  Returns false if no free entry was found.
__device__ __forceinline__ bool hash_insert(uint64_t *tab, uint32_t mask, uint32_t key,
                                            int32_t slot)
{
    const uint64_t want = ((uint64_t)key << 32) | (uint32_t)slot;
    uint32_t pos = hash_key(key) & mask;
    for (uint32_t n = 0; n <= mask + 64; ++n) {
        uint64_t e = load_entry(tab + pos);
        uint32_t k = (uint32_t)(e >> 32);
        if (k == KEY_EMPTY || k == KEY_TOMB) {
            if (atomicCAS((unsigned long long *)(tab + pos), (unsigned long long)e,
                          (unsigned long long)want) == (unsigned long long)e)
                return true;
            continue;  // lost the race for this entry: look at it again
        }
        pos = (pos + 1) & mask;
    }
    return false;
}

}  // namespace sp
