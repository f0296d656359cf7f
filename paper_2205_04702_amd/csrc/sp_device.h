// Device-side building blocks shared by the scratchpad kernels (CDNA4, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sp {

constexpr int WAVE = 64;
constexpr int BLOCK = 256;                 // 4 waves
constexpr int SCAN_ITEMS = 8;
constexpr int SCAN_TILE = BLOCK * SCAN_ITEMS;

__device__ __forceinline__ int lane_id() { return threadIdx.x & (WAVE - 1); }
__device__ __forceinline__ int wave_id() { return threadIdx.x / WAVE; }
__device__ __forceinline__ uint64_t lanemask_lt() { return (1ull << lane_id()) - 1ull; }

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

template <typename T>
__device__ __forceinline__ T block_sum(T v, T *lds)
{
    T total;
    (void)block_excl_scan(v, lds, total);
    return total;
}

// ---------------------------------------------------------------- segmented scan
//
// A segmented exclusive scan over index ranges.  Segment y covers
// [seg.beg(y), seg.end(y)); blockIdx.y selects the segment, blockIdx.x a tile
// of SCAN_TILE consecutive indices.  Three launches: tile sums, per-segment
// scan of tile sums (one block per segment), then per-index exclusive prefixes
// handed to out(i, prefix, value, y) in index order.  Values come from
// val(i, y).

template <class Seg, class Val, typename T>
__global__ void __launch_bounds__(BLOCK) k_seg_tile_sums(Seg seg, Val val, T *tile_sums,
                                                         int tiles)
{
    __shared__ T lds[BLOCK / WAVE];
    const int y = blockIdx.y;
    const int64_t beg = seg.beg(y), end = seg.end(y);
    const int64_t base = beg + (int64_t)blockIdx.x * SCAN_TILE;
    T acc = 0;
    for (int r = 0; r < SCAN_ITEMS; ++r) {
        int64_t i = base + (int64_t)r * BLOCK + threadIdx.x;
        if (i < end) acc += val(i, y);
    }
    T s = block_sum(acc, lds);
    if (threadIdx.x == 0) tile_sums[(int64_t)y * tiles + blockIdx.x] = s;
}

template <typename T>
__global__ void __launch_bounds__(1024) k_seg_scan_tiles(T *tile_sums, int tiles, T *totals)
{
    __shared__ T lds[1024 / WAVE];
    __shared__ T carry_s;
    T *row = tile_sums + (int64_t)blockIdx.x * tiles;
    if (threadIdx.x == 0) carry_s = 0;
    __syncthreads();
    for (int b = 0; b < tiles; b += 1024) {
        int i = b + threadIdx.x;
        T v = i < tiles ? row[i] : T(0);
        T incl = wave_incl_scan(v);
        if (lane_id() == WAVE - 1) lds[threadIdx.x / WAVE] = incl;
        __syncthreads();
        T base = 0, sum = 0;
        for (int w = 0; w < 1024 / WAVE; ++w) {
            T x = lds[w];
            if (w < (int)(threadIdx.x / WAVE)) base += x;
            sum += x;
        }
        T carry = carry_s;
        if (i < tiles) row[i] = carry + base + incl - v;
        __syncthreads();
        if (threadIdx.x == 0) carry_s = carry + sum;
        __syncthreads();
    }
    if (threadIdx.x == 0 && totals) totals[blockIdx.x] = carry_s;
}

template <class Seg, class Val, class Out, typename T>
__global__ void __launch_bounds__(BLOCK) k_seg_apply(Seg seg, Val val, Out out,
                                                     const T *tile_sums, int tiles)
{
    __shared__ T lds[BLOCK / WAVE];
    const int y = blockIdx.y;
    const int64_t beg = seg.beg(y), end = seg.end(y);
    const int64_t base = beg + (int64_t)blockIdx.x * SCAN_TILE;
    if (base >= end) return;  // uniform per block
    T carry = tile_sums[(int64_t)y * tiles + blockIdx.x];
    for (int r = 0; r < SCAN_ITEMS; ++r) {
        int64_t i = base + (int64_t)r * BLOCK + threadIdx.x;
        T v = i < end ? val(i, y) : T(0);
        T total;
        T e = block_excl_scan(v, lds, total);
        if (i < end) out(i, carry + e, v, y);
        carry += total;
    }
}

// One contiguous range [0, *n) whose length lives on the device.
struct SegDevN {
    const int32_t *n;
    __device__ int64_t beg(int) const { return 0; }
    __device__ int64_t end(int) const { return *n; }
};
// One contiguous range [0, n).
struct SegN {
    int64_t n;
    __device__ int64_t beg(int) const { return 0; }
    __device__ int64_t end(int) const { return n; }
};

// Small segments: one 1024-thread block per segment, each thread scanning
// SS_ITEMS consecutive values in registers, block-wide scan of the thread sums.
constexpr int SS_THREADS = 1024;
constexpr int SS_ITEMS = 16;
constexpr int64_t SMALL_SCAN = (int64_t)SS_THREADS * SS_ITEMS * 8;

template <class Seg, class Val, class Out, typename T>
__global__ void __launch_bounds__(SS_THREADS) k_scan_single(Seg seg, Val val, Out out)
{
    __shared__ T lds[SS_THREADS / WAVE];
    __shared__ T carry_s;
    const int y = blockIdx.x;
    const int64_t beg = seg.beg(y), end = seg.end(y);
    if (threadIdx.x == 0) carry_s = 0;
    __syncthreads();
    for (int64_t base = beg; base < end; base += (int64_t)SS_THREADS * SS_ITEMS) {
        const int64_t i0 = base + (int64_t)threadIdx.x * SS_ITEMS;
        T v[SS_ITEMS];
        T sum = 0;
#pragma unroll
        for (int q = 0; q < SS_ITEMS; ++q) {
            const int64_t i = i0 + q;
            v[q] = i < end ? val(i, y) : T(0);
            sum += v[q];
        }
        const T incl = wave_incl_scan(sum);
        if (lane_id() == WAVE - 1) lds[threadIdx.x / WAVE] = incl;
        __syncthreads();
        T wbase = 0, tot = 0;
        for (int w = 0; w < SS_THREADS / WAVE; ++w) {
            const T x = lds[w];
            if (w < (int)(threadIdx.x / WAVE)) wbase += x;
            tot += x;
        }
        const T carry = carry_s;
        T run = carry + wbase + incl - sum;
#pragma unroll
        for (int q = 0; q < SS_ITEMS; ++q) {
            const int64_t i = i0 + q;
            if (i < end) out(i, run, v[q], y);
            run += v[q];
        }
        __syncthreads();
        if (threadIdx.x == 0) carry_s = carry + tot;
        __syncthreads();
    }
}

// Launch the scan.  max_len bounds every segment's length; tile_sums needs
// nseg * ceil(max_len / SCAN_TILE) entries; totals (optional) gets each
// segment's sum (multi-block path only).  With one_block, segments of at most
// SMALL_SCAN values take the one-block-per-segment path: one launch instead
// of three, worth it only when val/out are cheap (no dependent global loads).
template <class Seg, class Val, class Out, typename T>
inline void seg_scan(Seg seg, int nseg, int64_t max_len, Val val, Out out, T *tile_sums,
                     T *totals, hipStream_t s, bool one_block = false)
{
    if (nseg <= 0 || max_len <= 0) return;
    if (one_block && max_len <= SMALL_SCAN && totals == nullptr) {
        hipLaunchKernelGGL((k_scan_single<Seg, Val, Out, T>), dim3(nseg), dim3(SS_THREADS), 0, s,
                           seg, val, out);
        return;
    }
    int tiles = (int)((max_len + SCAN_TILE - 1) / SCAN_TILE);
    dim3 grid(tiles, nseg);
    hipLaunchKernelGGL((k_seg_tile_sums<Seg, Val, T>), grid, dim3(BLOCK), 0, s, seg, val,
                       tile_sums, tiles);
    hipLaunchKernelGGL((k_seg_scan_tiles<T>), dim3(nseg), dim3(1024), 0, s, tile_sums, tiles,
                       totals);
    hipLaunchKernelGGL((k_seg_apply<Seg, Val, Out, T>), grid, dim3(BLOCK), 0, s, seg, val, out,
                       (const T *)tile_sums, tiles);
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

// Returns the slot of key, or -1.
__device__ __forceinline__ int32_t hash_find(const uint64_t *tab, uint32_t mask, uint32_t key)
{
    uint32_t pos = hash_key(key) & mask;
    for (uint32_t n = 0; n <= mask; ++n) {
        uint64_t e = load_entry(tab + pos);
        uint32_t k = (uint32_t)(e >> 32);
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
