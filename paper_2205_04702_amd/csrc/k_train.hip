// Data movement and training kernels over the scratchpad Storage.
//
// Row layout: Storage is fp32 [slots][D] in HBM; a row is D/4 float4 words
// and LPR = D/4 lanes cover one row, so one wave64 touches 64/LPR rows per
// pass with fully coalesced 16-byte loads.
#include <hip/hip_ext.h>

#include "sp_device.h"
#include "sp_internal.h"

namespace sp {

struct HostRows {
    const float4 *p[MAX_TABLES];  // device-visible pointers to the pinned host tables
};

// Loads and stores that do not keep the line in the caches: the update reads
// and writes each Storage row once, and streamed rows would otherwise evict
// the bag gradients it reads again for every chunk that uses them.
typedef float nv4f __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 nt_load(const float4 *p)
{
    const nv4f v = __builtin_nontemporal_load(reinterpret_cast<const nv4f *>(p));
    return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void nt_store(float4 *p, float4 x)
{
    nv4f v;
    v.x = x.x;
    v.y = x.y;
    v.z = x.z;
    v.w = x.w;
    __builtin_nontemporal_store(v, reinterpret_cast<nv4f *>(p));
}

__device__ __forceinline__ float4 f4_add(float4 a, float4 b)
{
    return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

__device__ __forceinline__ float4 f4_xor(float4 a, int o)
{
    return make_float4(__shfl_xor(a.x, o, WAVE), __shfl_xor(a.y, o, WAVE), __shfl_xor(a.z, o, WAVE),
                       __shfl_xor(a.w, o, WAVE));
}

// Sum the per-subgroup partial rows of a wave (lane groups of LPR lanes).
template <int LPR>
__device__ __forceinline__ float4 reduce_rows(float4 acc)
{
#pragma unroll
    for (int o = LPR; o < WAVE; o <<= 1) acc = f4_add(acc, f4_xor(acc, o));
    return acc;
}

// Sum of the rows src[idx[k]] for k in [beg, end), one wave, idx read 64 at a
// time (coalesced) and broadcast by shuffles; each lane group takes every
// RPP-th row in order and UNROLL rows are in flight per lane.
template <int LPR, int UNROLL>
__device__ __forceinline__ float4 gather_sum(const float4 *__restrict__ src, int64_t nrows,
                                             const int32_t *__restrict__ idx, int64_t beg,
                                             int64_t end)
{
    constexpr int RPP = WAVE / LPR;
    const int lane = lane_id(), sub = lane / LPR, c = lane % LPR;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int64_t base = beg; base < end; base += WAVE) {
        const int n = (int)((end - base) < WAVE ? (end - base) : WAVE);
        const int32_t my = lane < n ? idx[base + lane] : 0;
        for (int k0 = 0; k0 < n; k0 += RPP * UNROLL) {
            float4 v[UNROLL];
#pragma unroll
            for (int q = 0; q < UNROLL; ++q) {
                const int k = k0 + q * RPP + sub;
                int32_t r = __shfl(my, k < n ? k : 0, WAVE);
                r = (uint32_t)r < (uint64_t)nrows ? r : 0;  // never leave the array
                v[q] = k < n ? src[(int64_t)r * LPR + c] : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
            for (int q = 0; q < UNROLL; ++q) acc = f4_add(acc, v[q]);
        }
    }
    return acc;
}

// ---------------------------------------------------------------- forward

// out[g] = sum of Storage[slot_of[j]] over the positions j of bag g
// (Sec. II-B, gather then element-wise reduction per table).  One wave per bag.
template <int LPR>
__global__ void __launch_bounds__(BLOCK) k_forward(const float4 *__restrict__ storage,
                                                   const int32_t *__restrict__ slot_of,
                                                   const int32_t *__restrict__ bag_off,
                                                   int64_t nbags, int64_t nslots,
                                                   float4 *__restrict__ out)
{
    // consecutive bags (one table's) on one XCD: the table's hot rows share its L2
    const int64_t g = xcd_block(blockIdx.x, gridDim.x) * (BLOCK / WAVE) + wave_id();
    if (g >= nbags) return;
    // at least 8 rows in flight per wave (a wave covers 64/LPR rows per load)
    constexpr int UNROLL = LPR >= 32 ? 8 : 4;
    float4 acc = gather_sum<LPR, UNROLL>(storage, nslots, slot_of, bag_off[g], bag_off[g + 1]);
    acc = reduce_rows<LPR>(acc);
    const int lane = lane_id();
    if (lane < LPR) out[g * LPR + lane] = acc;
}

// ---------------------------------------------------------------- backward + SGD

__device__ __forceinline__ float4 sgd_step(float4 x, float4 g, float lr)
{
    x.x = fmaf(-lr, g.x, x.x);
    x.y = fmaf(-lr, g.y, x.y);
    x.z = fmaf(-lr, g.z, x.z);
    x.w = fmaf(-lr, g.w, x.w);
    return x;
}


// Gradient coalescing and SGD (Sec. II-B "Backpropagation").  The sorted
// positions of one batch form runs of equal keys; each run is cut into chunks
// of at most `chunk` positions.  One group of G = LPR / VPL lanes takes one
// chunk, each lane VPL of the row's LPR 16-byte words (word j * G + c for lane
// c), so a wave works on 64 / G chunks at once and each lane keeps VPL loads
// of every row in flight: more rows per memory round trip than one word per
// lane would give, which is what bounds this kernel (each chunk is a short
// chain of dependent loads: descriptor, then slot and bag indices, then the
// Storage row and gradient rows).  It sums the gradient rows of the bags at
// its positions in ascending position order.
//  * a run of one chunk updates its Storage row directly: W -= lr * g;
//  * a longer run stores per-chunk partial sums, which k_bwd_combine adds in
//    chunk order before updating the row (the kernel boundary orders the two).
constexpr int BWD_INFLIGHT = 8;  // gradient words in flight per lane (rows x VPL)

// Words per lane for rows of LPR words (the launch's grid follows it): two
// from rows of 64 floats up.  Measured alone on the 26x10M workload's update
// (128 floats): 0.80 ms with one word per lane, 0.69 ms with four (fewer
// waves fit: 97 registers), 0.63 ms with two (71 registers, 7 waves per SIMD).
constexpr int bwd_vpl(int lpr) { return lpr >= 16 ? 2 : 1; }

template <int LPR>
__global__ void __launch_bounds__(BLOCK) k_backward(float4 *__restrict__ storage,
                                                    const int4 *__restrict__ chunk_desc,
                                                    const int32_t *__restrict__ sbag,
                                                    const int32_t *__restrict__ slot_u,
                                                    int64_t n_chunks,
                                                    const float4 *__restrict__ grad,
                                                    int64_t nbags, int64_t nslots, float lr,
                                                    float4 *__restrict__ partial)
{
    constexpr int VPL = bwd_vpl(LPR);
    constexpr int G = LPR / VPL;                // lanes per chunk
    constexpr int INFL = BWD_INFLIGHT / VPL;    // gradient rows in flight per lane
    // consecutive chunks (one table's) on one XCD: the table's bag gradients
    // share its L2
    const int64_t t = xcd_block(blockIdx.x, gridDim.x) * BLOCK + threadIdx.x;
    const int64_t ch = t / G;
    const int c = (int)(t % G);
    if (ch >= n_chunks) return;  // whole lane groups leave together
    const int4 d = chunk_desc[ch];  // first position, end position, run, chunks of the run
    const int64_t p0 = d.x, p1 = d.y;
    const int32_t slot = slot_u[d.z];
    const int64_t nch = d.w;
    // a one-chunk run reads its Storage row beside its gradient rows rather
    // than after them: one memory round trip less on the lane's path
    const bool direct = nch == 1 && (uint32_t)slot < (uint64_t)nslots;
    float4 *const w = storage + (direct ? (int64_t)slot * LPR + c : 0);
    float4 w0[VPL];
#pragma unroll
    for (int j = 0; j < VPL; ++j) w0[j] = direct ? nt_load(w + j * G) : make_float4(0.f, 0.f, 0.f, 0.f);
    // A chunk's bag indices arrive in one coalesced load (lane c of the group
    // holds positions c, c+G, ...) and are broadcast by shuffles, so its
    // gradient rows are requested INFL at a time without waiting on further
    // index loads.  Sums stay in position order.
    constexpr int PER_LANE = BWD_CHUNK / G > 0 ? BWD_CHUNK / G : 1;
    const int gbase = lane_id() - c;
    // 32-bit byte offsets from the uniform base (the gradient array is far
    // below 4 GiB): one address register per load in flight
    const char *__restrict__ gbytes = reinterpret_cast<const char *>(grad);
    float4 acc[VPL];
#pragma unroll
    for (int j = 0; j < VPL; ++j) acc[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int64_t base = p0; base < p1; base += BWD_CHUNK) {
        const int n = (int)(p1 - base < BWD_CHUNK ? p1 - base : BWD_CHUNK);
        int32_t mine[PER_LANE];
#pragma unroll
        for (int l = 0; l < PER_LANE; ++l) {
            const int k = l * G + c;
            const int32_t b = k < n ? sbag[base + k] : 0;
            mine[l] = (uint32_t)b < (uint64_t)nbags ? b : 0;
        }
#pragma unroll
        for (int k0 = 0; k0 < BWD_CHUNK; k0 += INFL) {
            if (k0 >= n) break;  // uniform within the lane group
            float4 v[INFL][VPL];
#pragma unroll
            for (int q = 0; q < INFL; ++q) {
                const int k = k0 + q;
                // every lane of the group takes part in the shuffle; only the load is predicated
                const int32_t b = __shfl(mine[k / G], gbase + k % G, WAVE);
                const uint32_t off = (uint32_t)b * (uint32_t)(LPR * 16) + (uint32_t)c * 16u;
#pragma unroll
                for (int j = 0; j < VPL; ++j)
                    v[q][j] = k < n ? *reinterpret_cast<const float4 *>(gbytes + off + j * G * 16)
                                    : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
            for (int q = 0; q < INFL; ++q)
#pragma unroll
                for (int j = 0; j < VPL; ++j) acc[j] = f4_add(acc[j], v[q][j]);
        }
    }
    if (nch > 1) {
#pragma unroll
        for (int j = 0; j < VPL; ++j) partial[ch * LPR + j * G + c] = acc[j];
    } else if (direct) {
#pragma unroll
        for (int j = 0; j < VPL; ++j) nt_store(w + j * G, sgd_step(w0[j], acc[j], lr));
    }
}

// Runs longer than one chunk (listed in `multi`, any order), one block per
// run: the block's G lane groups add the run's chunk partials in a fixed
// strided order (group g takes chunks g, g+G, ...), four loads in flight per
// lane; group 0 then adds the G group sums in order and updates the row.
template <int LPR>
__global__ void __launch_bounds__(BLOCK) k_bwd_combine(float4 *__restrict__ storage,
                                                       const int32_t *__restrict__ multi,
                                                       int64_t n_multi,
                                                       const int32_t *__restrict__ seg_chunk0,
                                                       const int4 *__restrict__ chunk_desc,
                                                       const int32_t *__restrict__ slot_u,
                                                       const float4 *__restrict__ partial,
                                                       int64_t nslots, float lr)
{
    constexpr int G = BLOCK / LPR;
    __shared__ float4 red[G][LPR];
    const int64_t m = blockIdx.x;
    if (m >= n_multi) return;  // uniform per block
    const int g = threadIdx.x / LPR, c = threadIdx.x % LPR;
    const int32_t s = multi[m];
    const int64_t c0 = seg_chunk0[s];
    const int64_t nch = chunk_desc[c0].w;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    int64_t q = g;
    for (; q + 3 * G < nch; q += 4 * G) {
        float4 v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = partial[(c0 + q + k * G) * LPR + c];
#pragma unroll
        for (int k = 0; k < 4; ++k) acc = f4_add(acc, v[k]);
    }
    for (; q < nch; q += G) acc = f4_add(acc, partial[(c0 + q) * LPR + c]);
    red[g][c] = acc;
    __syncthreads();
    if (g != 0) return;
    float4 sum = red[0][c];
    for (int k = 1; k < G; ++k) sum = f4_add(sum, red[k][c]);
    const int32_t slot = slot_u[s];
    if ((uint32_t)slot < (uint64_t)nslots) {
        float4 *const w = storage + (int64_t)slot * LPR + c;
        nt_store(w, sgd_step(nt_load(w), sum, lr));
    }
}

// ---------------------------------------------------------------- evict / fill

// Victim i: copy the row its slot held (if any) to staging row i for the
// write-back, then fill the slot with the missing row m_key[i]: read straight
// from the pinned host table (zero-copy over the host link), or, with the
// staged fill, from row i of the rows already copied to the device.  The same
// lanes read the old row before writing the new one.  Every victim's previous
// key is stored after the n staging rows, so rows and keys leave the device
// in one copy.  For the zero-copy fill the grid is kept small and each lane
// group keeps MOVE_ROWS victims in flight: waves waiting on the host link
// then occupy few compute units, and the kernels running beside this one
// keep the rest.  The staged fill only moves rows within HBM and takes a
// full grid.
// Every row the move reads or writes is touched once, so none of its accesses
// keeps the line in the caches: cached stores of a large fill left the caches
// full of dirty lines, whose write-back then slowed the forward that follows
// (26x10M forward 0.350 ms after a cached fill, 0.317 ms after this one).
__device__ __forceinline__ nv4f nt_row(const float4 *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const nv4f *>(p));
}
__device__ __forceinline__ void nt_row_store(float4 *p, nv4f x)
{
    __builtin_nontemporal_store(x, reinterpret_cast<nv4f *>(p));
}

constexpr int MOVE_MAX_BLOCKS = 64;
constexpr int MOVE_ROWS = 4;

template <int LPR>
__global__ void __launch_bounds__(BLOCK) k_move(float4 *__restrict__ storage, Tables tb,
                                                HostRows hr, TicketDev tk, int64_t n,
                                                int64_t nslots, float4 *__restrict__ stage,
                                                const float4 *__restrict__ staged)
{
    const int c = (int)(threadIdx.x % LPR);
    const int64_t groups = (int64_t)gridDim.x * (BLOCK / LPR);
    const int64_t g = ((int64_t)blockIdx.x * BLOCK + threadIdx.x) / LPR;
    const uint32_t row_mask = (1u << tb.row_bits) - 1u;
    int32_t *const old_keys = reinterpret_cast<int32_t *>(stage + n * LPR);
    for (int64_t i0 = g; i0 < n; i0 += groups * MOVE_ROWS) {
        // Straight-line code over the pass's MOVE_ROWS victims, with no branch
        // around a load: an entry past n reads entry i0's indices, and one
        // with nothing to read reads row 0 of the scratchpad and drops it.
        // Each round of loads is then in flight together and the values stay
        // in registers until the stores.
        bool in[MOVE_ROWS];
        int32_t old[MOVE_ROWS], v[MOVE_ROWS];
        uint32_t key[MOVE_ROWS];
#pragma unroll
        for (int q = 0; q < MOVE_ROWS; ++q) {
            const int64_t i = i0 + q * groups;
            in[q] = i < n;
            const int64_t ic = in[q] ? i : i0;
            old[q] = tk.v_old_key[ic];
            v[q] = tk.v_slot[ic];
            key[q] = tk.m_key[ic];
        }
        const float4 *src[MOVE_ROWS];
        if (staged) {
#pragma unroll
            for (int q = 0; q < MOVE_ROWS; ++q) src[q] = staged + (i0 + q * groups) * LPR + c;
        } else {
            int tab[MOVE_ROWS];
            int64_t nrows[MOVE_ROWS];
            const float4 *base[MOVE_ROWS];
#pragma unroll
            for (int q = 0; q < MOVE_ROWS; ++q) {
                tab[q] = (int)(key[q] >> tb.row_bits);
                const int tc = tab[q] < tb.T ? tab[q] : 0;
                nrows[q] = tb.rows[tc];
                base[q] = hr.p[tc];
            }
#pragma unroll
            for (int q = 0; q < MOVE_ROWS; ++q) {
                const int64_t row = key[q] & row_mask;
                src[q] = tab[q] < tb.T && row < nrows[q] ? base[q] + row * LPR + c : nullptr;
            }
        }
#pragma unroll
        for (int q = 0; q < MOVE_ROWS; ++q) {
            if (!in[q] || (uint32_t)v[q] >= (uint64_t)nslots) v[q] = -1;
            if (v[q] < 0) src[q] = nullptr;
        }
        nv4f prev[MOVE_ROWS], next[MOVE_ROWS];
#pragma unroll
        for (int q = 0; q < MOVE_ROWS; ++q) {
            prev[q] = nt_row(storage + (v[q] >= 0 && old[q] >= 0 ? (int64_t)v[q] * LPR : 0) + c);
            next[q] = nt_row(src[q] ? src[q] : storage + c);
        }
#pragma unroll
        for (int q = 0; q < MOVE_ROWS; ++q) {
            const int64_t i = i0 + q * groups;
            if (in[q] && c == 0) old_keys[i] = old[q];
            if (v[q] >= 0 && old[q] >= 0) nt_row_store(stage + i * LPR + c, prev[q]);
            if (src[q]) nt_row_store(storage + (int64_t)v[q] * LPR + c, next[q]);
        }
    }
}

// ---------------------------------------------------------------- fixed scratch

// Partial sums of split runs for callers that cannot allocate: a fixed array
// per GPU, held until the process ends.  Host code never uses its name as an
// address; it takes the address hipGetSymbolAddress gives on each device.
static __device__ __align__(256) float4 scratch[STATIC_PARTIAL_BYTES / sizeof(float4)];

hipError_t static_partial_address(void **ptr)
{
    return hipGetSymbolAddress(ptr, HIP_SYMBOL(scratch));
}

// ---------------------------------------------------------------- dispatch

#define SP_DISPATCH_LPR(D4, KERNEL, GRID, ...)                                                   \
    switch (D4) {                                                                                \
    case 1: hipLaunchKernelGGL(KERNEL<1>, GRID, dim3(BLOCK), 0, s, __VA_ARGS__); break;          \
    case 2: hipLaunchKernelGGL(KERNEL<2>, GRID, dim3(BLOCK), 0, s, __VA_ARGS__); break;          \
    case 4: hipLaunchKernelGGL(KERNEL<4>, GRID, dim3(BLOCK), 0, s, __VA_ARGS__); break;          \
    case 8: hipLaunchKernelGGL(KERNEL<8>, GRID, dim3(BLOCK), 0, s, __VA_ARGS__); break;          \
    case 16: hipLaunchKernelGGL(KERNEL<16>, GRID, dim3(BLOCK), 0, s, __VA_ARGS__); break;        \
    case 32: hipLaunchKernelGGL(KERNEL<32>, GRID, dim3(BLOCK), 0, s, __VA_ARGS__); break;        \
    default: hipLaunchKernelGGL(KERNEL<64>, GRID, dim3(BLOCK), 0, s, __VA_ARGS__); break;        \
    }

static dim3 grid_rows(int64_t n, int D4)
{
    int64_t threads = n * D4;
    return dim3((unsigned)((threads + BLOCK - 1) / BLOCK));
}

static dim3 grid_waves(int64_t n)
{
    return dim3((unsigned)((n + BLOCK / WAVE - 1) / (BLOCK / WAVE)));
}

void launch_move(float *storage, int dim, const Tables &tb, float *const *host_dev, TicketDev tk,
                 int64_t n_miss, int32_t u, float *stage, const float *staged, hipStream_t s)
{
    if (n_miss <= 0) return;
    const int D4 = dim / 4;
    HostRows hr{};
    for (int t = 0; t < tb.T; ++t) hr.p[t] = (const float4 *)host_dev[t];
    // each lane group places MOVE_ROWS victims per pass
    dim3 grid = grid_rows((n_miss + MOVE_ROWS - 1) / MOVE_ROWS, D4);
    if (!staged) grid.x = grid.x < (unsigned)MOVE_MAX_BLOCKS ? grid.x : (unsigned)MOVE_MAX_BLOCKS;
    SP_DISPATCH_LPR(D4, k_move, grid, (float4 *)storage, tb, hr, tk, n_miss,
                    tb.slot_base[tb.T], (float4 *)stage, (const float4 *)staged);
}

// Launches that may carry start/stop events: the events then time the kernel's
// own execution on stream s (null events = plain launch).
#define SP_DISPATCH_LPR_EV(D4, KERNEL, GRID, E0, E1, ...)                                        \
    switch (D4) {                                                                                \
    case 1: hipExtLaunchKernelGGL(KERNEL<1>, GRID, dim3(BLOCK), 0, s, E0, E1, 0, __VA_ARGS__); break;   \
    case 2: hipExtLaunchKernelGGL(KERNEL<2>, GRID, dim3(BLOCK), 0, s, E0, E1, 0, __VA_ARGS__); break;   \
    case 4: hipExtLaunchKernelGGL(KERNEL<4>, GRID, dim3(BLOCK), 0, s, E0, E1, 0, __VA_ARGS__); break;   \
    case 8: hipExtLaunchKernelGGL(KERNEL<8>, GRID, dim3(BLOCK), 0, s, E0, E1, 0, __VA_ARGS__); break;   \
    case 16: hipExtLaunchKernelGGL(KERNEL<16>, GRID, dim3(BLOCK), 0, s, E0, E1, 0, __VA_ARGS__); break; \
    case 32: hipExtLaunchKernelGGL(KERNEL<32>, GRID, dim3(BLOCK), 0, s, E0, E1, 0, __VA_ARGS__); break; \
    default: hipExtLaunchKernelGGL(KERNEL<64>, GRID, dim3(BLOCK), 0, s, E0, E1, 0, __VA_ARGS__); break; \
    }

void launch_forward(const float *storage, int dim, int64_t nslots, const int32_t *slot_of,
                    const int32_t *bag_off, int64_t nbags, float *out, hipStream_t s,
                    hipEvent_t e0, hipEvent_t e1)
{
    if (nbags <= 0) return;
    SP_DISPATCH_LPR_EV(dim / 4, k_forward, grid_waves(nbags), e0, e1, (const float4 *)storage,
                       slot_of, bag_off, nbags, nslots, (float4 *)out);
}

void launch_backward(float *storage, int dim, int64_t nslots, const BatchDev &b,
                     const int32_t *slot_u, int64_t n_chunks, int64_t n_multi, int chunk,
                     const float *grad, int64_t nbags, float lr, float *partial, hipStream_t s,
                     hipEvent_t ev[4])
{
    if (n_chunks <= 0) return;
    const int D4 = dim / 4;
    (void)chunk;
    // one lane group of D4 / VPL lanes per chunk
    SP_DISPATCH_LPR_EV(D4, k_backward, grid_rows(n_chunks, D4 / bwd_vpl(D4)), ev[0], ev[1],
                       (float4 *)storage,
                       (const int4 *)b.chunk_desc, (const int32_t *)b.sbag, slot_u, n_chunks,
                       (const float4 *)grad, nbags, nslots, lr, (float4 *)partial);
    if (n_multi > 0)
        SP_DISPATCH_LPR_EV(D4, k_bwd_combine, dim3((unsigned)n_multi), ev[2], ev[3],
                           (float4 *)storage, (const int32_t *)b.multi, n_multi,
                           (const int32_t *)b.seg_chunk0, (const int4 *)b.chunk_desc, slot_u,
                           (const float4 *)partial, nslots, lr);
}

}  // namespace sp
