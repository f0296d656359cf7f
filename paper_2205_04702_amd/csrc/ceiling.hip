// Access-pattern ceilings for the roofline of the training kernels.
//
// The forward gathers, and the update reads and rewrites, rows of 4*D bytes
// at scattered places of the scratchpad Storage.  How fast HBM serves that
// pattern on this GPU is measured here with bare kernels that do nothing
// else, at a workload's own shape:
//   * rmw:    n distinct random rows of a [slots][D] fp32 array are each read,
//             decremented by a gradient row (one of `bags` rows) and written
//             back: 2*n*4D + bags*4D + 8n bytes;
//   * gather: the same n rows are copied to a dense [n][D] output:
//             2*n*4D + 4n bytes;
//   * copy:   a sequential copy of `copy_mib` MiB: 2*copy_mib MiB.
// Each is timed with HIP events, the best of five launches after one warm-up,
// with a 512 MiB fill before each launch so the rows come from HBM.
// Usage: ceiling <slots> <n> <dim> <bags> <copy_mib> [seed]; prints one JSON line.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <numeric>
#include <random>
#include <vector>

namespace {

constexpr int BLOCK = 256;

#define CK(x)                                                                            \
    do {                                                                                 \
        hipError_t e_ = (x);                                                             \
        if (e_ != hipSuccess) {                                                          \
            fprintf(stderr, "ceiling: %s at line %d\n", hipGetErrorString(e_), __LINE__); \
            return 1;                                                                    \
        }                                                                                \
    } while (0)

// one lane group of LPR lanes (one row) per listed row
template <int LPR>
__global__ void __launch_bounds__(BLOCK) k_rmw(float4 *__restrict__ st, const int32_t *__restrict__ slot,
                                               const int32_t *__restrict__ bag,
                                               const float4 *__restrict__ g, int64_t n, float lr)
{
    const int64_t t = (int64_t)blockIdx.x * BLOCK + threadIdx.x;
    const int64_t i = t / LPR;
    const int c = (int)(t % LPR);
    if (i >= n) return;
    const int64_t s = slot[i], b = bag[i];
    float4 w = st[s * LPR + c];
    const float4 v = g[b * LPR + c];
    w.x = fmaf(-lr, v.x, w.x);
    w.y = fmaf(-lr, v.y, w.y);
    w.z = fmaf(-lr, v.z, w.z);
    w.w = fmaf(-lr, v.w, w.w);
    st[s * LPR + c] = w;
}

template <int LPR>
__global__ void __launch_bounds__(BLOCK) k_gather(const float4 *__restrict__ st, const int32_t *__restrict__ slot,
                                                  float4 *__restrict__ out, int64_t n)
{
    const int64_t t = (int64_t)blockIdx.x * BLOCK + threadIdx.x;
    const int64_t i = t / LPR;
    const int c = (int)(t % LPR);
    if (i >= n) return;
    out[i * LPR + c] = st[(int64_t)slot[i] * LPR + c];
}

// four 16-byte loads in flight per lane, each wave touching 1 KiB per load
constexpr int COPY_UNROLL = 4;

__global__ void __launch_bounds__(BLOCK) k_copy(const float4 *__restrict__ a, float4 *__restrict__ b, int64_t n4)
{
    const int64_t stride = (int64_t)gridDim.x * BLOCK;
    int64_t t = (int64_t)blockIdx.x * BLOCK + threadIdx.x;
    for (; t + (COPY_UNROLL - 1) * stride < n4; t += COPY_UNROLL * stride) {
        float4 v[COPY_UNROLL];
#pragma unroll
        for (int q = 0; q < COPY_UNROLL; ++q) v[q] = a[t + q * stride];
#pragma unroll
        for (int q = 0; q < COPY_UNROLL; ++q) b[t + q * stride] = v[q];
    }
    for (; t < n4; t += stride) b[t] = a[t];
}

template <int LPR>
void launch_pattern(int which, float4 *st, const int32_t *slot, const int32_t *bag, const float4 *g,
                    float4 *out, int64_t n)
{
    const dim3 grid((unsigned)((n * LPR + BLOCK - 1) / BLOCK));
    if (which == 0)
        hipLaunchKernelGGL(k_rmw<LPR>, grid, dim3(BLOCK), 0, 0, st, slot, bag, g, n, 0.01f);
    else
        hipLaunchKernelGGL(k_gather<LPR>, grid, dim3(BLOCK), 0, 0, st, slot, out, n);
}

void launch_lpr(int lpr, int which, float4 *st, const int32_t *slot, const int32_t *bag, const float4 *g,
                float4 *out, int64_t n)
{
    switch (lpr) {
    case 1: launch_pattern<1>(which, st, slot, bag, g, out, n); break;
    case 2: launch_pattern<2>(which, st, slot, bag, g, out, n); break;
    case 4: launch_pattern<4>(which, st, slot, bag, g, out, n); break;
    case 8: launch_pattern<8>(which, st, slot, bag, g, out, n); break;
    case 16: launch_pattern<16>(which, st, slot, bag, g, out, n); break;
    case 32: launch_pattern<32>(which, st, slot, bag, g, out, n); break;
    default: launch_pattern<64>(which, st, slot, bag, g, out, n); break;
    }
}

}  // namespace

int main(int argc, char **argv)
{
    if (argc < 6) {
        fprintf(stderr, "usage: ceiling <slots> <n> <dim> <bags> <copy_mib> [seed]\n");
        return 2;
    }
    const int64_t slots = atoll(argv[1]), n = atoll(argv[2]), bags = atoll(argv[4]), copy_mib = atoll(argv[5]);
    const int dim = atoi(argv[3]);
    const uint64_t seed = argc > 6 ? strtoull(argv[6], nullptr, 10) : 1;
    if (slots < 1 || slots > INT32_MAX || n < 1 || n > slots || bags < 1 || bags > INT32_MAX || dim < 4 ||
        dim > 256 || (dim & (dim - 1)) != 0 || copy_mib < 1 || copy_mib > 8192) {
        fprintf(stderr, "ceiling: bad arguments\n");
        return 2;
    }
    const int lpr = dim / 4;
    // n distinct random rows, and a random gradient row for each
    std::mt19937_64 rng(seed);
    std::vector<int32_t> all((size_t)slots);
    std::iota(all.begin(), all.end(), 0);
    for (int64_t i = 0; i < n; ++i) {  // partial Fisher-Yates: the first n are a uniform sample
        const int64_t j = i + (int64_t)(rng() % (uint64_t)(slots - i));
        std::swap(all[(size_t)i], all[(size_t)j]);
    }
    std::vector<int32_t> slot(all.begin(), all.begin() + n), bag((size_t)n);
    for (auto &b : bag) b = (int32_t)(rng() % (uint64_t)bags);

    const size_t row = sizeof(float) * (size_t)dim;
    const int64_t copy4 = copy_mib * (1 << 20) / 16, flush4 = (512 << 20) / 16;
    float4 *st, *g, *out, *ca, *cb, *fl;
    int32_t *d_slot, *d_bag;
    CK(hipMalloc(&st, row * slots));
    CK(hipMalloc(&g, row * bags));
    CK(hipMalloc(&out, row * n));
    CK(hipMalloc(&ca, 16 * copy4));
    CK(hipMalloc(&cb, 16 * copy4));
    CK(hipMalloc(&fl, 16 * flush4));
    CK(hipMalloc(&d_slot, sizeof(int32_t) * n));
    CK(hipMalloc(&d_bag, sizeof(int32_t) * n));
    CK(hipMemset(st, 0, row * slots));
    CK(hipMemset(g, 0, row * bags));
    CK(hipMemset(ca, 0, 16 * copy4));
    CK(hipMemcpy(d_slot, slot.data(), sizeof(int32_t) * n, hipMemcpyHostToDevice));
    CK(hipMemcpy(d_bag, bag.data(), sizeof(int32_t) * n, hipMemcpyHostToDevice));
    hipEvent_t e0, e1;
    CK(hipEventCreate(&e0));
    CK(hipEventCreate(&e1));

    double best_ms[3] = {1e30, 1e30, 1e30};
    for (int which = 0; which < 3; ++which) {
        for (int r = 0; r < 6; ++r) {
            CK(hipMemsetAsync(fl, r, 16 * flush4, 0));
            CK(hipEventRecord(e0, 0));
            if (which < 2)
                launch_lpr(lpr, which, st, d_slot, d_bag, g, out, n);
            else
                hipLaunchKernelGGL(k_copy, dim3(8192), dim3(BLOCK), 0, 0, ca, cb, copy4);
            CK(hipGetLastError());
            CK(hipEventRecord(e1, 0));
            CK(hipEventSynchronize(e1));
            float ms = 0.f;
            CK(hipEventElapsedTime(&ms, e0, e1));
            if (r > 0) best_ms[which] = std::min(best_ms[which], (double)ms);
        }
    }
    const double bytes[3] = {2.0 * n * row + (double)bags * row + 8.0 * n, 2.0 * n * row + 4.0 * n,
                             2.0 * 16 * copy4};
    printf("{\"slots\": %lld, \"rows\": %lld, \"dim\": %d, \"bags\": %lld", (long long)slots, (long long)n, dim,
           (long long)bags);
    const char *names[3] = {"rmw", "gather", "copy"};
    for (int k = 0; k < 3; ++k)
        printf(", \"%s\": {\"bytes\": %.0f, \"us\": %.2f, \"GBps\": %.1f}", names[k], bytes[k], best_ms[k] * 1e3,
               bytes[k] / (best_ms[k] * 1e-3) / 1e9);
    printf("}\n");
    CK(hipFree(st));
    CK(hipFree(g));
    CK(hipFree(out));
    CK(hipFree(ca));
    CK(hipFree(cb));
    CK(hipFree(fl));
    CK(hipFree(d_slot));
    CK(hipFree(d_bag));
    return 0;
}
