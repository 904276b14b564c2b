// Quantile thermometer thresholds fitted on the device (Sec. 4
// "Initialization": fitted once from the empirical pixel quantiles of the
// training split; App. B: over the flattened pixel distribution).
//
// The d features are cut into n_groups contiguous groups (one group: the
// whole flattened distribution; one per colour channel for CHW images).  Per
// group, with cum(v) = number of the group's pixels <= v and total = n * d /
// n_groups, threshold i (i = 1..b) is the smallest v with
// (b + 1) * cum(v) >= i * total -- the exact integer form of
// cum(v) / total >= i / (b + 1) -- and every feature of the group receives
// the group's ladder.
//
// k_fit_hist: each block counts a run of rows into an LDS histogram per
// group (LDS atomics), then adds it into the global 64-bit histogram.  The
// LDS histogram holds R interleaved copies of every bin (lane l counts into
// copy l mod R, at word bin * R + l mod R), so that the 64 atomics of a wave
// spread over the banks and rarely hit the same word; the copies are summed
// before the global add.  Rows are read as coalesced dwords: a thread keeps
// its columns (and their groups) and walks the rows, kRowUnroll rows' loads
// at a time.  k_fit_select:
// one block per group turns the histogram into the ladder (a block prefix sum,
// one thread per bin).
#include "bl_internal.h"

namespace bl {
namespace {

constexpr int kThreads = 256;
constexpr int kHistBlocks = 1024;
#ifndef BL_FIT_UNROLL
#define BL_FIT_UNROLL 32
#endif
#ifndef BL_FIT_MAX_REP
#define BL_FIT_MAX_REP 32
#endif
constexpr int kRowUnroll = BL_FIT_UNROLL;
constexpr int kFitMaxRep = BL_FIT_MAX_REP;        // copies of each histogram bin
constexpr int kFitHistBytes = 48 << 10;           // LDS of one histogram block

__global__ __launch_bounds__(kThreads) void k_fit_clear(uint64_t *__restrict__ ws, int32_t n)
{
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i < n)
        ws[i] = 0;
}

__global__ __launch_bounds__(kThreads) void k_fit_hist(
    const uint8_t *__restrict__ x, int64_t n, int32_t d, int32_t per, int32_t n_groups,
    int64_t rows_per_block, int aligned4, int32_t rep_log2, uint64_t *__restrict__ ws)
{
    extern __shared__ uint32_t hist[];             // [n_groups][256][R], R = 2^rep_log2
    const int nbins = n_groups * 256;
    for (int i = threadIdx.x; i < nbins << rep_log2; i += kThreads)
        hist[i] = 0;
    __syncthreads();
    const uint32_t copy = threadIdx.x & ((1u << rep_log2) - 1);
    // LDS word of bin (g256 + v) in this lane's copy
    auto slot = [&](int g256, uint32_t v) { return (((uint32_t)g256 + v) << rep_log2) + copy; };
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t r1 = min(n, r0 + rows_per_block);
    if (aligned4) {
        const int32_t d4 = d / 4;
        const uint32_t *x32 = reinterpret_cast<const uint32_t *>(x);
        for (int32_t fq = threadIdx.x; fq < d4; fq += kThreads) {
            int g[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                g[u] = (4 * fq + u) / per * 256;
            // eight rows' loads in flight before their counts
            int64_t r = r0;
            for (; r + kRowUnroll <= r1; r += kRowUnroll) {
                uint32_t v[kRowUnroll];
#pragma unroll
                for (int q = 0; q < kRowUnroll; ++q)
                    v[q] = x32[(r + q) * d4 + fq];
#pragma unroll
                for (int q = 0; q < kRowUnroll; ++q)
#pragma unroll
                    for (int u = 0; u < 4; ++u)
                        atomicAdd(&hist[slot(g[u], (v[q] >> (8 * u)) & 0xFFu)], 1u);
            }
            for (; r < r1; ++r) {
                const uint32_t v = x32[r * d4 + fq];
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    atomicAdd(&hist[slot(g[u], (v >> (8 * u)) & 0xFFu)], 1u);
            }
        }
    } else {
        for (int32_t f = threadIdx.x; f < d; f += kThreads) {
            const int g = f / per * 256;
            int64_t r = r0;
            for (; r + kRowUnroll <= r1; r += kRowUnroll) {
                uint32_t v[kRowUnroll];
#pragma unroll
                for (int q = 0; q < kRowUnroll; ++q)
                    v[q] = x[(r + q) * d + f];
#pragma unroll
                for (int q = 0; q < kRowUnroll; ++q)
                    atomicAdd(&hist[slot(g, v[q])], 1u);
            }
            for (; r < r1; ++r)
                atomicAdd(&hist[slot(g, x[r * d + f])], 1u);
        }
    }
    __syncthreads();
    // sum the copies (each thread starts at another copy, so that the
    // threads of a wave read different banks), then one global add per bin
    const int nrep = 1 << rep_log2;
    for (int i = threadIdx.x; i < nbins; i += kThreads) {
        uint32_t sum = 0;
        for (int k = 0; k < nrep; ++k)
            sum += hist[((uint32_t)i << rep_log2) + ((uint32_t)(k + i) & (uint32_t)(nrep - 1))];
        if (sum)
            atomicAdd(reinterpret_cast<unsigned long long *>(&ws[i]), (unsigned long long)sum);
    }
}

__global__ __launch_bounds__(kThreads) void k_fit_select(
    const uint64_t *__restrict__ ws, int64_t total, int32_t per, int32_t b,
    uint8_t *__restrict__ th)
{
    static_assert(kThreads == 256, "one thread per histogram bin");
    __shared__ uint64_t cum[256];
    __shared__ uint8_t ladder[64];
    const int grp = blockIdx.x;
    const int v = threadIdx.x;
    // inclusive prefix sum of the 256 bins (Hillis-Steele, 8 steps)
    cum[v] = ws[grp * 256 + v];
    __syncthreads();
#pragma unroll
    for (int off = 1; off < 256; off <<= 1) {
        const uint64_t add = v >= off ? cum[v - off] : 0;
        __syncthreads();
        cum[v] += add;
        __syncthreads();
    }
    // threshold i is the smallest v with (b + 1) cum(v) >= i total (255 if
    // none): thread v sets it where the criterion first holds
    const uint64_t b1 = (uint64_t)(b + 1);
    for (int i = 1; i <= b; ++i) {
        const uint64_t need = (uint64_t)i * (uint64_t)total;
        const bool here = cum[v] * b1 >= need;
        const bool before = v > 0 && cum[v - 1] * b1 >= need;
        if ((here && !before) || (v == 255 && !here))
            ladder[i - 1] = (uint8_t)v;
    }
    __syncthreads();
    uint8_t *dst = th + (int64_t)grp * per * b;
    for (int64_t e = threadIdx.x; e < (int64_t)per * b; e += kThreads)
        dst[e] = ladder[e % b];
}

}  // namespace

hipError_t launch_fit_quantiles(const uint8_t *x, int64_t n, int32_t d, int32_t b,
                                int32_t n_groups, uint8_t *th, uint64_t *ws, hipStream_t stream)
{
    if (n_groups < 1 || n_groups > kFitMaxGroups || d % n_groups != 0 || b < 1 || b > 64 ||
        n < 1)
        return hipErrorInvalidValue;
    const int32_t per = d / n_groups;
    const int32_t bins = n_groups * 256;
    hipLaunchKernelGGL(k_fit_clear, dim3((bins + kThreads - 1) / kThreads), dim3(kThreads), 0,
                       stream, ws, bins);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    // rows per block: about kHistBlocks blocks, and a block's count of any
    // one bin (at most rows * per) stays below 2^31
    int64_t rows = (n + kHistBlocks - 1) / kHistBlocks;
    const int64_t cap = ((int64_t)1 << 31) / per;
    if (rows > cap)
        rows = cap < 1 ? 1 : cap;
    const int64_t blocks = (n + rows - 1) / rows;
    if (blocks > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    const int aligned4 = (d % 4 == 0) && ((uintptr_t)x % 4 == 0);
    // as many bin copies as the block's LDS budget allows (at least one)
    int32_t rep_log2 = 0;
    while ((2 << rep_log2) <= kFitMaxRep &&
           (size_t)bins * sizeof(uint32_t) * (2u << rep_log2) <= (size_t)kFitHistBytes)
        ++rep_log2;
    hipLaunchKernelGGL(k_fit_hist, dim3((unsigned)blocks), dim3(kThreads),
                       ((size_t)bins << rep_log2) * sizeof(uint32_t), stream, x, n, d, per,
                       n_groups, rows, aligned4, rep_log2, ws);
    e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_fit_select, dim3((unsigned)n_groups), dim3(kThreads), 0, stream, ws,
                       n * (int64_t)per, per, b, th);
    return hipGetLastError();
}

}  // namespace bl
