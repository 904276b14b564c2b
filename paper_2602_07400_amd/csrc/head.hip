// GroupSum popcount head + argmax on gfx950.
//
// score[s][i] = number of 1s among nodes [i*g, (i+1)*g) for sample s, and
// argmax[s] = lowest i with the largest score (Sec. 3 "Encoders and heads";
// Sec. 5 "Head"; App. C.2, where the deployed design outputs the class index).
//
// Packed words count *across* samples, but a score counts one sample
// *across* nodes: a positional ("vertical") popcount.  Stage 1 keeps, per
// 64-sample column, a bit-sliced counter (plane p holds bit p of 64 counts)
// and adds the group's words into it with a Harley-Seal carry-save tree
// (v_bitop3 full adders, ~2 ops per word per 32 samples), one lane per column
// so every row load is a coalesced 512-byte segment.  Long groups are split
// into row ranges so the launch fills the chip.  Stage 2 runs one lane per
// sample and one block per column: its waves share the classes, assemble each
// class score bit by bit from the column's planes (wave-uniform scalar loads)
// and sum the splits into an LDS score tile, from which the argmax is taken
// and the scores are written as one contiguous block.
#include "bl_internal.h"

namespace bl {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxPlanes = 16;

__device__ __forceinline__ void csa(uint64_t &h, uint64_t &l, uint64_t a, uint64_t b,
                                    uint64_t c)
{
    const uint64_t u = a ^ b;
    h = (a & b) | (u & c);
    l = u ^ c;
}

template <int P>
__device__ __forceinline__ void ripple_add(uint64_t (&cnt)[P], uint64_t carry, int from)
{
#pragma unroll
    for (int p = 0; p < P; ++p) {
        if (p < from)
            continue;
        const uint64_t t = cnt[p] & carry;
        cnt[p] ^= carry;
        carry = t;
    }
}

template <int P, int LAYOUT>
__global__ __launch_bounds__(kThreads) void k_head_planes(
    const uint64_t *__restrict__ bits, int64_t W, int32_t w, int32_t g, int32_t S,
    int32_t rps, int32_t c, uint64_t *__restrict__ planes, int64_t n_cb)
{
    const int lane = threadIdx.x % kWave;
    const int64_t task = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave;
    const int64_t cb = task % n_cb;
    const int64_t rest = task / n_cb;
    const int q = (int)(rest % S);
    const int i = (int)(rest / S);
    if (i >= c)
        return;
    const int64_t col = cb * kWave + lane;
    const int64_t colc = min(col, W - 1);
    const int64_t r0 = (int64_t)i * g + (int64_t)q * rps;
    const int64_t r1 = min(r0 + rps, (int64_t)(i + 1) * g);

    // word (r, colc) = src[r * stride]
    const uint64_t *src;
    int64_t stride;
    if constexpr (LAYOUT == kLayoutSlab) {
        src = bits + slab_index(0, colc, w);
        stride = kSlabWords;
    } else {
        src = bits + colc;
        stride = W;
    }

    uint64_t cnt[P];
#pragma unroll
    for (int p = 0; p < P; ++p)
        cnt[p] = 0;
    int64_t r = r0;
    if constexpr (P >= 4) {
        for (; r + 8 <= r1; r += 8) {
            uint64_t d[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                d[u] = src[(r + u) * stride];
            uint64_t twosA, twosB, foursA, foursB, eights;
            csa(twosA, cnt[0], cnt[0], d[0], d[1]);
            csa(twosB, cnt[0], cnt[0], d[2], d[3]);
            csa(foursA, cnt[1], cnt[1], twosA, twosB);
            csa(twosA, cnt[0], cnt[0], d[4], d[5]);
            csa(twosB, cnt[0], cnt[0], d[6], d[7]);
            csa(foursB, cnt[1], cnt[1], twosA, twosB);
            csa(eights, cnt[2], cnt[2], foursA, foursB);
            ripple_add<P>(cnt, eights, 3);
        }
    }
    for (; r < r1; ++r)
        ripple_add<P>(cnt, src[r * stride], 0);

    // planes of one column are contiguous: [col][class][split][plane]
    if (col < W) {
        uint64_t *dst = planes + ((col * c + i) * (int64_t)S + q) * P;
#pragma unroll
        for (int p = 0; p < P; ++p)
            dst[p] = cnt[p];
    }
}

constexpr int kFinishClasses = 128;   // classes per LDS score tile

// One block (4 waves) per 64-sample column, one lane per sample.  The waves
// take classes round-robin; a class score is assembled bit by bit from the
// column's planes (contiguous [class][split][plane], wave-uniform scalar
// loads) and parked in an LDS tile [64][classes]; then every lane scans its
// sample's row of the tile for the argmax (lowest index on ties) and the tile
// is written to scores as one contiguous block.
template <int P>
__global__ __launch_bounds__(kThreads) void k_head_finish(
    const uint64_t *__restrict__ planes, int64_t W, int64_t n, int32_t c, int32_t S,
    int32_t *__restrict__ scores, int32_t *__restrict__ argmax)
{
    extern __shared__ int32_t tile[];     // [64][min(c, kFinishClasses)]
    const int lane = threadIdx.x % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t col = blockIdx.x;
    const int64_t s0 = col * kWave;
    const uint64_t *pc = planes + col * (int64_t)c * S * P;
    int32_t best = -1, besti = 0;
    for (int c0 = 0; c0 < c; c0 += kFinishClasses) {
        const int cn = min(kFinishClasses, c - c0);
        for (int ii = wave; ii < cn; ii += kWaves) {
            const int i = c0 + ii;
            int32_t cnt = 0;
            for (int q = 0; q < S; ++q) {
                const uint64_t *pl = pc + ((int64_t)i * S + q) * P;
                int32_t part = 0;
#pragma unroll
                for (int p = 0; p < P; ++p)
                    part |= (int32_t)((pl[p] >> lane) & 1u) << p;
                cnt += part;
            }
            tile[lane * cn + ii] = cnt;
        }
        __syncthreads();
        if (wave == 0) {
            for (int ii = 0; ii < cn; ++ii) {
                const int32_t v = tile[lane * cn + ii];
                if (v > best) {
                    best = v;
                    besti = c0 + ii;
                }
            }
        }
        if (scores) {
            for (int e = threadIdx.x; e < kWave * cn; e += kThreads) {
                const int64_t ss = s0 + e / cn;
                if (ss < n)
                    scores[ss * c + c0 + e % cn] = tile[e];
            }
        }
        __syncthreads();
    }
    if (wave == 0 && argmax && s0 + lane < n)
        argmax[s0 + lane] = besti;
}

template <int P>
hipError_t launch_p(const uint64_t *bits, int32_t w, int64_t n, int32_t c,
                    int32_t *scores, int32_t *argmax, uint64_t *planes,
                    const HeadPlan &plan, int layout, hipStream_t stream)
{
    const int64_t W = (n + 63) / 64;
    const int64_t n_cb = (W + kWave - 1) / kWave;
    const int64_t tasks = n_cb * plan.splits * c;
    const int64_t blocks1 = (tasks + kWaves - 1) / kWaves;
    if (blocks1 > 0x7fffffff || W > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    if (layout == kLayoutSlab)
        hipLaunchKernelGGL((k_head_planes<P, kLayoutSlab>), dim3((unsigned)blocks1),
                           dim3(kThreads), 0, stream, bits, W, w, w / c, plan.splits,
                           plan.rows_per_split, c, planes, n_cb);
    else
        hipLaunchKernelGGL((k_head_planes<P, kLayoutRowMajor>), dim3((unsigned)blocks1),
                           dim3(kThreads), 0, stream, bits, W, w, w / c, plan.splits,
                           plan.rows_per_split, c, planes, n_cb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    const size_t lds = (size_t)kWave * (c < kFinishClasses ? c : kFinishClasses) * sizeof(int32_t);
    hipLaunchKernelGGL(k_head_finish<P>, dim3((unsigned)W), dim3(kThreads), lds, stream,
                       planes, W, n, c, plan.splits, scores, argmax);
    return hipGetLastError();
}

int bit_length(int64_t v)
{
    int b = 0;
    while (v > 0) {
        ++b;
        v >>= 1;
    }
    return b;
}

}  // namespace

HeadPlan plan_head(int32_t w, int64_t n, int32_t c)
{
    HeadPlan p{};
    const int64_t W = (n + 63) / 64;
    const int64_t n_cb = (W + kWave - 1) / kWave;
    const int32_t g = w / c;
    if (W == 0 || g == 0) {          // nothing to count
        p.splits = 1;
        p.rows_per_split = g;
        p.planes = bit_length(g);
        p.ws_bytes = 0;
        return p;
    }
    // enough (class, split, column block) waves to fill 256 CUs several
    // times, but keep at least 32 rows per split
    const int64_t want = (4096 + (int64_t)c * n_cb - 1) / ((int64_t)c * n_cb);
    int64_t S = want < 1 ? 1 : want;
    const int64_t max_s = (g + 31) / 32;
    if (S > max_s)
        S = max_s < 1 ? 1 : max_s;
    int64_t rps = (g + S - 1) / S;
    S = (g + rps - 1) / rps;
    p.splits = (int32_t)S;
    p.rows_per_split = (int32_t)rps;
    p.planes = bit_length(rps);
    p.ws_bytes = (size_t)c * S * p.planes * W * sizeof(uint64_t);
    return p;
}

HeadPlan plan_fused_head(int32_t w, int64_t n, int32_t c, int32_t nb)
{
    HeadPlan p{};
    const int64_t W = (n + 63) / 64;
    const int32_t g = w / c;
    p.splits = g / nb;
    p.rows_per_split = nb;
    p.planes = bit_length(nb);
    p.ws_bytes = (size_t)c * p.splits * p.planes * W * sizeof(uint64_t);
    return p;
}

template <int P>
hipError_t launch_finish_p(const uint64_t *planes, int64_t n, int32_t c, int32_t *scores,
                           int32_t *argmax, const HeadPlan &plan, hipStream_t stream)
{
    const int64_t W = (n + 63) / 64;
    if (W > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    const size_t lds = (size_t)kWave * (c < kFinishClasses ? c : kFinishClasses) * sizeof(int32_t);
    hipLaunchKernelGGL(k_head_finish<P>, dim3((unsigned)W), dim3(kThreads), lds, stream,
                       planes, W, n, c, plan.splits, scores, argmax);
    return hipGetLastError();
}

hipError_t launch_head_finish(const uint64_t *planes, int64_t n, int32_t c, int32_t *scores,
                              int32_t *argmax, const HeadPlan &plan, hipStream_t stream)
{
    switch (plan.planes) {
#define BL_CASE(P) \
    case P: return launch_finish_p<P>(planes, n, c, scores, argmax, plan, stream);
    BL_CASE(1) BL_CASE(2) BL_CASE(3) BL_CASE(4) BL_CASE(5) BL_CASE(6) BL_CASE(7) BL_CASE(8)
    BL_CASE(9) BL_CASE(10) BL_CASE(11) BL_CASE(12) BL_CASE(13) BL_CASE(14) BL_CASE(15)
    BL_CASE(16)
#undef BL_CASE
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_head(const uint64_t *bits, int32_t w, int64_t n, int32_t c,
                       int32_t *scores, int32_t *argmax, void *ws, const HeadPlan &plan,
                       int layout, hipStream_t stream)
{
    uint64_t *planes = static_cast<uint64_t *>(ws);
    switch (plan.planes) {
#define BL_CASE(P) \
    case P: return launch_p<P>(bits, w, n, c, scores, argmax, planes, plan, layout, stream);
    BL_CASE(1) BL_CASE(2) BL_CASE(3) BL_CASE(4) BL_CASE(5) BL_CASE(6) BL_CASE(7) BL_CASE(8)
    BL_CASE(9) BL_CASE(10) BL_CASE(11) BL_CASE(12) BL_CASE(13) BL_CASE(14) BL_CASE(15)
    BL_CASE(16)
#undef BL_CASE
    default: return hipErrorInvalidValue;
    }
}

static_assert(kMaxPlanes == 16, "plane count switch covers 1..16");

}  // namespace bl
