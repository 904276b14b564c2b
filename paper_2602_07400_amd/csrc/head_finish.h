// Finish step of the GroupSum head (Sec. 3 "Encoders and heads"; App. C.2):
// the counter planes of one 64-sample column -> scores and argmax, as a
// device function of one 256-thread block (the finish kernel in head.hip runs
// one block per column).
#pragma once

#include "bl_internal.h"

namespace bl {
namespace finish {

constexpr int kThreads = 256;                    // the block this runs in
constexpr int kWaves = kThreads / kWave;
constexpr int kClasses = 128;                    // classes per chunk
// LDS of the finish: the score tile [64][cs] (int32, cs = the odd stride >=
// the chunk's classes, so the tile has no bank conflicts).

__host__ __device__ inline int32_t stride(int32_t c)
{
    return (c < kClasses ? c : kClasses) | 1;
}

__host__ __device__ inline int64_t tile_words(int32_t c)
{
    return ((int64_t)kWave * stride(c) + 1) / 2;
}

// 2 v + bit `lane` of the 64-bit word w (wave-uniform, in an SGPR pair): one
// v_addc_co_u32 whose carry-in is w read as a lane mask.
__device__ __forceinline__ int32_t twice_plus_bit(int32_t v, uint64_t w)
{
    uint64_t carry_out;
    asm("v_addc_co_u32_e64 %0, %1, %0, %0, %2" : "+v"(v), "=s"(carry_out) : "s"(w));
    return v;
}

// Sum over splits q, q + 1, ... (while kQ more remain) of the lane's count
// from P plane words each, advancing q.  The kQ splits' words are loaded
// together, so a wave waits for one scalar-load latency per kQ splits.
template <int P, int kQ>
__device__ __forceinline__ int32_t add_splits(const uint64_t *__restrict__ pw, int &q, int S)
{
    int32_t cnt = 0;
    for (; q + kQ <= S; q += kQ) {
        uint64_t w[kQ][P];
#pragma unroll
        for (int u = 0; u < kQ; ++u)
#pragma unroll
            for (int p = 0; p < P; ++p)
                w[u][p] = pw[(q + u) * P + p];
#pragma unroll
        for (int u = 0; u < kQ; ++u) {
            int32_t v = 0;
#pragma unroll
            for (int p = P - 1; p >= 0; --p)
                v = twice_plus_bit(v, w[u][p]);
            cnt += v;
        }
    }
    return cnt;
}

// Store a score tile [64][cn] (LDS, row stride cs) into dst, the [64][c]
// block of a row-major [n][c] array that starts at the tile's first sample,
// of which `rows` rows are inside the batch: whole 16-byte stores where the
// block is contiguous (cn == c), complete and aligned, walking element
// e = r * c + k without a division per element; else one element at a time.
// All threads of the block; no barrier.
__device__ __forceinline__ void store_tile(const int32_t *tile, int32_t cs, int32_t *__restrict__ dst,
                                           int32_t c, int32_t cn, int64_t rows)
{
    const int total = kWave * cn;
    if (cn == c && rows >= kWave && ((uintptr_t)dst % 16) == 0) {
        const int e0 = 4 * threadIdx.x;
        int r = e0 / cn, k = e0 - r * cn;
        const int dr = 4 * kThreads / cn, dk = 4 * kThreads - dr * cn;
        for (int e = e0; e < total; e += 4 * kThreads) {
            int32_t v[4];
            int rr = r, kk = k;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                v[u] = tile[rr * cs + kk];
                if (++kk == cn) {
                    kk = 0;
                    ++rr;
                }
            }
            *reinterpret_cast<int4 *>(dst + e) = make_int4(v[0], v[1], v[2], v[3]);
            r += dr;
            k += dk;
            if (k >= cn) {
                k -= cn;
                ++r;
            }
        }
    } else {
        int r = threadIdx.x / cn, k = threadIdx.x - r * cn;
        const int dr = kThreads / cn, dk = kThreads - dr * cn;
        for (int e = threadIdx.x; e < total; e += kThreads) {
            if (r < rows)
                dst[(int64_t)r * c + k] = tile[r * cs + k];
            r += dr;
            k += dk;
            if (k >= cn) {
                k -= cn;
                ++r;
            }
        }
    }
}

// Column `col` of planes [W][c][S][P], one lane per sample.  A class's S * P
// plane words are wave-uniform, so they are read with scalar loads (several
// classes' or splits' words at a time), and bit `lane` of each word enters
// the lane's count through the word as a carry-in mask (Horner from the top
// plane): P VALU instructions per split and class instead of a shift, mask
// and merge per plane.  Wave w counts classes w, w + 4, ...; the counts go
// to the LDS tile [64][cs] (buf, tile_words(c) words), from which the scores
// leave as one contiguous block with 16-byte stores where the block is whole
// and aligned.  Each wave keeps a running argmax in class order, merged at
// the end (largest count, then lowest class).  Starts and ends with a barrier.
template <int P>
__device__ __forceinline__ void column_scalar(const uint64_t *__restrict__ planes, int64_t col,
                                              int64_t n, int32_t c, int32_t S, int32_t cs,
                                              uint64_t *buf, int32_t (*part)[kWaves][kWave],
                                              int32_t *__restrict__ scores,
                                              int32_t *__restrict__ argmax)
{
    int32_t *tile = reinterpret_cast<int32_t *>(buf);
    const int lane = threadIdx.x % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t s0 = col * kWave;
    const uint64_t *pc = planes + col * (int64_t)c * S * P;
    int32_t best = -1, besti = 0;
    __syncthreads();
    for (int c0 = 0; c0 < c; c0 += kClasses) {
        const int cn = min(kClasses, c - c0);
        int ii = wave;
        if (S == 1) {
            // kU classes at a time: their plane words are loaded together, so
            // a wave waits for one scalar-load latency per kU classes
            constexpr int kU = P <= 8 ? 4 : 2;
            for (; ii + (kU - 1) * kWaves < cn; ii += kU * kWaves) {
                uint64_t w[kU][P];
#pragma unroll
                for (int u = 0; u < kU; ++u)
#pragma unroll
                    for (int p = 0; p < P; ++p)
                        w[u][p] = pc[(int64_t)(c0 + ii + u * kWaves) * P + p];
#pragma unroll
                for (int u = 0; u < kU; ++u) {
                    int32_t v = 0;
#pragma unroll
                    for (int p = P - 1; p >= 0; --p)
                        v = twice_plus_bit(v, w[u][p]);
                    tile[lane * cs + ii + u * kWaves] = v;
                    if (v > best) {           // classes ascend within a wave
                        best = v;
                        besti = c0 + ii + u * kWaves;
                    }
                }
            }
        }
        for (; ii < cn; ii += kWaves) {
            const uint64_t *pw = pc + (int64_t)(c0 + ii) * S * P;
            int q = 0;
            const int32_t cnt =
                add_splits<P, (P <= 8 ? 4 : 2)>(pw, q, S) + add_splits<P, 1>(pw, q, S);
            tile[lane * cs + ii] = cnt;
            if (cnt > best) {
                best = cnt;
                besti = c0 + ii;
            }
        }
        __syncthreads();
        if (scores)
            store_tile(tile, cs, scores + s0 * c + c0, c, cn, n - s0);
        __syncthreads();
    }
    part[0][wave][lane] = best;
    part[1][wave][lane] = besti;
    __syncthreads();
    if (wave == 0 && argmax && s0 + lane < n) {
        int32_t b = part[0][0][lane], bi = part[1][0][lane];
        for (int w = 1; w < kWaves; ++w) {
            const int32_t v = part[0][w][lane], vi = part[1][w][lane];
            if (v > b || (v == b && vi < bi)) {
                b = v;
                bi = vi;
            }
        }
        argmax[s0 + lane] = bi;
    }
    __syncthreads();
}

}  // namespace finish
}  // namespace bl
