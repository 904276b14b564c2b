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
constexpr int kPerWave = kClasses / kWaves;
// LDS of the finish: one buffer that first stages plane words (uint64) and
// then holds the score tile [64][cs] (int32, cs = the odd stride >= the
// chunk's classes, so the tile has no bank conflicts).  Its size is the
// larger of the tile and the planes of one chunk, at most kMaxWords.
constexpr int kMaxWords = kWave * (kClasses + 1) / 2;   // uint64 words

__host__ __device__ inline int32_t stride(int32_t c)
{
    return (c < kClasses ? c : kClasses) | 1;
}

__host__ __device__ inline int64_t tile_words(int32_t c)
{
    return ((int64_t)kWave * stride(c) + 1) / 2;
}

__host__ __device__ inline int64_t lds_words(int32_t c, int32_t S, int32_t P)
{
    const int64_t stage = (int64_t)(c < kClasses ? c : kClasses) * S * P;
    const int64_t want = stage < kMaxWords ? stage : kMaxWords;
    return tile_words(c) > want ? tile_words(c) : want;
}

// Column `col` of planes [W][c][S][P]: all kThreads threads of the block, one
// lane per sample.  Per chunk of up to 128 classes, the block first copies
// the chunk's planes ([class][split][plane], contiguous) into buf with
// coalesced loads, all in flight at once (a class's planes are otherwise a
// chain of scalar loads, one latency per class); when a chunk's splits do
// not fit, it is copied in runs of splits.  Wave w counts classes w, w + 4,
// ...: bit `lane` of each plane word (a broadcast LDS read of the word's
// half) goes to bit p of the count, and the splits are summed in registers.
// The counts then go to the LDS tile [64][cs], from which the scores leave as
// one contiguous block.  Each wave keeps its own running argmax in class
// order; the four are merged at the end (largest count, then lowest class)
// through part.  buf holds buf_words >= tile_words(c) words.  Starts and ends
// with a barrier, so calls can follow each other.
template <int P>
__device__ __forceinline__ void column(const uint64_t *__restrict__ planes, int64_t col, int64_t n,
                                       int32_t c, int32_t S, int32_t cs, int32_t buf_words,
                                       uint64_t *buf, int32_t (*part)[kWaves][kWave],
                                       int32_t *__restrict__ scores, int32_t *__restrict__ argmax)
{
    const uint32_t *buf32 = reinterpret_cast<const uint32_t *>(buf);
    int32_t *tile = reinterpret_cast<int32_t *>(buf);
    const int lane = threadIdx.x % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int half = lane >> 5, bit = lane & 31;
    const int64_t s0 = col * kWave;
    const uint64_t *pc = planes + col * (int64_t)c * S * P;
    const int32_t sp_words = S * P;                   // one class's plane words
    int32_t best = -1, besti = 0;
    __syncthreads();
    for (int c0 = 0, cn = 0; c0 < c; c0 += cn) {
        // classes of this chunk, and splits per staged run
        cn = min(kClasses, c - c0);
        if ((int64_t)cn * sp_words > buf_words)
            cn = max(1, buf_words / sp_words);
        const int run = (int64_t)cn * sp_words <= buf_words ? S : buf_words / P;
        int32_t cnt[kPerWave];
#pragma unroll
        for (int j = 0; j < kPerWave; ++j)
            cnt[j] = 0;
        for (int q0 = 0; q0 < S; q0 += run) {
            const int qn = min(run, S - q0);
            // contiguous: either whole classes (qn == S) or one class (cn == 1)
            const uint64_t *src = pc + ((int64_t)c0 * S + q0) * P;
            const int words = cn * qn * P;
            for (int e = threadIdx.x; e < words; e += kThreads)
                buf[e] = src[e];
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kPerWave; ++j) {
                const int ii = wave + kWaves * j;
                if (ii < cn) {
                    int32_t acc = 0;
                    for (int q = 0; q < qn; ++q) {
                        const uint32_t *w = buf32 + 2 * (ii * qn + q) * P + half;
                        int32_t v = 0;
#pragma unroll
                        for (int p = 0; p < P; ++p)
                            v |= (int32_t)((w[2 * p] >> bit) & 1u) << p;
                        acc += v;
                    }
                    cnt[j] += acc;
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int j = 0; j < kPerWave; ++j) {
            const int ii = wave + kWaves * j;
            if (ii < cn) {
                tile[lane * cs + ii] = cnt[j];
                if (cnt[j] > best) {             // classes ascend within a wave
                    best = cnt[j];
                    besti = c0 + ii;
                }
            }
        }
        __syncthreads();
        if (scores) {
            // element e = r * cn + k of the contiguous block, walked without a
            // division per element
            const int e0 = threadIdx.x;
            int r = e0 / cn, k = e0 - r * cn;
            const int dr = kThreads / cn, dk = kThreads - dr * cn;
            for (int e = e0; e < kWave * cn; e += kThreads) {
                if (s0 + r < n)
                    scores[(s0 + r) * c + c0 + k] = tile[r * cs + k];
                r += dr;
                k += dk;
                if (k >= cn) {
                    k -= cn;
                    ++r;
                }
            }
        }
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
