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
// into row ranges so the launch fills the chip.  Stage 2 (head_finish.h) runs
// one lane per sample and one block per column: after one vector load per
// 128-byte line of the column's planes, its waves share the classes, read
// each class's plane words with scalar loads, assemble each score bit by bit
// (one v_addc per plane) and sum the splits into an LDS score tile, from
// which the scores are written as one contiguous block, and take the argmax.
//
// Quantized head (Sec. 3 "Encoders and heads"; Sec. 5 "Head", the DSP-backed
// head): logit i = sum_j Q[i][j] * count[j] with Q a c x c matrix of signed
// 8-bit weights.  Per 64-sample column this is a [64 x c] x [c x c] integer
// product, done on the matrix cores with v_mfma_i32_16x16x32_i8: a count
// (0..65535) is split into two offset bytes, count = 256 (h + 128) + (l + 128)
// with h, l in [-128, 127], so logit = 256 (Q h) + (Q l) + 32896 rowsum(Q),
// exact in 32-bit integers for c <= 128.
#include "bl_internal.h"
#include "head_finish.h"

namespace bl {

template <int P>
hipError_t launch_finish_p(const uint64_t *planes, int64_t n, int32_t c, int32_t *scores,
                           int32_t *argmax, const int8_t *dsp_weights, const HeadPlan &plan,
                           hipStream_t stream);

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxPlanes = 16;
constexpr int kDspMaxClasses = 128;   // logits stay below 2^31; tiles fit in LDS
// blocks of the quantized head: 4 per CU where a tile's product has several
// K steps, 16 where one K step (c <= 32) leaves each tile little work to
// cover its loads (2^18 x 100: 0.055 ms at 1024 blocks, 0.058 at 4096;
// 2^20 x 10: 0.058 ms at 1024, 0.050 at 4096)
constexpr int64_t kDspBlocks = 1024;
constexpr int64_t kDspBlocksOneK = 4096;

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

// One block (4 waves) per 64-sample column: finish::column_scalar (head_finish.h).
template <int P>
__global__ __launch_bounds__(kThreads) void k_head_finish(
    const uint64_t *__restrict__ planes, int64_t n, int32_t c, int32_t S, int32_t cs,
    int32_t buf_words, int32_t *__restrict__ scores, int32_t *__restrict__ argmax)
{
    extern __shared__ uint64_t buf[];                 // buf_words words
    __shared__ int32_t part[2][finish::kWaves][kWave];
    (void)buf_words;
    // Touch each 128-byte line of the column's planes with one vector load
    // per thread before the count loop.  The lines then arrive together, and
    // the loop's scalar loads, issued a few classes at a time, hit the L2
    // instead of waiting for memory once per batch.  The load is consumed
    // only after the column (into partials nothing reads any more), so it
    // stays in flight meanwhile.  Every thread loads (clamped index): under a
    // divergent branch the compiler reads the planes with vector loads.
    const int64_t nw = (int64_t)c * S * P;
    const int64_t e = min((int64_t)threadIdx.x * 16, nw - 1);
    const uint32_t touch = reinterpret_cast<const uint32_t *>(planes + blockIdx.x * nw + e)[0];
    finish::column_scalar<P>(planes, blockIdx.x, n, c, S, cs, buf, part, scores, argmax);
    part[0][threadIdx.x / kWave][threadIdx.x % kWave] ^= (int32_t)touch;
}

// ---------------------------------------------------------------------------
// Quantized head on the matrix cores.

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// LDS of the quantized head for c classes: Q padded to [cn][ckp] bytes
// (cn = c rounded up to 16 output classes, ck = c rounded up to the 32-deep
// K step, ckp = ck + 8 to spread the banks) and its row sums; for the fused
// finish also the two offset byte planes of a column's counts [64][ckp].
struct DspLayout {
    int cn, ck, ckp;
    size_t off_q, off_rs, off_lo, off_hi, bytes;
};

__host__ __device__ inline DspLayout dsp_layout(int c)
{
    DspLayout L;
    L.cn = (c + 15) / 16 * 16;
    L.ck = (c + 31) / 32 * 32;
    L.ckp = L.ck + 8;
    L.off_q = 0;
    L.off_rs = (size_t)L.cn * L.ckp;
    L.off_lo = L.off_rs + (size_t)L.cn * 4;
    L.off_hi = L.off_lo + (size_t)kWave * L.ckp;
    L.bytes = L.off_hi + (size_t)kWave * L.ckp;
    return L;
}

// Stage Q (zero padded to [cn][ckp]) and its row sums in LDS.  All threads;
// ends with a barrier.  Where c is a multiple of 4 and Q is 4-byte aligned,
// each LDS dword of a row is one dword of Q's row (or zero past it), walked
// without a division per dword; else byte by byte.
__device__ __forceinline__ void dsp_stage_q(const int8_t *__restrict__ weights, int c,
                                            const DspLayout &L, uint8_t *smem)
{
    int8_t *q = reinterpret_cast<int8_t *>(smem + L.off_q);
    int32_t *rs = reinterpret_cast<int32_t *>(smem + L.off_rs);
    uint32_t *q32 = reinterpret_cast<uint32_t *>(smem + L.off_q);
    const int rw = L.ckp / 4;                         // LDS dwords per row
    if (c % 4 == 0 && ((uintptr_t)weights % 4) == 0) {
        const uint32_t *w32 = reinterpret_cast<const uint32_t *>(weights);
        const int cw = c / 4;
        int i = threadIdx.x / rw, j = threadIdx.x - i * rw;
        const int di = kThreads / rw, dj = kThreads - di * rw;
        for (int e = threadIdx.x; e < L.cn * rw; e += kThreads) {
            q32[e] = (i < c && j < cw) ? w32[i * cw + j] : 0u;
            i += di;
            j += dj;
            if (j >= rw) {
                j -= rw;
                ++i;
            }
        }
        __syncthreads();
        for (int r = threadIdx.x; r < L.cn; r += kThreads) {
            int32_t sum = 0;
            for (int k = 0; k < cw; ++k) {
                const uint32_t v = q32[r * rw + k];
                sum += (int8_t)v + (int8_t)(v >> 8) + (int8_t)(v >> 16) + (int8_t)(v >> 24);
            }
            rs[r] = sum;
        }
    } else {
        for (int e = threadIdx.x; e < L.cn * rw; e += kThreads)
            q32[e] = 0;
        __syncthreads();
        for (int f = threadIdx.x; f < c * c; f += kThreads)
            q[(f / c) * L.ckp + f % c] = weights[f];
        __syncthreads();
        for (int r = threadIdx.x; r < L.cn; r += kThreads) {
            int32_t sum = 0;
            for (int k = 0; k < c; ++k)
                sum += q[r * L.ckp + k];
            rs[r] = sum;
        }
    }
    __syncthreads();
}

// Count of (sample row r, class k) into the two offset byte planes.
__device__ __forceinline__ void dsp_put_count(uint8_t *smem, const DspLayout &L, int r, int k,
                                              int32_t cnt)
{
    smem[L.off_lo + (size_t)r * L.ckp + k] = (uint8_t)((cnt & 0xFF) ^ 0x80);
    smem[L.off_hi + (size_t)r * L.ckp + k] = (uint8_t)(((cnt >> 8) & 0xFF) ^ 0x80);
}

constexpr int kDspMaxK = kDspMaxClasses / 32;      // K steps of 32 classes

// Merge (best, besti) with the lane that the DPP control CTL selects in the
// same 16-lane row: the larger value wins, the lower class on ties (besti = c
// marks "none yet").  The order is total, so any merge tree gives the same
// result.  All lanes of the wave.
template <int CTL>
__device__ __forceinline__ void dsp_argmax_step(int32_t &best, int32_t &besti, int c)
{
    const int32_t ov = __builtin_amdgcn_update_dpp(0, best, CTL, 0xF, 0xF, false);
    const int32_t oi = __builtin_amdgcn_update_dpp(0, besti, CTL, 0xF, 0xF, false);
    if (oi < c && (besti >= c || ov > best || (ov == best && oi < besti))) {
        best = ov;
        besti = oi;
    }
}

// One 16-sample M-tile of logits (samples s_first .. s_first + 15) from its
// A operands (8 K-consecutive counts per lane and K step, as the two offset
// bytes, in the MFMA layout), with Q and its row sums in LDS: each N tile's
// product over the K steps, its logits stored from the accumulators, and the
// argmax of each sample -- spread over the 16 lanes of a row and over the N
// tiles -- as a running maximum per lane followed by a 16-lane reduction
// (dsp_argmax_step) that prefers the lower class on ties.  One wave.  v_mfma_i32_16x16x32_i8
// takes in lane l the 8 K-consecutive bytes of row l % 16 at K offset
// 8 (l / 16) of A (counts) and of B^T (rows of Q), and returns
// D[4 (l / 16) + r][l % 16] in accumulator r.
__device__ __forceinline__ void dsp_mtile(const long (&a_lo)[kDspMaxK], const long (&a_hi)[kDspMaxK],
                                          int nks, int n_nt, const int8_t *q, int ckp,
                                          const int32_t *rs, int c, int64_t s_first, int64_t n,
                                          int32_t *__restrict__ logits,
                                          int32_t *__restrict__ argmax)
{
    const int lane = threadIdx.x % kWave;
    const int row = lane % 16, kg = lane / 16, kq = 8 * kg;
    int32_t best[4], besti[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        best[r] = INT32_MIN;
        besti[r] = c;
    }
    for (int nt = 0; nt < n_nt; ++nt) {
        i32x4 acc_lo = {0, 0, 0, 0}, acc_hi = {0, 0, 0, 0};
#pragma unroll
        for (int ks = 0; ks < kDspMaxK; ++ks) {
            if (ks >= nks)
                break;
            const long b = *reinterpret_cast<const long *>(
                q + (size_t)(16 * nt + row) * ckp + 32 * ks + kq);
            acc_lo = __builtin_amdgcn_mfma_i32_16x16x32_i8(a_lo[ks], b, acc_lo, 0, 0, 0);
            acc_hi = __builtin_amdgcn_mfma_i32_16x16x32_i8(a_hi[ks], b, acc_hi, 0, 0, 0);
        }
        const int cls = 16 * nt + row;               // output column of this lane
        if (cls < c) {
            const uint32_t corr = 32896u * (uint32_t)rs[cls];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int32_t v =
                    (int32_t)(256u * (uint32_t)acc_hi[r] + (uint32_t)acc_lo[r] + corr);
                const int64_t smp = s_first + 4 * kg + r;
                if (logits && smp < n)
                    logits[smp * c + cls] = v;
                if (v > best[r]) {                   // classes ascend with nt
                    best[r] = v;
                    besti[r] = cls;
                }
            }
        }
    }
    if (argmax) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            // the 16 lanes of a row: swap within quads (lane ^ 1, ^ 2), then
            // rotate the row by 4 and 8; every lane ends with the row's result
            dsp_argmax_step<0xB1>(best[r], besti[r], c);     // quad_perm [1, 0, 3, 2]
            dsp_argmax_step<0x4E>(best[r], besti[r], c);     // quad_perm [2, 3, 0, 1]
            dsp_argmax_step<0x124>(best[r], besti[r], c);    // row_ror:4
            dsp_argmax_step<0x128>(best[r], besti[r], c);    // row_ror:8
            const int64_t smp = s_first + 4 * kg + r;
            if (row == 0 && smp < n)
                argmax[smp] = besti[r];
        }
    }
}


// Fused finish of the quantized head, one block per 64-sample column: class
// counts from the bit planes as in k_head_finish (the column's lines touched
// first, then scalar plane loads and one v_addc per plane), written as the two
// offset byte planes, then the logits on the matrix cores, each wave one of
// the column's four 16-sample M-tiles (dsp_mtile).
template <int P>
__global__ __launch_bounds__(kThreads) void k_head_finish_dsp(
    const uint64_t *__restrict__ planes, int64_t n, int32_t c, int32_t S,
    const int8_t *__restrict__ weights, int32_t *__restrict__ logits,
    int32_t *__restrict__ argmax)
{
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    const DspLayout L = dsp_layout(c);
    const int lane = threadIdx.x % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t col = blockIdx.x;
    const int64_t nw = (int64_t)c * S * P;
    const int64_t e = min((int64_t)threadIdx.x * 16, nw - 1);
    const uint32_t touch = reinterpret_cast<const uint32_t *>(planes + col * nw + e)[0];
    dsp_stage_q(weights, c, L, smem);
    const uint64_t *pc = planes + col * nw;
    for (int i = wave; i < c; i += kWaves) {
        const uint64_t *pw = pc + (int64_t)i * S * P;
        int q = 0;
        const int32_t cnt = finish::add_splits<P, (P <= 8 ? 4 : 2)>(pw, q, S) +
                            finish::add_splits<P, 1>(pw, q, S);
        dsp_put_count(smem, L, lane, i, cnt);
    }
    __syncthreads();
    // wave w: samples 16 w .. 16 w + 15 of the column, its A operands from
    // its 16 rows of the byte planes
    const int row = lane % 16, kq = 8 * (lane / 16);
    const int nks = L.ck / 32;
    long a_lo[kDspMaxK], a_hi[kDspMaxK];
#pragma unroll
    for (int ks = 0; ks < kDspMaxK; ++ks) {
        if (ks >= nks)
            break;
        const size_t a_off = (size_t)(16 * wave + row) * L.ckp + 32 * ks + kq;
        a_lo[ks] = *reinterpret_cast<const long *>(smem + L.off_lo + a_off);
        a_hi[ks] = *reinterpret_cast<const long *>(smem + L.off_hi + a_off);
    }
    dsp_mtile(a_lo, a_hi, nks, L.cn / 16, reinterpret_cast<const int8_t *>(smem + L.off_q), L.ckp,
              reinterpret_cast<const int32_t *>(smem + L.off_rs), c, col * kWave + 16 * wave, n,
              logits, argmax);
    // the touch is consumed after the column, into a padding dword of one of
    // the wave's own rows (bytes ck .. ckp - 1, which no product reads)
    atomicXor(reinterpret_cast<uint32_t *>(smem + L.off_lo + (size_t)(16 * wave + row) * L.ckp +
                                           L.ck) + (lane / 16) % 2,
              touch);
}

// Standalone quantized head on counts [n][c] in device memory: only Q lives
// in LDS, and each wave takes 16-sample M-tiles and builds their A operands
// straight from the count rows (8 counts per lane and K step, split into the
// two offset bytes); dsp_mtile does the rest.
__device__ __forceinline__ uint32_t dsp_byte_pack(const int32_t (&v)[4], int shift)
{
    uint32_t r = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u)
        r |= (((uint32_t)v[u] >> shift) & 0xFFu) << (8 * u);
    return r ^ 0x80808080u;
}

__global__ __launch_bounds__(kThreads) void k_grouped_dsp(
    const int32_t *__restrict__ counts, int64_t n, int32_t c,
    const int8_t *__restrict__ weights, int32_t *__restrict__ logits,
    int32_t *__restrict__ argmax)
{
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    const DspLayout L = dsp_layout(c);
    dsp_stage_q(weights, c, L, smem);
    const int8_t *q = reinterpret_cast<const int8_t *>(smem + L.off_q);
    const int32_t *rs = reinterpret_cast<const int32_t *>(smem + L.off_rs);
    const int lane = threadIdx.x % kWave;
    const int row = lane % 16, kg = lane / 16, kq = 8 * kg;
    const int nks = L.ck / 32, n_nt = L.cn / 16;
    const int64_t n_mt = (n + 15) / 16;
    const int64_t stride = (int64_t)gridDim.x * kWaves;
    const bool vec = c % 4 == 0 && ((uintptr_t)counts % 16) == 0;   // rows 16-byte aligned
    for (int64_t mt = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave; mt < n_mt;
         mt += stride) {
        const int64_t sa = 16 * mt + row;                 // this lane's A row
        long a_lo[kDspMaxK], a_hi[kDspMaxK];
#pragma unroll
        for (int ks = 0; ks < kDspMaxK; ++ks) {
            if (ks >= nks)
                break;
            int32_t v[8];
            if (vec && sa < n && 32 * ks + 32 <= c) {
                // the K step lies inside the row: two 16-byte loads
                const int4 *src = reinterpret_cast<const int4 *>(counts + sa * c + 32 * ks + kq);
                const int4 x0 = src[0], x1 = src[1];
                v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w;
                v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int k = 32 * ks + kq + j;
                    v[j] = (sa < n && k < c) ? counts[sa * c + k] : 0;
                }
            }
            const int32_t v0[4] = {v[0], v[1], v[2], v[3]}, v1[4] = {v[4], v[5], v[6], v[7]};
            a_lo[ks] = (long)(((uint64_t)dsp_byte_pack(v1, 0) << 32) | dsp_byte_pack(v0, 0));
            a_hi[ks] = (long)(((uint64_t)dsp_byte_pack(v1, 8) << 32) | dsp_byte_pack(v0, 8));
        }
        dsp_mtile(a_lo, a_hi, nks, L.cn / 16, q, L.ckp, rs, c, 16 * mt, n, logits, argmax);
    }
}

template <int P>
hipError_t launch_p(const uint64_t *bits, int32_t w, int64_t n, int32_t c,
                    int32_t *scores, int32_t *argmax, const int8_t *dsp_weights,
                    uint64_t *planes, const HeadPlan &plan, int layout, hipStream_t stream)
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
    return launch_finish_p<P>(planes, n, c, scores, argmax, dsp_weights, plan, stream);
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
    p.splits = (g + nb - 1) / nb;                // the last block of a group may be short
    p.rows_per_split = nb;
    p.planes = bit_length(nb);
    p.ws_bytes = (size_t)c * p.splits * p.planes * W * sizeof(uint64_t);
    return p;
}

template <int P>
hipError_t launch_finish_p(const uint64_t *planes, int64_t n, int32_t c, int32_t *scores,
                           int32_t *argmax, const int8_t *dsp_weights, const HeadPlan &plan,
                           hipStream_t stream)
{
    const int64_t W = (n + 63) / 64;
    if (W > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    if (dsp_weights) {
        if (c > kDspMaxClasses)
            return hipErrorInvalidValue;
        hipLaunchKernelGGL(k_head_finish_dsp<P>, dim3((unsigned)W), dim3(kThreads),
                           dsp_layout(c).bytes, stream, planes, n, c, plan.splits, dsp_weights,
                           scores, argmax);
        return hipGetLastError();
    }
    const int64_t words = finish::tile_words(c);
    hipLaunchKernelGGL(k_head_finish<P>, dim3((unsigned)W), dim3(kThreads),
                       (size_t)words * sizeof(uint64_t), stream, planes, n, c, plan.splits,
                       finish::stride(c), (int32_t)words, scores, argmax);
    return hipGetLastError();
}

hipError_t launch_head_finish(const uint64_t *planes, int64_t n, int32_t c, int32_t *scores,
                              int32_t *argmax, const int8_t *dsp_weights, const HeadPlan &plan,
                              hipStream_t stream)
{
    switch (plan.planes) {
#define BL_CASE(P) \
    case P: return launch_finish_p<P>(planes, n, c, scores, argmax, dsp_weights, plan, stream);
    BL_CASE(1) BL_CASE(2) BL_CASE(3) BL_CASE(4) BL_CASE(5) BL_CASE(6) BL_CASE(7) BL_CASE(8)
    BL_CASE(9) BL_CASE(10) BL_CASE(11) BL_CASE(12) BL_CASE(13) BL_CASE(14) BL_CASE(15)
    BL_CASE(16)
#undef BL_CASE
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_head(const uint64_t *bits, int32_t w, int64_t n, int32_t c,
                       int32_t *scores, int32_t *argmax, const int8_t *dsp_weights, void *ws,
                       const HeadPlan &plan, int layout, hipStream_t stream)
{
    uint64_t *planes = static_cast<uint64_t *>(ws);
    switch (plan.planes) {
#define BL_CASE(P) \
    case P: return launch_p<P>(bits, w, n, c, scores, argmax, dsp_weights, planes, plan, \
                               layout, stream);
    BL_CASE(1) BL_CASE(2) BL_CASE(3) BL_CASE(4) BL_CASE(5) BL_CASE(6) BL_CASE(7) BL_CASE(8)
    BL_CASE(9) BL_CASE(10) BL_CASE(11) BL_CASE(12) BL_CASE(13) BL_CASE(14) BL_CASE(15)
    BL_CASE(16)
#undef BL_CASE
    default: return hipErrorInvalidValue;
    }
}

static_assert(kMaxPlanes == 16, "plane count switch covers 1..16");

hipError_t launch_grouped_dsp(const int32_t *counts, int64_t n, int32_t c,
                              const int8_t *weights, int32_t *logits, int32_t *argmax,
                              hipStream_t stream)
{
    const int64_t mtiles = (n + 15) / 16;
    const int64_t want = (mtiles + kWaves - 1) / kWaves;
    const int64_t cap = c <= 32 ? kDspBlocksOneK : kDspBlocks;
    const int64_t blocks = want < cap ? want : cap;
    if (c < 1 || c > kDspMaxClasses)
        return hipErrorInvalidConfiguration;
    // only Q and its row sums in LDS
    const DspLayout L = dsp_layout(c);
    hipLaunchKernelGGL(k_grouped_dsp, dim3((unsigned)blocks), dim3(kThreads), L.off_lo, stream,
                       counts, n, c, weights, logits, argmax);
    return hipGetLastError();
}

}  // namespace bl
