// The whole network in one kernel, for networks whose activations of 64
// samples fit in LDS (Sec. 3, Eq. 1: encoder -> D LUT layers -> GroupSum
// head; App. C.1).
//
// Small networks at small batches are latency-bound, and this kernel tries
// to remove the stage boundaries: one block of 512 threads takes a 64-sample
// column through every stage without leaving the CU (used on request; on
// MI355X the layered kernels measured faster, see the forward's planner):
//   1. encode: each wave packs 64-wire groups of the column's samples (codes
//      computed from the thresholds, or the binary code) and transposes them
//      across the wave (dev::transpose64) into one word per wire in LDS;
//   2. layers: one node per thread at a time, its k input words read from
//      the LDS activations, evaluated by the mux tree (dev::eval_node) on the
//      column's two half-words, the output word written to the other LDS
//      buffer; a barrier between layers;
//   3. head: the waves take (class, slice of nodes) items and each lane
//      counts its sample's set bits over the slice's node words into an LDS
//      score tile (LDS atomics), from which the argmax (lowest class on ties)
//      and the scores are written.
// Latency is what matters at these sizes: a wave loads the next group's
// pixels while it packs the current one, the thresholds sit in LDS, and a
// thread issues the connection and table loads of eight nodes before it
// waits for any of them.
// Global traffic is the pixels in and the scores out; the connections and
// tables of every layer are read by every block (they stay in L2).
#include "bl_device.h"

namespace bl {
namespace {

constexpr int kNetThreads = 512;
constexpr int kNetWaves = kNetThreads / kWave;
constexpr int32_t kNetSlice = 64;            // nodes per counting item of the head

// The thread's nodes j, j + 512, ... eight at a time: their connection
// indices and tables are loaded together before any is evaluated.
template <int K>
__device__ __forceinline__ void net_layer(const uint64_t *cur, uint64_t *nxt,
                                          const int32_t *__restrict__ conn,
                                          const uint64_t *__restrict__ tables, int32_t w_out)
{
    constexpr int U = 8;
    for (int32_t j0 = threadIdx.x; j0 < w_out; j0 += U * kNetThreads) {
        int32_t cn[U][K];
        uint64_t T[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t j = j0 + u * kNetThreads;
            const bool in = j < w_out;
            T[u] = in ? tables[j] : 0;
#pragma unroll
            for (int i = 0; i < K; ++i)
                cn[u][i] = in ? conn[(int64_t)j * K + i] : 0;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t j = j0 + u * kNetThreads;
            if (j >= w_out)
                break;
            uint32_t xv[2][K];
#pragma unroll
            for (int i = 0; i < K; ++i) {
                const uint64_t w = cur[cn[u][i]];
                xv[0][i] = (uint32_t)w;
                xv[1][i] = (uint32_t)(w >> 32);
            }
            uint32_t o[2];
            dev::eval_node<K, 1>(T[u], xv, o);
            nxt[j] = ((uint64_t)o[1] << 32) | o[0];
        }
    }
}

// This lane's kFPG pixel bytes of group gi (features gi*kFPG ..), packed four
// to a dword: dword loads when the group starts on a dword and the rows are
// whole dwords, else byte loads.
template <int B>
__device__ __forceinline__ void net_pixels(const uint8_t *__restrict__ row, int32_t d, int gi,
                                           bool live, bool rows4,
                                           uint32_t (&pw)[(64 / B + 3) / 4])
{
    constexpr int kFPG = 64 / B;
    constexpr int kPW = (kFPG + 3) / 4;
    const int f0 = gi * kFPG;
    if (kFPG % 4 == 0 && rows4 && f0 + kFPG <= d) {
#pragma unroll
        for (int q = 0; q < kPW; ++q)
            pw[q] = live ? reinterpret_cast<const uint32_t *>(row + f0)[q] : 0u;
    } else {
#pragma unroll
        for (int q = 0; q < kPW; ++q) {
            uint32_t v = 0;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int fl = 4 * q + u;
                if (fl < kFPG && live && f0 + fl < d)
                    v |= (uint32_t)row[f0 + fl] << (8 * u);
            }
            pw[q] = v;
        }
    }
}

// Encode sample s of this lane (64 samples per wave) into one word per wire:
// the waves take the 64-wire groups of floor(64/B) features; a lane loads its
// group's pixel bytes one group ahead of the one it packs, builds its row of
// wire bits (thresholds staged in LDS, or the binary code) and the wave
// transposes the 64 rows into 64 wire words.
template <int B>
__device__ __forceinline__ void net_encode(const uint8_t *__restrict__ x, int64_t n, int32_t d,
                                           const uint8_t *ths, int32_t kind, int64_t s,
                                           uint64_t *buf)
{
    constexpr int kFPG = 64 / B;
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    uint32_t amt[5], msk[5];
    dev::transpose_consts(lane, amt, msk);
    const int groups = (d + kFPG - 1) / kFPG;
    const int32_t D0 = d * B;
    const bool live = s < n;
    const uint8_t *row = x + (live ? s : n - 1) * d;
    const bool rows4 = (d % 4 == 0) && ((uintptr_t)x % 4 == 0);
    constexpr int kPW = (kFPG + 3) / 4;
    uint32_t px[kPW], nx[kPW];
    if (wave < groups)
        net_pixels<B>(row, d, wave, live, rows4, px);
    for (int gi = wave; gi < groups; gi += kNetWaves) {
        const bool more = gi + kNetWaves < groups;
        if (more)
            net_pixels<B>(row, d, gi + kNetWaves, live, rows4, nx);
        const int f0 = gi * kFPG;
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int fl = 0; fl < kFPG; ++fl) {
            const int f = f0 + fl;
            const uint32_t v = (px[fl / 4] >> (8 * (fl % 4))) & 0xFFu;
            uint32_t code = 0;
            if (kind == kEncBinary) {
                code = (2u * v * ((1u << B) - 1u) + 255u) / 510u;
            } else if (f < d) {
#pragma unroll
                for (int t = 0; t < B; ++t)
                    code |= (v > (uint32_t)ths[f * B + t] ? 1u : 0u) << t;
            }
            const int pos = fl * B;
            if (pos < 32)
                lo |= code << pos;
            if (pos + B > 32)
                hi |= pos >= 32 ? code << (pos - 32) : code >> (32 - pos);
        }
        dev::transpose64(lo, hi, amt, msk);
        const int32_t wire = f0 * B + lane;
        if (lane < kFPG * B && wire < D0)
            buf[wire] = ((uint64_t)hi << 32) | lo;
        if (more)
#pragma unroll
            for (int q = 0; q < kPW; ++q)
                px[q] = nx[q];
    }
}

__global__ __launch_bounds__(kNetThreads) void k_net_fused(
    const uint8_t *__restrict__ x, int64_t n, int32_t d, const uint8_t *__restrict__ th,
    int32_t b, int32_t kind, NetLayers P, int32_t c, int32_t rows_a, int32_t rows_b,
    int32_t tile_in_a, int32_t *__restrict__ scores, int32_t *__restrict__ argmax)
{
    extern __shared__ __attribute__((aligned(16))) uint64_t smem[];
    uint64_t *buf_a = smem;                     // encoded wires, odd layers' outputs
    uint64_t *buf_b = smem + rows_a;            // even layers' outputs
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    const int64_t s0 = (int64_t)blockIdx.x * kWave;
    const int64_t s = s0 + lane;

    // ---- 1. encode the column into buf_a; the thresholds wait in buf_b,
    // which the first layer writes only after the encoder is done
    uint8_t *ths = reinterpret_cast<uint8_t *>(buf_b);
    if (kind != kEncBinary) {
        for (int e = threadIdx.x; e < d * b; e += kNetThreads)
            ths[e] = th[e];
        __syncthreads();
    }
    switch (b) {
    case 1: net_encode<1>(x, n, d, ths, kind, s, buf_a); break;
    case 2: net_encode<2>(x, n, d, ths, kind, s, buf_a); break;
    case 3: net_encode<3>(x, n, d, ths, kind, s, buf_a); break;
    case 4: net_encode<4>(x, n, d, ths, kind, s, buf_a); break;
    case 5: net_encode<5>(x, n, d, ths, kind, s, buf_a); break;
    case 6: net_encode<6>(x, n, d, ths, kind, s, buf_a); break;
    case 7: net_encode<7>(x, n, d, ths, kind, s, buf_a); break;
    default: net_encode<8>(x, n, d, ths, kind, s, buf_a); break;
    }
    __syncthreads();

    // ---- 2. the layers, ping-pong between the two buffers
    const uint64_t *cur = buf_a;
    for (int32_t l = 0; l < P.n; ++l) {
        uint64_t *nxt = (l % 2 == 0) ? buf_b : buf_a;
        const int32_t *conn = P.conn[l];
        const uint64_t *tab = P.tables[l];
        const int32_t w = P.w_out[l];
        switch (P.k[l]) {
        case 1: net_layer<1>(cur, nxt, conn, tab, w); break;
        case 2: net_layer<2>(cur, nxt, conn, tab, w); break;
        case 3: net_layer<3>(cur, nxt, conn, tab, w); break;
        case 4: net_layer<4>(cur, nxt, conn, tab, w); break;
        case 5: net_layer<5>(cur, nxt, conn, tab, w); break;
        default: net_layer<6>(cur, nxt, conn, tab, w); break;
        }
        __syncthreads();
        cur = nxt;
    }

    // ---- 3. head: class counts per sample into the free buffer, then argmax
    const int32_t w_last = P.w_out[P.n - 1];
    const int32_t g = w_last / c;
    int32_t *tile = reinterpret_cast<int32_t *>(tile_in_a ? buf_a : buf_b);
    for (int e = threadIdx.x; e < kWave * c; e += kNetThreads)
        tile[e] = 0;
    __syncthreads();
    // (class, slice of at most kNetSlice nodes) items over the waves; lane =
    // sample; partial counts meet in the tile through LDS atomics
    const int32_t per_class = (g + kNetSlice - 1) / kNetSlice;
    for (int item = wave; item < c * per_class; item += kNetWaves) {
        const int32_t i = item / per_class, q = item % per_class;
        const int32_t j0 = i * g + q * kNetSlice;
        const int32_t j1 = min(j0 + kNetSlice, (i + 1) * g);
        int32_t cnt = 0;
        for (int32_t j = j0; j < j1; ++j)
            cnt += (int32_t)((cur[j] >> lane) & 1u);
        atomicAdd(&tile[lane * c + i], cnt);
    }
    __syncthreads();
    if (argmax && threadIdx.x < kWave && s < n) {
        int32_t best = tile[lane * c], besti = 0;
        for (int i = 1; i < c; ++i) {
            const int32_t v = tile[lane * c + i];
            if (v > best) {
                best = v;
                besti = i;
            }
        }
        argmax[s] = besti;
    }
    if (scores)
        for (int e = threadIdx.x; e < kWave * c; e += kNetThreads) {
            const int64_t ss = s0 + e / c;
            if (ss < n)
                scores[ss * c + e % c] = tile[e];
        }
}

}  // namespace

NetPlan plan_net_fused(int32_t d, int32_t b, int32_t kind, const int32_t *w_out, int32_t n_layers,
                       int32_t c)
{
    NetPlan p{};
    if (n_layers < 1 || n_layers > kNetMaxLayers || b < 1 || b > 8 || c < 1)
        return p;
    // layer l writes buffer B for even l and A for odd l; A first holds the wires
    int64_t rows_a = (int64_t)d * b, rows_b = 0;
    for (int32_t l = 0; l < n_layers; ++l) {
        int64_t &r = (l % 2 == 0) ? rows_b : rows_a;
        if (w_out[l] > r)
            r = w_out[l];
    }
    // buffer B holds the thresholds while the encoder runs
    if (kind != kEncBinary && rows_b * 8 < (int64_t)d * b)
        rows_b = ((int64_t)d * b + 7) / 8;
    // the score tile goes into the buffer the last layer did not write
    const bool last_in_b = (n_layers - 1) % 2 == 0;
    const int64_t tile_bytes = (int64_t)kWave * c * 4;
    int64_t &free_rows = last_in_b ? rows_a : rows_b;
    if (free_rows * 8 < tile_bytes)
        free_rows = (tile_bytes + 7) / 8;
    const int64_t bytes = (rows_a + rows_b) * 8;
    if (bytes > kNetMaxLds)
        return p;
    p.ok = true;
    p.rows_a = (int32_t)rows_a;
    p.rows_b = (int32_t)rows_b;
    p.tile_in_a = last_in_b;
    p.lds_bytes = (size_t)bytes;
    return p;
}

hipError_t launch_net_fused(const uint8_t *x, int64_t n, int32_t d, const uint8_t *th, int32_t b,
                            int32_t kind, const NetLayers &layers, int32_t c,
                            const NetPlan &plan, int32_t *scores, int32_t *argmax,
                            hipStream_t stream)
{
    const int64_t W = (n + kWave - 1) / kWave;
    if (!plan.ok || W > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_net_fused, dim3((unsigned)W), dim3(kNetThreads), plan.lds_bytes, stream,
                       x, n, d, th, b, kind, layers, c, plan.rows_a, plan.rows_b,
                       plan.tile_in_a ? 1 : 0, scores, argmax);
    return hipGetLastError();
}

}  // namespace bl
