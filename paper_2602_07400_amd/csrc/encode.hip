// Thermometer encoder + bit-pack on gfx950.
//
// Wire f*b + t of sample s is (x[s][f] > theta[f][t]) (Sec. 3 "Encoders and
// heads"; App. A "Initialization"), packed 64 samples per 64-bit word along
// the batch (App. C.1 "Bit-packed inference").
//
// Two kernels, one lane per sample and one wave per 64-sample column in both:
//
// k_encode_t (b <= 8, the hot path).  A block first fills an LDS code table
// code[f][v] = sum_t (v > theta[f][t]) << t for its tile of features and every
// pixel value v, then reuses it for several tiles of 16 columns (1024
// samples); each wave packs 4 of the 16 columns, one at a time (at small
// batches 2 or 4 blocks share a tile's columns, down to one per wave, so that
// more blocks share the latency).  The table is
// built four codes per thread at a time: a dword holds the codes of four
// consecutive values, and threshold t sets its bit from the first value above
// it on.  A lane loads
// its own sample's FT feature bytes (16-byte loads where rows and tiles allow;
// the next column's bytes are in flight while the current one is packed) and
// assembles, for a group of floor(64/b) features (8 at b = 7, 16 at b = 3),
// the 64-bit row of its sample's wires (one table read and one
// shift-or per feature), and a 64x64 bit transpose across the wave
// (v_permlane32_swap for the 32-lane halves, then five ds_swizzle xor stages,
// each a rotate (v_alignbit) and a bit-field merge (v_bfi) per register) turns
// rows of samples into packed words of wires: lane p ends with wire p's word.
// The words of a 16-column tile are collected in LDS and written as whole
// 128-byte row segments.
//
// k_encode_ballot (any b <= 64).  Each comparison is a wave64 ballot, i.e. the
// packed word of one wire; v_writelane collects 64 such words into one lane
// each before they are stored.
//
// Both write either the row-major layout [wires][W] of bitlogic_encode or the
// slab layout [Wp/S][wires][S] of bitlogic_forward's intermediates.
//
// The binary-coded uniform fixed-point encoder (Sec. 3 "Encoders and heads":
// 2^b levels on b wires; Sec. 5 "Encoder") is the same kernel with another
// code table: code[f][v] = round(v (2^b - 1) / 255), wire t = bit t.
#include "bl_device.h"

namespace bl {
namespace {

using dev::transpose64;
using dev::transpose_consts;

constexpr int kThreads = 256;

#ifndef BL_ENC_TPB
#define BL_ENC_TPB 2
#endif
#ifndef BL_ENC_NT_STORE
#define BL_ENC_NT_STORE 1
#endif

template <int LAYOUT>
__device__ __forceinline__ int64_t out_index(int64_t wire, int64_t wb, int64_t W, int64_t rows)
{
    if constexpr (LAYOUT == kLayoutSlab)
        return slab_index(wire, wb, rows);
    else
        return wire * W + wb;
}

template <int B>
struct EncGeom {
    // Features per 64-wire group: floor(64 / B), except at B = 7 and 3, which
    // take 8 and 16 (56 and 48 of the 64 wires) so that a tile is a whole
    // number of 16-byte pieces and four or two tiles share each 128-byte
    // pixel line, instead of 36- or 84-byte tiles straddling lines (encoder
    // 8-17% faster on 256K-1M samples x 784-3072 features, the transpose
    // then carries 8 or 16 idle rows).
    static constexpr int kFPG = (B == 7) ? 8 : (B == 3) ? 16 : 64 / B;
    static_assert(kFPG * B <= 64, "a group's wires fit one 64-bit row");
    static constexpr int kWPG = kFPG * B;                // wires per group (<= 64)
    static constexpr int kG = (B <= 2) ? 1 : (B == 4) ? 2 : (B == 5) ? 3 : 4;
    static constexpr int kFT = kFPG * kG;                // features per tile
    static constexpr int kDw = kFT / 4;                  // pixel dwords per sample
    static_assert(kFT % 4 == 0, "feature tile must be whole dwords");
};

constexpr int kEncCols = 16;     // columns per output tile: 128-byte row segments
constexpr int kOtRow = kEncCols + 1;   // LDS words per tile row (odd: no bank conflicts)

// This lane's kDw pixel dwords (features f0 .. f0 + 4*kDw - 1 of sample s);
// zero past the batch or past the last feature.  `full` (wave-uniform): the
// whole column is inside the batch, the tile holds kFT features and rows are
// dword aligned, so the loads need no guards.
template <int kDw>
__device__ __forceinline__ void load_pixels(const uint8_t *__restrict__ x, int64_t s, int64_t n,
                                            int32_t d, int f0, int nf, int aligned4, bool full,
                                            uint32_t (&px)[kDw])
{
    const uint8_t *row = x + s * d + f0;
    if constexpr (kDw % 4 == 0) {
        // tiles of whole 16-byte pieces in 16-byte aligned rows (aligned4 == 2)
        if (full && aligned4 == 2) {
#pragma unroll
            for (int q = 0; q < kDw / 4; ++q) {
                const u32x4 v = reinterpret_cast<const u32x4 *>(row)[q];
                px[4 * q + 0] = v.x;
                px[4 * q + 1] = v.y;
                px[4 * q + 2] = v.z;
                px[4 * q + 3] = v.w;
            }
            return;
        }
    }
    if (full) {
#pragma unroll
        for (int q = 0; q < kDw; ++q)
            px[q] = reinterpret_cast<const uint32_t *>(row)[q];
    } else if (s < n && aligned4) {
#pragma unroll
        for (int q = 0; q < kDw; ++q)
            px[q] = (4 * q < nf) ? reinterpret_cast<const uint32_t *>(row)[q] : 0u;
    } else if (s < n) {
#pragma unroll
        for (int q = 0; q < kDw; ++q) {
            uint32_t v = 0;
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (4 * q + u < nf)
                    v |= (uint32_t)row[4 * q + u] << (8 * u);
            px[q] = v;
        }
    } else {
#pragma unroll
        for (int q = 0; q < kDw; ++q)
            px[q] = 0;
    }
}

template <int B, int LAYOUT, int CS>
__global__ __launch_bounds__(kThreads) void k_encode_t(
    const uint8_t *__restrict__ x, int64_t n, int32_t d, const uint8_t *__restrict__ th,
    uint64_t *__restrict__ out, int64_t W, int64_t W_cols, int32_t n_ftiles,
    int32_t tiles_per_block, int64_t n_tiles, int64_t n_tgroups, int aligned4, int kind)
{
    using G = EncGeom<B>;
    constexpr int kWires = G::kG * G::kWPG;              // wire rows of one output tile
    __shared__ __attribute__((aligned(4))) uint8_t lut[G::kFT * 256];
    __shared__ uint8_t ths[G::kFT * B];
    __shared__ uint64_t otile[kWires * kOtRow];

    const int bid = blockIdx.x;
    const int64_t loc = local_of(bid);
    const int64_t tg = (int64_t)xcd_of(bid) + (int64_t)kXcds * (loc / n_ftiles);
    const int ft = (int)(loc % n_ftiles);
    if (tg >= n_tgroups)
        return;
    const int f0 = ft * G::kFT;
    const int nf = min(G::kFT, d - f0);
    const int64_t D0 = (int64_t)d * B;
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;

    // ---- code table for this feature tile: dword e holds the codes of values
    // 4*(e%64) .. +3 of tile feature e/64 (one feature per wave); bit t of a
    // code is set from byte position p on, p = clamp(theta_t - v0 + 1, 0, 4)
    if (kind == kEncThermometer)
        for (int q = threadIdx.x; q < nf * B; q += kThreads)
            ths[q] = th[(int64_t)f0 * B + q];
    __syncthreads();
    for (int e = threadIdx.x; e < G::kFT * 64; e += kThreads) {
        const int f = e >> 6;
        const int v0 = 4 * (e & 63);
        uint32_t codes = 0;
        if (f < nf && kind == kEncThermometer) {
#pragma unroll
            for (int t = 0; t < B; ++t) {
                const int p = min(max((int)ths[f * B + t] - v0 + 1, 0), 4);
                const uint32_t m = (p >= 4) ? 0u : (0xFFFFFFFFu << (8 * p));
                codes |= m & (0x01010101u << t);
            }
        } else if (f < nf) {
            // binary code: q = round(v (2^B - 1) / 255), no ties since 255 is odd
#pragma unroll
            for (int u = 0; u < 4; ++u)
                codes |= (uint32_t)((2u * (uint32_t)(v0 + u) * ((1u << B) - 1u) + 255u) / 510u)
                         << (8 * u);
        }
        reinterpret_cast<uint32_t *>(lut)[e] = codes;
    }
    __syncthreads();

    // per-lane constants of the transpose stages
    uint32_t amt[5], msk[5];
    transpose_consts(lane, amt, msk);

    // block tg covers part (tg % CS) of the columns of tile group tg / CS:
    // cpb columns per tile, cpw consecutive columns per wave
    constexpr int cpb = kEncCols / CS;
    constexpr int cpw = cpb / (kThreads / kWave);
    static_assert(cpw >= 1, "at least one column per wave");
    const int part = (int)(tg % CS);
    const int c_first = part * cpb + wave * cpw;      // this wave's first column of a tile
    const int64_t t0 = (tg / CS) * tiles_per_block;
    const int64_t t1 = min(t0 + tiles_per_block, n_tiles);
    // columns whose 64 samples are all in the batch, in a full aligned tile
    const bool tile_full = aligned4 && nf == G::kFT;
    auto col_full = [&](int64_t gcol) { return tile_full && (gcol + 1) * kWave <= n; };
    uint32_t px[G::kDw];
    {
        const int64_t gcol = t0 * kEncCols + c_first;
        load_pixels<G::kDw>(x, gcol * kWave + lane, n, d, f0, nf, aligned4, col_full(gcol), px);
    }
    for (int64_t tile = t0; tile < t1; ++tile) {
        for (int cw = 0; cw < cpw; ++cw) {
            const int col = c_first + cw;                  // column inside the tile
            // prefetch the next column's pixels while this one is packed
            uint32_t nx[G::kDw];
            const bool more = cw + 1 < cpw || tile + 1 < t1;
            if (more) {
                const int64_t ncol = (cw + 1 < cpw) ? tile * kEncCols + col + 1
                                                    : (tile + 1) * kEncCols + c_first;
                load_pixels<G::kDw>(x, ncol * kWave + lane, n, d, f0, nf, aligned4, col_full(ncol),
                                    nx);
            }
#pragma unroll
            for (int gi = 0; gi < G::kG; ++gi) {
                uint32_t lo = 0, hi = 0;
#pragma unroll
                for (int fl = 0; fl < G::kFPG; ++fl) {
                    const int f = gi * G::kFPG + fl;
                    const uint32_t byte = (px[f / 4] >> (8 * (f % 4))) & 0xFFu;
                    const uint32_t code = lut[f * 256 + byte];
                    const int pos = fl * B;
                    if (pos + B <= 32) {
                        lo |= code << pos;
                    } else if (pos >= 32) {
                        hi |= code << (pos - 32);
                    } else {
                        lo |= code << pos;
                        hi |= code >> (32 - pos);
                    }
                }
                transpose64(lo, hi, amt, msk);
                if (lane < G::kWPG)
                    otile[(gi * G::kWPG + lane) * kOtRow + col] = ((uint64_t)hi << 32) | lo;
            }
            if (more) {
#pragma unroll
                for (int q = 0; q < G::kDw; ++q)
                    px[q] = nx[q];
            }
        }
        __syncthreads();
        // write the tile: each wire's 16 words are one contiguous row segment
        const int64_t wb0 = tile * kEncCols;
        for (int e = threadIdx.x; e < kWires * (cpb / 2); e += kThreads) {
            const int r = e / (cpb / 2);                   // tile wire row
            const int c2 = part * cpb + 2 * (e % (cpb / 2));   // even column
            const int gi = r / G::kWPG, p = r % G::kWPG;
            const int fg = gi * G::kFPG + p / B;           // feature of this wire in the tile
            const int64_t wb = wb0 + c2;
            if (fg >= nf || wb >= W_cols)
                continue;
            const int64_t wire = (int64_t)(f0 + gi * G::kFPG) * B + p;
            const uint64_t w0 = otile[r * kOtRow + c2], w1 = otile[r * kOtRow + c2 + 1];
            uint64_t *q = out + out_index<LAYOUT>(wire, wb, W, D0);
            if (wb + 1 < W_cols && (LAYOUT == kLayoutSlab || ((uintptr_t)q % 16) == 0)) {
                const u32x4 v = u32x4{(uint32_t)w0, (uint32_t)(w0 >> 32), (uint32_t)w1,
                                      (uint32_t)(w1 >> 32)};
                if (BL_ENC_NT_STORE)
                    __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(q));
                else
                    *reinterpret_cast<u32x4 *>(q) = v;
            } else {
                q[0] = w0;
                if (wb + 1 < W_cols)
                    out[out_index<LAYOUT>(wire, wb + 1, W, D0)] = w1;
            }
        }
        __syncthreads();       // tile written before the next one reuses it
    }
}

// Write a wave-uniform value into one lane of a VGPR (v_writelane_b32).  The
// lane select goes through M0: with the value already in an SGPR, a second
// SGPR operand would exceed the one-SGPR constant-bus limit of GFX9-family
// VOP3 encodings.
__device__ __forceinline__ uint32_t write_lane(uint32_t acc, uint32_t value, int lane)
{
    asm("s_mov_b32 m0, %2\n\tv_writelane_b32 %0, %1, m0"
        : "+v"(acc) : "s"(value), "s"(lane) : "m0");
    return acc;
}

constexpr int kBFeat = 32;             // features per tile
constexpr int kBRow = kBFeat + 4;      // LDS bytes per staged sample row (9 dwords)
constexpr int kBCols = 16;             // 64-sample columns per tile
constexpr int kBSamples = kBCols * kWave;

template <bool kAligned4, int LAYOUT>
__global__ __launch_bounds__(kThreads) void k_encode_ballot(
    const uint8_t *__restrict__ x, int64_t n, int32_t d,
    const uint8_t *__restrict__ th, int32_t b, uint64_t *__restrict__ out,
    int64_t W, int64_t W_cols, int32_t n_ftiles, int64_t n_cgroups)
{
    __shared__ uint8_t xs[kBSamples * kBRow];
    __shared__ uint8_t ths[kBFeat * 64];

    const int bid = blockIdx.x;
    const int64_t loc = local_of(bid);
    const int64_t cg = (int64_t)xcd_of(bid) + (int64_t)kXcds * (loc / n_ftiles);
    const int ft = (int)(loc % n_ftiles);
    if (cg >= n_cgroups)
        return;
    const int f0 = ft * kBFeat;
    const int nf = min(kBFeat, d - f0);
    const int64_t s0 = cg * kBSamples;
    const int64_t D0 = (int64_t)d * b;

    for (int q = threadIdx.x; q < nf * b; q += kThreads)
        ths[q] = th[(int64_t)f0 * b + q];
    if (kAligned4) {
        for (int q = threadIdx.x; q < kBSamples * (kBFeat / 4); q += kThreads) {
            const int r = q / (kBFeat / 4), dw = q % (kBFeat / 4);
            const int64_t s = s0 + r;
            uint32_t v = 0;
            if (s < n && 4 * dw < nf)
                v = *reinterpret_cast<const uint32_t *>(x + s * d + f0 + 4 * dw);
            *reinterpret_cast<uint32_t *>(&xs[r * kBRow + 4 * dw]) = v;
        }
    } else {
        for (int q = threadIdx.x; q < kBSamples * kBFeat; q += kThreads) {
            const int r = q / kBFeat, f = q % kBFeat;
            const int64_t s = s0 + r;
            xs[r * kBRow + f] = (s < n && f < nf) ? x[s * d + f0 + f] : 0;
        }
    }
    __syncthreads();

    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    const int nwires = nf * b;
    const int64_t wire0 = (int64_t)f0 * b;
    for (int c = wave; c < kBCols; c += kThreads / kWave) {
        const int64_t col = cg * kBCols + c;
        if (col >= W_cols)
            break;
        const uint8_t *xrow = &xs[(c * kWave + lane) * kBRow];
        uint32_t acc_lo = 0, acc_hi = 0;
        int q = 0;
        for (int f = 0; f < nf; ++f) {
            const uint32_t xv = xrow[f];
            for (int t = 0; t < b; ++t, ++q) {
                const uint64_t m = __ballot(xv > (uint32_t)ths[f * b + t]);
                const int pos = q & (kWave - 1);
                acc_lo = write_lane(acc_lo, (uint32_t)m, pos);
                acc_hi = write_lane(acc_hi, (uint32_t)(m >> 32), pos);
                if (pos == kWave - 1) {
                    const int64_t wire = wire0 + (q - (kWave - 1)) + lane;
                    out[out_index<LAYOUT>(wire, col, W, D0)] = ((uint64_t)acc_hi << 32) | acc_lo;
                }
            }
        }
        const int rem = nwires & (kWave - 1);
        if (rem != 0 && lane < rem) {
            const int64_t wire = wire0 + (nwires - rem) + lane;
            out[out_index<LAYOUT>(wire, col, W, D0)] = ((uint64_t)acc_hi << 32) | acc_lo;
        }
    }
}

template <int B, int LAYOUT>
hipError_t launch_t(const uint8_t *x, int64_t n, int32_t d, const uint8_t *th, uint64_t *out,
                    int64_t W_cols, int kind, hipStream_t stream)
{
    using G = EncGeom<B>;
    const int64_t W = (n + 63) / 64;
    const int64_t n_tiles = (W_cols + kEncCols - 1) / kEncCols;
    const int32_t n_ftiles = (d + G::kFT - 1) / G::kFT;
    // enough blocks to fill the chip; at most BL_ENC_TPB column tiles reuse one
    // code table (longer runs let the blocks that share pixel lines drift
    // apart, and the lines are fetched again: 2 tiles a block beat 1, 3, 4
    // and 8 on 256K-1M samples x 784-3072 features)
    int64_t tpb = n_tiles * n_ftiles / 2048;
    tpb = tpb < 1 ? 1 : (tpb > BL_ENC_TPB ? BL_ENC_TPB : tpb);
    // small batches: split each tile's 16 columns over 2 or 4 blocks (down to
    // one column per wave), so that more blocks share the latency
    int32_t csplit = 1;
    while (csplit < 4 && n_tiles * n_ftiles * csplit < 1024)
        csplit *= 2;
    const int64_t n_tg = (n_tiles + tpb - 1) / tpb * csplit;
    const int64_t n_tg_pad = (n_tg + kXcds - 1) / kXcds * kXcds;
    const int64_t blocks = n_tg_pad * n_ftiles;
    if (blocks > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    // 2: rows 16-byte aligned, 1: 4-byte aligned, 0: neither
    const int aligned4 = ((d % 16 == 0) && ((uintptr_t)x % 16 == 0))  ? 2
                         : ((d % 4 == 0) && ((uintptr_t)x % 4 == 0)) ? 1
                                                                      : 0;
    if (csplit == 4)
        hipLaunchKernelGGL((k_encode_t<B, LAYOUT, 4>), dim3((unsigned)blocks), dim3(kThreads), 0,
                           stream, x, n, d, th, out, W, W_cols, n_ftiles, (int32_t)tpb, n_tiles,
                           n_tg, aligned4, kind);
    else if (csplit == 2)
        hipLaunchKernelGGL((k_encode_t<B, LAYOUT, 2>), dim3((unsigned)blocks), dim3(kThreads), 0,
                           stream, x, n, d, th, out, W, W_cols, n_ftiles, (int32_t)tpb, n_tiles,
                           n_tg, aligned4, kind);
    else
        hipLaunchKernelGGL((k_encode_t<B, LAYOUT, 1>), dim3((unsigned)blocks), dim3(kThreads), 0,
                           stream, x, n, d, th, out, W, W_cols, n_ftiles, (int32_t)tpb, n_tiles,
                           n_tg, aligned4, kind);
    return hipGetLastError();
}

template <int LAYOUT>
hipError_t launch_ballot(const uint8_t *x, int64_t n, int32_t d, const uint8_t *th, int32_t b,
                         uint64_t *out, int64_t W_cols, hipStream_t stream)
{
    const int64_t W = (n + 63) / 64;
    const int32_t n_ftiles = (d + kBFeat - 1) / kBFeat;
    const int64_t n_cg = (W_cols + kBCols - 1) / kBCols;
    const int64_t n_cg_pad = (n_cg + kXcds - 1) / kXcds * kXcds;
    const int64_t blocks = n_cg_pad * n_ftiles;
    if (blocks > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    const bool aligned4 = (d % 4 == 0) && ((uintptr_t)x % 4 == 0);
    if (aligned4)
        hipLaunchKernelGGL((k_encode_ballot<true, LAYOUT>), dim3((unsigned)blocks), dim3(kThreads),
                           0, stream, x, n, d, th, b, out, W, W_cols, n_ftiles, n_cg);
    else
        hipLaunchKernelGGL((k_encode_ballot<false, LAYOUT>), dim3((unsigned)blocks),
                           dim3(kThreads), 0, stream, x, n, d, th, b, out, W, W_cols, n_ftiles,
                           n_cg);
    return hipGetLastError();
}

template <int LAYOUT>
hipError_t launch_layout(const uint8_t *x, int64_t n, int32_t d, const uint8_t *th, int32_t b,
                         uint64_t *out, int64_t W_cols, int kind, hipStream_t stream)
{
    switch (b) {
    case 1: return launch_t<1, LAYOUT>(x, n, d, th, out, W_cols, kind, stream);
    case 2: return launch_t<2, LAYOUT>(x, n, d, th, out, W_cols, kind, stream);
    case 3: return launch_t<3, LAYOUT>(x, n, d, th, out, W_cols, kind, stream);
    case 4: return launch_t<4, LAYOUT>(x, n, d, th, out, W_cols, kind, stream);
    case 5: return launch_t<5, LAYOUT>(x, n, d, th, out, W_cols, kind, stream);
    case 6: return launch_t<6, LAYOUT>(x, n, d, th, out, W_cols, kind, stream);
    case 7: return launch_t<7, LAYOUT>(x, n, d, th, out, W_cols, kind, stream);
    case 8: return launch_t<8, LAYOUT>(x, n, d, th, out, W_cols, kind, stream);
    default:
        if (kind != kEncThermometer)
            return hipErrorInvalidValue;          // binary codes have at most 8 bits
        return launch_ballot<LAYOUT>(x, n, d, th, b, out, W_cols, stream);
    }
}

}  // namespace

hipError_t launch_encode(const uint8_t *x, int64_t n, int32_t d, const uint8_t *thresholds,
                         int32_t b, uint64_t *out, int layout, int64_t W_cols,
                         hipStream_t stream, int kind)
{
    if (layout == kLayoutSlab)
        return launch_layout<kLayoutSlab>(x, n, d, thresholds, b, out, W_cols, kind, stream);
    return launch_layout<kLayoutRowMajor>(x, n, d, thresholds, b, out, W_cols, kind, stream);
}

}  // namespace bl
