// Thermometer encoder + bit-pack on gfx950.
//
// Wire f*b + t of sample s is (x[s][f] > theta[f][t]) (Sec. 3 "Encoders and
// heads"; App. A "Initialization"), packed 64 samples per 64-bit word along
// the batch (App. C.1 "Bit-packed inference").
//
// Mapping: one lane per sample, one wave per 64-sample column, so a wave64
// ballot of the comparison is exactly the packed word of one wire.  Ballots
// land in SGPRs; v_writelane moves wire q's word into lane (q mod 64) of an
// accumulator pair, and once 64 wires are collected every lane stores the
// word of "its" wire, so each wave writes 64 rows at one column.
//
// Tile: 32 features x 16 columns (1024 samples).  The 1024 x 32-byte pixel
// tile is staged in LDS with coalesced loads (rows are read as 32 contiguous
// bytes), then lanes read their own sample's byte from LDS.  The row stride
// is padded to 36 bytes (9 dwords, odd) so the 64 lanes of a wave spread
// over the LDS banks.  16 columns per tile make each wire's output segment
// 128 bytes, one full cache line.
//
// XCD-aware order: tile (column group cg, feature tile ft) runs on
// XCD cg % 8, and each XCD walks the feature tiles of one column group in
// order, so the pixel lines shared by neighbouring feature tiles are
// fetched once into that XCD's L2.
#include "bl_internal.h"

namespace bl {
namespace {

constexpr int kThreads = 256;
constexpr int kFeat = 32;              // features per tile
constexpr int kRow = kFeat + 4;        // LDS bytes per staged sample row
constexpr int kCols = 16;              // 64-sample columns per tile
constexpr int kSamples = kCols * kWave;

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

template <bool kAligned4>
__global__ __launch_bounds__(kThreads) void k_encode(
    const uint8_t *__restrict__ x, int64_t n, int32_t d,
    const uint8_t *__restrict__ th, int32_t b, uint64_t *__restrict__ out,
    int64_t W, int32_t n_ftiles, int64_t n_cgroups)
{
    __shared__ uint8_t xs[kSamples * kRow];
    __shared__ uint8_t ths[kFeat * 64];

    const int bid = blockIdx.x;
    const int64_t loc = local_of(bid);
    const int64_t cg = (int64_t)xcd_of(bid) + (int64_t)kXcds * (loc / n_ftiles);
    const int ft = (int)(loc % n_ftiles);
    if (cg >= n_cgroups)
        return;
    const int f0 = ft * kFeat;
    const int nf = min(kFeat, d - f0);
    const int64_t s0 = cg * kSamples;

    // ---- stage thresholds and the pixel tile in LDS
    for (int q = threadIdx.x; q < nf * b; q += kThreads)
        ths[q] = th[(int64_t)f0 * b + q];
    if (kAligned4) {
        // 8 dwords per sample row; features >= d are zero (never read)
        for (int q = threadIdx.x; q < kSamples * (kFeat / 4); q += kThreads) {
            const int r = q / (kFeat / 4), dw = q % (kFeat / 4);
            const int64_t s = s0 + r;
            uint32_t v = 0;
            if (s < n && 4 * dw < nf)
                v = *reinterpret_cast<const uint32_t *>(x + s * d + f0 + 4 * dw);
            *reinterpret_cast<uint32_t *>(&xs[r * kRow + 4 * dw]) = v;
        }
    } else {
        for (int q = threadIdx.x; q < kSamples * kFeat; q += kThreads) {
            const int r = q / kFeat, f = q % kFeat;
            const int64_t s = s0 + r;
            xs[r * kRow + f] = (s < n && f < nf) ? x[s * d + f0 + f] : 0;
        }
    }
    __syncthreads();

    // ---- ballots: wave w handles columns w, w+4, w+8, w+12 of the tile
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    const int nwires = nf * b;
    const int64_t wire0 = (int64_t)f0 * b;
    for (int c = wave; c < kCols; c += kThreads / kWave) {
        const int64_t col = cg * kCols + c;
        if (col >= W)
            break;
        const uint8_t *xrow = &xs[(c * kWave + lane) * kRow];
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
                    out[wire * W + col] = ((uint64_t)acc_hi << 32) | acc_lo;
                }
            }
        }
        const int rem = nwires & (kWave - 1);
        if (rem != 0 && lane < rem) {
            const int64_t wire = wire0 + (nwires - rem) + lane;
            out[wire * W + col] = ((uint64_t)acc_hi << 32) | acc_lo;
        }
    }
}

}  // namespace

hipError_t launch_encode(const uint8_t *x, int64_t n, int32_t d,
                         const uint8_t *thresholds, int32_t b, uint64_t *out,
                         hipStream_t stream)
{
    const int64_t W = (n + 63) / 64;
    const int32_t n_ftiles = (d + kFeat - 1) / kFeat;
    const int64_t n_cg = (W + kCols - 1) / kCols;
    const int64_t n_cg_pad = (n_cg + kXcds - 1) / kXcds * kXcds;
    const int64_t blocks = n_cg_pad * n_ftiles;
    if (blocks > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    const bool aligned4 = (d % 4 == 0) && ((uintptr_t)x % 4 == 0);
    if (aligned4)
        hipLaunchKernelGGL(k_encode<true>, dim3((unsigned)blocks), dim3(kThreads), 0, stream,
                           x, n, d, thresholds, b, out, W, n_ftiles, n_cg);
    else
        hipLaunchKernelGGL(k_encode<false>, dim3((unsigned)blocks), dim3(kThreads), 0, stream,
                           x, n, d, thresholds, b, out, W, n_ftiles, n_cg);
    return hipGetLastError();
}

}  // namespace bl
