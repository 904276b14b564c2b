// Peak probes: the device's sustained integer VALU rate and HBM streaming
// rates (read-only, write-only, copy), measured with the instruction and
// access types of the hot path (v_bitop3_b32 multiplexers; 16-byte
// non-temporal loads and stores), so that
// roofline fractions can be read against measured as well as published
// peaks.
#include "bl_internal.h"

namespace bl {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeChains = 8;

// Each lane runs `iters` rounds over 8 words; word c becomes the bit-wise
// multiplexer of words c+1 (selector), c (ones) and c+2 (zeros): 8
// v_bitop3_b32 per round (table 0xCA, the LUT layers' multiplexer), written
// as volatile asm so that the compiler cannot merge steps across rounds.
__global__ __launch_bounds__(kProbeThreads) void k_probe_valu(uint32_t *__restrict__ out,
                                                              int32_t iters, uint32_t seed)
{
    const uint32_t gid = blockIdx.x * kProbeThreads + threadIdx.x;
    uint32_t a[kProbeChains];
#pragma unroll
    for (int c = 0; c < kProbeChains; ++c)
        a[c] = (gid + 1u) * 0x9E3779B1u ^ (seed + (uint32_t)c) * 0x85EBCA77u;
#pragma unroll 4
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int c = 0; c < kProbeChains; ++c)
            asm volatile("v_bitop3_b32 %0, %1, %0, %2 bitop3:0xca"
                         : "+v"(a[c])
                         : "v"(a[(c + 1) % kProbeChains]), "v"(a[(c + 2) % kProbeChains]));
    }
    uint32_t r = 0;
#pragma unroll
    for (int c = 0; c < kProbeChains; ++c)
        r ^= a[c];
    out[gid] = r;
}

// HBM streaming probes over n 16-byte pieces.  A block covers U * 256
// consecutive pieces per step (each wave instruction a contiguous 1 KB), its
// U loads all issued before any is used, then strides over the grid.
//   kHbmCopy:  out[i] = in[i]
//   kHbmRead:  xr (16 bytes, cleared by k_probe_clear) ^= every in[i], one
//              set of atomics per wave
//   kHbmWrite: out[i] = (i, i >> 32, ~i, ~(i >> 32)) as four 32-bit words
__device__ __forceinline__ u32x4 piece_pattern(int64_t i)
{
    const uint32_t lo = (uint32_t)i, hi = (uint32_t)((uint64_t)i >> 32);
    return u32x4{lo, hi, ~lo, ~hi};
}

__global__ void k_probe_clear(uint32_t *xr)
{
    if (threadIdx.x < 4)
        xr[threadIdx.x] = 0;
}

template <int MODE, int U>
__global__ __launch_bounds__(kProbeThreads) void k_probe_hbm(const u32x4 *__restrict__ in,
                                                             u32x4 *__restrict__ out, int64_t n)
{
    constexpr int64_t kStep = (int64_t)U * kProbeThreads;
    const int64_t stride = (int64_t)gridDim.x * kStep;
    u32x4 acc = u32x4{0, 0, 0, 0};
    for (int64_t base = (int64_t)blockIdx.x * kStep + threadIdx.x; base < n; base += stride) {
        if (base + (U - 1) * kProbeThreads < n) {
            if constexpr (MODE == kHbmWrite) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int64_t i = base + u * kProbeThreads;
                    __builtin_nontemporal_store(piece_pattern(i), out + i);
                }
            } else {
                u32x4 v[U];
#pragma unroll
                for (int u = 0; u < U; ++u)
                    v[u] = __builtin_nontemporal_load(in + base + u * kProbeThreads);
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    if constexpr (MODE == kHbmCopy)
                        __builtin_nontemporal_store(v[u], out + base + u * kProbeThreads);
                    else
                        acc ^= v[u];
                }
            }
        } else {
            // the ragged last step, piece by piece
            for (int u = 0; u < U; ++u) {
                const int64_t i = base + u * kProbeThreads;
                if (i >= n)
                    break;
                if constexpr (MODE == kHbmWrite)
                    out[i] = piece_pattern(i);
                else if constexpr (MODE == kHbmCopy)
                    out[i] = in[i];
                else
                    acc ^= in[i];
            }
        }
    }
    if constexpr (MODE == kHbmRead) {
        // xor over the wave, then one lane adds it into xr
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            acc.x ^= (uint32_t)__shfl_xor((int)acc.x, off);
            acc.y ^= (uint32_t)__shfl_xor((int)acc.y, off);
            acc.z ^= (uint32_t)__shfl_xor((int)acc.z, off);
            acc.w ^= (uint32_t)__shfl_xor((int)acc.w, off);
        }
        if ((threadIdx.x & (kWave - 1)) == 0 && (acc.x | acc.y | acc.z | acc.w)) {
            uint32_t *xr = reinterpret_cast<uint32_t *>(out);
            atomicXor(xr + 0, acc.x);
            atomicXor(xr + 1, acc.y);
            atomicXor(xr + 2, acc.z);
            atomicXor(xr + 3, acc.w);
        }
    }
}

template <int MODE>
hipError_t launch_hbm_mode(const u32x4 *in, u32x4 *out, int64_t n, int32_t unroll,
                           int32_t blocks, hipStream_t stream)
{
    switch (unroll) {
    case 1: hipLaunchKernelGGL((k_probe_hbm<MODE, 1>), dim3(blocks), dim3(kProbeThreads), 0, stream, in, out, n); break;
    case 2: hipLaunchKernelGGL((k_probe_hbm<MODE, 2>), dim3(blocks), dim3(kProbeThreads), 0, stream, in, out, n); break;
    case 4: hipLaunchKernelGGL((k_probe_hbm<MODE, 4>), dim3(blocks), dim3(kProbeThreads), 0, stream, in, out, n); break;
    case 8: hipLaunchKernelGGL((k_probe_hbm<MODE, 8>), dim3(blocks), dim3(kProbeThreads), 0, stream, in, out, n); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_probe_valu(uint32_t *out, int32_t blocks, int32_t iters, uint32_t seed,
                             hipStream_t stream)
{
    hipLaunchKernelGGL(k_probe_valu, dim3((unsigned)blocks), dim3(kProbeThreads), 0, stream, out,
                       iters, seed);
    return hipGetLastError();
}

hipError_t launch_probe_hbm(int32_t mode, const void *in, void *out, int64_t n_bytes,
                            int32_t unroll, int32_t blocks, hipStream_t stream)
{
    const int64_t n = n_bytes / 16;
    const int64_t step = (int64_t)unroll * kProbeThreads;
    int64_t need = (n + step - 1) / step;                 // blocks that have work
    if (blocks <= 0)
        blocks = 256 * 8;                                 // 8 blocks a CU, grid-stride
    const int32_t grid = (int32_t)(need < blocks ? (need > 0 ? need : 1) : blocks);
    const u32x4 *src = static_cast<const u32x4 *>(in);
    u32x4 *dst = static_cast<u32x4 *>(out);
    switch (mode) {
    case kHbmCopy:
        if (n == 0)
            return hipSuccess;
        return launch_hbm_mode<kHbmCopy>(src, dst, n, unroll, grid, stream);
    case kHbmRead:
        hipLaunchKernelGGL(k_probe_clear, dim3(1), dim3(kWave), 0, stream,
                           reinterpret_cast<uint32_t *>(out));
        if (n == 0)
            return hipGetLastError();
        return launch_hbm_mode<kHbmRead>(src, dst, n, unroll, grid, stream);
    case kHbmWrite:
        if (n == 0)
            return hipSuccess;
        return launch_hbm_mode<kHbmWrite>(src, dst, n, unroll, grid, stream);
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace bl
