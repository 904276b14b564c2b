// Peak probes: the device's sustained integer VALU rate and HBM streaming
// rate, measured with the instruction and access types of the hot path
// (v_bitop3_b32 multiplexers; 16-byte non-temporal loads and stores), so that
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

// Grid-stride copy of n 16-byte pieces.
__global__ __launch_bounds__(kProbeThreads) void k_probe_copy(const u32x4 *__restrict__ in,
                                                              u32x4 *__restrict__ out, int64_t n)
{
    const int64_t stride = (int64_t)gridDim.x * kProbeThreads;
    for (int64_t i = (int64_t)blockIdx.x * kProbeThreads + threadIdx.x; i < n; i += stride)
        __builtin_nontemporal_store(__builtin_nontemporal_load(in + i), out + i);
}

}  // namespace

hipError_t launch_probe_valu(uint32_t *out, int32_t blocks, int32_t iters, uint32_t seed,
                             hipStream_t stream)
{
    hipLaunchKernelGGL(k_probe_valu, dim3((unsigned)blocks), dim3(kProbeThreads), 0, stream, out,
                       iters, seed);
    return hipGetLastError();
}

hipError_t launch_probe_copy(const void *in, void *out, int64_t n_bytes, hipStream_t stream)
{
    const int64_t n = n_bytes / 16;
    int64_t blocks = (n + kProbeThreads - 1) / kProbeThreads;
    blocks = blocks < 256 * 16 ? blocks : 256 * 16;          // 16 blocks per CU, grid-stride
    if (blocks == 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_probe_copy, dim3((unsigned)blocks), dim3(kProbeThreads), 0, stream,
                       static_cast<const u32x4 *>(in), static_cast<u32x4 *>(out), n);
    return hipGetLastError();
}

}  // namespace bl
