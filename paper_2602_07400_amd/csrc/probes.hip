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

// ---- instruction-rate probe: one VALU instruction form repeated ----------
// A self-contained asm loop on fixed registers, so that the VGPR banks of
// the operands are known (v[n] is in bank n % 4): eight chains in v40, v44,
// ..., v68 (bank 0), the selector in v41 (bank 1) and the zero operand in
// v42 (bank 2) or v45 (bank 1).  Each round issues 64 instructions:
//   kOpMux:      v_bitop3_b32 c, v41, c, v42 (table 0xCA: c = (v41 & c) | (~v41 & v42)),
//                three source banks: the LUT layers' multiplexer at full rate
//   kOpMuxBank:  the same with v45 in place of v42: two sources in bank 1
//   kOpBfe:      v_bfe_i32 c, v41, 5, 1 (the mask of one table bit)
// The lane's result is the sum of the eight chain registers afterwards.
constexpr int kOpMux = 0, kOpMuxBank = 1, kOpBfe = 2;

#define BL_PV8(INS) INS(40) INS(44) INS(48) INS(52) INS(56) INS(60) INS(64) INS(68)
#define BL_MUX(R) "v_bitop3_b32 v" #R ", v41, v" #R ", v42 bitop3:0xca\n\t"
#define BL_MUXB(R) "v_bitop3_b32 v" #R ", v41, v" #R ", v45 bitop3:0xca\n\t"
#define BL_BFE(R) "v_bfe_i32 v" #R ", v41, 5, 1\n\t"
#define BL_INIT(R) "v_mov_b32 v" #R ", %[c0]\n\t"
#define BL_FOLD(R) "v_add_u32 %[r], %[r], v" #R "\n\t"
#define BL_ROUND(X) BL_PV8(X) BL_PV8(X) BL_PV8(X) BL_PV8(X) BL_PV8(X) BL_PV8(X) BL_PV8(X) BL_PV8(X)

template <int OP>
__global__ __launch_bounds__(kProbeThreads) void k_probe_valu_op(uint32_t *__restrict__ out,
                                                                 int32_t iters, uint32_t seed)
{
    const uint32_t gid = blockIdx.x * kProbeThreads + threadIdx.x;
    const uint32_t c0 = (gid + 1u) * 0x9E3779B1u ^ seed;
    const uint32_t sel = c0 * 0x85EBCA77u, zero = ~c0;
    uint32_t r = 0;
    uint32_t cnt = (uint32_t)iters;           // >= 1 (the launcher checks)
    if constexpr (OP == kOpMux)
        asm volatile(BL_PV8(BL_INIT) "v_mov_b32 v41, %[s]\n\tv_mov_b32 v42, %[z]\n\t"
                     "1:\n\t" BL_ROUND(BL_MUX)
                     "s_sub_u32 %[n], %[n], 1\n\ts_cmp_lg_u32 %[n], 0\n\ts_cbranch_scc1 1b\n\t"
                     BL_PV8(BL_FOLD)
                     : [r] "+v"(r), [n] "+s"(cnt)
                     : [c0] "v"(c0), [s] "v"(sel), [z] "v"(zero)
                     : "v40", "v41", "v42", "v44", "v48", "v52", "v56", "v60", "v64", "v68",
                       "scc");
    else if constexpr (OP == kOpMuxBank)
        asm volatile(BL_PV8(BL_INIT) "v_mov_b32 v41, %[s]\n\tv_mov_b32 v45, %[z]\n\t"
                     "1:\n\t" BL_ROUND(BL_MUXB)
                     "s_sub_u32 %[n], %[n], 1\n\ts_cmp_lg_u32 %[n], 0\n\ts_cbranch_scc1 1b\n\t"
                     BL_PV8(BL_FOLD)
                     : [r] "+v"(r), [n] "+s"(cnt)
                     : [c0] "v"(c0), [s] "v"(sel), [z] "v"(zero)
                     : "v40", "v41", "v44", "v45", "v48", "v52", "v56", "v60", "v64", "v68",
                       "scc");
    else
        asm volatile(BL_PV8(BL_INIT) "v_mov_b32 v41, %[s]\n\t"
                     "1:\n\t" BL_ROUND(BL_BFE)
                     "s_sub_u32 %[n], %[n], 1\n\ts_cmp_lg_u32 %[n], 0\n\ts_cbranch_scc1 1b\n\t"
                     BL_PV8(BL_FOLD)
                     : [r] "+v"(r), [n] "+s"(cnt)
                     : [c0] "v"(c0), [s] "v"(sel)
                     : "v40", "v41", "v44", "v48", "v52", "v56", "v60", "v64", "v68", "scc");
    out[gid] = r;
}

#undef BL_PV8
#undef BL_MUX
#undef BL_MUXB
#undef BL_BFE
#undef BL_INIT
#undef BL_FOLD
#undef BL_ROUND

// ---- gather probe: the LUT layers' row gathers without their arithmetic --
// Per pass, wave w of block b gathers 6 rows of 128 bytes for each of 16
// nodes j = (b * passes + pass) * 64 + w * 16 + m, row (j, i) =
// probe_row(seed, 6 j + i) mod n_rows, with the lane split of the layer
// kernels: LPR = 4 lanes per node, each loading two 16-byte halves of its
// 32 bytes of every row (16 rows per load instruction, as at 5 and 6
// inputs), or LPR = 8 lanes per row, one 16-byte piece each (a whole line
// per 8 lanes, 8 rows per instruction; a lane then serves nodes m and m + 8).
// V v_bitop3_b32 per lane and pass then run on the loaded words (their
// results are dropped: they only occupy the VALU as the multiplexers do);
// with a sink, each wave also stores 2 KB per pass (the lane's first two
// pieces, non-temporal), as the layer kernel stores its output.
__device__ __forceinline__ uint32_t probe_row(uint32_t seed, uint32_t x)
{
    uint32_t h = (x ^ seed) * 0x9E3779B1u;
    return h ^ (h >> 16);
}

template <int LPR, int V, bool SINK>
__global__ __launch_bounds__(kProbeThreads) void k_probe_gather(
    const u32x4 *__restrict__ rows, uint32_t n_rows, uint32_t seed, int32_t passes,
    uint32_t *__restrict__ out, u32x4 *__restrict__ sink)
{
    extern __shared__ uint32_t pad[];            // occupancy limiter only
    (void)pad;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int sub = lane % LPR;
    u32x4 acc = u32x4{0, 0, 0, 0};
#pragma unroll 1
    for (int pass = 0; pass < passes; ++pass) {
        const uint32_t j0 = ((uint32_t)blockIdx.x * (uint32_t)passes + (uint32_t)pass) * 64u +
                            (uint32_t)wave * 16u;
        u32x4 v[12];
#pragma unroll
        for (int i = 0; i < 6; ++i) {
            if constexpr (LPR == 4) {
                const uint32_t j = j0 + (uint32_t)(lane / 4);
                const uint32_t r = probe_row(seed, 6u * j + (uint32_t)i) % n_rows;
                v[2 * i] = rows[(size_t)r * 8 + 2 * sub];
                v[2 * i + 1] = rows[(size_t)r * 8 + 2 * sub + 1];
            } else {
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const uint32_t j = j0 + (uint32_t)(h * 8 + lane / 8);
                    const uint32_t r = probe_row(seed, 6u * j + (uint32_t)i) % n_rows;
                    v[6 * h + i] = rows[(size_t)r * 8 + sub];
                }
            }
        }
        if constexpr (V > 0) {
            uint32_t a = v[0].x, b = v[1].y;
#pragma unroll
            for (int t = 0; t < V / 2; ++t) {
                asm volatile("v_bitop3_b32 %0, %1, %0, %2 bitop3:0xca"
                             : "+v"(a) : "v"(v[t % 12].z), "v"(b));
                asm volatile("v_bitop3_b32 %0, %1, %0, %2 bitop3:0xca"
                             : "+v"(b) : "v"(v[(t + 5) % 12].w), "v"(a));
            }
        }
#pragma unroll
        for (int k = 0; k < 12; ++k)
            acc ^= v[k];
        if constexpr (SINK) {
            u32x4 *q = sink + (((size_t)blockIdx.x * passes + pass) * 4 + wave) * 128 + lane * 2;
            __builtin_nontemporal_store(v[0], q);
            __builtin_nontemporal_store(v[1], q + 1);
        }
    }
    out[blockIdx.x * kProbeThreads + threadIdx.x] = acc.x ^ acc.y ^ acc.z ^ acc.w;
}

template <int LPR, int V>
hipError_t launch_gather_v(const u32x4 *rows, uint32_t n_rows, uint32_t seed, int32_t passes,
                           int32_t blocks, size_t lds, uint32_t *out, u32x4 *sink,
                           hipStream_t stream)
{
    if (sink)
        hipLaunchKernelGGL((k_probe_gather<LPR, V, true>), dim3(blocks), dim3(kProbeThreads), lds,
                           stream, rows, n_rows, seed, passes, out, sink);
    else
        hipLaunchKernelGGL((k_probe_gather<LPR, V, false>), dim3(blocks), dim3(kProbeThreads),
                           lds, stream, rows, n_rows, seed, passes, out, sink);
    return hipGetLastError();
}

template <int LPR>
hipError_t launch_gather_l(const u32x4 *rows, uint32_t n_rows, uint32_t seed, int32_t passes,
                           int32_t blocks, size_t lds, int32_t valu, uint32_t *out, u32x4 *sink,
                           hipStream_t stream)
{
    switch (valu) {
    case 0: return launch_gather_v<LPR, 0>(rows, n_rows, seed, passes, blocks, lds, out, sink, stream);
    case 256: return launch_gather_v<LPR, 256>(rows, n_rows, seed, passes, blocks, lds, out, sink, stream);
    case 512: return launch_gather_v<LPR, 512>(rows, n_rows, seed, passes, blocks, lds, out, sink, stream);
    case 768: return launch_gather_v<LPR, 768>(rows, n_rows, seed, passes, blocks, lds, out, sink, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_probe_valu(uint32_t *out, int32_t blocks, int32_t iters, uint32_t seed,
                             hipStream_t stream)
{
    hipLaunchKernelGGL(k_probe_valu, dim3((unsigned)blocks), dim3(kProbeThreads), 0, stream, out,
                       iters, seed);
    return hipGetLastError();
}

hipError_t launch_probe_valu_op(int32_t op, uint32_t *out, int32_t blocks, int32_t iters,
                                uint32_t seed, hipStream_t stream)
{
    if (iters < 1)
        return hipErrorInvalidValue;
    switch (op) {
    case kOpMux:
        hipLaunchKernelGGL(k_probe_valu_op<kOpMux>, dim3(blocks), dim3(kProbeThreads), 0, stream,
                           out, iters, seed);
        break;
    case kOpMuxBank:
        hipLaunchKernelGGL(k_probe_valu_op<kOpMuxBank>, dim3(blocks), dim3(kProbeThreads), 0,
                           stream, out, iters, seed);
        break;
    case kOpBfe:
        hipLaunchKernelGGL(k_probe_valu_op<kOpBfe>, dim3(blocks), dim3(kProbeThreads), 0, stream,
                           out, iters, seed);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_probe_gather(const void *rows, int64_t n_rows, int32_t lanes_per_row,
                               int32_t valu, int32_t blocks, int32_t passes,
                               int32_t waves_per_simd, uint32_t seed, uint32_t *out, void *sink,
                               hipStream_t stream)
{
    // a block is one wave per SIMD: waves_per_simd blocks fit one CU's LDS
    const size_t lds = waves_per_simd > 0 ? (size_t)(160 * 1024 / waves_per_simd) - 256 : 0;
    const u32x4 *r = static_cast<const u32x4 *>(rows);
    u32x4 *k = static_cast<u32x4 *>(sink);
    if (lanes_per_row == 4)
        return launch_gather_l<4>(r, (uint32_t)n_rows, seed, passes, blocks, lds, valu, out, k,
                                  stream);
    if (lanes_per_row == 8)
        return launch_gather_l<8>(r, (uint32_t)n_rows, seed, passes, blocks, lds, valu, out, k,
                                  stream);
    return hipErrorInvalidValue;
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
