// Device helpers shared by the kernels of libbitlogic (internal).
//
//  * bfi_asm, swap_stage, transpose64: the 64x64 bit transpose across a wave
//    that turns per-sample rows of wire bits into per-wire words of 64
//    samples (the encoders);
//  * mux_tree, subtree, eval_node: a LUT node on bit-sliced words, its 2^K
//    table entries as all-0/all-1 masks folded by K levels of bitwise
//    multiplexers (Sec. 3 "Nodes are parameterizations"; App. C.1).
#pragma once

#include "bl_internal.h"

#ifndef BL_K6_QUARTERS
#define BL_K6_QUARTERS 1
#endif
#ifndef BL_MUX_BITOP3
#define BL_MUX_BITOP3 1
#endif

namespace bl {
namespace dev {

// (sel & one) | (~sel & zero) as a single v_bfi_b32 (left to itself the
// compiler splits it into and/or with an extra inverted-mask register)
__device__ __forceinline__ uint32_t bfi_asm(uint32_t sel, uint32_t one, uint32_t zero)
{
    uint32_t r;
    asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "v"(sel), "v"(one), "v"(zero));
    return r;
}

// One block-swap stage of the 32x32 transpose inside each 32-lane half: lanes
// l and l^S exchange the S-bit blocks that sit off the diagonal.
template <int S, int K>
__device__ __forceinline__ void swap_stage(uint32_t &v, const uint32_t (&amt)[5],
                                           const uint32_t (&msk)[5])
{
    constexpr int kPattern = 0x1F | (S << 10);     // ds_swizzle bit mode: lane ^ S
    const uint32_t y = (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, kPattern);
    v = bfi_asm(msk[K], v, __builtin_amdgcn_alignbit(y, y, amt[K]));
}

// 64x64 bit transpose across a wave.  In: lane l holds bits (lo, hi) = row l.
// Out: lane p holds column p (bit l of (lo, hi) = old bit p of lane l).
__device__ __forceinline__ void transpose64(uint32_t &lo, uint32_t &hi,
                                            const uint32_t (&amt)[5], const uint32_t (&msk)[5])
{
    // off-diagonal 32x32 blocks: hi of lanes 0..31 <-> lo of lanes 32..63
    const auto sw = __builtin_amdgcn_permlane32_swap(lo, hi, false, false);
    lo = sw[0];
    hi = sw[1];
    // each register is now a 32x32 block per 32-lane half: recursive block swap
    swap_stage<16, 0>(lo, amt, msk); swap_stage<16, 0>(hi, amt, msk);
    swap_stage<8, 1>(lo, amt, msk);  swap_stage<8, 1>(hi, amt, msk);
    swap_stage<4, 2>(lo, amt, msk);  swap_stage<4, 2>(hi, amt, msk);
    swap_stage<2, 3>(lo, amt, msk);  swap_stage<2, 3>(hi, amt, msk);
    swap_stage<1, 4>(lo, amt, msk);  swap_stage<1, 4>(hi, amt, msk);
}

// Per-lane constants of transpose64: rotate amounts and merge masks of its
// five block-swap stages.
__device__ __forceinline__ void transpose_consts(int lane, uint32_t (&amt)[5], uint32_t (&msk)[5])
{
    const uint32_t low[5] = {0x0000FFFFu, 0x00FF00FFu, 0x0F0F0F0Fu, 0x33333333u, 0x55555555u};
#pragma unroll
    for (int k = 0; k < 5; ++k) {
        const int s = 16 >> k;
        const bool up = (lane & s) != 0;
        amt[k] = up ? s : 32 - s;
        msk[k] = up ? ~low[k] : low[k];
    }
}

// The bitwise multiplexer (sel & one) | (~sel & zero).  As v_bitop3_b32 with
// truth table 0xCA (bit (sel << 2 | one << 1 | zero) of the table is the
// result): chains of it sustain about 59 T lane-ops/s on gfx950 (75% of the
// 78.6 T VALU peak) in the instruction-rate probe of probes.hip, and the k = 6
// layers ran 8-10% faster with it than with v_bfi_b32.
__device__ __forceinline__ uint32_t bfi(uint32_t sel, uint32_t one, uint32_t zero)
{
#if BL_MUX_BITOP3
    return __builtin_amdgcn_bitop3_b32(sel, one, zero, 0xCA);
#else
    return (sel & one) | (~sel & zero);
#endif
}

// Fold 2^K masks with K select words: level i pairs entries that differ in
// address bit i, so the address bit order is slot 0 = least significant.
template <int K>
__device__ __forceinline__ uint32_t mux_tree(const uint32_t (&sel)[K],
                                             const uint32_t (&m)[1 << K])
{
    uint32_t v[1 << (K - 1)];
#pragma unroll
    for (int a = 0; a < (1 << (K - 1)); ++a)
        v[a] = bfi(sel[0], m[2 * a + 1], m[2 * a]);
#pragma unroll
    for (int i = 1; i < K; ++i) {
#pragma unroll
        for (int a = 0; a < (1 << (K - 1 - i)); ++a)
            v[a] = bfi(sel[i], v[2 * a + 1], v[2 * a]);
    }
    return v[0];
}

// Fold a K-input subtree whose 2^K leaf masks come from bits [base, base + 2^K)
// of the table word t (a 32-bit half of the table).
template <int K, int H>
__device__ __forceinline__ void subtree(uint32_t t, const uint32_t (&xv)[H][6], uint32_t (&o)[H])
{
    uint32_t m[1 << K];
#pragma unroll
    for (int a = 0; a < (1 << K); ++a)
        m[a] = 0u - ((t >> a) & 1u);
#pragma unroll
    for (int h = 0; h < H; ++h) {
        uint32_t sel[K];
#pragma unroll
        for (int i = 0; i < K; ++i)
            sel[i] = xv[h][i];
        o[h] = mux_tree<K>(sel, m);
    }
}

// Evaluate one node on 2R half-words (32 samples each).
template <int K, int R>
__device__ __forceinline__ void eval_node(uint64_t T, const uint32_t (&xv)[2 * R][K],
                                          uint32_t (&o)[2 * R])
{
    if constexpr (K == 6 && BL_K6_QUARTERS) {
        // Shannon split on x4 and x5: the four 4-input quarters of the table
        // are folded one after the other, so only 16 masks are live at a time
        // (the same 63 multiplexers per half-word as the split on x5 alone,
        // 16 fewer live registers; measured 2-4% faster in the LUT kernels)
        uint32_t a[2 * R], b[2 * R], r01[2 * R];
        const uint32_t t_lo = (uint32_t)T, t_hi = (uint32_t)(T >> 32);
        subtree<4, 2 * R>(t_lo, xv, a);
        __builtin_amdgcn_sched_barrier(0);
        subtree<4, 2 * R>(t_lo >> 16, xv, b);
#pragma unroll
        for (int h = 0; h < 2 * R; ++h)
            r01[h] = bfi(xv[h][4], b[h], a[h]);
        __builtin_amdgcn_sched_barrier(0);
        subtree<4, 2 * R>(t_hi, xv, a);
        __builtin_amdgcn_sched_barrier(0);
        subtree<4, 2 * R>(t_hi >> 16, xv, b);
#pragma unroll
        for (int h = 0; h < 2 * R; ++h)
            o[h] = bfi(xv[h][5], bfi(xv[h][4], b[h], a[h]), r01[h]);
    } else if constexpr (K == 6) {
        // Shannon split on x5: the two 5-input halves of the table are folded
        // one after the other, so only 32 masks are live at a time
        uint32_t lo[2 * R], hi[2 * R];
        subtree<5, 2 * R>((uint32_t)T, xv, lo);
        __builtin_amdgcn_sched_barrier(0);   // keep the two halves' masks apart
        subtree<5, 2 * R>((uint32_t)(T >> 32), xv, hi);
#pragma unroll
        for (int h = 0; h < 2 * R; ++h)
            o[h] = (xv[h][5] & hi[h]) | (~xv[h][5] & lo[h]);
    } else {
        const uint32_t t_lo = (uint32_t)T, t_hi = (uint32_t)(T >> 32);
        uint32_t m[1 << K];
#pragma unroll
        for (int a = 0; a < (1 << K); ++a)
            m[a] = 0u - (((a < 32 ? t_lo : t_hi) >> (a & 31)) & 1u);
#pragma unroll
        for (int h = 0; h < 2 * R; ++h)
            o[h] = mux_tree<K>(xv[h], m);
    }
}

}  // namespace dev
}  // namespace bl
