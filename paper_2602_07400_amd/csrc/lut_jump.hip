// One LUT layer of fan-in 5 or 6 with a node per wave (slab layout), gfx950.
//
// The function is the one of lut_layer.hip (Sec. 3 "Nodes are
// parameterizations", "Connectivity is the main per-layer design choice";
// App. C.1 "Bit-packed inference"): node j outputs entry a of its truth
// table, a = sum_i bit_s(in[conn[j][i]]) << i, for every sample s.  Here a
// whole wave evaluates one node, so the node's table is the same for all 64
// lanes and can steer control flow instead of being turned into masks:
//
//  * Shannon expansion on the three upper inputs splits the 64-entry table
//    into 8 bytes; byte t is the 3-input function g_t(x0, x1, x2) =
//    T[8t + (x0 + 2 x1 + 4 x2)].  A 3-input function with a constant truth
//    table is exactly one v_bitop3_b32 (operands x2, x1, x0, table = the
//    byte).  The truth table is an instruction immediate, so the kernel keeps
//    8 x 256 prebuilt "leaves", one per (byte position, byte value): a leaf
//    is one v_bitop3_b32 followed by an s_setpc_b64 to the next leaf.  Per
//    node, the wave jumps through the 8 leaves its table selects and comes
//    back with g_0..g_7.
//  * Three levels of multiplexers on x3, x4, x5 fold g_0..g_7 (7 more
//    v_bitop3_b32, table 0xCA).
//  Per 32 samples that is 15 VALU instructions against 63 multiplexers plus
//  the table-to-mask extraction of the per-lane layout, and 9 jumps.
//
// Mapping: a wave covers a pair of 16-word slabs (lanes 0-31: slab 2p,
// lanes 32-63: slab 2p + 1; one 32-bit half-word, 32 samples, a lane), so
// every gather is a coalesced 128-byte row segment per half wave and every
// store two whole lines.  A wave walks kJumpNodesPerWave consecutive nodes;
// the next node's 6 rows are in flight while the current one is evaluated.
// Each node's output goes to LDS, and the wave stores its nodes' outputs
// after its last gather: its vector-memory counter retires loads and stores
// in issue order, so a gather issued after a store would wait for that
// store's acknowledgement (against a store per node in the loop: C2's layer
// 1 0.651 -> 0.628 ms, C3's 0.538 -> 0.527 ms, ABBA).
// The cost is the working set: a slab pair of w_in rows is w_in * 256
// bytes per XCD, twice the per-lane layout's.  The layer is therefore used
// only where that fits the 4 MB L2 with room to spare (w_in <= 12288, e.g.
// the 9216-wire encoder outputs of the CIFAR-shaped networks); for wider
// inputs (21504 or 64000 rows) both layouts take the same time, bound by
// the gathers.
//
// Per-node records.  A prep kernel turns (conn, tables) into one 128-byte
// record per node: the 8 leaf addresses (64-bit, absolute) followed by the
// 6 row byte offsets conn * 128 within a slab.  The layer kernel reads a
// record with two scalar loads and jumps to the addresses it holds: no
// address arithmetic per node on the scalar unit.
//
// The leaves are assembled once, inside the prep kernel's code (jumped
// over there), under the hidden symbol bl_jump_leaves; both kernels sit in
// this translation unit and so in one code object, and reach the symbol
// PC-relative.  A second copy of that asm block would redefine the symbol
// and fail the build, so the addresses the prep kernel writes always point
// into the one table the layer kernel was built against.  The leaves name
// fixed registers: inputs x0..x2 in v14..v16, outputs g_t in v(20 + t),
// leaf t jumps to s[66 + 2t : 67 + 2t] (t < 7) or to the return address
// in s[80:81] (t = 7).  The layer kernel keeps exactly that assignment.
#include "bl_device.h"

namespace bl {
namespace {

constexpr int kJumpThreads = 256;
constexpr int kJumpLeafBytes = 12;                   // v_bitop3_b32 (8) + s_setpc_b64 (4)
constexpr int kJumpTableBytes = 256 * kJumpLeafBytes;
constexpr int kJumpRecWords = kJumpRecBytes / 4;

// One leaf: g = bitop3(x2, x1, x0) with truth table tt, then jump on.
#define BL_LEAF(tt, G, NEXT) "v_bitop3_b32 " G ", v16, v15, v14 bitop3:" #tt "\n" NEXT "\n"
#define BL_LEAF16(G, NEXT, h)                                                               \
    BL_LEAF(0x##h##0, G, NEXT) BL_LEAF(0x##h##1, G, NEXT) BL_LEAF(0x##h##2, G, NEXT)        \
    BL_LEAF(0x##h##3, G, NEXT) BL_LEAF(0x##h##4, G, NEXT) BL_LEAF(0x##h##5, G, NEXT)        \
    BL_LEAF(0x##h##6, G, NEXT) BL_LEAF(0x##h##7, G, NEXT) BL_LEAF(0x##h##8, G, NEXT)        \
    BL_LEAF(0x##h##9, G, NEXT) BL_LEAF(0x##h##a, G, NEXT) BL_LEAF(0x##h##b, G, NEXT)        \
    BL_LEAF(0x##h##c, G, NEXT) BL_LEAF(0x##h##d, G, NEXT) BL_LEAF(0x##h##e, G, NEXT)        \
    BL_LEAF(0x##h##f, G, NEXT)
// The 256 leaves of one byte position, in byte-value order.
#define BL_LEAF_TABLE(G, NEXT)                                                              \
    BL_LEAF16(G, NEXT, 0) BL_LEAF16(G, NEXT, 1) BL_LEAF16(G, NEXT, 2) BL_LEAF16(G, NEXT, 3) \
    BL_LEAF16(G, NEXT, 4) BL_LEAF16(G, NEXT, 5) BL_LEAF16(G, NEXT, 6) BL_LEAF16(G, NEXT, 7) \
    BL_LEAF16(G, NEXT, 8) BL_LEAF16(G, NEXT, 9) BL_LEAF16(G, NEXT, a) BL_LEAF16(G, NEXT, b) \
    BL_LEAF16(G, NEXT, c) BL_LEAF16(G, NEXT, d) BL_LEAF16(G, NEXT, e) BL_LEAF16(G, NEXT, f)

// Records of nodes [0, n_rec): nodes j >= w are padding (rows 0, and each
// leaf address the first leaf of its table, a chain that ends at the return
// address like any other; the layer kernel reads but never runs them).
// k = 5: slot 5 repeats slot 0 and the table is extended over a sixth input
// it ignores (upper half = lower half).
__global__ __launch_bounds__(kJumpThreads) void k_jump_prep(
    const int32_t *__restrict__ conn, const uint64_t *__restrict__ tables, int32_t k,
    int32_t w, uint32_t *__restrict__ rec, int32_t n_rec)
{
    uint64_t base;
    asm volatile(
        "s_getpc_b64 s[40:41]\n"
        "s_add_u32 s40, s40, bl_jump_leaves@rel32@lo+4\n"
        "s_addc_u32 s41, s41, bl_jump_leaves@rel32@hi+12\n"
        "s_mov_b64 %0, s[40:41]\n"
        "s_branch L_jump_prep_body%=\n"
        ".p2align 6\n"
        ".globl bl_jump_leaves\n"
        ".hidden bl_jump_leaves\n"
        "bl_jump_leaves:\n"
        BL_LEAF_TABLE("v20", "s_setpc_b64 s[66:67]")
        BL_LEAF_TABLE("v21", "s_setpc_b64 s[68:69]")
        BL_LEAF_TABLE("v22", "s_setpc_b64 s[70:71]")
        BL_LEAF_TABLE("v23", "s_setpc_b64 s[72:73]")
        BL_LEAF_TABLE("v24", "s_setpc_b64 s[74:75]")
        BL_LEAF_TABLE("v25", "s_setpc_b64 s[76:77]")
        BL_LEAF_TABLE("v26", "s_setpc_b64 s[78:79]")
        BL_LEAF_TABLE("v27", "s_setpc_b64 s[80:81]")
        "L_jump_prep_body%=:\n"
        : "=s"(base)
        :
        : "s40", "s41");
    const int j = blockIdx.x * kJumpThreads + threadIdx.x;
    if (j >= n_rec)
        return;
    uint32_t r[kJumpRecWords];
#pragma unroll
    for (int i = 0; i < kJumpRecWords; ++i)
        r[i] = 0;
    const bool node = j < w;
    uint64_t T = node ? tables[j] : 0;
    if (k == 5)
        T = (T & 0xFFFFFFFFull) | (T << 32);
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const uint64_t a = base + (uint64_t)(t * kJumpTableBytes) +
                           (node ? ((T >> (8 * t)) & 0xFF) * kJumpLeafBytes : 0);
        r[2 * t] = (uint32_t)a;
        r[2 * t + 1] = (uint32_t)(a >> 32);
    }
    if (node) {
#pragma unroll
        for (int i = 0; i < 6; ++i)
            r[16 + i] = (uint32_t)conn[(int64_t)j * k + (i < k ? i : 0)] * (uint32_t)(kSlabWords * 8);
    }
    u32x4 *dst = reinterpret_cast<u32x4 *>(rec + (int64_t)j * kJumpRecWords);
#pragma unroll
    for (int q = 0; q < kJumpRecWords / 4; ++q)
        dst[q] = u32x4{r[4 * q], r[4 * q + 1], r[4 * q + 2], r[4 * q + 3]};
}

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer resource over [base, base + bytes) (gfx9 layout: stride 0, 32-bit
// data format word).
__device__ __forceinline__ i32x4 buffer_rsrc(const void *base, uint32_t bytes)
{
    const uint64_t b = (uint64_t)base;
    i32x4 r;
    r.x = (int32_t)(uint32_t)b;
    r.y = (int32_t)((uint32_t)(b >> 32) & 0xFFFFu);
    r.z = (int32_t)bytes;
    r.w = 0x00020000;
    return r;
}

// Node loop of one wave (registers as in the file comment):
//   v8..v13   the next node's x0..x5 (gathered while the current one runs)
//   v14..v19  the current node's x0..x5; v20..v27 g_0..g_7, then the tree
//   s[48:55]  row offsets of the node after next; s[64:79] leaf addresses of
//             the current node; s[80:81] return address (label L_ret)
//   s45       byte offset of the current node's record, s46 of its output
//             row within the slab pair (the loop counter), s44 the end of the
//             wave's rows; the lds operand: this lane's slot for the node
// Records are read up to two past the wave's last node, which the caller's
// record array holds (kJumpPadRecs).
__global__ __launch_bounds__(kJumpThreads) void k_jump_layer(
    const uint64_t *__restrict__ in, int32_t w_in, const uint32_t *__restrict__ rec,
    int32_t w_out, uint64_t *__restrict__ out, int32_t n_nblk, int32_t n_pairs)
{
    constexpr int kRow = kSlabWords * 8;          // bytes of one row segment
    const int bid = blockIdx.x;
    const int loc = local_of(bid);
    const int pair = (loc / n_nblk) * kXcds + xcd_of(bid);
    const int nblk = loc % n_nblk;
    if (pair >= n_pairs)
        return;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int n0 = (nblk * (kJumpThreads / kWave) + wave) * kJumpNodesPerWave;
    const int cnt = min(kJumpNodesPerWave, w_out - n0);
    if (cnt <= 0)
        return;
    const char *ib = reinterpret_cast<const char *>(in) + (int64_t)pair * 2 * w_in * kRow;
    char *ob = reinterpret_cast<char *>(out) + (int64_t)pair * 2 * w_out * kRow;
    const i32x4 rin = buffer_rsrc(ib, (uint32_t)(2 * w_in * kRow));
    const uint32_t vin = (uint32_t)(lane / 32) * (uint32_t)w_in * kRow + (lane % 32) * 4u;
    const uint32_t vout = (uint32_t)(lane / 32) * (uint32_t)w_out * kRow + (lane % 32) * 4u;
    // each node's output half-word goes to LDS in the loop (ds_write, counted
    // by lgkmcnt), and the wave stores its nodes after its last gather
    __shared__ uint32_t s_out[kJumpThreads / kWave][kJumpNodesPerWave][kWave];
    uint32_t lds = (uint32_t)reinterpret_cast<uintptr_t>(&s_out[wave][0][lane]);
    const uint32_t roff = __builtin_amdgcn_readfirstlane((uint32_t)n0 * kJumpRecBytes);
    const uint32_t ooff = __builtin_amdgcn_readfirstlane((uint32_t)n0 * kRow);
    const uint32_t oend = __builtin_amdgcn_readfirstlane((uint32_t)(n0 + cnt) * kRow);
    static_assert(kJumpRecBytes == 128 && kRow == 128, "offsets below assume 128-byte records and rows");
    asm volatile(
        "s_mov_b32 s45, %[roff]\n"
        "s_mov_b32 s46, %[ooff]\n"
        "s_mov_b32 s44, %[oend]\n"
        "s_getpc_b64 s[40:41]\n"
        "L_pc%=:\n"
        "s_add_u32 s80, s40, L_ret%= - L_pc%=\n"
        "s_addc_u32 s81, s41, 0\n"
        // first node: rows, gathers, leaf addresses; rows of the second
        "s_load_dwordx8 s[48:55], %[rec], s45 offset:0x40\n"
        "s_waitcnt lgkmcnt(0)\n"
        "buffer_load_dword v8, %[vin], %[rin], s48 offen\n"
        "buffer_load_dword v9, %[vin], %[rin], s49 offen\n"
        "buffer_load_dword v10, %[vin], %[rin], s50 offen\n"
        "buffer_load_dword v11, %[vin], %[rin], s51 offen\n"
        "buffer_load_dword v12, %[vin], %[rin], s52 offen\n"
        "buffer_load_dword v13, %[vin], %[rin], s53 offen\n"
        "s_load_dwordx8 s[48:55], %[rec], s45 offset:0xc0\n"
        "s_load_dwordx16 s[64:79], %[rec], s45\n"
        "s_waitcnt vmcnt(0)\n"
        "s_branch L_first%=\n"
        // only this node's gathers are outstanding: the outputs go to LDS,
        // so no store sits ahead of a gather in the wave's vector-memory
        // counter (it retires in issue order)
        "L_node%=:\n"
        "s_waitcnt vmcnt(0)\n"
        "L_first%=:\n"
        "v_mov_b32 v14, v8\n"
        "v_mov_b32 v15, v9\n"
        "v_mov_b32 v16, v10\n"
        "v_mov_b32 v17, v11\n"
        "v_mov_b32 v18, v12\n"
        "v_mov_b32 v19, v13\n"
        "s_waitcnt lgkmcnt(0)\n"
        // the next node's gathers, then the rows of the node after it
        "buffer_load_dword v8, %[vin], %[rin], s48 offen\n"
        "buffer_load_dword v9, %[vin], %[rin], s49 offen\n"
        "buffer_load_dword v10, %[vin], %[rin], s50 offen\n"
        "buffer_load_dword v11, %[vin], %[rin], s51 offen\n"
        "buffer_load_dword v12, %[vin], %[rin], s52 offen\n"
        "buffer_load_dword v13, %[vin], %[rin], s53 offen\n"
        "s_load_dwordx8 s[48:55], %[rec], s45 offset:0x140\n"
        // g_0..g_7 through the node's 8 leaves
        "s_setpc_b64 s[64:65]\n"
        "L_ret%=:\n"
        "s_load_dwordx16 s[64:79], %[rec], s45 offset:0x80\n"
        "v_bitop3_b32 v20, v17, v21, v20 bitop3:0xca\n"
        "v_bitop3_b32 v22, v17, v23, v22 bitop3:0xca\n"
        "v_bitop3_b32 v24, v17, v25, v24 bitop3:0xca\n"
        "v_bitop3_b32 v26, v17, v27, v26 bitop3:0xca\n"
        "v_bitop3_b32 v20, v18, v22, v20 bitop3:0xca\n"
        "v_bitop3_b32 v24, v18, v26, v24 bitop3:0xca\n"
        "v_bitop3_b32 v20, v19, v24, v20 bitop3:0xca\n"
        "ds_write_b32 %[lds], v20\n"
        "v_add_u32_e32 %[lds], 0x100, %[lds]\n"
        "s_add_u32 s46, s46, 0x80\n"
        "s_add_u32 s45, s45, 0x80\n"
        "s_cmp_lg_u32 s46, s44\n"
        "s_cbranch_scc1 L_node%=\n"
        "s_waitcnt vmcnt(0) lgkmcnt(0)\n"
        : [lds] "+v"(lds)
        : [roff] "s"(roff), [ooff] "s"(ooff), [oend] "s"(oend), [rec] "s"(rec),
          [rin] "s"(rin), [vin] "v"(vin)
        : "memory", "scc", "s40", "s41", "s44", "s45", "s46", "s48", "s49", "s50", "s51", "s52",
          "s53", "s54", "s55", "s64", "s65", "s66", "s67", "s68", "s69", "s70", "s71", "s72",
          "s73", "s74", "s75", "s76", "s77", "s78", "s79", "s80", "s81", "v8", "v9", "v10",
          "v11", "v12", "v13", "v14", "v15", "v16", "v17", "v18", "v19", "v20", "v21", "v22",
          "v23", "v24", "v25", "v26", "v27");
    // the wave's outputs, one half-word a lane and node: nodes n0 .. n0 + cnt
    // are rows of the slab pair's output, 128 bytes apart
    char *o = ob + vout + (uint32_t)n0 * kRow;
    for (int i = 0; i < cnt; ++i)
        __builtin_nontemporal_store(s_out[wave][i][lane],
                                    reinterpret_cast<uint32_t *>(o + (uint32_t)i * kRow));
}

}  // namespace

bool jump_layer_fits(int32_t w_in, int32_t w_out, int32_t k, int64_t n_slabs, bool forced)
{
    if (k != 5 && k != 6)
        return false;
    if (n_slabs < 2 || n_slabs % 2 != 0)
        return false;
    if (w_in > kJumpMaxRows || w_out > kJumpMaxRows)
        return false;
    if (forced)
        return true;
    if ((int64_t)w_in * 2 * kSlabWords * 8 > kJumpMaxPairBytes)
        return false;
    const int64_t nblk = (w_out + kJumpNodesPerBlock - 1) / kJumpNodesPerBlock;
    return (n_slabs / 2) * nblk >= kJumpMinBlocks;
}

size_t jump_records_bytes(int32_t w_out)
{
    return (size_t)(w_out + kJumpPadRecs) * kJumpRecBytes;
}

hipError_t launch_jump_layer(const uint64_t *in, int32_t w_in, int64_t n_slabs,
                             const int32_t *conn, const uint64_t *tables, int32_t w_out,
                             int32_t k, uint64_t *out, uint32_t *rec, hipStream_t stream)
{
    if (!jump_layer_fits(w_in, w_out, k, n_slabs, true))
        return hipErrorInvalidValue;
    const int32_t n_rec = w_out + kJumpPadRecs;
    hipLaunchKernelGGL(k_jump_prep, dim3((n_rec + kJumpThreads - 1) / kJumpThreads),
                       dim3(kJumpThreads), 0, stream, conn, tables, k, w_out, rec, n_rec);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    const int64_t n_pairs = n_slabs / 2;
    const int32_t n_nblk = (w_out + kJumpNodesPerBlock - 1) / kJumpNodesPerBlock;
    const int64_t blocks = (n_pairs + kXcds - 1) / kXcds * kXcds * n_nblk;
    if (blocks > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_jump_layer, dim3((unsigned)blocks), dim3(kJumpThreads), 0, stream, in,
                       w_in, rec, w_out, out, n_nblk, (int32_t)n_pairs);
    return hipGetLastError();
}

}  // namespace bl
