// One LUT layer on packed bits, gfx950.
//
// Node j outputs, for every sample s, entry a of its truth table with
// a = sum_i bit_s(in[conn[j][i]]) << i (Sec. 3 "Nodes are
// parameterizations", "Connectivity is the main per-layer design choice";
// App. C.1 "Bit-packed inference").  On packed words this is a Shannon
// expansion: the 2^k table entries become all-0 / all-1 masks and k levels
// of bitwise multiplexers, level i selected by input word i, fold them to
// one word -- 2^k - 1 v_bitop3_b32 (table 0xCA) per 32 samples, no
// per-sample work.
//
// Mapping (K = fan-in, LPN lanes per node, R words per lane):
//  * a wave holds 64/LPN nodes; the LPN lanes of a node cover a window of
//    LPN*R consecutive words (LPN*R*8 bytes of each input row);
//  * each lane evaluates R words of its node, so the 2^K masks it derives
//    from the node's table with v_bfe_i32 are reused 2R times (two 32-bit
//    halves per word);
//  * connection indices and tables of the block's NB nodes are staged in
//    LDS with coalesced loads; lanes read their node's entries from LDS.
//
// Locality: input rows are gathered at random (fixed random routing has no
// spatial locality), so the cache working set of one window is w_in rows x
// window bytes.  Windows are dealt to the 8 XCDs round-robin and each XCD
// walks all node blocks of one window before the next.  A slab of up to
// ~32k rows (4 MB at 128 bytes a row) stays in that XCD's L2 while every
// node reading it runs; a 64000-row slab (8.2 MB) does not, and its rows are
// fetched about four times from HBM and the MALL.
#include "bl_device.h"

namespace bl {
namespace {

using dev::eval_node;
using dev::mux_tree;

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;

// Access modes: whole windows with 16-byte or 8-byte accesses, or the one
// ragged last window with per-word guards.  Separate instantiations keep the
// guards out of the hot loop.
enum Mode { kFull16 = 0, kFull8 = 1, kTail = 2 };

template <int K, int LPN, int R, int NB, int MODE>
__global__ __launch_bounds__(kThreads) void k_lut_layer(
    const uint64_t *__restrict__ in, int64_t W, const int32_t *__restrict__ conn,
    const uint64_t *__restrict__ tables, int32_t w_out, uint64_t *__restrict__ out,
    int32_t n_nblk, int32_t n_win, int32_t win_base)
{
    constexpr int kGroups = kWave / LPN;                  // nodes per wave per pass
    constexpr int kPassNodes = kGroups * kWavesPerBlock;  // nodes per block per pass
    constexpr int kWin = LPN * R;                         // words per window
    static_assert(NB % kPassNodes == 0, "node block must be whole passes");
    static_assert(MODE != kFull16 || R % 2 == 0, "16-byte path needs an even R");

    __shared__ int32_t s_conn[NB * K];
    __shared__ uint64_t s_tab[NB];

    const int bid = blockIdx.x;
    const int loc = local_of(bid);
    const int win = win_base + (loc / n_nblk) * kXcds + xcd_of(bid);
    const int nblk = loc % n_nblk;
    if (win >= n_win)
        return;
    const int node0 = nblk * NB;
    const int nodes = min(NB, w_out - node0);

    for (int q = threadIdx.x; q < NB * K; q += kThreads)
        s_conn[q] = (q < nodes * K) ? conn[(int64_t)node0 * K + q] : 0;
    for (int q = threadIdx.x; q < NB; q += kThreads)
        s_tab[q] = (q < nodes) ? tables[node0 + q] : 0;
    __syncthreads();

    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    const int grp = lane / LPN;
    const int sub = lane % LPN;
    const int64_t wb0 = (int64_t)win * kWin + (int64_t)sub * R;

#pragma unroll 1
    for (int pass = 0; pass < NB / kPassNodes; ++pass) {
        if (pass * kPassNodes >= nodes)
            break;
        const int jl = pass * kPassNodes + wave * kGroups + grp;

        // gather the K input words of each of this lane's R words
        uint32_t xv[2 * R][K];
#pragma unroll
        for (int i = 0; i < K; ++i) {
            const uint64_t *src = in + (int64_t)s_conn[jl * K + i] * W + wb0;
            if constexpr (MODE == kFull16) {
#pragma unroll
                for (int r = 0; r < R; r += 2) {
                    const uint4 v = reinterpret_cast<const uint4 *>(src)[r / 2];
                    xv[2 * r + 0][i] = v.x;
                    xv[2 * r + 1][i] = v.y;
                    xv[2 * r + 2][i] = v.z;
                    xv[2 * r + 3][i] = v.w;
                }
            } else if constexpr (MODE == kFull8) {
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const uint2 v = reinterpret_cast<const uint2 *>(src)[r];
                    xv[2 * r + 0][i] = v.x;
                    xv[2 * r + 1][i] = v.y;
                }
            } else {
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    // words past the end read the row's last word (discarded)
                    const int64_t idx = min(wb0 + r, W - 1) - wb0;
                    const uint2 v = reinterpret_cast<const uint2 *>(src)[idx];
                    xv[2 * r + 0][i] = v.x;
                    xv[2 * r + 1][i] = v.y;
                }
            }
        }

        // table entries -> full-word masks (one v_bfe_i32 each)
        const uint64_t T = s_tab[jl];
        const uint32_t t_lo = (uint32_t)T, t_hi = (uint32_t)(T >> 32);
        uint32_t m[1 << K];
#pragma unroll
        for (int a = 0; a < (1 << K); ++a)
            m[a] = 0u - (((a < 32 ? t_lo : t_hi) >> (a & 31)) & 1u);

        uint32_t o[2 * R];
#pragma unroll
        for (int h = 0; h < 2 * R; ++h)
            o[h] = mux_tree<K>(xv[h], m);

        if (jl < nodes) {
            uint64_t *dst = out + (int64_t)(node0 + jl) * W + wb0;
            if constexpr (MODE == kFull16) {
#pragma unroll
                for (int r = 0; r < R; r += 2)
                    reinterpret_cast<uint4 *>(dst)[r / 2] =
                        make_uint4(o[2 * r], o[2 * r + 1], o[2 * r + 2], o[2 * r + 3]);
            } else if constexpr (MODE == kFull8) {
#pragma unroll
                for (int r = 0; r < R; ++r)
                    reinterpret_cast<uint2 *>(dst)[r] = make_uint2(o[2 * r], o[2 * r + 1]);
            } else {
#pragma unroll
                for (int r = 0; r < R; ++r)
                    if (wb0 + r < W)
                        reinterpret_cast<uint2 *>(dst)[r] = make_uint2(o[2 * r], o[2 * r + 1]);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Slab layout (used for the intermediate tensors of bitlogic_forward): the
// batch is cut into slabs of S = kSlabWords words; within a slab the rows are
// contiguous, S * 8 bytes each:
//     word (row r, column wb) at ((wb / S) * rows + r) * S + wb % S
// The LPN lanes of a node split its S words (R = S / LPN words each, loaded
// as 16-byte pieces); a block handles one slab and NB nodes, so a wave's
// stores are contiguous.  The per-XCD working set of a slab is w_in * S * 8
// bytes.  Output stores are non-temporal so the output stream does not evict
// the input slab from L2.
#ifndef BL_NT_STORE
#define BL_NT_STORE 1
#endif

template <int K, int R>
__device__ __forceinline__ void gather(const uint64_t *src, const int32_t *c, int S,
                                       uint32_t (&xv)[2 * R][K])
{
#pragma unroll
    for (int i = 0; i < K; ++i) {
        const uint64_t *p = src + (int64_t)c[i] * S;
        if constexpr (R == 1) {
            const uint2 a = *reinterpret_cast<const uint2 *>(p);
            xv[0][i] = a.x;
            xv[1][i] = a.y;
        } else {
#pragma unroll
            for (int r = 0; r < R; r += 2) {
                const u32x4 a = reinterpret_cast<const u32x4 *>(p)[r / 2];
                xv[2 * r + 0][i] = a.x;
                xv[2 * r + 1][i] = a.y;
                xv[2 * r + 2][i] = a.z;
                xv[2 * r + 3][i] = a.w;
            }
        }
    }
}

// The same gather with each row address formed as a wave-uniform slab base
// plus a 32-bit byte offset (global loads with an SGPR base: one 32-bit
// shift-add per input instead of 64-bit address arithmetic).  Used by the
// fused last layer at 5 and 6 inputs: 3-5% faster there on C3, C4 and C5
// k = 6 in ABBA runs, but 4% slower at k = 4 and 1% at k = 2; the layer
// kernel measured slower with it (1.34 against 1.25 ms on C4).
template <int K, int R>
__device__ __forceinline__ void gather_off(const char *slab_base, uint32_t lane_off,
                                           const int32_t *c, int S, uint32_t (&xv)[2 * R][K])
{
#pragma unroll
    for (int i = 0; i < K; ++i) {
        const uint64_t *p = reinterpret_cast<const uint64_t *>(
            slab_base + ((uint32_t)c[i] * (uint32_t)(S * 8) + lane_off));
        if constexpr (R == 1) {
            const uint2 a = *reinterpret_cast<const uint2 *>(p);
            xv[0][i] = a.x;
            xv[1][i] = a.y;
        } else {
#pragma unroll
            for (int r = 0; r < R; r += 2) {
                const u32x4 a = reinterpret_cast<const u32x4 *>(p)[r / 2];
                xv[2 * r + 0][i] = a.x;
                xv[2 * r + 1][i] = a.y;
                xv[2 * r + 2][i] = a.z;
                xv[2 * r + 3][i] = a.w;
            }
        }
    }
}

template <int R>
__device__ __forceinline__ void store_out(const uint32_t (&o)[2 * R], uint64_t *q, bool ok)
{
    if (ok) {
        if constexpr (R == 1) {
            const uint64_t v = (uint64_t)o[1] << 32 | o[0];
            if (BL_NT_STORE)
                __builtin_nontemporal_store(v, q);
            else
                *q = v;
        } else {
#pragma unroll
            for (int r = 0; r < R; r += 2) {
                const u32x4 v = u32x4{o[2 * r], o[2 * r + 1], o[2 * r + 2], o[2 * r + 3]};
                if (BL_NT_STORE)
                    __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(q) + r / 2);
                else
                    reinterpret_cast<u32x4 *>(q)[r / 2] = v;
            }
        }
    }
}

template <int K, int R>
__device__ __forceinline__ void eval_store(uint64_t T, const uint32_t (&xv)[2 * R][K],
                                           uint64_t *q, bool ok)
{
    uint32_t o[2 * R];
    eval_node<K, R>(T, xv, o);
    store_out<R>(o, q, ok);
}

// Specialized layers (table specialization, see specialize.hip): the nodes of
// a pass share one evaluated fan-in kp <= K, taken from the layer's fan-in
// array (one entry per kSpecPass nodes; a pass spanning several entries
// takes their maximum) and staged per pass in LDS (stage_fanin below).  kp
// is uniform over the block, so the dispatch below is a scalar branch: the
// pass gathers kp wires and runs the 2^kp - 1 multiplexer tree; kp = 0 is a
// constant node (table bit 0).
template <int KQ, int K, int R>
__device__ __forceinline__ void spec_eval(int kp, const uint64_t *src, const int32_t *c, int S,
                                          uint64_t T, uint32_t (&o)[2 * R])
{
    if constexpr (KQ == 0) {
        if (kp == 0) {
            const uint32_t m = 0u - (uint32_t)(T & 1u);
#pragma unroll
            for (int h = 0; h < 2 * R; ++h)
                o[h] = m;
            return;
        }
    } else {
        if (kp == KQ) {
            uint32_t xv[2 * R][KQ];
            gather<KQ, R>(src, c, S, xv);
            eval_node<KQ, R>(T, xv, o);
            return;
        }
    }
    if constexpr (KQ < K)
        spec_eval<KQ + 1, K, R>(kp, src, c, S, T, o);
}

// evaluated fan-in of the PN nodes from node n0: the largest entry of the
// runs of kSpecPass nodes they touch (n0 need not start a run), at most K
template <int PN, int K>
__device__ __forceinline__ int pass_fanin(const uint8_t *fanin, int32_t n_fanin, int n0)
{
    static_assert(PN % kSpecPass == 0, "passes are whole fan-in entries");
    const int e0 = n0 / kSpecPass;
    int kp = 0;
#pragma unroll
    for (int e = 0; e <= PN / kSpecPass; ++e)
        if (e0 + e < n_fanin && (e < PN / kSpecPass || n0 % kSpecPass != 0))
            kp = max(kp, (int)fanin[e0 + e]);
    return min(kp, K);
}

// A specialized block's fan-ins, staged with its connections (before the
// block's barrier): s_kp[p] = the fan-in of pass p (PN nodes from n0 + p *
// PN) for p < npass, s_kp[slot] and s_kp[slot + 1] the smallest and largest
// of them.  Wave 0 reads the passes' entries at once, a lane a pass, and
// takes the extremes with ballots; the pass loops then read their fan-in
// from LDS instead of waiting for a global load before each pass's gathers.
template <int PN, int K>
__device__ __forceinline__ void stage_fanin(const uint8_t *fanin, int32_t n_fanin, int n0,
                                            int npass, int slot, int *s_kp)
{
    if (threadIdx.x >= kWave)
        return;
    const int p = threadIdx.x;
    const int kp = p < npass ? pass_fanin<PN, K>(fanin, n_fanin, n0 + p * PN) : -1;
    if (p < npass)
        s_kp[p] = kp;
    int lo = K, hi = 0;
#pragma unroll
    for (int v = 0; v <= K; ++v)
        if (__ballot(kp == v)) {
            lo = min(lo, v);
            hi = max(hi, v);
        }
    if (p == 0) {
        s_kp[slot] = lo;
        s_kp[slot + 1] = hi;
    }
}

// In a partial node block (fewer than NB nodes; full blocks take the split
// phases below) the next pass's gathers issue at a raised wave priority, so
// that they leave ahead of other waves' evaluation: C5 layer 1 at k = 4 0.807
// -> 0.786 ms, k = 2 0.665 -> 0.660 ms when every block ran this loop (ABBA
// runs on one set of buffers).  The memory clobbers keep the loads between
// the two s_setprio.
#ifndef BL_PF_SETPRIO
#define BL_PF_SETPRIO 1
#endif
#ifndef BL_LUT_MINWAVES
#define BL_LUT_MINWAVES 1
#endif
// Up to 4 inputs, the slab kernel loads rows ahead of the evaluation: in
// full blocks the split phases below, in a partial block the next pass's
// rows while it evaluates the current pass (two register sets; C5 layer 1,
// when every block ran that loop: k = 2 0.69 -> 0.665 ms, k = 4 0.84 -> 0.81
// ms).  At 5 and 6 inputs the second set would
// cost occupancy: 4 lanes a node with prefetch need ~170 VGPRs (C4 layer 1
// 1.23 -> 1.63 ms), 8 lanes with prefetch ran 1.34 ms.
template <int K>
constexpr bool slab_prefetch()
{
    return K <= 4;
}

// A wave's vector-memory counter retires loads and stores in issue order, so
// a gather issued after a store is seen complete only once that store has
// been acknowledged, and while the output stream saturates the HBM write path
// the acknowledgements come late: a loop that stores each pass before the
// next pass's gather waits on its own stores.  A block whose NB nodes all
// exist therefore runs in two phases: every pass's rows are gathered
// (split_depth passes ahead of the evaluation, which takes each pass as its
// rows arrive) and the outputs are held in registers, then all passes are
// stored.  No load ever follows a store in the wave.  The depth trades
// registers for loads in flight: all passes up to 2 inputs, 10 at 3, 4 at 4
// (C5 layer 1, 2^18 samples into 64000 nodes: k = 2 0.642 -> 0.540 ms, k = 4
// 0.773 -> 0.669 ms; k = 1 and 3 at that shape 0.585 -> 0.498 and 0.71 ->
// 0.61 ms).  At 5 and 6 inputs the held outputs would cost occupancy (k = 6
// holding one pass: 1.21 -> 1.32 ms).  The scheduling barriers keep the
// compiler from regrouping the gathers, which shortens their distance ahead
// (k = 2 0.600 ms without them).
template <int K>
constexpr int split_depth()
{
    return K <= 2 ? 15 : K == 3 ? 10 : 4;
}

// The two phases for nodes of KP inputs whose connections are KS apart in
// s_conn (KS = KP, or the layer's fan-in for a specialized block of fan-in
// KP: the first KP slots give each node's output); KP = 0 is a constant node
// (table bit 0).
template <int KP, int KS, int R, int NPASS, int kPassNodes>
__device__ __forceinline__ void split_passes(const uint64_t *src, const int32_t *s_conn,
                                             const uint64_t *s_tab, int lnode, int S,
                                             uint64_t *dst)
{
    uint32_t o[NPASS][2 * R];
    if constexpr (KP == 0) {
#pragma unroll
        for (int p = 0; p < NPASS; ++p) {
            const uint32_t m = 0u - (uint32_t)(s_tab[p * kPassNodes + lnode] & 1u);
#pragma unroll
            for (int h = 0; h < 2 * R; ++h)
                o[p][h] = m;
        }
    } else {
        constexpr int D = split_depth<KP>() < NPASS - 1 ? split_depth<KP>() : NPASS - 1;
        uint32_t xs[D + 1][2 * R][KP];
#pragma unroll
        for (int p = 0; p < D; ++p)
            gather<KP, R>(src, &s_conn[(p * kPassNodes + lnode) * KS], S, xs[p]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int p = 0; p < NPASS; ++p) {
            if (p + D < NPASS)
                gather<KP, R>(src, &s_conn[((p + D) * kPassNodes + lnode) * KS], S,
                              xs[(p + D) % (D + 1)]);
            __builtin_amdgcn_sched_barrier(0);
            eval_node<KP, R>(s_tab[p * kPassNodes + lnode], xs[p % (D + 1)], o[p]);
            // pins the evaluation here: without it instruction selection
            // sinks every pass's evaluation to the stores, after all the
            // gathers
#pragma unroll
            for (int w = 0; w < 2 * R; ++w)
                asm volatile("" : "+v"(o[p][w]));
            __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int p = 0; p < NPASS; ++p)
        store_out<R>(o[p], dst + (int64_t)(p * kPassNodes + lnode) * S, true);
}

// split_passes at the block's fan-in kp (wave-uniform, 0 <= kp <= K).
template <int KQ, int K, int R, int NPASS, int kPassNodes>
__device__ __forceinline__ void split_passes_kp(int kp, const uint64_t *src,
                                                const int32_t *s_conn, const uint64_t *s_tab,
                                                int lnode, int S, uint64_t *dst)
{
    if (kp == KQ) {
        split_passes<KQ, K, R, NPASS, kPassNodes>(src, s_conn, s_tab, lnode, S, dst);
        return;
    }
    if constexpr (KQ < K)
        split_passes_kp<KQ + 1, K, R, NPASS, kPassNodes>(kp, src, s_conn, s_tab, lnode, S, dst);
}

template <int K, int S, int LPN, int NB, bool SPEC>
__global__ __launch_bounds__(kThreads, BL_LUT_MINWAVES) void k_lut_slab(
    const uint64_t *__restrict__ in, int32_t w_in, const int32_t *__restrict__ conn,
    const uint64_t *__restrict__ tables, int32_t w_out, uint64_t *__restrict__ out,
    int32_t n_nblk, int32_t n_slabs, const uint8_t *__restrict__ fanin)
{
    constexpr int R = S / LPN;                         // words per lane
    constexpr int kPassNodes = kThreads / LPN;
    static_assert(NB % kPassNodes == 0, "node block must be whole passes");
    static_assert(R == 1 || R % 2 == 0, "R words are loaded as 8- or 16-byte pieces");
    constexpr int kPasses = NB / kPassNodes;
    static_assert(kPasses <= kWave, "a lane per pass stages the fan-ins");
    __shared__ int32_t s_conn[NB * K];
    __shared__ uint64_t s_tab[NB];
    __shared__ int s_kp[SPEC ? kPasses + 2 : 1];

    const int bid = blockIdx.x;
    const int loc = local_of(bid);
    const int slab = (loc / n_nblk) * kXcds + xcd_of(bid);
    const int nblk = loc % n_nblk;
    if (slab >= n_slabs)
        return;
    const int node0 = nblk * NB;
    const int nodes = min(NB, w_out - node0);

    for (int q = threadIdx.x; q < NB * K; q += kThreads)
        s_conn[q] = (q < nodes * K) ? conn[(int64_t)node0 * K + q] : 0;
    for (int q = threadIdx.x; q < NB; q += kThreads)
        s_tab[q] = (q < nodes) ? tables[node0 + q] : 0;
    if constexpr (SPEC)
        stage_fanin<kPassNodes, K>(fanin, (w_out + kSpecPass - 1) / kSpecPass, node0,
                                   (nodes + kPassNodes - 1) / kPassNodes, kPasses, s_kp);
    __syncthreads();

    const int sub = threadIdx.x % LPN;
    const int lnode = threadIdx.x / LPN;
    const uint64_t *src = in + (int64_t)slab * w_in * S + sub * R;
    uint64_t *dst = out + ((int64_t)slab * w_out + node0) * S + sub * R;
    const int npass = (nodes + kPassNodes - 1) / kPassNodes;

    if constexpr (slab_prefetch<K>() && kPasses >= 2) {
        if (nodes == NB) {
            if constexpr (SPEC) {
                // a specialized block of one fan-in runs as a plain block of
                // that fan-in
                const int kmin = __builtin_amdgcn_readfirstlane(s_kp[kPasses]);
                const int kmax = __builtin_amdgcn_readfirstlane(s_kp[kPasses + 1]);
                if (kmin == kmax) {
                    split_passes_kp<0, K, R, kPasses, kPassNodes>(kmax, src, s_conn, s_tab, lnode,
                                                                  S, dst);
                    return;
                }
            } else {
                split_passes<K, K, R, kPasses, kPassNodes>(src, s_conn, s_tab, lnode, S, dst);
                return;
            }
        }
    }
    if constexpr (!SPEC && slab_prefetch<K>()) {
        // a partial block: two register sets, the next pass's rows are in
        // flight while this pass is evaluated
        uint32_t xa[2 * R][K], xb[2 * R][K];
        if (npass > 0)
            gather<K, R>(src, &s_conn[lnode * K], S, xa);
#pragma unroll 1
        for (int pass = 0; pass < npass; pass += 2) {
            const int jl = pass * kPassNodes + lnode;
            const int jl1 = jl + kPassNodes;
            if (pass + 1 < npass) {
                if (BL_PF_SETPRIO)
                    asm volatile("s_setprio 2" ::: "memory");
                gather<K, R>(src, &s_conn[jl1 * K], S, xb);
                if (BL_PF_SETPRIO)
                    asm volatile("s_setprio 0" ::: "memory");
            }
            eval_store<K, R>(s_tab[jl], xa, dst + (int64_t)jl * S, jl < nodes);
            if (pass + 1 < npass) {
                if (pass + 2 < npass) {
                    if (BL_PF_SETPRIO)
                        asm volatile("s_setprio 2" ::: "memory");
                    gather<K, R>(src, &s_conn[(jl1 + kPassNodes) * K], S, xa);
                    if (BL_PF_SETPRIO)
                        asm volatile("s_setprio 0" ::: "memory");
                }
                eval_store<K, R>(s_tab[jl1], xb, dst + (int64_t)jl1 * S, jl1 < nodes);
            }
        }
        return;
    }
#pragma unroll 1
    for (int pass = 0; pass < npass; ++pass) {
        const int jl = pass * kPassNodes + lnode;
        if constexpr (SPEC) {
            const int kp = __builtin_amdgcn_readfirstlane(s_kp[pass]);
            uint32_t o[2 * R];
            spec_eval<0, K, R>(kp, src, &s_conn[jl * K], S, s_tab[jl], o);
            store_out<R>(o, dst + (int64_t)jl * S, jl < nodes);
        } else {
            uint32_t xv[2 * R][K];
            gather<K, R>(src, &s_conn[jl * K], S, xv);
            eval_store<K, R>(s_tab[jl], xv, dst + (int64_t)jl * S, jl < nodes);
        }
    }
}

// Nodes per block: 512 (8 passes over one staging of connections and
// tables) when the launch has blocks to spare; one pass per block when the
// batch is so small that 512-node blocks would leave most CUs idle and each
// block's passes would run one gather latency after another.
constexpr int kSlabNB = 512;
constexpr int64_t kSlabSmallBlocks = 2048;

// Lanes per node: 4 (8 half-words each) for 5 and 6 inputs, where the masks'
// reuse matters; 8 (one full 128-byte line per node in each gather
// instruction) for up to 4 inputs, whose layers are bound by the gathers'
// L1-miss path rather than the VALU (C5: layer 1 5% faster at k = 2, 2.5%
// at k = 4; 4% slower at k = 6).
template <int K>
constexpr int slab_lanes()
{
    return K <= 4 ? 8 : kSlabLanes;
}

template <int K, int NB>
hipError_t launch_slab_kn(const uint64_t *in, int32_t w_in, int64_t n_slabs,
                          const int32_t *conn, const uint64_t *tables, int32_t w_out,
                          uint64_t *out, const uint8_t *fanin, hipStream_t stream)
{
    const int32_t n_nblk = (w_out + NB - 1) / NB;
    const int64_t slabs_pad = (n_slabs + kXcds - 1) / kXcds * kXcds;
    const int64_t blocks = slabs_pad * n_nblk;
    if (blocks > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    if (fanin)
        hipLaunchKernelGGL((k_lut_slab<K, kSlabWords, slab_lanes<K>(), NB, true>),
                           dim3((unsigned)blocks), dim3(kThreads), 0, stream, in, w_in, conn,
                           tables, w_out, out, n_nblk, (int32_t)n_slabs, fanin);
    else
        hipLaunchKernelGGL((k_lut_slab<K, kSlabWords, slab_lanes<K>(), NB, false>),
                           dim3((unsigned)blocks), dim3(kThreads), 0, stream, in, w_in, conn,
                           tables, w_out, out, n_nblk, (int32_t)n_slabs, fanin);
    return hipGetLastError();
}

template <int K>
hipError_t launch_slab_k(const uint64_t *in, int32_t w_in, int64_t n_slabs,
                         const int32_t *conn, const uint64_t *tables, int32_t w_out,
                         uint64_t *out, const uint8_t *fanin, hipStream_t stream)
{
    const int64_t big = n_slabs * ((w_out + kSlabNB - 1) / kSlabNB);
    if (big < kSlabSmallBlocks)     // one pass per block
        return launch_slab_kn<K, kThreads / slab_lanes<K>()>(in, w_in, n_slabs, conn, tables,
                                                             w_out, out, fanin, stream);
    return launch_slab_kn<K, kSlabNB>(in, w_in, n_slabs, conn, tables, w_out, out, fanin,
                                      stream);
}

// ---------------------------------------------------------------------------
// Last LUT layer fused with the GroupSum head (Sec. 3 "Encoders and heads";
// Sec. 5 "Head").  Instead of storing the last layer's bits, every block
// counts them: its NB nodes lie inside one class group, each lane adds the
// output bits of the nodes it evaluates into bit-sliced counters (plane p =
// bit p of 32 per-sample counts per half-word), and at the end the block's
// lanes are summed through LDS and ds_swizzle into the same per-column bit
// planes ([column][class][split][plane], split = block within the class)
// that the head's finish kernel turns into scores and argmax.  The last
// layer's output tensor is never written or read back.
//
// Mapping: slab width 16 words; 4 lanes share a node (4 words = 8 half-words
// each, 64 nodes per pass of the 256-thread block, at most 15 passes per
// block, 4 counter planes), so each node's 64 table masks serve 8 half-words.
// A class group of g nodes is split into ceil(g / nb) blocks of nb nodes (a
// multiple of 64); the last block of a group, and its last pass, may be
// short: its padding nodes get connections 0 and a constant-0 table, so they
// evaluate to 0 and add nothing to the counters.  A C4 class group of 640
// nodes is one block, so the finish reads one counter per class.  The kernel
// is held to 128 VGPRs (4 waves per SIMD; it takes 126 at K = 6, with no
// spills).
#ifndef BL_HEAD_CP
#define BL_HEAD_CP 4
#endif
#ifndef BL_HEAD_MINWAVES
#define BL_HEAD_MINWAVES 4
#endif
constexpr int kHeadLPN = 4;
constexpr int kHeadR = kSlabWords / kHeadLPN;
constexpr int kHeadPassNodes = kThreads / kHeadLPN;          // 64
constexpr int kHeadCP = BL_HEAD_CP;                          // counter planes
constexpr int kHeadMaxPasses = (1 << BL_HEAD_CP) - 1;         // passes per block
constexpr int kHeadHalves = 2 * kSlabWords;                  // 32 half-words per slab

// Bit-sliced counter ctr (CP planes) += one bit per lane of o, ripple carry,
// two planes per step with 3-input v_bitop3_b32 (operand S0 is the most
// significant bit of the truth-table index): with carry k into plane p,
//   k'      = c[p] & c[p+1] & k          (table 0x80)
//   c[p+1] ^= c[p] & k                   (table 0x78, old c[p])
//   c[p]   ^= k
// 3 ops per pair of planes, 2 for a top pair, 1 for an odd top plane (4
// planes: 5 ops instead of 7).  Each plane is updated in place (a tied asm
// operand), so the counters keep their registers from one pass to the next
// instead of being rotated by moves at the loop edge.
template <int CP>
__device__ __forceinline__ void bs_count(uint32_t (&ctr)[CP], uint32_t o)
{
    uint32_t k = o;
#pragma unroll
    for (int p = 0; p + 1 < CP; p += 2) {
        if (p + 2 < CP) {
            uint32_t kn;
            asm("v_bitop3_b32 %2, %0, %1, %3 bitop3:0x80\n\t"
                "v_bitop3_b32 %1, %1, %0, %3 bitop3:0x78\n\t"
                "v_xor_b32 %0, %0, %3"
                : "+v"(ctr[p]), "+v"(ctr[p + 1]), "=&v"(kn)
                : "v"(k));
            k = kn;
        } else {
            asm("v_bitop3_b32 %1, %1, %0, %2 bitop3:0x78\n\t"
                "v_xor_b32 %0, %0, %2"
                : "+v"(ctr[p]), "+v"(ctr[p + 1])
                : "v"(k));
        }
    }
    if constexpr (CP % 2 == 1)
        asm("v_xor_b32 %0, %0, %1" : "+v"(ctr[CP - 1]) : "v"(k));
}

// acc (NP planes) += v (NQ planes), bit-sliced ripple carry
template <int NP, int NQ>
__device__ __forceinline__ void bs_add(uint32_t (&acc)[NP], const uint32_t (&v)[NQ])
{
    uint32_t carry = 0;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        const uint32_t b = (p < NQ) ? v[p < NQ ? p : 0] : 0u;
        const uint32_t a = acc[p];
        acc[p] = a ^ b ^ carry;
        carry = (a & b) | (carry & (a ^ b));
    }
}

// The specialized kernel at 6 inputs dispatches over every fan-in up to 6 and
// does not fit 128 VGPRs: held to 4 waves per SIMD it spilled 80 bytes per
// lane and its layer ran 2.00 ms on C4 forced through it, against 1.50 ms at
// 3 waves per SIMD (138 VGPRs, no spills; ABBA runs).
template <int K, bool SPEC>
constexpr int head_min_waves()
{
    return (SPEC && K == 6) ? 3 : BL_HEAD_MINWAVES;
}

// The fused layer's pass loop for nodes of KP inputs whose connections are
// KS apart in s_conn (KS = KP, or the layer's fan-in for a specialized block
// of fan-in KP); KP = 0 is a constant node (table bit 0).  Each pass's output
// bits go into the lane's bit-sliced counters.
template <int KP, int KS>
__device__ __forceinline__ void head_passes(int passes, const uint64_t *src,
                                            const char *slab_base, uint32_t lane_off, bool off32,
                                            const int32_t *s_conn, const uint64_t *s_tab,
                                            int lnode, uint32_t (&ctr)[2 * kHeadR][kHeadCP])
{
    // Up to 4 inputs the next pass's rows are in flight while this pass is
    // evaluated and counted (two register sets, 87-128 VGPRs; the loop taken
    // two passes at a time so that the compiler can count the outstanding
    // gathers): C5's fused layer at k = 2 0.487 -> 0.474 ms, k = 4 0.768 ->
    // 0.749 ms (ABBA, four alternations).  At 5 and 6 inputs the second set
    // costs occupancy (C4's fused layer 1.91 against 1.25 ms).
    if constexpr (KP >= 1 && KP <= 4) {
        auto gat = [&](int pass, uint32_t (&xv)[2 * kHeadR][KP]) {
            gather<KP, kHeadR>(src, &s_conn[(pass * kHeadPassNodes + lnode) * KS], kSlabWords, xv);
        };
        auto run = [&](int pass, const uint32_t (&xv)[2 * kHeadR][KP]) {
            uint32_t o[2 * kHeadR];
            eval_node<KP, kHeadR>(s_tab[pass * kHeadPassNodes + lnode], xv, o);
#pragma unroll
            for (int h = 0; h < 2 * kHeadR; ++h)
                bs_count<kHeadCP>(ctr[h], o[h]);
        };
        uint32_t xa[2 * kHeadR][KP], xb[2 * kHeadR][KP];
        gat(0, xa);
        int pass = 0;
#pragma unroll 1
        for (; pass + 2 < passes; pass += 2) {
            gat(pass + 1, xb);
            run(pass, xa);
            gat(pass + 2, xa);
            run(pass + 1, xb);
        }
        if (pass + 1 < passes) {
            gat(pass + 1, xb);
            run(pass, xa);
            run(pass + 1, xb);
        } else {
            run(pass, xa);
        }
        return;
    }
#pragma unroll 1
    for (int pass = 0; pass < passes; ++pass) {
        const int jl = pass * kHeadPassNodes + lnode;
        uint32_t o[2 * kHeadR];
        if constexpr (KP == 0) {
            const uint32_t m = 0u - (uint32_t)(s_tab[jl] & 1u);
#pragma unroll
            for (int h = 0; h < 2 * kHeadR; ++h)
                o[h] = m;
        } else {
            uint32_t xv[2 * kHeadR][KP];
            if (KP >= 5 && off32)
                gather_off<KP, kHeadR>(slab_base, lane_off, &s_conn[jl * KS], kSlabWords, xv);
            else
                gather<KP, kHeadR>(src, &s_conn[jl * KS], kSlabWords, xv);
            eval_node<KP, kHeadR>(s_tab[jl], xv, o);
        }
#pragma unroll
        for (int h = 0; h < 2 * kHeadR; ++h)
            bs_count<kHeadCP>(ctr[h], o[h]);
    }
}

// head_passes at fan-in kp (wave-uniform, 0 <= kp <= K).
template <int KQ, int K>
__device__ __forceinline__ void head_passes_kp(int kp, int passes, const uint64_t *src,
                                               const char *slab_base, uint32_t lane_off,
                                               bool off32, const int32_t *s_conn,
                                               const uint64_t *s_tab, int lnode,
                                               uint32_t (&ctr)[2 * kHeadR][kHeadCP])
{
    if (kp == KQ) {
        head_passes<KQ, K>(passes, src, slab_base, lane_off, off32, s_conn, s_tab, lnode, ctr);
        return;
    }
    if constexpr (KQ < K)
        head_passes_kp<KQ + 1, K>(kp, passes, src, slab_base, lane_off, off32, s_conn, s_tab,
                                  lnode, ctr);
}

template <int K, int P, bool SPEC>
__global__ __launch_bounds__(kThreads, (head_min_waves<K, SPEC>())) void k_lut_slab_head(
    const uint64_t *__restrict__ in, int32_t w_in, const int32_t *__restrict__ conn,
    const uint64_t *__restrict__ tables, int32_t g, int32_t nb, int32_t n_nblk,
    int32_t n_slabs, int64_t W, int32_t c, int32_t splits, uint64_t *__restrict__ planes,
    const uint8_t *__restrict__ fanin)
{
    static_assert(kSlabWords == 16 && kSlabWords == kHeadLPN * kHeadR, "slab of 16 words");
    static_assert(P >= kHeadCP, "final planes hold the per-lane counters");
    static_assert(kHeadPassNodes % 8 == 0, "8 threads per half-word sum the node lanes");
    // connections and tables while the nodes run, then the counter reduction
    constexpr int kStageBytes = kHeadMaxPasses * kHeadPassNodes * (K * 4 + 8);
    constexpr int kRedBytes = kHeadHalves * kHeadPassNodes * kHeadCP * 4;
    __shared__ __attribute__((aligned(16))) uint8_t s_mem[kStageBytes > kRedBytes ? kStageBytes
                                                                                  : kRedBytes];
    uint64_t *s_tab = reinterpret_cast<uint64_t *>(s_mem);
    int32_t *s_conn = reinterpret_cast<int32_t *>(s_mem + kHeadMaxPasses * kHeadPassNodes * 8);
    auto s_red = reinterpret_cast<uint32_t (*)[kHeadPassNodes][kHeadCP]>(s_mem);
    static_assert(kHeadMaxPasses <= kWave, "a lane per pass stages the fan-ins");
    __shared__ int s_kp[SPEC ? kHeadMaxPasses + 2 : 1];

    const int bid = blockIdx.x;
    const int loc = local_of(bid);
    const int slab = (loc / n_nblk) * kXcds + xcd_of(bid);
    const int nblk = loc % n_nblk;
    if (slab >= n_slabs)
        return;
    const int cls = nblk / splits;               // one class per block
    const int split = nblk % splits;
    const int nodes = min(nb, g - split * nb);   // the group's last block may be short
    const int node0 = cls * g + split * nb;
    const int passes = (nodes + kHeadPassNodes - 1) / kHeadPassNodes;

    // padding nodes of a short last pass: wire 0 and the constant-0 table
    const int staged = passes * kHeadPassNodes;
    for (int q = threadIdx.x; q < staged * K; q += kThreads)
        s_conn[q] = q < nodes * K ? conn[(int64_t)node0 * K + q] : 0;
    for (int q = threadIdx.x; q < staged; q += kThreads)
        s_tab[q] = q < nodes ? tables[node0 + q] : 0;
    if constexpr (SPEC)
        stage_fanin<kHeadPassNodes, K>(fanin, (g * c + kSpecPass - 1) / kSpecPass, node0, passes,
                                       kHeadMaxPasses, s_kp);
    __syncthreads();

    const int sub = threadIdx.x % kHeadLPN;
    const int lnode = threadIdx.x / kHeadLPN;
    const uint64_t *src = in + (int64_t)slab * w_in * kSlabWords + sub * kHeadR;
    const char *slab_base = reinterpret_cast<const char *>(in + (int64_t)slab * w_in * kSlabWords);
    const uint32_t lane_off = (uint32_t)(sub * kHeadR * 8);
    // a slab's rows span w_in * 128 bytes: 32-bit offsets while that fits
    const bool off32 = (int64_t)w_in * kSlabWords * 8 <= 0xFFFFFFFFll;

    uint32_t ctr[2 * kHeadR][kHeadCP];
#pragma unroll
    for (int h = 0; h < 2 * kHeadR; ++h)
#pragma unroll
        for (int p = 0; p < kHeadCP; ++p)
            ctr[h][p] = 0;
    int kmin = K, kmax = K;
    if constexpr (SPEC) {
        kmin = __builtin_amdgcn_readfirstlane(s_kp[kHeadMaxPasses]);
        kmax = __builtin_amdgcn_readfirstlane(s_kp[kHeadMaxPasses + 1]);
    }
    if constexpr (!SPEC && K >= 5) {
        // the plain loop of 5 and 6 inputs written out here rather than
        // through head_passes: the same instructions, but the helper's loop
        // entry moved the register allocation, and C3's fused layer (k = 6)
        // measured 2% slower with it (ABBA)
#pragma unroll 1
        for (int pass = 0; pass < passes; ++pass) {
            const int jl = pass * kHeadPassNodes + lnode;
            uint32_t o[2 * kHeadR];
            uint32_t xv[2 * kHeadR][K];
            if (off32)
                gather_off<K, kHeadR>(slab_base, lane_off, &s_conn[jl * K], kSlabWords, xv);
            else
                gather<K, kHeadR>(src, &s_conn[jl * K], kSlabWords, xv);
            eval_node<K, kHeadR>(s_tab[jl], xv, o);
#pragma unroll
            for (int h = 0; h < 2 * kHeadR; ++h)
                bs_count<kHeadCP>(ctr[h], o[h]);
        }
    } else if constexpr (!SPEC) {
        head_passes<K, K>(passes, src, slab_base, lane_off, off32, s_conn, s_tab, lnode, ctr);
    } else if (kmin == kmax) {
        // a specialized block of one fan-in runs the plain loop of that fan-in
        head_passes_kp<0, K>(kmax, passes, src, slab_base, lane_off, off32, s_conn, s_tab, lnode,
                             ctr);
    } else {
#pragma unroll 1
        for (int pass = 0; pass < passes; ++pass) {
            const int jl = pass * kHeadPassNodes + lnode;
            uint32_t o[2 * kHeadR];
            const int kp = __builtin_amdgcn_readfirstlane(s_kp[pass]);
            spec_eval<0, K, kHeadR>(kp, src, &s_conn[jl * K], kSlabWords, s_tab[jl], o);
#pragma unroll
            for (int h = 0; h < 2 * kHeadR; ++h)
                bs_count<kHeadCP>(ctr[h], o[h]);
        }
    }

    // lane counters -> LDS (over the staging area), one row of 32 node lanes
    // per half-word
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2 * kHeadR; ++h)
#pragma unroll
        for (int p = 0; p < kHeadCP; ++p)
            s_red[sub * 2 * kHeadR + h][lnode][p] = ctr[h][p];
    __syncthreads();

    // thread t sums PN/8 node lanes of half-word t/8; the 8 threads of a
    // half-word then combine with xor swizzles over lanes 1, 2, 4
    constexpr int kPerThread = kHeadPassNodes / 8;
    const int hw = threadIdx.x / 8;
    const int part = threadIdx.x % 8;
    uint32_t acc[P];
#pragma unroll
    for (int p = 0; p < P; ++p)
        acc[p] = 0;
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) {
        uint32_t v[kHeadCP];
#pragma unroll
        for (int p = 0; p < kHeadCP; ++p)
            v[p] = s_red[hw][part * kPerThread + q][p];
        bs_add<P, kHeadCP>(acc, v);
    }
    {
        uint32_t v[P];
#pragma unroll
        for (int p = 0; p < P; ++p)
            v[p] = (uint32_t)__builtin_amdgcn_ds_swizzle((int)acc[p], 0x1F | (1 << 10));
        bs_add<P, P>(acc, v);
#pragma unroll
        for (int p = 0; p < P; ++p)
            v[p] = (uint32_t)__builtin_amdgcn_ds_swizzle((int)acc[p], 0x1F | (2 << 10));
        bs_add<P, P>(acc, v);
#pragma unroll
        for (int p = 0; p < P; ++p)
            v[p] = (uint32_t)__builtin_amdgcn_ds_swizzle((int)acc[p], 0x1F | (4 << 10));
        bs_add<P, P>(acc, v);
    }
    // half-words 2m and 2m+1 (8 lanes apart) form word m of the slab
    uint32_t odd[P];
#pragma unroll
    for (int p = 0; p < P; ++p)
        odd[p] = (uint32_t)__builtin_amdgcn_ds_swizzle((int)acc[p], 0x1F | (8 << 10));
    const int64_t col = (int64_t)slab * kSlabWords + hw / 2;
    if (part == 0 && (hw % 2) == 0 && col < W) {
        uint64_t *dst = planes + ((col * c + cls) * (int64_t)splits + split) * P;
#pragma unroll
        for (int p = 0; p < P; ++p)
            dst[p] = ((uint64_t)odd[p] << 32) | acc[p];
    }
}

template <int K, int P>
hipError_t launch_slab_head_kp(const uint64_t *in, int32_t w_in, int64_t n_slabs,
                               const int32_t *conn, const uint64_t *tables, int32_t w_out,
                               int32_t g, int32_t nb, int64_t W, int32_t c, uint64_t *planes,
                               const uint8_t *fanin, hipStream_t stream)
{
    if (nb <= 0 || nb % kHeadPassNodes != 0 || nb / kHeadPassNodes > kHeadMaxPasses || g <= 0)
        return hipErrorInvalidValue;
    const int32_t splits = (g + nb - 1) / nb;
    const int64_t n_nblk = (int64_t)c * splits;
    const int64_t slabs_pad = (n_slabs + kXcds - 1) / kXcds * kXcds;
    const int64_t blocks = slabs_pad * n_nblk;
    if (blocks > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    if (fanin)
        hipLaunchKernelGGL((k_lut_slab_head<K, P, true>), dim3((unsigned)blocks), dim3(kThreads),
                           0, stream, in, w_in, conn, tables, g, nb, (int32_t)n_nblk,
                           (int32_t)n_slabs, W, c, splits, planes, fanin);
    else
        hipLaunchKernelGGL((k_lut_slab_head<K, P, false>), dim3((unsigned)blocks),
                           dim3(kThreads), 0, stream, in, w_in, conn, tables, g, nb,
                           (int32_t)n_nblk, (int32_t)n_slabs, W, c, splits, planes, fanin);
    return hipGetLastError();
}

template <int K>
hipError_t launch_slab_head_k(const uint64_t *in, int32_t w_in, int64_t n_slabs,
                              const int32_t *conn, const uint64_t *tables, int32_t w_out,
                              int32_t g, int32_t nb, int32_t P, int64_t W, int32_t c,
                              uint64_t *planes, const uint8_t *fanin, hipStream_t stream)
{
    switch (P) {
    case 6: return launch_slab_head_kp<K, 6>(in, w_in, n_slabs, conn, tables, w_out, g, nb, W, c, planes, fanin, stream);
    case 7: return launch_slab_head_kp<K, 7>(in, w_in, n_slabs, conn, tables, w_out, g, nb, W, c, planes, fanin, stream);
    case 8: return launch_slab_head_kp<K, 8>(in, w_in, n_slabs, conn, tables, w_out, g, nb, W, c, planes, fanin, stream);
    case 9: return launch_slab_head_kp<K, 9>(in, w_in, n_slabs, conn, tables, w_out, g, nb, W, c, planes, fanin, stream);
    case 10: return launch_slab_head_kp<K, 10>(in, w_in, n_slabs, conn, tables, w_out, g, nb, W, c, planes, fanin, stream);
    default: return hipErrorInvalidValue;
    }
}

constexpr int kLPN = 4;
constexpr int kR = 4;
constexpr int kNB = 256;

template <int K, int MODE>
hipError_t launch_mode(const uint64_t *in, int64_t W, const int32_t *conn,
                       const uint64_t *tables, int32_t w_out, uint64_t *out,
                       int64_t win_base, int64_t n_win, hipStream_t stream)
{
    const int32_t n_nblk = (w_out + kNB - 1) / kNB;
    const int64_t span = n_win - win_base;
    const int64_t span_pad = (span + kXcds - 1) / kXcds * kXcds;
    const int64_t blocks = span_pad * n_nblk;
    if (blocks > 0x7fffffff || n_win > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((k_lut_layer<K, kLPN, kR, kNB, MODE>), dim3((unsigned)blocks),
                       dim3(kThreads), 0, stream, in, W, conn, tables, w_out, out, n_nblk,
                       (int32_t)n_win, (int32_t)win_base);
    return hipGetLastError();
}

template <int K>
hipError_t launch_k(const uint64_t *in, int64_t W, const int32_t *conn,
                    const uint64_t *tables, int32_t w_out, uint64_t *out,
                    hipStream_t stream)
{
    constexpr int kWin = kLPN * kR;
    const int64_t n_full = W / kWin;
    hipError_t e = hipSuccess;
    if (n_full > 0) {
        const bool vec16 = (W % 2 == 0) && ((uintptr_t)in % 16 == 0) &&
                           ((uintptr_t)out % 16 == 0);
        e = vec16 ? launch_mode<K, kFull16>(in, W, conn, tables, w_out, out, 0, n_full, stream)
                  : launch_mode<K, kFull8>(in, W, conn, tables, w_out, out, 0, n_full, stream);
        if (e != hipSuccess)
            return e;
    }
    if (W % kWin != 0)
        e = launch_mode<K, kTail>(in, W, conn, tables, w_out, out, n_full, n_full + 1, stream);
    return e;
}

}  // namespace

hipError_t launch_lut_layer_slab(const uint64_t *in, int32_t w_in, int64_t n_slabs,
                                 const int32_t *conn, const uint64_t *tables, int32_t w_out,
                                 int32_t k, uint64_t *out, hipStream_t stream,
                                 const uint8_t *fanin)
{
    switch (k) {
    case 1: return launch_slab_k<1>(in, w_in, n_slabs, conn, tables, w_out, out, fanin, stream);
    case 2: return launch_slab_k<2>(in, w_in, n_slabs, conn, tables, w_out, out, fanin, stream);
    case 3: return launch_slab_k<3>(in, w_in, n_slabs, conn, tables, w_out, out, fanin, stream);
    case 4: return launch_slab_k<4>(in, w_in, n_slabs, conn, tables, w_out, out, fanin, stream);
    case 5: return launch_slab_k<5>(in, w_in, n_slabs, conn, tables, w_out, out, fanin, stream);
    case 6: return launch_slab_k<6>(in, w_in, n_slabs, conn, tables, w_out, out, fanin, stream);
    default: return hipErrorInvalidValue;
    }
}

int32_t fused_head_nodes(int32_t g, int32_t c, int64_t n_slabs)
{
    if (kSlabWords != 16 || g <= 0 || c <= 0)
        return 0;
    const int32_t units = (g + kHeadPassNodes - 1) / kHeadPassNodes;
    // small batches: fewer passes per block until the launch has
    // kSlabSmallBlocks blocks (n_slabs * c * ceil(units / p) of them)
    int max_p = kHeadMaxPasses;
    while (max_p > 1 &&
           n_slabs * c * (int64_t)((units + max_p - 1) / max_p) < kSlabSmallBlocks)
        --max_p;
    // whole blocks of equal size when a divisor of the passes allows it (it
    // measured faster than fewer, longer blocks: C5's 100 passes as 10 x 10
    // against 6 x 15 + 10), else the fewest blocks with balanced passes
    for (int p = max_p; 2 * p >= max_p; --p)
        if (units % p == 0)
            return p * kHeadPassNodes;
    const int32_t splits = (units + max_p - 1) / max_p;
    return (units + splits - 1) / splits * kHeadPassNodes;
}

hipError_t launch_lut_slab_head(const uint64_t *in, int32_t w_in, int64_t n_slabs,
                                const int32_t *conn, const uint64_t *tables, int32_t w_out,
                                int32_t k, int32_t c, int64_t W, uint64_t *planes, int32_t P,
                                hipStream_t stream, const uint8_t *fanin)
{
    const int32_t g = w_out / c;
    const int32_t nb = fused_head_nodes(g, c, n_slabs);
    if (nb == 0)
        return hipErrorInvalidValue;
    switch (k) {
    case 1: return launch_slab_head_k<1>(in, w_in, n_slabs, conn, tables, w_out, g, nb, P, W, c, planes, fanin, stream);
    case 2: return launch_slab_head_k<2>(in, w_in, n_slabs, conn, tables, w_out, g, nb, P, W, c, planes, fanin, stream);
    case 3: return launch_slab_head_k<3>(in, w_in, n_slabs, conn, tables, w_out, g, nb, P, W, c, planes, fanin, stream);
    case 4: return launch_slab_head_k<4>(in, w_in, n_slabs, conn, tables, w_out, g, nb, P, W, c, planes, fanin, stream);
    case 5: return launch_slab_head_k<5>(in, w_in, n_slabs, conn, tables, w_out, g, nb, P, W, c, planes, fanin, stream);
    case 6: return launch_slab_head_k<6>(in, w_in, n_slabs, conn, tables, w_out, g, nb, P, W, c, planes, fanin, stream);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_lut_layer(const uint64_t *in, int32_t w_in, int64_t n_words,
                            const int32_t *conn, const uint64_t *tables,
                            int32_t w_out, int32_t k, uint64_t *out,
                            hipStream_t stream)
{
    (void)w_in;
    switch (k) {
    case 1: return launch_k<1>(in, n_words, conn, tables, w_out, out, stream);
    case 2: return launch_k<2>(in, n_words, conn, tables, w_out, out, stream);
    case 3: return launch_k<3>(in, n_words, conn, tables, w_out, out, stream);
    case 4: return launch_k<4>(in, n_words, conn, tables, w_out, out, stream);
    case 5: return launch_k<5>(in, n_words, conn, tables, w_out, out, stream);
    case 6: return launch_k<6>(in, n_words, conn, tables, w_out, out, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace bl
