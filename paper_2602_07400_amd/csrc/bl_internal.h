// Library-internal declarations shared by the kernel translation units and
// the C-ABI front end.  Nothing here is part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace bl {

constexpr int kWave = 64;       // CDNA wavefront width
constexpr int kXcds = 8;        // MI355X: 8 accelerator dies, each with its own L2
#ifndef BL_SLAB_WORDS
#define BL_SLAB_WORDS 16
#endif
#ifndef BL_SLAB_LPN
#define BL_SLAB_LPN 4
#endif
// Words per row segment in the slab layout (BL_SLAB_WORDS * 64 samples) and
// lanes that share one node's segment in the slab LUT kernel.
constexpr int kSlabWords = BL_SLAB_WORDS;
constexpr int kSlabLanes = BL_SLAB_LPN;
static_assert(kSlabWords % kSlabLanes == 0, "each lane takes whole words");

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Layouts of packed bit tensors: row-major [rows][W] (the public calls) or
// slabs (bitlogic_forward's intermediates in its workspace).
constexpr int kLayoutRowMajor = 0;
constexpr int kLayoutSlab = 1;

// Word (row r, column wb) of a packed tensor with `rows` rows in the slab
// layout of bitlogic_forward's intermediates, [W / kSlabWords][rows][kSlabWords].
__host__ __device__ inline int64_t slab_index(int64_t r, int64_t wb, int64_t rows)
{
    return ((wb / kSlabWords) * rows + r) * kSlabWords + (wb % kSlabWords);
}

// Workgroups are dealt to the XCDs round-robin by workgroup id.  These helpers
// turn a linear id into (xcd, index within that xcd).
__device__ __forceinline__ int xcd_of(int bid) { return bid % kXcds; }
__device__ __forceinline__ int local_of(int bid) { return bid / kXcds; }

// ---- launchers (each returns the hipError_t of its launch) ----

// Encoder into either layout; W_cols = columns (words) to write: W for the
// row-major layout, W rounded up to whole slabs for the slab layout (columns
// past the batch get zero bits).
// kind: kEncThermometer (thresholds [d][b]) or kEncBinary (b <= 8, thresholds
// unused).
constexpr int kEncThermometer = 0;
constexpr int kEncBinary = 1;
hipError_t launch_encode(const uint8_t *x, int64_t n, int32_t d,
                         const uint8_t *thresholds, int32_t b, uint64_t *out, int layout,
                         int64_t W_cols, hipStream_t stream, int kind = kEncThermometer);

// Quantile thresholds from data: histograms of n_groups contiguous feature
// groups (ws: n_groups * 256 uint64, cleared here), then per group the
// smallest v with (b + 1) * cum(v) >= i * total for i = 1..b into th [d][b].
constexpr int kFitMaxGroups = 32;
hipError_t launch_fit_quantiles(const uint8_t *x, int64_t n, int32_t d, int32_t b,
                                int32_t n_groups, uint8_t *th, uint64_t *ws, hipStream_t stream);

// Nodes per entry of a specialized layer's fan-in array.
constexpr int kSpecPass = 32;

// Slab-layout LUT layer over n_slabs slabs (bitlogic_forward's intermediates).
// fanin: NULL, or a specialized layer's evaluated fan-in per kSpecPass nodes
// (device; connections [w_out][k] then use the first fan-in slots).
hipError_t launch_lut_layer_slab(const uint64_t *in, int32_t w_in, int64_t n_slabs,
                                 const int32_t *conn, const uint64_t *tables, int32_t w_out,
                                 int32_t k, uint64_t *out, hipStream_t stream,
                                 const uint8_t *fanin = nullptr);

hipError_t launch_lut_layer(const uint64_t *in, int32_t w_in, int64_t n_words,
                            const int32_t *conn, const uint64_t *tables,
                            int32_t w_out, int32_t k, uint64_t *out,
                            hipStream_t stream);

// Table specialization of one node (host): merges tied slots and drops
// inputs the table ignores; returns the effective fan-in k' and writes the
// k' remaining connections and the table over them.
int specialize_node(const int32_t *conn, uint64_t T, int k, int32_t *conn_out, uint64_t *T_out);

// Table specialization of a network (host): every node specialized, each
// layer's nodes reordered by effective fan-in (within class groups for the
// last layer, of c classes), the next layer's connections relabelled, and per
// kSpecPass nodes the largest fan-in, to which the pass's nodes are padded.
// w[l], k[l]: layer widths and fan-ins; conn/tables: the network (host);
// min_gain: the least fraction of multiplexers a layer must save to be
// specialized; outputs per layer: k_out (the largest effective fan-in, at
// least 1; k for a layer left as is), applied_out (1 if specialized),
// conn_out [w][k_out], tables_out [w] (over k_out slots), fanin_out
// [ceil(w / kSpecPass)], order_out [w] (original node at each position; may
// be NULL).  Connections must be in range (the caller checks).
void specialize_network(int32_t w_in, int32_t L, const int32_t *w, const int32_t *k,
                        const int32_t *const *conn, const uint64_t *const *tables, int32_t c,
                        double min_gain, int32_t *k_out, int32_t *applied_out,
                        int32_t *const *conn_out, uint64_t *const *tables_out,
                        uint8_t *const *fanin_out, int32_t *const *order_out);

// Node-per-wave LUT layer with jump-table leaves (lut_jump.hip), fan-in 5 or
// 6, slab layout.  Its prep step writes one kJumpRecBytes record per node
// (and kJumpPadRecs past the last) into `rec` (jump_records_bytes(w_out)
// bytes, 128-byte aligned), then the layer runs; both on `stream`.
// jump_layer_fits: the kernel can run the layer (fan-in 5 or 6, an even slab
// count, rows within 2^23) and, unless `forced`, is the faster choice (the
// input slab pair, w_in * 256 bytes, within kJumpMaxPairBytes, and at least
// kJumpMinBlocks blocks).
constexpr int kJumpRecBytes = 128;
constexpr int kJumpPadRecs = 2;
constexpr int kJumpNodesPerWave = 16;
constexpr int kJumpNodesPerBlock = 4 * kJumpNodesPerWave;
constexpr int64_t kJumpMaxPairBytes = 3 << 20;
constexpr int32_t kJumpMaxRows = 1 << 23;
constexpr int64_t kJumpMinBlocks = 4096;
bool jump_layer_fits(int32_t w_in, int32_t w_out, int32_t k, int64_t n_slabs, bool forced);
size_t jump_records_bytes(int32_t w_out);
hipError_t launch_jump_layer(const uint64_t *in, int32_t w_in, int64_t n_slabs,
                             const int32_t *conn, const uint64_t *tables, int32_t w_out,
                             int32_t k, uint64_t *out, uint32_t *rec, hipStream_t stream);

// Last LUT layer fused with the GroupSum head (slab layout): writes the head's
// bit planes instead of the layer's bits.  fused_head_nodes(g, c, n_slabs) is the
// node count nb of one block (a multiple of 64; a class group of g nodes takes
// ceil(g / nb) blocks, the last one possibly short; fewer passes per block for
// small batches), or 0 when the shape does not allow the fused kernel.
int32_t fused_head_nodes(int32_t g, int32_t c, int64_t n_slabs);
hipError_t launch_lut_slab_head(const uint64_t *in, int32_t w_in, int64_t n_slabs,
                                const int32_t *conn, const uint64_t *tables, int32_t w_out,
                                int32_t k, int32_t c, int64_t W, uint64_t *planes, int32_t P,
                                hipStream_t stream, const uint8_t *fanin = nullptr);

struct HeadPlan {
    int32_t splits;        // row splits per class group
    int32_t planes;        // bit planes per split counter
    int32_t rows_per_split;
    size_t ws_bytes;       // scratch bytes
};
HeadPlan plan_head(int32_t w, int64_t n, int32_t c);
// Plan of the fused last layer + head: splits = ceil(g / nb), planes = bit length of nb.
HeadPlan plan_fused_head(int32_t w, int64_t n, int32_t c, int32_t nb);
// Finish step only (planes -> scores, argmax).  With dsp_weights (int8
// [c][c], c <= 128) the quantized head's logits replace the scores.
hipError_t launch_head_finish(const uint64_t *planes, int64_t n, int32_t c, int32_t *scores,
                              int32_t *argmax, const int8_t *dsp_weights, const HeadPlan &plan,
                              hipStream_t stream);

hipError_t launch_head(const uint64_t *bits, int32_t w, int64_t n, int32_t c,
                       int32_t *scores, int32_t *argmax, const int8_t *dsp_weights, void *ws,
                       const HeadPlan &plan, int layout, hipStream_t stream);

// Quantized head on counts [n][c] (0..65535 each), c <= 128.
hipError_t launch_grouped_dsp(const int32_t *counts, int64_t n, int32_t c,
                              const int8_t *weights, int32_t *logits, int32_t *argmax,
                              hipStream_t stream);

// Peak probes (probes.hip): kProbeThreads = 256 lanes a block.
hipError_t launch_probe_valu(uint32_t *out, int32_t blocks, int32_t iters, uint32_t seed,
                             hipStream_t stream);
hipError_t launch_probe_valu_op(int32_t op, uint32_t *out, int32_t blocks, int32_t iters,
                                uint32_t seed, hipStream_t stream);
hipError_t launch_probe_gather(const void *rows, int64_t n_rows, int32_t lanes_per_row,
                               int32_t valu, int32_t blocks, int32_t passes,
                               int32_t waves_per_simd, uint32_t seed, uint32_t *out, void *sink,
                               hipStream_t stream);
constexpr int kHbmCopy = 0;     // bitlogic_probe_hbm modes
constexpr int kHbmRead = 1;
constexpr int kHbmWrite = 2;
hipError_t launch_probe_hbm(int32_t mode, const void *in, void *out, int64_t n_bytes,
                            int32_t unroll, int32_t blocks, hipStream_t stream);

}  // namespace bl
