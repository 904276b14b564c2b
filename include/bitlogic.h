/*
 * bitlogic.h -- C ABI of the bit-packed LUT-network inference path for
 * AMD Instinct MI355X (gfx950).
 *
 * The network is the paper's forward composition (Sec. 3, Eq. 1):
 *
 *     encoder E : R^d -> {0,1}^{d b}          (thermometer, Sec. 3 "Encoders
 *                                               and heads")
 *     D layers  : node j of a layer reads k wires through its connection map
 *                 M_j and outputs entry a of its 2^k-entry truth table, where
 *                 a = sum_i x_{M_j(i)} 2^i   (Sec. 3 "Nodes are
 *                 parameterizations", "Connectivity is the main per-layer
 *                 design choice"; App. C.1 "Bit-packed inference")
 *     head H    : class i scores the number of 1s among its group of g = w/c
 *                 final-layer nodes; argmax is the predicted class
 *                 (Sec. 3 "Encoders and heads", Sec. 5 "Head"; App. C.2)
 *
 * evaluated on bit-packed activations: 64 samples per 64-bit word along the
 * batch (App. C.1 "Bit-packed inference").
 *
 * ---------------------------------------------------------------- layouts
 * N = n_samples, W = ceil(N / 64) words.
 * Packed bit tensor  uint64 [rows][W], row-major (row stride W words).  Bit
 *                    (s % 64) of word [r][s / 64] is the value of row r for
 *                    sample s.  Bits of samples s >= N ("padding") are
 *                    written as 0 by bitlogic_encode; LUT layers compute
 *                    whatever their tables give there; the head ignores them.
 * Pixels             uint8 [N][d], row-major.
 * Thresholds         uint8 [d][b]; wire f*b + t of sample s is
 *                    (x[s][f] > thresholds[f][t]) -- a strict comparison on
 *                    the raw 0..255 pixel scale.
 * Connections        int32 [w_out][k]; entry [j][i] is the wire feeding
 *                    address bit i of node j; 0 <= conn < w_in, repeats
 *                    allowed.
 * Truth tables       uint64 [w_out]; entry a of node j is bit a of
 *                    tables[j]; bits >= 2^k are ignored.
 * Scores             int32 [N][c], row-major; class i of sample s.
 * Argmax             int32 [N]; lowest class index among the maxima.
 *
 * ------------------------------------------------------------ conventions
 * - Every array argument is a DEVICE pointer (memory the GPU can read or
 *   write), except the bitlogic_layer descriptor array of bitlogic_forward,
 *   which is a HOST array (its members are device pointers).
 * - The caller owns every buffer.  No entry point allocates or frees device
 *   memory; scratch comes from a caller-supplied workspace of at least the
 *   size the matching *_workspace_bytes query returns.
 * - Calls are asynchronous: work is enqueued on `stream` (a hipStream_t
 *   passed as void*; NULL is the null stream) and BITLOGIC_OK means "validated
 *   and enqueued".  Inputs must stay valid until the stream has run the work.
 * - Arguments are checked on the host before anything is enqueued; a failed
 *   check returns an error code, launches nothing and touches no memory.
 *   Connection indices are device data and are NOT range-checked: an index
 *   outside [0, w_in) is undefined behaviour.  The Python binding checks
 *   them on the host when it builds a model.
 * - Packed bit buffers (bits_in, bits_out, bits) must be 8-byte aligned
 *   (16-byte alignment together with an even word count W lets the kernels
 *   use 16-byte accesses); the workspace must be 256-byte aligned.  Pixels,
 *   thresholds, connections, tables, scores and argmax need only their
 *   natural alignment.
 * - Buffers written by a call must not overlap any buffer it reads.
 * - A HIP launch failure returns BITLOGIC_ERR_HIP; bitlogic_last_error()
 *   then names the runtime's error.
 * - Limits: 1 <= k <= 6; n_samples >= 0 (0 enqueues nothing);
 *   1 <= n_thresholds <= 64; every row count fits in int32; the head needs
 *   w % n_classes == 0 and g = w / n_classes <= 65535.
 * - Entry points are thread-safe; calls on one stream run in order.
 *
 * ---------------------------------------------------- environment switches
 * Read at every forward call; it changes which kernels run, never results.
 *   BITLOGIC_UNFUSED_HEAD=1   the forward stores the last layer's bits and
 *                             runs the separate head kernels instead of the
 *                             last layer fused with the GroupSum counting.
 *   BITLOGIC_JUMP_LAYER=0     every stored layer runs on the per-lane
 *                             multiplexer kernel, none on the node-per-wave
 *                             kernel (bitlogic_forward_info.jump_layers);
 *                       =1    the node-per-wave kernel runs every stored,
 *                             unspecialized layer of fan-in 5 or 6 when the
 *                             batch fills an even number of 1024-sample slabs,
 *                             also where it is not the faster kernel.
 */
#ifndef BITLOGIC_H
#define BITLOGIC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum bitlogic_status {
    BITLOGIC_OK = 0,
    BITLOGIC_ERR_NULL = 1,         /* a required pointer is NULL */
    BITLOGIC_ERR_SHAPE = 2,        /* a size is out of range or inconsistent */
    BITLOGIC_ERR_ALIGN = 3,        /* a buffer is not aligned as required */
    BITLOGIC_ERR_UNSUPPORTED = 4,  /* e.g. k outside 1..6 */
    BITLOGIC_ERR_HIP = 5,          /* the HIP runtime reported an error */
    BITLOGIC_ERR_WORKSPACE = 6     /* workspace smaller than required */
} bitlogic_status;

/* Thermometer encoder and bit-pack (Sec. 3 "Encoders and heads"; App. A
 * "Initialization": linear or quantile threshold ladders; App. C.1: 64
 * samples per 64-bit word).
 *   x           uint8 [n_samples][n_features]
 *   thresholds  uint8 [n_features][n_thresholds]
 *   bits_out    uint64 [n_features * n_thresholds][W]; padding bits are 0.
 * Any threshold values are accepted (they need not be sorted). */
int bitlogic_encode(const uint8_t *x, int64_t n_samples, int32_t n_features,
                    const uint8_t *thresholds, int32_t n_thresholds,
                    uint64_t *bits_out, void *stream);

/* One LUT layer on packed bits (Sec. 3: connection map M_j, fan-in n = k,
 * 2^k-entry truth table; App. C.1: bitwise evaluation of 64 samples per op).
 *   bits_in   uint64 [w_in][n_words]
 *   conn      int32  [w_out][k]
 *   tables    uint64 [w_out]
 *   bits_out  uint64 [w_out][n_words]
 * Bit s of bits_out[j][.] = (tables[j] >> a) & 1 with
 * a = sum_i bit_s(bits_in[conn[j][i]][.]) << i. */
int bitlogic_lut_layer(const uint64_t *bits_in, int32_t w_in, int64_t n_words,
                       const int32_t *conn, const uint64_t *tables,
                       int32_t w_out, int32_t k, uint64_t *bits_out,
                       void *stream);

/* Scratch bytes bitlogic_groupsum_head needs for these sizes. */
size_t bitlogic_groupsum_head_workspace_bytes(int32_t w, int64_t n_samples,
                                              int32_t n_classes);

/* GroupSum popcount head and argmax (Sec. 3 "Encoders and heads"; Sec. 5
 * "Head"; App. C.2: the deployed design outputs the class index).
 *   bits     uint64 [w][W], the last layer's output
 *   scores   int32 [n_samples][n_classes], or NULL to skip
 *   argmax   int32 [n_samples], or NULL to skip (not both NULL)
 * Class i owns nodes [i*g, (i+1)*g), g = w / n_classes. */
int bitlogic_groupsum_head(const uint64_t *bits, int32_t w, int64_t n_samples,
                           int32_t n_classes, int32_t *scores, int32_t *argmax,
                           void *workspace, size_t workspace_bytes,
                           void *stream);

/* One layer of a network: device pointers plus its shape. */
typedef struct bitlogic_layer {
    const int32_t *conn;      /* int32 [w_out][k] */
    const uint64_t *tables;   /* uint64 [w_out] */
    int32_t w_out;
    int32_t k;
} bitlogic_layer;

/* Scratch bytes bitlogic_forward needs for these sizes (0 on bad shapes). */
size_t bitlogic_forward_workspace_bytes(int64_t n_samples, int32_t n_features,
                                        int32_t n_thresholds,
                                        const bitlogic_layer *layers,
                                        int32_t n_layers, int32_t n_classes);

/* How bitlogic_forward runs a network of this shape (host only, no HIP
 * call, nothing enqueued).  Fills *info and returns BITLOGIC_OK, or returns
 * the status bitlogic_forward would return for these sizes and descriptors
 * (info untouched).  Device pointers in `layers` are not dereferenced. */
typedef struct bitlogic_forward_info {
    size_t workspace_bytes;   /* = bitlogic_forward_workspace_bytes(...)          */
    int32_t slab_words;       /* intermediates are stored in slabs of this many
                                 64-sample words: [W_pad / slab][rows][slab]     */
    int32_t fused_head;       /* 1: the last LUT layer and the GroupSum head run
                                 as one kernel; the last layer's bits are never
                                 written to memory                                */
    int32_t head_splits;      /* partial counters per (sample word, class)       */
    int32_t head_planes;      /* bit planes per partial counter                  */
    uint32_t jump_layers;     /* bit l (l < 32): layer l is stored by the
                                 node-per-wave kernel whose table bytes select
                                 prebuilt 3-input leaves (fan-in 5 or 6, input
                                 slab pair within the L2); other stored layers
                                 use the per-lane multiplexer kernel          */
} bitlogic_forward_info;

int bitlogic_forward_plan(int64_t n_samples, int32_t n_features, int32_t n_thresholds,
                          const bitlogic_layer *layers, int32_t n_layers,
                          int32_t n_classes, bitlogic_forward_info *info);

/* Whole forward pass, encoder -> n_layers LUT layers -> head (Sec. 3,
 * Eq. 1; App. C.1): pixels in device memory to scores and argmax in
 * device memory.  Layer 0 reads the n_features * n_thresholds encoder wires
 * and layer l > 0 reads layer l-1, so w_in(l) = layers[l-1].w_out.
 * `layers` is a host array of n_layers >= 1 descriptors.  The encoded and
 * intermediate bit tensors live in the workspace. */
int bitlogic_forward(const uint8_t *x, int64_t n_samples, int32_t n_features,
                     const uint8_t *thresholds, int32_t n_thresholds,
                     const bitlogic_layer *layers, int32_t n_layers,
                     int32_t n_classes, int32_t *scores, int32_t *argmax,
                     void *workspace, size_t workspace_bytes, void *stream);

/* bitlogic_forward plus stage timing, for profiling: the same kernels on the
 * same stream, and hipEventRecord(events[i], stream) at every stage boundary:
 * events[0] before the encoder, events[1] after it, events[1 + l] after
 * layer l (l = 1..n_layers), events[n_layers + 2] after the head.
 * `events` is a host array of n_events = n_layers + 3 hipEvent_t handles
 * (passed as void*) created by the caller; the timing is read with
 * hipEventElapsedTime.  Errors as bitlogic_forward, plus BITLOGIC_ERR_SHAPE
 * if n_events is wrong and BITLOGIC_ERR_NULL if an event is NULL. */
int bitlogic_forward_timed(const uint8_t *x, int64_t n_samples, int32_t n_features,
                           const uint8_t *thresholds, int32_t n_thresholds,
                           const bitlogic_layer *layers, int32_t n_layers,
                           int32_t n_classes, int32_t *scores, int32_t *argmax,
                           void *workspace, size_t workspace_bytes, void *stream,
                           void *const *events, int32_t n_events);

/* Quantized class head (Sec. 3 "Encoders and heads": the quantized variant of
 * the popcount head; Sec. 5 "Head", the DSP-backed head of the head sweep):
 * a c x c matrix Q of signed 8-bit weights (trained heads snap them to the
 * grid [-127, 127]) multiplies the length-c vector of group sums,
 *     logits[s][i] = sum_j Q[i][j] * counts[s][j]
 * (row i of Q produces class i, no bias), and argmax[s] = lowest i with the
 * largest logit.  Any positive output scale leaves the argmax unchanged, so
 * logits are returned as exact int32 integers.
 *   counts   [n_samples][n_classes] int32, each in 0..65535 (a group sum;
 *            values outside that range give undefined logits)
 *   weights  [n_classes][n_classes] int8, row-major
 *   logits   [n_samples][n_classes] int32 or NULL; argmax [n_samples] or NULL
 *            (not both NULL)
 * Needs 1 <= n_classes <= 128 (BITLOGIC_ERR_UNSUPPORTED otherwise).  Runs on
 * the matrix cores (8-bit integer MFMA). */
int bitlogic_grouped_dsp_head(const int32_t *counts, int64_t n_samples, int32_t n_classes,
                              const int8_t *weights, int32_t *logits, int32_t *argmax,
                              void *stream);

/* bitlogic_forward with the quantized head in place of the popcount scores:
 * the same encoder, layers, workspace (bitlogic_forward_workspace_bytes) and
 * checks, then logits = Q * (group sums) and argmax over the logits, as in
 * bitlogic_grouped_dsp_head.  weights [n_classes][n_classes] int8, device
 * memory; n_classes <= 128; the group size is at most 65535 as for the
 * popcount head, so every count is in range. */
int bitlogic_forward_grouped_dsp(const uint8_t *x, int64_t n_samples, int32_t n_features,
                                 const uint8_t *thresholds, int32_t n_thresholds,
                                 const bitlogic_layer *layers, int32_t n_layers,
                                 int32_t n_classes, const int8_t *weights, int32_t *logits,
                                 int32_t *argmax, void *workspace, size_t workspace_bytes,
                                 void *stream);

/* ---- Encoder family and quantile fitting -------------------------------- */

/* Binary-coded uniform fixed-point encoder (Sec. 3 "Encoders and heads": the
 * integer quantizer with 2^b levels on b wires; Sec. 5 "Encoder", the encoder
 * sweep table).  Pixel v (0..255, read as v/255 in [0, 1]) is quantized to
 * the nearest of 2^b equispaced levels, q = round(v * (2^b - 1) / 255) (no
 * ties occur), and wire f * n_bits + t carries bit t of q, least significant
 * first:
 *     bit (s % 64) of bits_out[f * n_bits + t][s / 64] = (q(x[s][f]) >> t) & 1
 * Layout, padding and alignment as bitlogic_encode; 1 <= n_bits <= 8. */
int bitlogic_encode_binary(const uint8_t *x, int64_t n_samples, int32_t n_features,
                           int32_t n_bits, uint64_t *bits_out, void *stream);

/* Quantile thermometer thresholds fitted from data (Sec. 4 "Initialization":
 * fitted once from the empirical pixel quantiles of the training split;
 * App. B: over the flattened pixel distribution).  The n_features features
 * are cut into n_groups contiguous groups of n_features / n_groups (1: the
 * whole flattened distribution; 3 for CHW colour images: one ladder per
 * channel).  For each group, with cum(v) = number of its pixels <= v and
 * total = n_samples * n_features / n_groups, threshold i (i = 1..b) is the
 * smallest v with (b + 1) * cum(v) >= i * total, and every feature of the
 * group gets that ladder:
 *   x               [n_samples][n_features] uint8 pixels (device)
 *   thresholds_out  [n_features][n_thresholds] uint8 (device), ready for
 *                   bitlogic_encode / bitlogic_forward
 *   workspace       bitlogic_fit_quantile_thresholds_workspace_bytes(n_groups)
 *                   bytes of device memory, 8-byte aligned (a histogram)
 * Needs n_samples >= 1, 1 <= n_thresholds <= 64, 1 <= n_groups <= 32,
 * n_features % n_groups == 0 and n_samples * n_features <= 2^56. */
size_t bitlogic_fit_quantile_thresholds_workspace_bytes(int32_t n_groups);
int bitlogic_fit_quantile_thresholds(const uint8_t *x, int64_t n_samples, int32_t n_features,
                                     int32_t n_thresholds, int32_t n_groups,
                                     uint8_t *thresholds_out, void *workspace,
                                     size_t workspace_bytes, void *stream);

/* ---- Network descriptor: any encoder, any head --------------------------- */

/* ---- Table specialization ------------------------------------------------ */

/* Table specialization of a layer (host arrays, no HIP call): the collapse
 * the paper's synthesis flow applies to the per-node tables it emits (Sec. 5
 * "Connectivity": slots tied to the same wire reduce a table to a function of
 * fewer effective inputs; App. C.2, one table per node).  For every node j:
 * connection slots that repeat an earlier slot's wire are merged (only
 * addresses whose bits agree can occur), slots the table does not depend on
 * are dropped, and the table is rewritten over the k_eff[j] remaining slots,
 * which keep their order (k_eff = 0: a constant node, output bit = table
 * bit 0).  Evaluating conn_out[j][0..k_eff-1] with tables_out[j] gives the
 * node's output for every input, with 2^k_eff - 1 multiplexers instead of
 * 2^k - 1.
 *   conn [w_out][k], tables [w_out] in; k_eff [w_out], conn_out [w_out][k]
 *   (slots past k_eff are 0), tables_out [w_out] out.
 * Returns BITLOGIC_ERR_SHAPE if a connection is outside [0, w_in). */
int bitlogic_specialize_layer(const int32_t *conn, const uint64_t *tables, int32_t w_out,
                              int32_t k, int32_t w_in, int32_t *k_eff, int32_t *conn_out,
                              uint64_t *tables_out);

/* Table specialization of a whole network (host arrays, no HIP call), ready
 * for bitlogic_network_forward.  Every node is specialized as above; then
 * each layer's nodes are reordered by effective fan-in, largest first
 * (within each class group of the last layer, so every class keeps its
 * nodes), the next layer's connections are relabelled to the new order, and
 * every run of BITLOGIC_SPECIALIZE_PASS positions records its largest
 * fan-in in fanin_out.  The specialized layer's fan-in k_out[l] is the
 * largest effective fan-in of its nodes (at least 1).  Slots past a node's
 * effective fan-in repeat its first wire (wire 0 for a constant node) and
 * its table is extended over all k_out[l] slots so that it ignores them:
 * evaluating the first kp slots, for any kp from the node's effective fan-in
 * up to k_out[l], gives the node's output.  The result computes the same
 * scores as the original network; its hidden activations are the original
 * ones permuted.  A layer whose multiplexer count (runs of
 * BITLOGIC_SPECIALIZE_PASS nodes at their largest fan-in) would fall by less
 * than the fraction min_gain is left as it is (applied_out[l] = 0: original
 * nodes, order and tables, connections relabelled only), since the
 * specialized kernels cost a little more than the plain ones at equal work;
 * min_gain = 0 specializes every layer.
 *   w_in: encoder wires (n_features * n_bits); per layer l (host arrays of
 *   n_layers pointers): conn[l] [w_out[l]][k[l]], tables[l] [w_out[l]] in;
 *   k_out [n_layers], applied_out [n_layers]; conn_out[l]
 *   [w_out[l]][k_out[l]] (allocate w_out[l] * k[l] entries), tables_out[l]
 *   [w_out[l]], fanin_out[l] [ceil(w_out[l] / BITLOGIC_SPECIALIZE_PASS)]
 *   out; order_out: NULL, or per layer [w_out[l]] (the original node at each
 *   position).  The specialized network for bitlogic_network_forward has
 *   layers {conn_out[l], tables_out[l], w_out[l], k_out[l]} and pass_fanin
 *   fanin_out[l] on the device where applied_out[l] is 1, NULL elsewhere.
 * Returns BITLOGIC_ERR_SHAPE if a connection is out of range, the last width
 * is not a multiple of n_classes or min_gain is outside [0, 1]. */
#define BITLOGIC_SPECIALIZE_PASS 32
int bitlogic_specialize_network(int32_t w_in, const int32_t *const *conn,
                                const uint64_t *const *tables, const int32_t *w_out,
                                const int32_t *k, int32_t n_layers, int32_t n_classes,
                                double min_gain, int32_t *k_out, int32_t *applied_out,
                                int32_t *const *conn_out, uint64_t *const *tables_out,
                                uint8_t *const *fanin_out, int32_t *const *order_out);

enum { BITLOGIC_ENCODER_THERMOMETER = 0, BITLOGIC_ENCODER_BINARY = 1 };
enum { BITLOGIC_HEAD_GROUPSUM = 0, BITLOGIC_HEAD_GROUPED_DSP = 1 };

/* A whole network (Sec. 3, Eq. 1): encoder -> n_layers LUT layers -> head.
 * Host struct; its pointers are device memory except `layers` (a host array
 * of n_layers descriptors, as for bitlogic_forward). */
typedef struct bitlogic_network {
    int32_t n_features;             /* d                                          */
    int32_t encoder;                /* BITLOGIC_ENCODER_*                         */
    int32_t n_bits;                 /* b: thresholds per feature (thermometer,
                                       1..64) or code bits (binary, 1..8)         */
    const uint8_t *thresholds;      /* [d][b], thermometer only (else ignored)    */
    const bitlogic_layer *layers;   /* host array; layer 0 reads the d * b wires  */
    int32_t n_layers;
    int32_t n_classes;              /* c; the last width is a multiple of c       */
    int32_t head;                   /* BITLOGIC_HEAD_*                            */
    const int8_t *head_weights;     /* [c][c] int8, GROUPED_DSP only (c <= 128)   */
    const uint8_t *const *pass_fanin;
                                    /* NULL, or a host array of n_layers device
                                       pointers (entries may be NULL): a
                                       non-NULL entry marks layer l
                                       as specialized (bitlogic_specialize_network)
                                       and holds its fan-in per run of
                                       BITLOGIC_SPECIALIZE_PASS nodes: each
                                       node's output is read from its first
                                       fan-in slots (values above k[l] are
                                       clamped to it)                            */
} bitlogic_network;

/* Workspace bytes of bitlogic_network_forward for n_samples (0 if the
 * descriptor is invalid). */
size_t bitlogic_network_workspace_bytes(const bitlogic_network *net, int64_t n_samples);

/* bitlogic_forward_plan for a network descriptor. */
int bitlogic_network_plan(const bitlogic_network *net, int64_t n_samples,
                          bitlogic_forward_info *info);

/* The forward of a network descriptor: out [n_samples][c] int32 receives the
 * GroupSum scores or, with the quantized head, its logits; argmax [n_samples]
 * the lowest class holding the largest value (either may be NULL, not both).
 * events: NULL, or n_layers + 3 HIP events recorded as in
 * bitlogic_forward_timed.  Conventions and errors as bitlogic_forward, plus
 * BITLOGIC_ERR_UNSUPPORTED for an unknown encoder or head kind, a binary code
 * wider than 8 bits or a quantized head with more than 128 classes. */
int bitlogic_network_forward(const bitlogic_network *net, const uint8_t *x, int64_t n_samples,
                             int32_t *out, int32_t *argmax, void *workspace,
                             size_t workspace_bytes, void *stream, void *const *events,
                             int32_t n_events);

/* ---- Forward without allocation ----------------------------------------
 * For callers that cannot allocate device memory or hand in a workspace:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Computes exactly what bitlogic_network_forward computes (same
 * kernels, same results), but its scratch is a static device array inside
 * the library, BITLOGIC_NOALLOC_SCRATCH_BYTES per GPU, which each GPU the
 * library runs on holds from load until the process ends.  The call makes no
 * hipMalloc, hipFree or other allocating call.
 *   net, x, n_samples, out, argmax, stream: as bitlogic_network_forward
 *   (out and argmax are the caller's device buffers; no events).
 * Errors: as bitlogic_network_forward, plus
 *   BITLOGIC_ERR_WORKSPACE    bitlogic_network_workspace_bytes(net, n_samples)
 *                             exceeds BITLOGIC_NOALLOC_SCRATCH_BYTES (nothing
 *                             is enqueued; split the batch or use
 *                             bitlogic_network_forward);
 *   BITLOGIC_ERR_UNSUPPORTED  `stream` belongs to another device than the
 *                             current one.
 * All calls on one GPU share that GPU's array, which keeps the previous
 * call's contents (every byte a call reads it has written itself first).
 * Calls that overlap in time on one GPU -- on different streams, or from
 * threads that do not order them -- race on the array and their results are
 * undefined; calls in order on one stream are safe. */
#define BITLOGIC_NOALLOC_SCRATCH_BYTES (64u << 20)
int bitlogic_network_forward_noalloc(const bitlogic_network *net, const uint8_t *x,
                                     int64_t n_samples, int32_t *out, int32_t *argmax,
                                     void *stream);

/* ---- Peak probes (measurement, not part of the inference path) ---------- */

/* Integer VALU probe: `blocks` blocks of 256 lanes.  Lane l (global index)
 * starts from 8 words a[c] = (l + 1) * 0x9E3779B1 ^ (seed + c) * 0x85EBCA77
 * (32-bit wrap-around), runs `iters` rounds of
 *     for c = 0..7:  s = a[(c + 1) % 8];  a[c] = (s & a[c]) | (~s & a[(c + 2) % 8])
 * (each one v_bitop3_b32, the multiplexer of the LUT layers) and writes the XOR of
 * its 8 words to out[l].  A call performs blocks * 256 * iters * 8 32-bit
 * lane-ops; timing it on `stream` gives the sustained integer VALU rate.
 *   out  uint32 [blocks * 256], device memory; blocks >= 1, iters >= 0. */
int bitlogic_probe_valu(uint32_t *out, int32_t blocks, int32_t iters, uint32_t seed,
                        void *stream);

/* Instruction-rate probe: `blocks` blocks of 256 lanes, each lane running
 * `iters` rounds of 64 instructions of one form on fixed registers, so that
 * the VGPR banks of the operands are known (register v[n] is in bank n % 4).
 * Lane l (global index) starts from c0 = ((l + 1) * 0x9E3779B1) ^ seed,
 * s = c0 * 0x85EBCA77 and z = ~c0 (32-bit wrap-around) in eight chains
 * c[0..7] = c0, then every round applies to each chain:
 *   BITLOGIC_PROBE_OP_MUX       c = (s & c) | (~s & z), one v_bitop3_b32 whose
 *                               three sources sit in three VGPR banks
 *   BITLOGIC_PROBE_OP_MUX_BANK  the same with two sources in one bank
 *   BITLOGIC_PROBE_OP_BFE       c = -((s >> 5) & 1) (v_bfe_i32, the mask of
 *                               one table bit)
 * and writes the sum of the eight chains (mod 2^32) to out[l].  A call issues
 * blocks * 4 * iters * 64 wave instructions.
 *   out  uint32 [blocks * 256]; blocks >= 1, iters >= 1. */
#define BITLOGIC_PROBE_OP_MUX 0
#define BITLOGIC_PROBE_OP_MUX_BANK 1
#define BITLOGIC_PROBE_OP_BFE 2
int bitlogic_probe_valu_op(int32_t op, uint32_t *out, int32_t blocks, int32_t iters,
                           uint32_t seed, void *stream);

/* Gather probe: the LUT layers' random row gathers (App. C.1: every node
 * reads whole 1024-sample row segments of 128 bytes) without their
 * multiplexers.  Per pass, wave w of block b gathers, for the 16 nodes
 * j = (b * passes + pass) * 64 + w * 16 + m (m = 0..15), rows
 * r(j, i) = h(6 j + i) mod n_rows for i = 0..5, where
 * h(x) = y ^ (y >> 16), y = (x ^ seed) * 0x9E3779B1 (32-bit).
 *   lanes_per_row 4: lane t serves node m = t / 4 and loads 16-byte pieces
 *                    2 q and 2 q + 1 (q = t % 4) of each of its 6 rows (the
 *                    split of the 5- and 6-input layer kernels: 16 rows per
 *                    load instruction);
 *   lanes_per_row 8: lane t serves nodes m = t / 8 and m = 8 + t / 8 and
 *                    loads piece t % 8 of each of their rows (a whole line
 *                    per 8 lanes: 8 rows per load instruction).
 * Each lane then issues valu_per_pass (0, 256, 512 or 768) v_bitop3_b32 on
 * the loaded words, whose results are dropped (they occupy the VALU as the
 * multiplexers do), and XORs its 12 pieces into a 16-byte accumulator;
 * out[b * 256 + t] = the XOR of the accumulator's four words.  With a sink,
 * wave w of block b also stores, per pass, its lanes' first two pieces to
 * sink 16-byte pieces ((b * passes + pass) * 4 + w) * 128 + 2 t and + 1,
 * non-temporally (2 KB per wave and pass, as the layer kernel's output).
 * waves_per_simd 1..8 limits the resident waves through the block's LDS
 * size (0: no limit).
 *   rows  n_rows * 128 bytes (16-byte aligned), 1 <= n_rows < 2^32
 *   out   uint32 [blocks * 256];  sink  NULL or blocks * passes * 8 KB. */
int bitlogic_probe_gather(const void *rows, int64_t n_rows, int32_t lanes_per_row,
                          int32_t valu_per_pass, int32_t blocks, int32_t passes,
                          int32_t waves_per_simd, uint32_t seed, uint32_t *out, void *sink,
                          void *stream);

/* HBM streaming probes over n_bytes (a multiple of 16) in 16-byte pieces,
 * with non-temporal 16-byte loads and stores; a block of 256 lanes covers
 * unroll * 256 consecutive pieces per step with its `unroll` loads in
 * flight before any is used (unroll 1, 2, 4 or 8), over a grid of `blocks`
 * blocks (0: 8 per CU) that strides over the buffer.  Modes:
 *   BITLOGIC_PROBE_HBM_COPY   out[0, n_bytes) = in[0, n_bytes)    (2 n_bytes moved)
 *   BITLOGIC_PROBE_HBM_READ   out[0, 16) = XOR of every 16-byte piece of in
 *                             (n_bytes read; out is cleared first, so
 *                             n_bytes = 0 gives 16 zero bytes)
 *   BITLOGIC_PROBE_HBM_WRITE  piece i of out (bytes 16 i .. 16 i + 15) = the
 *                             32-bit words (i, i >> 32, ~i, ~(i >> 32)),
 *                             little-endian; `in` unused (n_bytes written)
 * in, out: 16-byte aligned device memory; for COPY they must not overlap
 * (BITLOGIC_ERR_SHAPE).  An unknown mode or unroll is
 * BITLOGIC_ERR_UNSUPPORTED.  0 bytes enqueue nothing except READ's clear. */
#define BITLOGIC_PROBE_HBM_COPY 0
#define BITLOGIC_PROBE_HBM_READ 1
#define BITLOGIC_PROBE_HBM_WRITE 2
int bitlogic_probe_hbm(int32_t mode, const void *in, void *out, int64_t n_bytes,
                       int32_t unroll, int32_t blocks, void *stream);

/* Static description of a status code. */
const char *bitlogic_status_string(int status);

/* Detail of the last failing call on this host thread ("" if none). */
const char *bitlogic_last_error(void);

/* Library version, major * 10000 + minor * 100 + patch.  A caller built
 * against this header can check bitlogic_version() == BITLOGIC_VERSION
 * before using the structs above (0.3.0 added bitlogic_network.pass_fanin and
 * the specialization calls; 0.4.0 the peak probes; 0.5.0
 * bitlogic_network_forward_noalloc, and bitlogic_probe_hbm in
 * place of the copy-only probe; 0.6.0 bitlogic_forward_info without the
 * fused_network member (the whole-network kernel was removed), and the
 * instruction-rate and gather probes; 0.7.0 bitlogic_forward_info.jump_layers
 * and the node-per-wave layer kernel, whose per-node records enlarge the
 * forward workspace of networks that use it). */
#define BITLOGIC_VERSION 700
int bitlogic_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BITLOGIC_H */
