// C-ABI front end of libbitlogic: argument checks on the host, workspace
// carving, launches.  Every check runs before any HIP runtime call, so a
// rejected call enqueues nothing (and needs no GPU to be rejected).
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

#include <algorithm>
#include <atomic>
#include <mutex>

#include "bitlogic.h"
#include "bl_internal.h"

// Scratch of bitlogic_network_forward_noalloc: one copy of this array per GPU
// the library runs on, held until the process ends.  In host code `scratch`
// only names the symbol for hipGetSymbolAddress; the array's device address on
// each GPU is looked up once and kept in g_scratch_ptr below.
static __device__ __align__(256) unsigned char scratch[BITLOGIC_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local char g_last_error[256] = "";

int fail(int status, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return status;
}

int ok()
{
    g_last_error[0] = '\0';
    return BITLOGIC_OK;
}

int hip_status(hipError_t e, const char *what)
{
    if (e != hipSuccess)
        return fail(BITLOGIC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p % a) == 0; }

constexpr int64_t kMaxRows = 0x7fffffff;
constexpr int32_t kDspMaxClasses = 128;   // quantized head: logits below 2^31
constexpr size_t kWsAlign = 256;

size_t round_up(size_t v) { return (v + kWsAlign - 1) / kWsAlign * kWsAlign; }

int64_t words_of(int64_t n) { return (n + 63) / 64; }

int check_encode(const uint8_t *x, int64_t n, int32_t d, const uint8_t *th, int32_t b,
                 const uint64_t *out)
{
    if (!x || !th || !out)
        return fail(BITLOGIC_ERR_NULL, "encode: NULL pointer");
    if (n < 0 || d <= 0 || b <= 0 || b > 64)
        return fail(BITLOGIC_ERR_SHAPE, "encode: need n >= 0, d > 0, 1 <= b <= 64");
    if ((int64_t)d * b > kMaxRows)
        return fail(BITLOGIC_ERR_SHAPE, "encode: d * b exceeds int32");
    if (!aligned(out, 8))
        return fail(BITLOGIC_ERR_ALIGN, "encode: bits_out not 8-byte aligned");
    return BITLOGIC_OK;
}

int check_layer(const uint64_t *in, int32_t w_in, int64_t n_words, const int32_t *conn,
                const uint64_t *tables, int32_t w_out, int32_t k, const uint64_t *out,
                const char *who)
{
    if (!in || !conn || !tables || !out)
        return fail(BITLOGIC_ERR_NULL, "%s: NULL pointer", who);
    if (k < 1 || k > 6)
        return fail(BITLOGIC_ERR_UNSUPPORTED, "%s: fan-in k=%d outside 1..6", who, k);
    if (w_in <= 0 || w_out <= 0 || n_words < 0)
        return fail(BITLOGIC_ERR_SHAPE, "%s: need w_in > 0, w_out > 0, n_words >= 0", who);
    if (n_words > ((int64_t)1 << 40))
        return fail(BITLOGIC_ERR_SHAPE, "%s: n_words too large", who);
    if (!aligned(in, 8) || !aligned(out, 8))
        return fail(BITLOGIC_ERR_ALIGN, "%s: bit buffers must be 8-byte aligned", who);
    if (!aligned(conn, 4) || !aligned(tables, 8))
        return fail(BITLOGIC_ERR_ALIGN, "%s: conn/tables misaligned", who);
    return BITLOGIC_OK;
}

int check_head(const uint64_t *bits, int32_t w, int64_t n, int32_t c, const int32_t *scores,
               const int32_t *argmax)
{
    if (!bits || (!scores && !argmax))
        return fail(BITLOGIC_ERR_NULL, "head: NULL bits, or both outputs NULL");
    if (w <= 0 || c <= 0 || n < 0)
        return fail(BITLOGIC_ERR_SHAPE, "head: need w > 0, c > 0, n >= 0");
    if (w % c != 0)
        return fail(BITLOGIC_ERR_SHAPE, "head: w=%d not a multiple of n_classes=%d", w, c);
    if (w / c > 65535)
        return fail(BITLOGIC_ERR_SHAPE, "head: group size %d > 65535", w / c);
    if (n > ((int64_t)1 << 40))
        return fail(BITLOGIC_ERR_SHAPE, "head: n_samples too large");
    if (!aligned(bits, 8) || (scores && !aligned(scores, 4)) || (argmax && !aligned(argmax, 4)))
        return fail(BITLOGIC_ERR_ALIGN, "head: misaligned buffer");
    return BITLOGIC_OK;
}

// BITLOGIC_UNFUSED_HEAD=1 in the environment runs the last layer and the head
// as separate kernels (for comparison; results are identical).
bool fused_head_enabled()
{
    const char *e = getenv("BITLOGIC_UNFUSED_HEAD");
    return !(e && e[0] == '1');
}

// BITLOGIC_JUMP_LAYER=0 keeps every stored layer on the per-lane slab kernel,
// =1 runs the node-per-wave kernel wherever it can (also where it is not the
// faster choice); unset, it runs where it is faster.  Results are identical.
enum JumpMode { kJumpOff, kJumpAuto, kJumpForced };
JumpMode jump_mode()
{
    const char *e = getenv("BITLOGIC_JUMP_LAYER");
    if (e && e[0] == '0')
        return kJumpOff;
    if (e && e[0] == '1')
        return kJumpForced;
    return kJumpAuto;
}

// bitlogic_forward keeps its encoded and intermediate bit tensors in the slab
// layout [Wp / S][rows][S] (S = kSlabWords, Wp = W rounded up to whole slabs),
// which bounds the LUT-layer gathers' per-XCD working set (see lut_layer.hip).
struct ForwardPlan {
    int64_t W;
    int64_t n_slabs;
    int32_t widest;
    size_t off_enc, off_a, off_b, off_head, total;
    bl::HeadPlan head;
    bool fused;            // last layer + head in one kernel
    uint64_t jump_mask;    // bit l: layer l runs on the node-per-wave kernel
    size_t off_rec;        // its per-node records (shared by those layers)
};

bitlogic_network legacy_net(int32_t n_features, const uint8_t *thresholds, int32_t n_thresholds,
                            const bitlogic_layer *layers, int32_t n_layers, int32_t n_classes,
                            const int8_t *dsp_weights);

int plan_forward(int64_t n, int32_t d, int32_t b, const bitlogic_layer *layers, int32_t L,
                 int32_t c, const uint8_t *const *pass_fanin, ForwardPlan *fp)
{
    if (!layers)
        return fail(BITLOGIC_ERR_NULL, "forward: NULL layer array");
    if (L < 1)
        return fail(BITLOGIC_ERR_SHAPE, "forward: need n_layers >= 1");
    if (n < 0 || d <= 0 || b <= 0 || b > 64 || c <= 0)
        return fail(BITLOGIC_ERR_SHAPE, "forward: need n >= 0, d > 0, 1 <= b <= 64, c > 0");
    if ((int64_t)d * b > kMaxRows)
        return fail(BITLOGIC_ERR_SHAPE, "forward: d * b exceeds int32");
    if (n > ((int64_t)1 << 40))
        return fail(BITLOGIC_ERR_SHAPE, "forward: n_samples too large");
    int32_t widest = 0;
    for (int32_t l = 0; l < L; ++l) {
        if (!layers[l].conn || !layers[l].tables)
            return fail(BITLOGIC_ERR_NULL, "forward: layer %d has a NULL pointer", l);
        if (layers[l].k < 1 || layers[l].k > 6)
            return fail(BITLOGIC_ERR_UNSUPPORTED, "forward: layer %d fan-in %d outside 1..6",
                        l, layers[l].k);
        if (layers[l].w_out <= 0)
            return fail(BITLOGIC_ERR_SHAPE, "forward: layer %d width %d", l, layers[l].w_out);
        if (!aligned(layers[l].conn, 4) || !aligned(layers[l].tables, 8))
            return fail(BITLOGIC_ERR_ALIGN, "forward: layer %d conn/tables misaligned", l);
        if (layers[l].w_out > widest)
            widest = layers[l].w_out;
    }
    const int32_t w_last = layers[L - 1].w_out;
    if (w_last % c != 0)
        return fail(BITLOGIC_ERR_SHAPE, "forward: last width %d not a multiple of %d classes",
                    w_last, c);
    if (w_last / c > 65535)
        return fail(BITLOGIC_ERR_SHAPE, "forward: group size %d > 65535", w_last / c);
    fp->W = words_of(n);
    fp->n_slabs = (fp->W + bl::kSlabWords - 1) / bl::kSlabWords;
    fp->widest = widest;
    const int64_t Wp = fp->n_slabs * bl::kSlabWords;
    const size_t enc = (size_t)d * b * Wp * sizeof(uint64_t);
    const size_t act = (size_t)widest * Wp * sizeof(uint64_t);
    // the last layer and the head run fused when the group size allows it
    const int32_t nb = bl::fused_head_nodes(w_last / c, c, fp->n_slabs);
    fp->fused = nb > 0 && fused_head_enabled();
    fp->head = fp->fused ? bl::plan_fused_head(w_last, n, c, nb) : bl::plan_head(w_last, n, c);
    // layer l writes activation buffer l % 2, except a last layer fused with
    // the head, which writes nothing: allocate only the buffers some layer writes
    const int32_t stored = fp->fused ? L - 1 : L;     // layers whose bits are stored
    const bool need_a = stored >= 1, need_b = stored >= 2;
    fp->off_enc = 0;
    fp->off_a = round_up(enc);
    fp->off_b = fp->off_a + (need_a ? round_up(act) : 0);
    fp->off_head = fp->off_b + (need_b ? round_up(act) : 0);
    // stored, unspecialized layers of fan-in 5 or 6 whose input slab pair
    // fits the L2 run with a node per wave (lut_jump.hip); they share one
    // record array, sized for the widest of them
    fp->jump_mask = 0;
    int32_t rec_w = 0;
    int32_t w_in = d * b;
    const JumpMode jm = jump_mode();
    for (int32_t l = 0; l < L; ++l) {
        const bool last_fused = fp->fused && l == L - 1;
        const bool spec = pass_fanin && pass_fanin[l];
        if (l < 64 && !last_fused && !spec && jm != kJumpOff &&
            bl::jump_layer_fits(w_in, layers[l].w_out, layers[l].k, fp->n_slabs,
                                jm == kJumpForced)) {
            fp->jump_mask |= 1ull << l;
            rec_w = std::max(rec_w, layers[l].w_out);
        }
        w_in = layers[l].w_out;
    }
    fp->off_rec = fp->off_head + round_up(fp->head.ws_bytes);
    fp->total = fp->off_rec + (fp->jump_mask ? round_up(bl::jump_records_bytes(rec_w)) : 0);
    return BITLOGIC_OK;
}

}  // namespace

extern "C" {

int bitlogic_encode(const uint8_t *x, int64_t n_samples, int32_t n_features,
                    const uint8_t *thresholds, int32_t n_thresholds, uint64_t *bits_out,
                    void *stream)
{
    int st = check_encode(x, n_samples, n_features, thresholds, n_thresholds, bits_out);
    if (st != BITLOGIC_OK)
        return st;
    if (n_samples == 0)
        return ok();
    return hip_status(bl::launch_encode(x, n_samples, n_features, thresholds, n_thresholds,
                                        bits_out, bl::kLayoutRowMajor, words_of(n_samples),
                                        (hipStream_t)stream),
                      "encode launch");
}

int bitlogic_lut_layer(const uint64_t *bits_in, int32_t w_in, int64_t n_words,
                       const int32_t *conn, const uint64_t *tables, int32_t w_out, int32_t k,
                       uint64_t *bits_out, void *stream)
{
    int st = check_layer(bits_in, w_in, n_words, conn, tables, w_out, k, bits_out, "lut_layer");
    if (st != BITLOGIC_OK)
        return st;
    if (n_words == 0)
        return ok();
    return hip_status(bl::launch_lut_layer(bits_in, w_in, n_words, conn, tables, w_out, k,
                                           bits_out, (hipStream_t)stream),
                      "lut_layer launch");
}

size_t bitlogic_groupsum_head_workspace_bytes(int32_t w, int64_t n_samples, int32_t n_classes)
{
    if (w <= 0 || n_classes <= 0 || n_samples < 0 || w % n_classes != 0 ||
        w / n_classes > 65535 || n_samples > ((int64_t)1 << 40))
        return 0;
    return bl::plan_head(w, n_samples, n_classes).ws_bytes;
}

int bitlogic_groupsum_head(const uint64_t *bits, int32_t w, int64_t n_samples,
                           int32_t n_classes, int32_t *scores, int32_t *argmax,
                           void *workspace, size_t workspace_bytes, void *stream)
{
    int st = check_head(bits, w, n_samples, n_classes, scores, argmax);
    if (st != BITLOGIC_OK)
        return st;
    const bl::HeadPlan plan = bl::plan_head(w, n_samples, n_classes);
    if (plan.ws_bytes > 0 && !workspace)
        return fail(BITLOGIC_ERR_NULL, "head: NULL workspace");
    if (workspace_bytes < plan.ws_bytes)
        return fail(BITLOGIC_ERR_WORKSPACE, "head: workspace %zu < %zu bytes", workspace_bytes,
                    plan.ws_bytes);
    if (workspace && !aligned(workspace, kWsAlign))
        return fail(BITLOGIC_ERR_ALIGN, "head: workspace not 256-byte aligned");
    if (n_samples == 0)
        return ok();
    return hip_status(bl::launch_head(bits, w, n_samples, n_classes, scores, argmax, nullptr,
                                      workspace, plan, bl::kLayoutRowMajor,
                                      (hipStream_t)stream),
                      "head launch");
}

size_t bitlogic_forward_workspace_bytes(int64_t n_samples, int32_t n_features,
                                        int32_t n_thresholds, const bitlogic_layer *layers,
                                        int32_t n_layers, int32_t n_classes)
{
    ForwardPlan fp;
    if (plan_forward(n_samples, n_features, n_thresholds, layers, n_layers, n_classes, nullptr,
                     &fp) != BITLOGIC_OK)
        return 0;
    return fp.total;
}

int bitlogic_forward_plan(int64_t n_samples, int32_t n_features, int32_t n_thresholds,
                          const bitlogic_layer *layers, int32_t n_layers, int32_t n_classes,
                          bitlogic_forward_info *info)
{
    // the descriptor bitlogic_forward builds; a placeholder stands in for the
    // threshold pointer, which planning never reads
    static const uint8_t kPlaceholder = 0;
    const bitlogic_network net =
        legacy_net(n_features, &kPlaceholder, n_thresholds, layers, n_layers, n_classes, nullptr);
    return bitlogic_network_plan(&net, n_samples, info);
}

}  // extern "C"

namespace {

// Checks of a network descriptor beyond the shapes that plan_forward checks.
int check_network(const bitlogic_network *net)
{
    if (!net)
        return fail(BITLOGIC_ERR_NULL, "network: NULL descriptor");
    if (net->encoder == BITLOGIC_ENCODER_THERMOMETER) {
        if (!net->thresholds)
            return fail(BITLOGIC_ERR_NULL, "network: thermometer needs thresholds");
    } else if (net->encoder == BITLOGIC_ENCODER_BINARY) {
        if (net->n_bits < 1 || net->n_bits > 8)
            return fail(BITLOGIC_ERR_UNSUPPORTED, "network: binary code of %d bits (1..8)",
                        net->n_bits);
    } else {
        return fail(BITLOGIC_ERR_UNSUPPORTED, "network: unknown encoder %d", net->encoder);
    }
    if (net->head == BITLOGIC_HEAD_GROUPED_DSP) {
        if (!net->head_weights)
            return fail(BITLOGIC_ERR_NULL, "network: quantized head needs weights");
        if (net->n_classes > kDspMaxClasses)
            return fail(BITLOGIC_ERR_UNSUPPORTED, "network: quantized head needs n_classes <= %d",
                        kDspMaxClasses);
    } else if (net->head != BITLOGIC_HEAD_GROUPSUM) {
        return fail(BITLOGIC_ERR_UNSUPPORTED, "network: unknown head %d", net->head);
    }
    return BITLOGIC_OK;
}

int plan_network(const bitlogic_network *net, int64_t n, ForwardPlan *fp)
{
    int st = check_network(net);
    if (st != BITLOGIC_OK)
        return st;
    st = plan_forward(n, net->n_features, net->n_bits, net->layers, net->n_layers,
                      net->n_classes, net->pass_fanin, fp);
    if (st != BITLOGIC_OK)
        return st;
    return BITLOGIC_OK;
}

int forward_impl(const bitlogic_network *net, const uint8_t *x, int64_t n_samples,
                 int32_t *scores, int32_t *argmax, void *workspace, size_t workspace_bytes,
                 void *stream, void *const *events, int32_t n_events)
{
    ForwardPlan fp;
    int st = plan_network(net, n_samples, &fp);
    if (st != BITLOGIC_OK)
        return st;
    if (!x || (!scores && !argmax))
        return fail(BITLOGIC_ERR_NULL, "forward: NULL pixels or both outputs NULL");
    if (!workspace)
        return fail(BITLOGIC_ERR_NULL, "forward: NULL workspace");
    if (workspace_bytes < fp.total)
        return fail(BITLOGIC_ERR_WORKSPACE, "forward: workspace %zu < %zu bytes",
                    workspace_bytes, fp.total);
    if (!aligned(workspace, kWsAlign))
        return fail(BITLOGIC_ERR_ALIGN, "forward: workspace not 256-byte aligned");
    if ((scores && !aligned(scores, 4)) || (argmax && !aligned(argmax, 4)))
        return fail(BITLOGIC_ERR_ALIGN, "forward: misaligned output");
    const int32_t n_layers = net->n_layers;
    if (events) {
        if (n_events != n_layers + 3)
            return fail(BITLOGIC_ERR_SHAPE, "forward_timed: need %d events, got %d",
                        n_layers + 3, n_events);
        for (int32_t i = 0; i < n_events; ++i)
            if (!events[i])
                return fail(BITLOGIC_ERR_NULL, "forward_timed: event %d is NULL", i);
    }
    if (n_samples == 0)
        return ok();

    const bitlogic_layer *layers = net->layers;
    const int32_t n_classes = net->n_classes;
    const int8_t *dsp = net->head == BITLOGIC_HEAD_GROUPED_DSP ? net->head_weights : nullptr;
    hipStream_t s = (hipStream_t)stream;
    auto mark = [&](int i) -> hipError_t {
        return events ? hipEventRecord((hipEvent_t)events[i], s) : hipSuccess;
    };
    char *ws = static_cast<char *>(workspace);
    uint64_t *enc = reinterpret_cast<uint64_t *>(ws + fp.off_enc);
    uint64_t *act[2] = {reinterpret_cast<uint64_t *>(ws + fp.off_a),
                        reinterpret_cast<uint64_t *>(ws + fp.off_b)};
    hipError_t e = mark(0);
    if (e == hipSuccess)
        e = bl::launch_encode(x, n_samples, net->n_features, net->thresholds, net->n_bits, enc,
                              bl::kLayoutSlab, fp.n_slabs * bl::kSlabWords, s,
                              net->encoder == BITLOGIC_ENCODER_BINARY ? bl::kEncBinary
                                                                      : bl::kEncThermometer);
    if (e == hipSuccess)
        e = mark(1);
    if (e != hipSuccess)
        return hip_status(e, "forward: encode launch");
    const uint64_t *cur = enc;
    int32_t w_in = net->n_features * net->n_bits;
    uint64_t *planes = reinterpret_cast<uint64_t *>(ws + fp.off_head);
    uint32_t *rec = reinterpret_cast<uint32_t *>(ws + fp.off_rec);
    for (int32_t l = 0; l < n_layers; ++l) {
        const bool last_fused = fp.fused && l == n_layers - 1;
        uint64_t *dst = act[l & 1];
        const uint8_t *fanin = net->pass_fanin ? net->pass_fanin[l] : nullptr;
        if (last_fused)
            e = bl::launch_lut_slab_head(cur, w_in, fp.n_slabs, layers[l].conn, layers[l].tables,
                                         layers[l].w_out, layers[l].k, n_classes, fp.W, planes,
                                         fp.head.planes, s, fanin);
        else if ((fp.jump_mask >> l) & 1)
            e = bl::launch_jump_layer(cur, w_in, fp.n_slabs, layers[l].conn, layers[l].tables,
                                      layers[l].w_out, layers[l].k, dst, rec, s);
        else
            e = bl::launch_lut_layer_slab(cur, w_in, fp.n_slabs, layers[l].conn,
                                          layers[l].tables, layers[l].w_out, layers[l].k, dst, s,
                                          fanin);
        if (e == hipSuccess)
            e = mark(2 + l);
        if (e != hipSuccess)
            return fail(BITLOGIC_ERR_HIP, "forward: layer %d launch: %s", l, hipGetErrorString(e));
        cur = dst;
        w_in = layers[l].w_out;
    }
    if (fp.fused)
        e = bl::launch_head_finish(planes, n_samples, n_classes, scores, argmax, dsp, fp.head, s);
    else
        e = bl::launch_head(cur, w_in, n_samples, n_classes, scores, argmax, dsp, planes,
                            fp.head, bl::kLayoutSlab, s);
    if (e == hipSuccess)
        e = mark(n_layers + 2);
    return hip_status(e, "forward: head launch");
}

// The descriptor of the legacy entry points' arguments.
bitlogic_network legacy_net(int32_t n_features, const uint8_t *thresholds, int32_t n_thresholds,
                            const bitlogic_layer *layers, int32_t n_layers, int32_t n_classes,
                            const int8_t *dsp_weights)
{
    bitlogic_network net;
    net.n_features = n_features;
    net.encoder = BITLOGIC_ENCODER_THERMOMETER;
    net.n_bits = n_thresholds;
    net.thresholds = thresholds;
    net.layers = layers;
    net.n_layers = n_layers;
    net.n_classes = n_classes;
    net.head = dsp_weights ? BITLOGIC_HEAD_GROUPED_DSP : BITLOGIC_HEAD_GROUPSUM;
    net.head_weights = dsp_weights;
    net.pass_fanin = nullptr;
    return net;
}

}  // namespace

extern "C" {

int bitlogic_forward(const uint8_t *x, int64_t n_samples, int32_t n_features,
                     const uint8_t *thresholds, int32_t n_thresholds,
                     const bitlogic_layer *layers, int32_t n_layers, int32_t n_classes,
                     int32_t *scores, int32_t *argmax, void *workspace, size_t workspace_bytes,
                     void *stream)
{
    if (!thresholds)
        return fail(BITLOGIC_ERR_NULL, "forward: NULL thresholds");
    const bitlogic_network net =
        legacy_net(n_features, thresholds, n_thresholds, layers, n_layers, n_classes, nullptr);
    return forward_impl(&net, x, n_samples, scores, argmax, workspace, workspace_bytes, stream,
                        nullptr, 0);
}

int bitlogic_forward_grouped_dsp(const uint8_t *x, int64_t n_samples, int32_t n_features,
                                 const uint8_t *thresholds, int32_t n_thresholds,
                                 const bitlogic_layer *layers, int32_t n_layers,
                                 int32_t n_classes, const int8_t *weights, int32_t *logits,
                                 int32_t *argmax, void *workspace, size_t workspace_bytes,
                                 void *stream)
{
    if (!weights)
        return fail(BITLOGIC_ERR_NULL, "forward_grouped_dsp: NULL weights");
    if (!thresholds)
        return fail(BITLOGIC_ERR_NULL, "forward: NULL thresholds");
    const bitlogic_network net =
        legacy_net(n_features, thresholds, n_thresholds, layers, n_layers, n_classes, weights);
    return forward_impl(&net, x, n_samples, logits, argmax, workspace, workspace_bytes, stream,
                        nullptr, 0);
}

int bitlogic_grouped_dsp_head(const int32_t *counts, int64_t n_samples, int32_t n_classes,
                              const int8_t *weights, int32_t *logits, int32_t *argmax,
                              void *stream)
{
    if (!counts || !weights || (!logits && !argmax))
        return fail(BITLOGIC_ERR_NULL, "grouped_dsp_head: NULL counts/weights or both outputs");
    if (n_samples < 0 || n_classes < 1 || n_samples > ((int64_t)1 << 40))
        return fail(BITLOGIC_ERR_SHAPE, "grouped_dsp_head: need n_samples >= 0, n_classes >= 1");
    if (n_classes > kDspMaxClasses)
        return fail(BITLOGIC_ERR_UNSUPPORTED, "grouped_dsp_head: n_classes %d > %d", n_classes,
                    kDspMaxClasses);
    if (!aligned(counts, 4) || (logits && !aligned(logits, 4)) || (argmax && !aligned(argmax, 4)))
        return fail(BITLOGIC_ERR_ALIGN, "grouped_dsp_head: misaligned buffer");
    if (n_samples == 0)
        return ok();
    return hip_status(bl::launch_grouped_dsp(counts, n_samples, n_classes, weights, logits, argmax,
                                             (hipStream_t)stream),
                      "grouped_dsp_head launch");
}

int bitlogic_forward_timed(const uint8_t *x, int64_t n_samples, int32_t n_features,
                           const uint8_t *thresholds, int32_t n_thresholds,
                           const bitlogic_layer *layers, int32_t n_layers, int32_t n_classes,
                           int32_t *scores, int32_t *argmax, void *workspace,
                           size_t workspace_bytes, void *stream, void *const *events,
                           int32_t n_events)
{
    if (!events)
        return fail(BITLOGIC_ERR_NULL, "forward_timed: NULL event array");
    if (!thresholds)
        return fail(BITLOGIC_ERR_NULL, "forward: NULL thresholds");
    const bitlogic_network net =
        legacy_net(n_features, thresholds, n_thresholds, layers, n_layers, n_classes, nullptr);
    return forward_impl(&net, x, n_samples, scores, argmax, workspace, workspace_bytes, stream,
                        events, n_events);
}

size_t bitlogic_network_workspace_bytes(const bitlogic_network *net, int64_t n_samples)
{
    ForwardPlan fp;
    if (plan_network(net, n_samples, &fp) != BITLOGIC_OK)
        return 0;
    return fp.total;
}

int bitlogic_network_plan(const bitlogic_network *net, int64_t n_samples,
                          bitlogic_forward_info *info)
{
    if (!info)
        return fail(BITLOGIC_ERR_NULL, "network_plan: NULL info");
    ForwardPlan fp;
    int st = plan_network(net, n_samples, &fp);
    if (st != BITLOGIC_OK)
        return st;
    info->workspace_bytes = fp.total;
    info->slab_words = bl::kSlabWords;
    info->fused_head = fp.fused ? 1 : 0;
    info->head_splits = fp.head.splits;
    info->head_planes = fp.head.planes;
    info->jump_layers = (uint32_t)(fp.jump_mask & 0xFFFFFFFFu);
    return ok();
}

int bitlogic_network_forward(const bitlogic_network *net, const uint8_t *x, int64_t n_samples,
                             int32_t *out, int32_t *argmax, void *workspace,
                             size_t workspace_bytes, void *stream, void *const *events,
                             int32_t n_events)
{
    return forward_impl(net, x, n_samples, out, argmax, workspace, workspace_bytes, stream,
                        events, events ? n_events : 0);
}

}  // extern "C"

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void *> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of `scratch` on device dev (the current device), looked up
// on the first call for that device.
int scratch_address(int dev, void **ptr)
{
    void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
        if (!p) {
            hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess || !p)
                return fail(BITLOGIC_ERR_HIP, "forward_noalloc: scratch address on device %d: %s",
                            dev, hipGetErrorString(e));
            g_scratch_ptr[dev].store(p, std::memory_order_release);
        }
    }
    *ptr = p;
    return BITLOGIC_OK;
}

}  // namespace

extern "C" {

int bitlogic_network_forward_noalloc(const bitlogic_network *net, const uint8_t *x,
                                     int64_t n_samples, int32_t *out, int32_t *argmax,
                                     void *stream)
{
    // every argument check before the first HIP call
    ForwardPlan fp;
    int st = plan_network(net, n_samples, &fp);
    if (st != BITLOGIC_OK)
        return st;
    if (!x || (!out && !argmax))
        return fail(BITLOGIC_ERR_NULL, "forward_noalloc: NULL pixels or both outputs NULL");
    if ((out && !aligned(out, 4)) || (argmax && !aligned(argmax, 4)))
        return fail(BITLOGIC_ERR_ALIGN, "forward_noalloc: misaligned output");
    if (fp.total > (size_t)BITLOGIC_NOALLOC_SCRATCH_BYTES)
        return fail(BITLOGIC_ERR_WORKSPACE,
                    "forward_noalloc: %lld samples need %zu bytes of scratch, the static buffer "
                    "holds %zu (use bitlogic_network_forward with a workspace)",
                    (long long)n_samples, fp.total, (size_t)BITLOGIC_NOALLOC_SCRATCH_BYTES);
    if (n_samples == 0)
        return ok();
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_status(e, "forward_noalloc: current device");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(BITLOGIC_ERR_UNSUPPORTED, "forward_noalloc: device %d beyond %d", dev,
                    kMaxDevices);
    if (stream) {
        hipDevice_t sdev = 0;
        e = hipStreamGetDevice((hipStream_t)stream, &sdev);
        if (e != hipSuccess)
            return hip_status(e, "forward_noalloc: stream device");
        if (sdev != dev)
            return fail(BITLOGIC_ERR_UNSUPPORTED,
                        "forward_noalloc: stream of device %d, current device %d", (int)sdev, dev);
    }
    void *ws = nullptr;
    st = scratch_address(dev, &ws);
    if (st != BITLOGIC_OK)
        return st;
    return forward_impl(net, x, n_samples, out, argmax, ws, BITLOGIC_NOALLOC_SCRATCH_BYTES,
                        stream, nullptr, 0);
}

int bitlogic_encode_binary(const uint8_t *x, int64_t n_samples, int32_t n_features,
                           int32_t n_bits, uint64_t *bits_out, void *stream)
{
    if (!x || !bits_out)
        return fail(BITLOGIC_ERR_NULL, "encode_binary: NULL pointer");
    if (n_samples < 0 || n_features <= 0 || n_bits < 1 || n_bits > 8)
        return fail(BITLOGIC_ERR_SHAPE, "encode_binary: need n >= 0, d > 0, 1 <= n_bits <= 8");
    if ((int64_t)n_features * n_bits > kMaxRows)
        return fail(BITLOGIC_ERR_SHAPE, "encode_binary: d * n_bits exceeds int32");
    if (!aligned(bits_out, 8))
        return fail(BITLOGIC_ERR_ALIGN, "encode_binary: bits_out not 8-byte aligned");
    if (n_samples == 0)
        return ok();
    return hip_status(bl::launch_encode(x, n_samples, n_features, nullptr, n_bits, bits_out,
                                        bl::kLayoutRowMajor, words_of(n_samples),
                                        (hipStream_t)stream, bl::kEncBinary),
                      "encode_binary launch");
}

int bitlogic_specialize_layer(const int32_t *conn, const uint64_t *tables, int32_t w_out,
                              int32_t k, int32_t w_in, int32_t *k_eff, int32_t *conn_out,
                              uint64_t *tables_out)
{
    if (!conn || !tables || !k_eff || !conn_out || !tables_out)
        return fail(BITLOGIC_ERR_NULL, "specialize_layer: NULL pointer");
    if (k < 1 || k > 6)
        return fail(BITLOGIC_ERR_UNSUPPORTED, "specialize_layer: fan-in %d outside 1..6", k);
    if (w_out < 0 || w_in <= 0)
        return fail(BITLOGIC_ERR_SHAPE, "specialize_layer: need w_out >= 0, w_in > 0");
    for (int64_t q = 0; q < (int64_t)w_out * k; ++q)
        if (conn[q] < 0 || conn[q] >= w_in)
            return fail(BITLOGIC_ERR_SHAPE, "specialize_layer: connection %lld = %d outside [0, %d)",
                        (long long)q, conn[q], w_in);
    for (int32_t j = 0; j < w_out; ++j) {
        int32_t *co = conn_out + (int64_t)j * k;
        k_eff[j] = bl::specialize_node(conn + (int64_t)j * k, tables[j], k, co, &tables_out[j]);
        for (int i = k_eff[j]; i < k; ++i)
            co[i] = 0;
    }
    return ok();
}

int bitlogic_specialize_network(int32_t w_in, const int32_t *const *conn,
                                const uint64_t *const *tables, const int32_t *w_out,
                                const int32_t *k, int32_t n_layers, int32_t n_classes,
                                double min_gain, int32_t *k_out, int32_t *applied_out,
                                int32_t *const *conn_out, uint64_t *const *tables_out,
                                uint8_t *const *fanin_out, int32_t *const *order_out)
{
    if (!conn || !tables || !w_out || !k || !k_out || !applied_out || !conn_out || !tables_out ||
        !fanin_out)
        return fail(BITLOGIC_ERR_NULL, "specialize_network: NULL pointer");
    if (n_layers < 1 || w_in <= 0 || n_classes < 1)
        return fail(BITLOGIC_ERR_SHAPE, "specialize_network: need n_layers, w_in, n_classes > 0");
    int32_t wi = w_in;
    for (int32_t l = 0; l < n_layers; ++l) {
        if (!conn[l] || !tables[l] || !conn_out[l] || !tables_out[l] || !fanin_out[l] ||
            (order_out && !order_out[l]))
            return fail(BITLOGIC_ERR_NULL, "specialize_network: layer %d NULL pointer", l);
        if (k[l] < 1 || k[l] > 6)
            return fail(BITLOGIC_ERR_UNSUPPORTED, "specialize_network: layer %d fan-in %d", l,
                        k[l]);
        if (w_out[l] <= 0)
            return fail(BITLOGIC_ERR_SHAPE, "specialize_network: layer %d width %d", l, w_out[l]);
        for (int64_t q = 0; q < (int64_t)w_out[l] * k[l]; ++q)
            if (conn[l][q] < 0 || conn[l][q] >= wi)
                return fail(BITLOGIC_ERR_SHAPE,
                            "specialize_network: layer %d connection %lld = %d outside [0, %d)",
                            l, (long long)q, conn[l][q], wi);
        wi = w_out[l];
    }
    if (wi % n_classes != 0)
        return fail(BITLOGIC_ERR_SHAPE, "specialize_network: last width %d not a multiple of %d",
                    wi, n_classes);
    if (!(min_gain >= 0.0 && min_gain <= 1.0))
        return fail(BITLOGIC_ERR_SHAPE, "specialize_network: min_gain outside [0, 1]");
    bl::specialize_network(w_in, n_layers, w_out, k, conn, tables, n_classes, min_gain, k_out,
                           applied_out, conn_out, tables_out, fanin_out, order_out);
    return ok();
}

size_t bitlogic_fit_quantile_thresholds_workspace_bytes(int32_t n_groups)
{
    if (n_groups < 1 || n_groups > bl::kFitMaxGroups)
        return 0;
    return (size_t)n_groups * 256 * sizeof(uint64_t);
}

int bitlogic_fit_quantile_thresholds(const uint8_t *x, int64_t n_samples, int32_t n_features,
                                     int32_t n_thresholds, int32_t n_groups,
                                     uint8_t *thresholds_out, void *workspace,
                                     size_t workspace_bytes, void *stream)
{
    if (!x || !thresholds_out || !workspace)
        return fail(BITLOGIC_ERR_NULL, "fit_quantiles: NULL pointer");
    if (n_samples < 1 || n_features < 1 || n_thresholds < 1 || n_thresholds > 64)
        return fail(BITLOGIC_ERR_SHAPE, "fit_quantiles: need n >= 1, d >= 1, 1 <= b <= 64");
    if (n_groups < 1 || n_groups > bl::kFitMaxGroups || n_features % n_groups != 0)
        return fail(BITLOGIC_ERR_SHAPE, "fit_quantiles: %d groups of %d features", n_groups,
                    n_features);
    if (n_samples > ((int64_t)1 << 56) / n_features)
        return fail(BITLOGIC_ERR_SHAPE, "fit_quantiles: n * d exceeds 2^56");
    if (workspace_bytes < bitlogic_fit_quantile_thresholds_workspace_bytes(n_groups))
        return fail(BITLOGIC_ERR_WORKSPACE, "fit_quantiles: workspace too small");
    if (!aligned(workspace, 8))
        return fail(BITLOGIC_ERR_ALIGN, "fit_quantiles: workspace not 8-byte aligned");
    return hip_status(bl::launch_fit_quantiles(x, n_samples, n_features, n_thresholds, n_groups,
                                               thresholds_out,
                                               static_cast<uint64_t *>(workspace),
                                               (hipStream_t)stream),
                      "fit_quantiles launch");
}

const char *bitlogic_status_string(int status)
{
    switch (status) {
    case BITLOGIC_OK: return "ok";
    case BITLOGIC_ERR_NULL: return "a required pointer is NULL";
    case BITLOGIC_ERR_SHAPE: return "a size is out of range or inconsistent";
    case BITLOGIC_ERR_ALIGN: return "a buffer is not aligned as required";
    case BITLOGIC_ERR_UNSUPPORTED: return "unsupported parameter";
    case BITLOGIC_ERR_HIP: return "HIP runtime error";
    case BITLOGIC_ERR_WORKSPACE: return "workspace too small";
    default: return "unknown status";
    }
}

const char *bitlogic_last_error(void) { return g_last_error; }

int bitlogic_version(void) { return BITLOGIC_VERSION; }

int bitlogic_probe_valu(uint32_t *out, int32_t blocks, int32_t iters, uint32_t seed,
                        void *stream)
{
    if (!out)
        return fail(BITLOGIC_ERR_NULL, "probe_valu: NULL output");
    if (blocks < 1 || iters < 0)
        return fail(BITLOGIC_ERR_SHAPE, "probe_valu: need blocks >= 1, iters >= 0");
    if (!aligned(out, 4))
        return fail(BITLOGIC_ERR_ALIGN, "probe_valu: output not 4-byte aligned");
    return hip_status(bl::launch_probe_valu(out, blocks, iters, seed, (hipStream_t)stream),
                      "probe_valu launch");
}

int bitlogic_probe_valu_op(int32_t op, uint32_t *out, int32_t blocks, int32_t iters,
                           uint32_t seed, void *stream)
{
    if (op < BITLOGIC_PROBE_OP_MUX || op > BITLOGIC_PROBE_OP_BFE)
        return fail(BITLOGIC_ERR_UNSUPPORTED, "probe_valu_op: unknown op %d", op);
    if (!out)
        return fail(BITLOGIC_ERR_NULL, "probe_valu_op: NULL output");
    if (blocks < 1 || iters < 1)
        return fail(BITLOGIC_ERR_SHAPE, "probe_valu_op: need blocks >= 1, iters >= 1");
    if (!aligned(out, 4))
        return fail(BITLOGIC_ERR_ALIGN, "probe_valu_op: output not 4-byte aligned");
    return hip_status(bl::launch_probe_valu_op(op, out, blocks, iters, seed, (hipStream_t)stream),
                      "probe_valu_op launch");
}

int bitlogic_probe_gather(const void *rows, int64_t n_rows, int32_t lanes_per_row,
                          int32_t valu_per_pass, int32_t blocks, int32_t passes,
                          int32_t waves_per_simd, uint32_t seed, uint32_t *out, void *sink,
                          void *stream)
{
    if (lanes_per_row != 4 && lanes_per_row != 8)
        return fail(BITLOGIC_ERR_UNSUPPORTED, "probe_gather: lanes_per_row %d not 4 or 8",
                    lanes_per_row);
    if (valu_per_pass != 0 && valu_per_pass != 256 && valu_per_pass != 512 &&
        valu_per_pass != 768)
        return fail(BITLOGIC_ERR_UNSUPPORTED, "probe_gather: valu_per_pass %d not 0, 256, 512 "
                    "or 768", valu_per_pass);
    if (!rows || !out)
        return fail(BITLOGIC_ERR_NULL, "probe_gather: NULL rows or output");
    if (n_rows < 1 || n_rows > 0xFFFFFFFFll || blocks < 1 || passes < 1 || waves_per_simd < 0 ||
        waves_per_simd > 8)
        return fail(BITLOGIC_ERR_SHAPE, "probe_gather: need 1 <= n_rows < 2^32, blocks >= 1, "
                    "passes >= 1, 0 <= waves_per_simd <= 8");
    if ((int64_t)blocks * passes * 64 * 6 > 0xFFFFFFFFll)
        return fail(BITLOGIC_ERR_SHAPE, "probe_gather: blocks * passes too large");
    if (!aligned(rows, 16) || !aligned(out, 4) || (sink && !aligned(sink, 16)))
        return fail(BITLOGIC_ERR_ALIGN, "probe_gather: rows and sink need 16-byte alignment");
    return hip_status(bl::launch_probe_gather(rows, n_rows, lanes_per_row, valu_per_pass, blocks,
                                              passes, waves_per_simd, seed, out, sink,
                                              (hipStream_t)stream),
                      "probe_gather launch");
}

int bitlogic_probe_hbm(int32_t mode, const void *in, void *out, int64_t n_bytes,
                       int32_t unroll, int32_t blocks, void *stream)
{
    if (mode != BITLOGIC_PROBE_HBM_COPY && mode != BITLOGIC_PROBE_HBM_READ &&
        mode != BITLOGIC_PROBE_HBM_WRITE)
        return fail(BITLOGIC_ERR_UNSUPPORTED, "probe_hbm: unknown mode %d", mode);
    if (unroll != 1 && unroll != 2 && unroll != 4 && unroll != 8)
        return fail(BITLOGIC_ERR_UNSUPPORTED, "probe_hbm: unroll %d not 1, 2, 4 or 8", unroll);
    if (n_bytes < 0 || n_bytes % 16 != 0 || blocks < 0)
        return fail(BITLOGIC_ERR_SHAPE, "probe_hbm: n_bytes %lld not a multiple of 16, or "
                    "blocks < 0", (long long)n_bytes);
    const bool reads = mode != BITLOGIC_PROBE_HBM_WRITE;
    if (mode == BITLOGIC_PROBE_HBM_READ) {
        if (!out || (n_bytes > 0 && !in))
            return fail(BITLOGIC_ERR_NULL, "probe_hbm: NULL buffer");
        if ((in && !aligned(in, 16)) || !aligned(out, 16))
            return fail(BITLOGIC_ERR_ALIGN, "probe_hbm: buffers not 16-byte aligned");
        return hip_status(bl::launch_probe_hbm(bl::kHbmRead, in, out, n_bytes, unroll, blocks,
                                               (hipStream_t)stream),
                          "probe_hbm launch");
    }
    if (n_bytes == 0)
        return ok();
    if (!out || (reads && !in))
        return fail(BITLOGIC_ERR_NULL, "probe_hbm: NULL buffer");
    if (!aligned(out, 16) || (reads && !aligned(in, 16)))
        return fail(BITLOGIC_ERR_ALIGN, "probe_hbm: buffers not 16-byte aligned");
    if (reads) {
        const char *a = static_cast<const char *>(in), *b = static_cast<const char *>(out);
        if (a < b + n_bytes && b < a + n_bytes)
            return fail(BITLOGIC_ERR_SHAPE, "probe_hbm: buffers overlap");
    }
    return hip_status(bl::launch_probe_hbm(mode == BITLOGIC_PROBE_HBM_COPY ? bl::kHbmCopy
                                                                            : bl::kHbmWrite,
                                           in, out, n_bytes, unroll, blocks,
                                           (hipStream_t)stream),
                      "probe_hbm launch");
}

}  // extern "C"
