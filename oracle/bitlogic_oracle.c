/*
 * BitLogic CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, per-sample implementation of the forward pass of a
 * two-layer (or D-layer) LUT network, written directly from the paper's
 * definitions, used only to check the HIP path.  Only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark may load it; the
 * product library never links or calls it, and the two share no code.
 *
 * Representation: every Boolean value is one byte (0 or 1), samples are
 * processed one at a time, and nothing is bit-packed, so that each step
 * can be checked against the paper by eye.
 *
 *   Forward composition  E -> [L_M(f^(n))]^D -> H          (Sec. 3, Eq. 1)
 *   Encoder   R^d -> {0,1}^{d b}, thermometer wires        (Sec. 3, "Encoders
 *             and heads"; App. A "Initialization";
 *             App. B "MNIST-specific encoder collapse")
 *   Layer     node j reads inputs through its map M_j and
 *             indexes its 2^n-entry truth table            (Sec. 3, "Nodes are
 *             parameterizations", "Connectivity is the main per-layer
 *             design choice"; App. C.1 "Bit-packed inference")
 *   Head      popcount GroupSum, c class scores            (Sec. 3, "Encoders
 *             and heads"; Sec. 5 "Head")
 *   DSP head  c x c signed 8-bit matrix on the group sums  (Sec. 3, "Encoders
 *             and heads"; Sec. 5 "Head", head sweep table)
 *   Binary    uniform fixed-point code, 2^b levels on b    (Sec. 3, "Encoders
 *   encoder   wires                                        and heads"; Sec. 5
 *                                                          "Encoder")
 *   Quantile  thresholds fitted from the data's quantiles  (Sec. 4
 *   fitting                                                "Initialization";
 *                                                          App. B)
 *   Argmax    predicted class index                        (App. C.2 "HDL
 *             export and emission modes": the top module outputs it)
 *
 * Readings where the paper is silent (each one also listed in the design
 * notes): comparison is strict (x > theta), thresholds are integers on the
 * raw 0..255 pixel scale, encoder wire of (feature f, threshold t) is
 * f*b + t, LUT address bit i comes from connection slot i (entry a of the
 * table is bit a of a 64-bit word), class i owns the contiguous nodes
 * [i*g, (i+1)*g) with g = w/c, argmax breaks ties toward the lowest class
 * index, and the quantized head computes logit i from row i of its matrix
 * (the convention of a linear layer's weight) with no bias term.
 *
 * Parity status: every function here is pinned by the CPU tests against
 * closed forms, textbook truth tables, brute force over all inputs of tiny
 * networks and invariants of the paper's definitions.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_ERR_ARG 1
#define ORACLE_ERR_RANGE 2
#define ORACLE_ERR_NOMEM 3

/* Thermometer encoder of one sample (Sec. 3 "Encoders and heads"): each of
 * the d input dimensions emits b wires; wire (f, t) is 1 when the pixel
 * exceeds the t-th threshold of feature f. */
static void encode_one(const uint8_t *x_row, int32_t d, const uint8_t *theta,
                       int32_t b, uint8_t *e)
{
    for (int32_t f = 0; f < d; ++f)
        for (int32_t t = 0; t < b; ++t)
            e[(int64_t)f * b + t] = (x_row[f] > theta[(int64_t)f * b + t]) ? 1 : 0;
}

/* Binary-coded uniform fixed-point encoder of one sample (Sec. 3 "Encoders and
 * heads": the integer quantizer with 2^b levels on b wires; Sec. 5 "Encoder",
 * the encoder sweep table).  The pixel v/255 in [0, 1] is quantized to the
 * nearest of the 2^b equispaced levels q/(2^b - 1), q = round(v (2^b-1) / 255)
 * (no ties occur: 255 is odd), and wire (f, t) carries bit t of q, least
 * significant first. */
static void encode_binary_one(const uint8_t *x_row, int32_t d, int32_t b, uint8_t *e)
{
    const int64_t top = ((int64_t)1 << b) - 1;
    for (int32_t f = 0; f < d; ++f) {
        const int64_t q = (2 * (int64_t)x_row[f] * top + 255) / 510;
        for (int32_t t = 0; t < b; ++t)
            e[(int64_t)f * b + t] = (uint8_t)((q >> t) & 1);
    }
}

/* One LUT layer on one sample (Sec. 3, connection map M_j and the 2^n-entry
 * truth table; App. C.1, table plus routing indices in a common input bit
 * order).  Node j forms the address a = sum_i v[M_j(i)] * 2^i and outputs
 * entry a of its table. */
static void layer_one(const uint8_t *v_in, const int32_t *conn,
                      const uint64_t *tables, int32_t w_out, int32_t k,
                      uint8_t *v_out)
{
    for (int32_t j = 0; j < w_out; ++j) {
        uint32_t a = 0;
        for (int32_t i = 0; i < k; ++i)
            a += (uint32_t)v_in[conn[(int64_t)j * k + i]] << i;
        v_out[j] = (uint8_t)((tables[j] >> a) & 1u);
    }
}

/* GroupSum head plus argmax on one sample (Sec. 3 "Encoders and heads",
 * Sec. 5 "Head"): class i sums the bits of its node group; the prediction is
 * the first class holding the largest score. */
static void head_one(const uint8_t *v, int32_t w, int32_t c,
                     int32_t *scores, int32_t *pred)
{
    const int32_t g = w / c;
    int32_t best = 0;
    for (int32_t i = 0; i < c; ++i) {
        int32_t s = 0;
        for (int32_t j = i * g; j < (i + 1) * g; ++j)
            s += v[j];
        scores[i] = s;
        if (s > scores[best])
            best = i;
    }
    *pred = best;
}

/* Quantized class head on one sample (Sec. 3 "Encoders and heads": the
 * quantized variant of the popcount head; Sec. 5 "Head", the DSP-backed head
 * of the head sweep table): a c x c matrix of signed 8-bit weights multiplies
 * the length-c group-sum vector, logit i = sum_j q[i][j] * count[j] (row i of
 * q produces class i, no bias), and the prediction is the first class holding
 * the largest logit.  Logits are exact in 64-bit integers. */
static void dsp_one(const int32_t *counts, int32_t c, const int8_t *q, int64_t *logits,
                    int32_t *pred)
{
    int32_t best = 0;
    for (int32_t i = 0; i < c; ++i) {
        int64_t acc = 0;
        for (int32_t j = 0; j < c; ++j)
            acc += (int64_t)q[(int64_t)i * c + j] * counts[j];
        logits[i] = acc;
        if (acc > logits[best])
            best = i;
    }
    *pred = best;
}

static int check_conn(const int32_t *conn, int32_t w_out, int32_t k, int32_t w_in)
{
    for (int64_t q = 0; q < (int64_t)w_out * k; ++q)
        if (conn[q] < 0 || conn[q] >= w_in)
            return ORACLE_ERR_RANGE;
    return ORACLE_OK;
}

static void set_threads(int32_t n_threads)
{
#ifdef _OPENMP
    if (n_threads > 0)
        omp_set_num_threads(n_threads);
#else
    (void)n_threads;
#endif
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* e [n][d*b] bytes */
int oracle_encode(const uint8_t *x, int64_t n, int32_t d, const uint8_t *theta,
                  int32_t b, uint8_t *e)
{
    if (!x || !theta || !e || n < 0 || d <= 0 || b <= 0)
        return ORACLE_ERR_ARG;
    for (int64_t s = 0; s < n; ++s)
        encode_one(x + s * d, d, theta, b, e + s * (int64_t)d * b);
    return ORACLE_OK;
}

/* v_in [n][w_in] bytes -> v_out [n][w_out] bytes */
int oracle_lut_layer(const uint8_t *v_in, int64_t n, int32_t w_in,
                     const int32_t *conn, const uint64_t *tables, int32_t w_out,
                     int32_t k, uint8_t *v_out)
{
    if (!v_in || !conn || !tables || !v_out || n < 0 || w_in <= 0 || w_out <= 0 ||
        k < 1 || k > 6)
        return ORACLE_ERR_ARG;
    if (check_conn(conn, w_out, k, w_in) != ORACLE_OK)
        return ORACLE_ERR_RANGE;
    for (int64_t s = 0; s < n; ++s)
        layer_one(v_in + s * w_in, conn, tables, w_out, k, v_out + s * w_out);
    return ORACLE_OK;
}

/* v [n][w] bytes -> scores [n][c], pred [n] */
int oracle_groupsum(const uint8_t *v, int64_t n, int32_t w, int32_t c,
                    int32_t *scores, int32_t *pred)
{
    if (!v || !scores || !pred || n < 0 || w <= 0 || c <= 0 || w % c != 0)
        return ORACLE_ERR_ARG;
    for (int64_t s = 0; s < n; ++s)
        head_one(v + s * w, w, c, scores + s * c, pred + s);
    return ORACLE_OK;
}

/* e [n][d*b] bytes, binary-coded encoder, 1 <= b <= 16 */
int oracle_encode_binary(const uint8_t *x, int64_t n, int32_t d, int32_t b, uint8_t *e)
{
    if (!x || !e || n < 0 || d <= 0 || b < 1 || b > 16)
        return ORACLE_ERR_ARG;
    for (int64_t s = 0; s < n; ++s)
        encode_binary_one(x + s * d, d, b, e + s * (int64_t)d * b);
    return ORACLE_OK;
}

/* Quantile thermometer thresholds fitted from data (Sec. 4 "Initialization":
 * fitted once from the empirical pixel quantiles of the training split;
 * App. B: over the flattened pixel distribution).  The d features are cut
 * into n_groups contiguous groups of d / n_groups features (1 group: the
 * whole flattened distribution; one group per colour channel for CHW
 * images); in each group, with cum(v) = number of pixels <= v among the
 * group's n * d / n_groups pixels, threshold i (i = 1..b) is the smallest v
 * with cum(v) / total >= i / (b + 1), compared exactly in integers.  Every
 * feature of the group receives the group's b thresholds: th [d][b]. */
int oracle_fit_quantiles(const uint8_t *x, int64_t n, int32_t d, int32_t b, int32_t n_groups,
                         uint8_t *th)
{
    if (!x || !th || n <= 0 || d <= 0 || b < 1 || b > 64 || n_groups < 1 || d % n_groups != 0)
        return ORACLE_ERR_ARG;
    const int32_t per = d / n_groups;
    for (int32_t grp = 0; grp < n_groups; ++grp) {
        int64_t hist[256];
        memset(hist, 0, sizeof hist);
        for (int64_t s = 0; s < n; ++s)
            for (int32_t f = grp * per; f < (grp + 1) * per; ++f)
                hist[x[s * d + f]] += 1;
        const int64_t total = n * per;
        for (int32_t i = 1; i <= b; ++i) {
            int64_t cum = 0;
            int32_t v = 0;
            for (v = 0; v < 256; ++v) {
                cum += hist[v];
                if (cum * (b + 1) >= (int64_t)i * total)
                    break;
            }
            for (int32_t f = grp * per; f < (grp + 1) * per; ++f)
                th[(int64_t)f * b + (i - 1)] = (uint8_t)v;
        }
    }
    return ORACLE_OK;
}

/* counts [n][c] int32, q [c][c] int8 -> logits [n][c] int64, pred [n] */
int oracle_grouped_dsp(const int32_t *counts, int64_t n, int32_t c, const int8_t *q,
                       int64_t *logits, int32_t *pred)
{
    if (!counts || !q || !logits || !pred || n < 0 || c <= 0)
        return ORACLE_ERR_ARG;
    for (int64_t s = 0; s < n; ++s)
        dsp_one(counts + s * c, c, q, logits + s * c, pred + s);
    return ORACLE_OK;
}

/* Whole forward, one sample at a time, OpenMP over samples.
 * conn[l] [w_out[l]][k[l]], tables[l] [w_out[l]]; layer 0 reads the d*b
 * encoder wires, layer l > 0 reads layer l-1. */
static int forward_impl(const uint8_t *x, int64_t n, int32_t d, const uint8_t *theta,
                        int32_t b, int binary, int32_t n_layers, const int32_t *const *conn,
                        const uint64_t *const *tables, const int32_t *w_out,
                        const int32_t *k, int32_t c, int32_t *scores, int32_t *pred,
                        int32_t n_threads);

int oracle_forward(const uint8_t *x, int64_t n, int32_t d, const uint8_t *theta,
                   int32_t b, int32_t n_layers, const int32_t *const *conn,
                   const uint64_t *const *tables, const int32_t *w_out,
                   const int32_t *k, int32_t c, int32_t *scores, int32_t *pred,
                   int32_t n_threads)
{
    if (!theta)
        return ORACLE_ERR_ARG;
    return forward_impl(x, n, d, theta, b, 0, n_layers, conn, tables, w_out, k, c, scores,
                        pred, n_threads);
}

/* The forward with the binary-coded encoder (b code bits per feature). */
int oracle_forward_binary(const uint8_t *x, int64_t n, int32_t d, int32_t b,
                          int32_t n_layers, const int32_t *const *conn,
                          const uint64_t *const *tables, const int32_t *w_out,
                          const int32_t *k, int32_t c, int32_t *scores, int32_t *pred,
                          int32_t n_threads)
{
    if (b > 16)
        return ORACLE_ERR_ARG;
    return forward_impl(x, n, d, NULL, b, 1, n_layers, conn, tables, w_out, k, c, scores, pred,
                        n_threads);
}

static int forward_impl(const uint8_t *x, int64_t n, int32_t d, const uint8_t *theta,
                        int32_t b, int binary, int32_t n_layers, const int32_t *const *conn,
                        const uint64_t *const *tables, const int32_t *w_out,
                        const int32_t *k, int32_t c, int32_t *scores, int32_t *pred,
                        int32_t n_threads)
{
    if (!x || !conn || !tables || !w_out || !k || !scores || !pred ||
        n < 0 || d <= 0 || b <= 0 || n_layers < 1 || c <= 0)
        return ORACLE_ERR_ARG;
    int32_t w_in = d * b, widest = d * b;
    for (int32_t l = 0; l < n_layers; ++l) {
        if (!conn[l] || !tables[l] || w_out[l] <= 0 || k[l] < 1 || k[l] > 6)
            return ORACLE_ERR_ARG;
        if (check_conn(conn[l], w_out[l], k[l], w_in) != ORACLE_OK)
            return ORACLE_ERR_RANGE;
        w_in = w_out[l];
        if (w_in > widest)
            widest = w_in;
    }
    if (w_in % c != 0)
        return ORACLE_ERR_ARG;
    const int32_t w_last = w_in;
    int status = ORACLE_OK;
    set_threads(n_threads);
#pragma omp parallel
    {
        uint8_t *cur = (uint8_t *)malloc((size_t)widest);
        uint8_t *nxt = (uint8_t *)malloc((size_t)widest);
        if (!cur || !nxt) {
#pragma omp atomic write
            status = ORACLE_ERR_NOMEM;
        } else {
#pragma omp for schedule(dynamic, 16)
            for (int64_t s = 0; s < n; ++s) {
                if (binary)
                    encode_binary_one(x + s * d, d, b, cur);
                else
                    encode_one(x + s * d, d, theta, b, cur);
                for (int32_t l = 0; l < n_layers; ++l) {
                    layer_one(cur, conn[l], tables[l], w_out[l], k[l], nxt);
                    uint8_t *t = cur; cur = nxt; nxt = t;
                }
                head_one(cur, w_last, c, scores + s * c, pred + s);
            }
        }
        free(cur);
        free(nxt);
    }
    return status;
}
