// A plain C-ABI consumer of libbitlogic (test infrastructure): it builds a
// small seeded network, runs bitlogic_forward and bitlogic_network_forward
// (binary encoder + quantized head) on the GPU through nothing but the
// entry points of bitlogic.h and the HIP runtime, and compares scores and
// argmax with the CPU oracle (liboracle, linked only into this test).
// Exit status 0 and a final "c abi ok" line when every comparison is exact.
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "bitlogic.h"

extern "C" {
int oracle_forward(const uint8_t *x, int64_t n, int32_t d, const uint8_t *theta, int32_t b,
                   int32_t n_layers, const int32_t *const *conn, const uint64_t *const *tables,
                   const int32_t *w_out, const int32_t *k, int32_t c, int32_t *scores,
                   int32_t *pred, int32_t n_threads);
int oracle_forward_binary(const uint8_t *x, int64_t n, int32_t d, int32_t b, int32_t n_layers,
                          const int32_t *const *conn, const uint64_t *const *tables,
                          const int32_t *w_out, const int32_t *k, int32_t c, int32_t *scores,
                          int32_t *pred, int32_t n_threads);
int oracle_grouped_dsp(const int32_t *counts, int64_t n, int32_t c, const int8_t *q,
                       int64_t *logits, int32_t *pred);
}

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next_u64()       // splitmix64
{
    uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

#define HIP_OK(call)                                                                 \
    do {                                                                             \
        hipError_t e_ = (call);                                                      \
        if (e_ != hipSuccess) {                                                      \
            std::fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));   \
            std::exit(2);                                                            \
        }                                                                            \
    } while (0)

#define BL_OK(call)                                                                  \
    do {                                                                             \
        int s_ = (call);                                                             \
        if (s_ != BITLOGIC_OK) {                                                     \
            std::fprintf(stderr, "%s: %s (%s)\n", #call, bitlogic_status_string(s_),  \
                         bitlogic_last_error());                                     \
            std::exit(3);                                                            \
        }                                                                            \
    } while (0)

template <typename T>
T *to_device(const std::vector<T> &h)
{
    T *d = nullptr;
    HIP_OK(hipMalloc(&d, h.size() * sizeof(T) + 16));
    HIP_OK(hipMemcpy(d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice));
    return d;
}

int mismatches(const std::vector<int32_t> &a, const std::vector<int32_t> &b)
{
    int bad = 0;
    for (size_t i = 0; i < a.size(); ++i)
        bad += a[i] != b[i];
    return bad;
}

}  // namespace

int main()
{
    std::printf("c abi: library version %d (header %d)\n", bitlogic_version(), BITLOGIC_VERSION);
    if (bitlogic_version() != BITLOGIC_VERSION)
        return 4;
    const int64_t n = 64 * 16 * 3 + 37;      // three slabs and a ragged tail
    const int32_t d = 100, b = 3, c = 10;
    const int32_t L = 2, widths[L] = {512, 320}, ks[L] = {6, 5};

    std::vector<uint8_t> x(n * d), th(d * b);
    for (auto &v : x)
        v = (uint8_t)next_u64();
    for (int32_t f = 0; f < d; ++f) {         // sorted ladders
        uint8_t t[3] = {(uint8_t)next_u64(), (uint8_t)next_u64(), (uint8_t)next_u64()};
        for (int i = 0; i < 3; ++i)
            for (int j = i + 1; j < 3; ++j)
                if (t[j] < t[i]) {
                    uint8_t s = t[i];
                    t[i] = t[j];
                    t[j] = s;
                }
        std::memcpy(&th[f * b], t, 3);
    }
    std::vector<std::vector<int32_t>> conn(L);
    std::vector<std::vector<uint64_t>> tab(L);
    int32_t w_in = d * b;
    for (int l = 0; l < L; ++l) {
        conn[l].resize((size_t)widths[l] * ks[l]);
        for (auto &v : conn[l])
            v = (int32_t)(next_u64() % (uint64_t)w_in);
        tab[l].resize(widths[l]);
        for (auto &v : tab[l])
            v = next_u64();
        w_in = widths[l];
    }
    std::vector<int8_t> q(c * c);
    for (auto &v : q)
        v = (int8_t)(next_u64() % 255 - 127);

    // ---- oracle
    const int32_t *cp[L] = {conn[0].data(), conn[1].data()};
    const uint64_t *tp[L] = {tab[0].data(), tab[1].data()};
    std::vector<int32_t> ref_s(n * c), ref_p(n), ref_bs(n * c), ref_bp(n), ref_dp(n);
    std::vector<int64_t> ref_dl(n * c);
    if (oracle_forward(x.data(), n, d, th.data(), b, L, cp, tp, widths, ks, c, ref_s.data(),
                       ref_p.data(), 0) ||
        oracle_forward_binary(x.data(), n, d, b, L, cp, tp, widths, ks, c, ref_bs.data(),
                              ref_bp.data(), 0) ||
        oracle_grouped_dsp(ref_bs.data(), n, c, q.data(), ref_dl.data(), ref_dp.data()))
        return 5;

    // ---- device
    uint8_t *dx = to_device(x), *dth = to_device(th);
    int8_t *dq = to_device(q);
    int32_t *dconn[L];
    uint64_t *dtab[L];
    bitlogic_layer layers[L];
    for (int l = 0; l < L; ++l) {
        dconn[l] = to_device(conn[l]);
        dtab[l] = to_device(tab[l]);
        layers[l] = bitlogic_layer{dconn[l], dtab[l], widths[l], ks[l]};
    }
    int32_t *dscores = nullptr, *dargmax = nullptr;
    HIP_OK(hipMalloc(&dscores, n * c * sizeof(int32_t)));
    HIP_OK(hipMalloc(&dargmax, n * sizeof(int32_t)));

    // a failed check enqueues nothing and says why
    if (bitlogic_forward(nullptr, n, d, dth, b, layers, L, c, dscores, dargmax, nullptr, 0,
                         nullptr) != BITLOGIC_ERR_NULL || std::strlen(bitlogic_last_error()) == 0)
        return 6;

    const size_t ws = bitlogic_forward_workspace_bytes(n, d, b, layers, L, c);
    void *dws = nullptr;
    HIP_OK(hipMalloc(&dws, ws));
    hipStream_t stream;
    HIP_OK(hipStreamCreate(&stream));
    BL_OK(bitlogic_forward(dx, n, d, dth, b, layers, L, c, dscores, dargmax, dws, ws, stream));
    HIP_OK(hipStreamSynchronize(stream));
    std::vector<int32_t> got_s(n * c), got_p(n);
    HIP_OK(hipMemcpy(got_s.data(), dscores, got_s.size() * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(got_p.data(), dargmax, got_p.size() * 4, hipMemcpyDeviceToHost));
    const int bad1 = mismatches(got_s, ref_s) + mismatches(got_p, ref_p);
    std::printf("c abi: bitlogic_forward, %lld samples: %d mismatches\n", (long long)n, bad1);

    // the network descriptor: binary encoder and the quantized head
    bitlogic_network net;
    std::memset(&net, 0, sizeof net);
    net.n_features = d;
    net.encoder = BITLOGIC_ENCODER_BINARY;
    net.n_bits = b;
    net.thresholds = nullptr;
    net.layers = layers;
    net.n_layers = L;
    net.n_classes = c;
    net.head = BITLOGIC_HEAD_GROUPED_DSP;
    net.head_weights = dq;
    net.pass_fanin = nullptr;
    const size_t ws2 = bitlogic_network_workspace_bytes(&net, n);
    void *dws2 = nullptr;
    HIP_OK(hipMalloc(&dws2, ws2));
    BL_OK(bitlogic_network_forward(&net, dx, n, dscores, dargmax, dws2, ws2, stream, nullptr, 0));
    HIP_OK(hipStreamSynchronize(stream));
    HIP_OK(hipMemcpy(got_s.data(), dscores, got_s.size() * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(got_p.data(), dargmax, got_p.size() * 4, hipMemcpyDeviceToHost));
    int bad2 = mismatches(got_p, ref_dp);
    for (size_t i = 0; i < got_s.size(); ++i)
        bad2 += (int64_t)got_s[i] != ref_dl[i];
    std::printf("c abi: bitlogic_network_forward (binary encoder, quantized head): %d "
                "mismatches\n", bad2);

    HIP_OK(hipStreamDestroy(stream));
    for (int l = 0; l < L; ++l) {
        HIP_OK(hipFree(dconn[l]));
        HIP_OK(hipFree(dtab[l]));
    }
    for (void *p : {(void *)dx, (void *)dth, (void *)dq, (void *)dscores, (void *)dargmax, dws, dws2})
        HIP_OK(hipFree(p));
    if (bad1 || bad2)
        return 1;
    std::printf("c abi ok\n");
    return 0;
}
