// Table specialization of LUT nodes (host code).
//
// The paper's synthesis flow emits one truth table per node and lets the
// logic synthesis tool collapse it: inputs tied to the same wire shrink a
// node to a function of fewer effective inputs, and gates on irrelevant
// inputs disappear (Sec. 5 "Connectivity", the full-candidate-pool routing
// whose tied slots reduce a 16-entry table to an effective function of at
// most 3 inputs; App. C.2, one table per node in the emitted design).  This
// is the same collapse for the GPU path, per node:
//   1. tied slots: when slots i < j read the same wire, only addresses whose
//      bits i and j agree can occur, so slot j is removed and the table
//      restricted to those addresses;
//   2. irrelevant slots: slot i is removed when the table is unchanged by
//      flipping address bit i;
//   3. the remaining k' slots keep their order, and the table is rewritten
//      over the k' remaining address bits (least significant = first slot);
//      k' = 0 is a constant node.
// A node with k' effective inputs then costs 2^k' - 1 multiplexers and k'
// gathers instead of 2^k - 1 and k.
//
// For the GPU the whole network is then rearranged so that a kernel pass
// evaluates nodes of one fan-in: each layer's nodes are ordered by effective
// fan-in, largest first (within each class group for the last layer, so the
// GroupSum of every class reads the same nodes), the next layer's
// connections are relabelled to the new positions, and every run of
// kSpecPass positions records its largest fan-in kp.  The specialized layer
// has fan-in kn, the largest effective fan-in of its nodes (at least 1), so
// its kernels are instantiated for kn inputs, not k.  Every node keeps kn
// slots: the slots past its effective fan-in repeat its first wire (wire 0
// for a constant node) and its table is extended over all kn slots so that
// it ignores them, so evaluating any kp' with k' <= kp' <= kn slots gives the
// node's output (a kernel pass spanning several runs takes their maximum).
// A layer whose multiplexer count would fall by less than min_gain keeps its
// nodes, order and tables: the specialized kernels cost a little more than
// the plain ones at equal work.
#include <algorithm>
#include <numeric>
#include <vector>

#include "bl_internal.h"

namespace bl {

namespace {

// Entry a' of the table after removing address bit `bit`, where the removed
// bit takes the value of address bit `src` (tied slot) or 0 (src < 0).
uint64_t remove_bit(uint64_t T, int k, int bit, int src)
{
    uint64_t out = 0;
    for (int a2 = 0; a2 < (1 << (k - 1)); ++a2) {
        const int low = a2 & ((1 << bit) - 1);
        const int high = (a2 >> bit) << (bit + 1);
        int a = high | low;
        if (src >= 0) {
            // bit src of the full address: src < bit keeps its position
            const int s = src < bit ? src : src + 1;
            if ((a >> s) & 1)
                a |= 1 << bit;
        }
        out |= ((T >> a) & 1u) << a2;
    }
    return out;
}

// Table over k inputs rewritten over K >= k inputs, slots k..K-1 ignored.
uint64_t extend(uint64_t T, int k, int K)
{
    uint64_t out = 0;
    const int mask = (1 << k) - 1;
    for (int a = 0; a < (1 << K); ++a)
        out |= ((T >> (a & mask)) & 1u) << a;
    return out;
}

bool irrelevant(uint64_t T, int k, int bit)
{
    for (int a = 0; a < (1 << k); ++a)
        if (!((a >> bit) & 1) && ((T >> a) & 1u) != ((T >> (a | (1 << bit))) & 1u))
            return false;
    return true;
}

}  // namespace

int specialize_node(const int32_t *conn, uint64_t T, int k, int32_t *conn_out, uint64_t *T_out)
{
    int32_t c[6];
    for (int i = 0; i < k; ++i)
        c[i] = conn[i];
    if (k < 6)
        T &= ((uint64_t)1 << (1 << k)) - 1;
    // 1. tied slots
    for (int j = 1; j < k; ++j) {
        int i = 0;
        while (i < j && c[i] != c[j])
            ++i;
        if (i < j) {
            T = remove_bit(T, k, j, i);
            for (int q = j; q + 1 < k; ++q)
                c[q] = c[q + 1];
            --k;
            --j;
        }
    }
    // 2. irrelevant slots
    for (int i = 0; i < k;) {
        if (irrelevant(T, k, i)) {
            T = remove_bit(T, k, i, -1);
            for (int q = i; q + 1 < k; ++q)
                c[q] = c[q + 1];
            --k;
        } else {
            ++i;
        }
    }
    for (int i = 0; i < k; ++i)
        conn_out[i] = c[i];
    *T_out = k < 6 ? T & (((uint64_t)1 << (1 << k)) - 1) : T;
    return k;
}

void specialize_network(int32_t w_in, int32_t L, const int32_t *w, const int32_t *k,
                        const int32_t *const *conn, const uint64_t *const *tables, int32_t c,
                        double min_gain, int32_t *k_out, int32_t *applied_out,
                        int32_t *const *conn_out, uint64_t *const *tables_out,
                        uint8_t *const *fanin_out, int32_t *const *order_out)
{
    (void)w_in;
    std::vector<int32_t> pos_prev;      // new position of each previous-layer node
    for (int32_t l = 0; l < L; ++l) {
        const int32_t wl = w[l], kl = k[l];
        std::vector<int32_t> ke(wl), ce((size_t)wl * kl);
        std::vector<uint64_t> te(wl);
        for (int32_t j = 0; j < wl; ++j)
            ke[j] = specialize_node(conn[l] + (int64_t)j * kl, tables[l][j], kl,
                                    &ce[(size_t)j * kl], &te[j]);
        const int32_t seg = (l == L - 1 && c > 0 && wl % c == 0) ? wl / c : wl;
        std::vector<int32_t> order(wl);
        std::iota(order.begin(), order.end(), 0);
        for (int32_t s0 = 0; s0 < wl; s0 += seg)
            std::stable_sort(order.begin() + s0, order.begin() + std::min(wl, s0 + seg),
                             [&](int32_t a, int32_t b) { return ke[a] > ke[b]; });
        const int32_t n_pass = (wl + kSpecPass - 1) / kSpecPass;
        std::vector<int> run_k(n_pass, 0);
        double mux_spec = 0;
        for (int32_t q = 0; q < n_pass; ++q) {
            const int32_t p0 = q * kSpecPass, p1 = std::min(wl, p0 + kSpecPass);
            for (int32_t p = p0; p < p1; ++p)
                run_k[q] = std::max(run_k[q], ke[order[p]]);
            mux_spec += (double)(p1 - p0) * ((1 << run_k[q]) - 1);
        }
        const double mux_orig = (double)wl * ((1 << kl) - 1);
        if (mux_spec > (1.0 - min_gain) * mux_orig) {
            // too little to gain: the layer stays as it is (connections
            // relabelled to the previous layer's order only)
            applied_out[l] = 0;
            k_out[l] = kl;
            for (int64_t q = 0; q < (int64_t)wl * kl; ++q) {
                const int32_t v = conn[l][q];
                conn_out[l][q] = pos_prev.empty() ? v : pos_prev[v];
            }
            std::copy(tables[l], tables[l] + wl, tables_out[l]);
            std::fill(fanin_out[l], fanin_out[l] + n_pass, (uint8_t)kl);
            if (order_out && order_out[l])
                std::iota(order_out[l], order_out[l] + wl, 0);
            pos_prev.clear();
            continue;
        }
        applied_out[l] = 1;
        // the specialized layer's fan-in: its largest effective fan-in
        int32_t kn = 1;
        for (int32_t j = 0; j < wl; ++j)
            kn = std::max(kn, ke[j]);
        k_out[l] = kn;
        for (int32_t q = 0; q < n_pass; ++q) {
            const int32_t p0 = q * kSpecPass, p1 = std::min(wl, p0 + kSpecPass);
            const int kp = run_k[q];
            fanin_out[l][q] = (uint8_t)kp;
            for (int32_t p = p0; p < p1; ++p) {
                const int32_t j = order[p];
                const int32_t *cj = &ce[(size_t)j * kl];
                int32_t *co = conn_out[l] + (int64_t)p * kn;
                for (int i = 0; i < kn; ++i) {
                    const int32_t v = i < ke[j] ? cj[i] : (ke[j] > 0 ? cj[0] : 0);
                    co[i] = pos_prev.empty() ? v : pos_prev[v];
                }
                tables_out[l][p] = extend(te[j], ke[j], kn);
            }
        }
        if (order_out && order_out[l])
            std::copy(order.begin(), order.end(), order_out[l]);
        pos_prev.assign(wl, 0);
        for (int32_t p = 0; p < wl; ++p)
            pos_prev[order[p]] = p;
    }
}

}  // namespace bl
