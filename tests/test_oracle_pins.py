"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

None of these checks re-types the oracle's formulas: each compares the oracle
with a closed form, a textbook truth table, a case the paper states, a brute
force over every input of a tiny network built in a different formulation
(truth tables composed as big integers), or an invariant.  A plausible slip in
the oracle -- address bit order, connection indexing, comparison strictness,
wire order, group assignment, argmax tie-break -- fails at least one test.
"""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _truth_tables():
    rows = []
    with open(os.path.join(GOLDEN, "truth_tables.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, k, table = line.split()[:3]
            rows.append((name, int(k), int(table, 16)))
    return rows


def _distinct_conn(rng, w, k, w_in):
    return np.stack([rng.choice(w_in, size=k, replace=False) for _ in range(w)]).astype(np.int32)


# ---------------------------------------------------------------- LUT layer

def _reference_function(name, xs):
    """xs: list of k boolean arrays.  Independent numpy definitions."""
    if name.startswith("proj"):
        i = int(name[4])
        return xs[i]
    if name.startswith("and"):
        return np.logical_and.reduce(xs)
    if name.startswith("or"):
        return np.logical_or.reduce(xs)
    if name.startswith("parity") or name.startswith("xor"):
        return np.logical_xor.reduce(xs)
    if name == "maj3":
        return (xs[0].astype(int) + xs[1] + xs[2]) >= 2
    if name == "nand2":
        return ~np.logical_and(xs[0], xs[1])
    raise KeyError(name)


@pytest.mark.parametrize("name,k,table", _truth_tables())
def test_textbook_tables(name, k, table):
    rng = np.random.default_rng(11)
    n, w_in, w = 300, 23, 17
    v = rng.integers(0, 2, size=(n, w_in), dtype=np.uint8)
    conn = _distinct_conn(rng, w, k, w_in)
    tables = np.full(w, table, dtype=np.uint64)
    out = oracle.lut_layer(v, conn, tables)
    for j in range(w):
        xs = [v[:, conn[j, i]].astype(bool) for i in range(k)]
        np.testing.assert_array_equal(out[:, j].astype(bool), _reference_function(name, xs),
                                      err_msg=f"{name} node {j}")


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5, 6])
def test_projection_tables_all_k(k):
    """Closed form: the table whose entry a is bit i of a reproduces input slot i."""
    rng = np.random.default_rng(k)
    n, w_in = 200, 40
    v = rng.integers(0, 2, size=(n, w_in), dtype=np.uint8)
    for i in range(k):
        proj = sum(1 << a for a in range(1 << k) if (a >> i) & 1)
        conn = _distinct_conn(rng, 13, k, w_in)
        out = oracle.lut_layer(v, conn, np.full(13, proj, dtype=np.uint64))
        np.testing.assert_array_equal(out, v[:, conn[:, i]])


@pytest.mark.parametrize("k", [1, 2, 4, 6])
def test_constant_tables(k):
    rng = np.random.default_rng(5)
    v = rng.integers(0, 2, size=(128, 30), dtype=np.uint8)
    conn = _distinct_conn(rng, 20, k, 30)
    ones = np.full(20, (1 << (1 << k)) - 1, dtype=np.uint64)
    assert not oracle.lut_layer(v, conn, np.zeros(20, np.uint64)).any()
    assert oracle.lut_layer(v, conn, ones).all()
    # the unused high bits of the table word never matter for k < 6
    if k < 6:
        junk = np.uint64(((1 << 64) - 1) ^ ((1 << (1 << k)) - 1))
        assert not oracle.lut_layer(v, conn, np.full(20, junk, dtype=np.uint64)).any()


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5, 6])
def test_enumeration_reads_table(k):
    """A node wired to inputs 0..k-1, fed every pattern a, outputs entry a."""
    rng = np.random.default_rng(100 + k)
    a = np.arange(1 << k)
    v = ((a[:, None] >> np.arange(k)[None, :]) & 1).astype(np.uint8)
    conn = np.arange(k, dtype=np.int32)[None, :]
    for _ in range(8):
        t = int(rng.integers(0, 1 << 63)) * 2 + int(rng.integers(0, 2))
        out = oracle.lut_layer(v, conn, np.array([t], dtype=np.uint64))[:, 0]
        expect = np.array([(t >> int(q)) & 1 for q in a], dtype=np.uint8)
        np.testing.assert_array_equal(out, expect)
        if k == 6:
            # 64 samples packed LSB-first reproduce the table word itself
            assert sum(int(bit) << q for q, bit in enumerate(out)) == t


def test_repeated_inputs():
    """Slots wired to the same wire can only reach addresses with equal bits."""
    v = np.array([[0, 1], [1, 0]], dtype=np.uint8)
    # k = 2, both slots on wire 0: only entries 0 (x=0) and 3 (x=1) are reachable
    conn = np.array([[0, 0]], dtype=np.int32)
    for t in range(16):
        out = oracle.lut_layer(v, conn, np.array([t], dtype=np.uint64))[:, 0]
        assert out[0] == (t >> 0) & 1 and out[1] == (t >> 3) & 1
    # xor of a wire with itself is constant 0; xnor constant 1
    assert not oracle.lut_layer(v, conn, np.array([0x6], dtype=np.uint64)).any()
    assert oracle.lut_layer(v, conn, np.array([0x9], dtype=np.uint64)).all()
    # k = 6 with a triple repeat: x0 = x1 = x2 = wire 1, x3..x5 = wires 0,0,0
    conn6 = np.array([[1, 1, 1, 0, 0, 0]], dtype=np.int32)
    t = 0x8000000000000001  # entries 0 and 63: and6 | nor6
    out = oracle.lut_layer(v, conn6, np.array([t], dtype=np.uint64))[:, 0]
    # sample 0: wire0=0, wire1=1 -> address 0b000111 = 7 -> 0
    # sample 1: wire0=1, wire1=0 -> address 0b111000 = 56 -> 0
    assert list(out) == [0, 0]


def test_layer_rejects_out_of_range():
    v = np.zeros((4, 8), dtype=np.uint8)
    with pytest.raises(ValueError):
        oracle.lut_layer(v, np.array([[0, 8]], dtype=np.int32), np.zeros(1, np.uint64))


# ------------------------------------------------------------------ encoder

def test_encoder_exhaustive_counts():
    """Wire count per feature = #{t : theta_t < x}; strict comparison."""
    rng = np.random.default_rng(3)
    x = np.arange(256, dtype=np.uint8)[:, None]
    for b in (1, 3, 7, 8):
        for _ in range(5):
            th = np.sort(rng.integers(0, 256, size=b)).astype(np.uint8)[None, :]
            e = oracle.encode(x, th)
            counts = e.sum(axis=1)
            expect = np.array([int((th[0] < v).sum()) for v in range(256)])
            np.testing.assert_array_equal(counts, expect)
            # each wire is a step function switching on just above its threshold
            for t in range(b):
                assert not e[: int(th[0, t]) + 1, t].any()
                assert e[int(th[0, t]) + 1:, t].all()


def test_encoder_edges():
    x = np.arange(256, dtype=np.uint8)[:, None]
    # x = 0 never fires; theta = 255 never fires; theta = x does not fire
    assert not oracle.encode(np.zeros((1, 5), np.uint8), np.zeros((5, 2), np.uint8)).any()
    assert not oracle.encode(x, np.full((1, 4), 255, np.uint8)).any()
    for v in range(256):
        assert oracle.encode(np.array([[v]], np.uint8), np.array([[v]], np.uint8))[0, 0] == 0


def test_encoder_wire_order():
    """Wire f*b + t belongs to feature f, threshold t."""
    d, b = 5, 3
    th = (np.arange(d * b).reshape(d, b) * 7 + 10).astype(np.uint8)
    rng = np.random.default_rng(9)
    x = rng.integers(0, 256, size=(50, d), dtype=np.uint8)
    e = oracle.encode(x, th)
    for f in range(d):
        for t in range(b):
            np.testing.assert_array_equal(e[:, f * b + t], (x[:, f] > th[f, t]).astype(np.uint8))


def test_encoder_collapse_golden():
    """The quantile-threshold collapse on MNIST stated in App. B."""
    with open(os.path.join(GOLDEN, "encoder_collapse.txt")) as f:
        rows = [l.split() for l in f if l.strip() and not l.startswith("#")]
    for b, ladder, px, bits in rows:
        th = np.array([[int(v) for v in ladder.split(",")]], dtype=np.uint8)
        assert th.shape[1] == int(b)
        e = oracle.encode(np.array([[int(px)]], np.uint8), th)[0]
        assert "".join(str(int(q)) for q in e) == bits
    # b = 4 collapses to one effective bit, b = 8 to three levels (2 bits)
    x = np.arange(256, dtype=np.uint8)[:, None]
    codes4 = {tuple(r) for r in oracle.encode(x, np.zeros((1, 4), np.uint8))}
    codes8 = {tuple(r) for r in oracle.encode(x, np.array([[0] * 7 + [180]], np.uint8))}
    assert len(codes4) == 2 and len(codes8) == 3


# --------------------------------------------------------------------- head

def test_head_counts_by_packed_popcount():
    rng = np.random.default_rng(21)
    n, c, g = 100, 7, 13
    v = rng.integers(0, 2, size=(n, c * g), dtype=np.uint8)
    scores, pred = oracle.groupsum(v, c)
    for s in range(n):
        for i in range(c):
            word = sum(int(v[s, i * g + q]) << q for q in range(g))
            assert scores[s, i] == bin(word).count("1")
    np.testing.assert_array_equal(scores.sum(axis=1), v.sum(axis=1))


def test_head_groups_are_contiguous():
    n, c, g = 1, 4, 5
    for hot in range(c):
        v = np.zeros((n, c * g), np.uint8)
        v[0, hot * g:(hot + 1) * g] = 1
        scores, pred = oracle.groupsum(v, c)
        assert list(scores[0]) == [g if i == hot else 0 for i in range(c)]
        assert pred[0] == hot


def test_head_argmax_ties_lowest_index():
    c, g = 6, 3
    v = np.zeros((4, c * g), np.uint8)
    v[1, 2 * g:2 * g + 2] = 1          # class 2: 2
    v[1, 5 * g:5 * g + 2] = 1          # class 5: 2 (tie)
    v[2, :] = 1                        # all classes g
    v[3, 4 * g:5 * g] = 1
    v[3, 1 * g] = 1
    scores, pred = oracle.groupsum(v, c)
    assert list(pred) == [0, 2, 0, 4]
    # single class: score is the total count, prediction is always 0
    s1, p1 = oracle.groupsum(v, 1)
    np.testing.assert_array_equal(s1[:, 0], v.sum(axis=1))
    assert not p1.any()


# ------------------------------------------------- whole network, brute force

def _tt_compose(w_in, layers):
    """Truth tables over all 2^w_in input patterns, as Python big integers.

    Wire i's table has bit p set when bit i of pattern p is set.  A node's
    table is the OR over the table entries a that are 1 of the AND over its
    slots of the slot table (bit i of a set) or its complement.
    """
    P = 1 << w_in
    full = (1 << P) - 1
    wires = []
    for i in range(w_in):
        tt = 0
        for p in range(P):
            if (p >> i) & 1:
                tt |= 1 << p
        wires.append(tt)
    for conn, tables in layers:
        nxt = []
        for j in range(conn.shape[0]):
            k = conn.shape[1]
            acc = 0
            for a in range(1 << k):
                if (int(tables[j]) >> a) & 1:
                    term = full
                    for i in range(k):
                        src = wires[int(conn[j, i])]
                        term &= src if (a >> i) & 1 else (full ^ src)
                    acc |= term
            nxt.append(acc)
        wires = nxt
    return wires


@pytest.mark.parametrize("seed", range(6))
def test_tiny_networks_brute_force(seed):
    rng = np.random.default_rng(1000 + seed)
    w_in = int(rng.integers(6, 11))
    k1, k2 = int(rng.integers(1, 7)), int(rng.integers(1, 7))
    c = int(rng.integers(1, 3))
    w1 = int(rng.integers(max(k2, 2), 9))
    w2 = c * int(rng.integers(1, 5))
    k1 = min(k1, w_in)
    repeats = seed % 2 == 1
    def conn_for(w, k, wi):
        if repeats:   # learnable routing may wire one input twice
            return rng.integers(0, wi, size=(w, k)).astype(np.int32)
        return _distinct_conn(rng, w, k, wi)
    layers = [(conn_for(w1, k1, w_in), rng.integers(0, 1 << 62, size=w1).astype(np.uint64) * 3),
              (conn_for(w2, k2, w1), rng.integers(0, 1 << 62, size=w2).astype(np.uint64) * 5)]
    P = 1 << w_in
    # input pattern p on the wires via the encoder: x in {0,1}, threshold 0
    x = ((np.arange(P)[:, None] >> np.arange(w_in)[None, :]) & 1).astype(np.uint8)
    th = np.zeros((w_in, 1), np.uint8)
    scores, pred = oracle.forward(x, th, layers, c)
    outs = _tt_compose(w_in, layers)
    g = w2 // c
    for p in range(P):
        bits = [(outs[j] >> p) & 1 for j in range(w2)]
        expect = [sum(bits[i * g:(i + 1) * g]) for i in range(c)]
        assert list(scores[p]) == expect, p
        assert pred[p] == expect.index(max(expect))


def test_forward_equals_staged_and_thread_invariant():
    rng = np.random.default_rng(77)
    n, d, b, c = 257, 40, 3, 5
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = np.sort(rng.integers(0, 256, size=(d, b)), axis=1).astype(np.uint8)
    layers = [(_distinct_conn(rng, 60, 6, d * b), rng.integers(0, 1 << 63, size=60).astype(np.uint64)),
              (_distinct_conn(rng, 45, 4, 60), rng.integers(0, 1 << 16, size=45).astype(np.uint64))]
    s1, p1 = oracle.forward(x, th, layers, c, n_threads=1)
    s4, p4 = oracle.forward(x, th, layers, c, n_threads=4)
    v = oracle.encode(x, th)
    for conn, tab in layers:
        v = oracle.lut_layer(v, conn, tab)
    s0, p0 = oracle.groupsum(v, c)
    np.testing.assert_array_equal(s1, s0)
    np.testing.assert_array_equal(p1, p0)
    np.testing.assert_array_equal(s4, s0)
    np.testing.assert_array_equal(p4, p0)


# ---------------------------------------------------------------------------
# Quantized (DSP-backed) head on the group sums (Sec. 3 "Encoders and heads";
# Sec. 5 "Head")

def _dsp_golden():
    rows = []
    for line in open(os.path.join(GOLDEN, "grouped_dsp.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        cnt, q, lg, pr = [f.strip() for f in line.split("|")]
        counts = np.array([int(v) for v in cnt.split(",")], np.int32)
        Q = np.array([[int(v) for v in r.split(",")] for r in q.split(";")], np.int8)
        rows.append((counts, Q, np.array([int(v) for v in lg.split(",")], np.int64), int(pr)))
    return rows


@pytest.mark.parametrize("case", range(6))
def test_grouped_dsp_golden(case):
    counts, Q, logits, pred = _dsp_golden()[case]
    got, p = oracle.grouped_dsp(counts[None, :], Q)
    assert np.array_equal(got[0], logits)
    assert p[0] == pred


def test_grouped_dsp_identity_is_groupsum():
    # Q = identity reduces the quantized head to the popcount head
    rng = np.random.default_rng(3)
    counts = rng.integers(0, 50, (500, 10)).astype(np.int32)
    logits, pred = oracle.grouped_dsp(counts, np.eye(10, dtype=np.int8))
    assert np.array_equal(logits, counts)
    assert np.array_equal(pred, np.argmax(counts, axis=1))


def test_grouped_dsp_positive_scale_and_negation():
    rng = np.random.default_rng(4)
    counts = rng.integers(0, 20, (400, 7)).astype(np.int32)
    for a in (1, 3, 127):
        _, pred = oracle.grouped_dsp(counts, (a * np.eye(7)).astype(np.int8))
        assert np.array_equal(pred, np.argmax(counts, axis=1))
    _, pred = oracle.grouped_dsp(counts, (-np.eye(7)).astype(np.int8))
    assert np.array_equal(pred, np.argmin(counts, axis=1))


def test_grouped_dsp_rank_one_closed_form():
    # Q[i][j] = u[i] * v[j]: logit i = u[i] * (v . counts); catches a
    # transposed weight matrix (that gives v[i] * (u . counts))
    rng = np.random.default_rng(5)
    u = rng.integers(-11, 12, 9)
    v = rng.integers(-11, 12, 9)
    Q = np.outer(u, v).astype(np.int8)
    counts = rng.integers(0, 1000, (300, 9)).astype(np.int32)
    logits, _ = oracle.grouped_dsp(counts, Q)
    dot = counts.astype(np.int64) @ v.astype(np.int64)
    assert np.array_equal(logits, dot[:, None] * u[None, :].astype(np.int64))


def test_grouped_dsp_linear_in_counts():
    rng = np.random.default_rng(6)
    Q = rng.integers(-127, 128, (12, 12)).astype(np.int8)
    a = rng.integers(0, 3000, (200, 12)).astype(np.int32)
    b = rng.integers(0, 3000, (200, 12)).astype(np.int32)
    la, _ = oracle.grouped_dsp(a, Q)
    lb, _ = oracle.grouped_dsp(b, Q)
    lab, _ = oracle.grouped_dsp(a + b, Q)
    assert np.array_equal(lab, la + lb)


def test_grouped_dsp_extremes_exact():
    c = 100
    counts = np.full((2, c), 65535, np.int32)
    lp, _ = oracle.grouped_dsp(counts, np.full((c, c), 127, np.int8))
    ln, pred = oracle.grouped_dsp(counts, np.full((c, c), -128, np.int8))
    assert (lp == 100 * 127 * 65535).all() and (ln == -100 * 128 * 65535).all()
    assert (pred == 0).all()          # all logits equal: lowest index


# ---------------------------------------------------------------------------
# Binary-coded uniform fixed-point encoder (Sec. 3 "Encoders and heads";
# Sec. 5 "Encoder") and quantile-threshold fitting (Sec. 4 "Initialization";
# App. B)

def _binary_golden():
    rows = []
    for line in open(os.path.join(GOLDEN, "binary_encoder.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        b, v, bits = line.split()
        rows.append((int(b), int(v), [int(ch) for ch in bits]))
    return rows


def test_binary_encoder_golden():
    rows = _binary_golden()
    assert len(rows) >= 18
    for b, v, bits in rows:
        e = oracle.encode_binary(np.array([[v]], np.uint8), b)
        assert e[0].tolist() == bits, (b, v)


@pytest.mark.parametrize("b", range(1, 9))
def test_binary_encoder_levels_and_exact_rounding(b):
    from fractions import Fraction
    v = np.arange(256, dtype=np.uint8)[:, None]
    e = oracle.encode_binary(v, b)                       # [256][b]
    q = (e.astype(np.int64) << np.arange(b)).sum(axis=1)
    # the paper's count: 2^b distinct levels, in order, from 0 to 2^b - 1
    assert len(set(q.tolist())) == 2 ** b
    assert (np.diff(q) >= 0).all() and q[0] == 0 and q[255] == 2 ** b - 1
    top = 2 ** b - 1
    for val in range(256):
        exact = Fraction(val * top, 255)
        lo = exact.numerator // exact.denominator
        assert exact - lo != Fraction(1, 2)                 # no ties
        assert q[val] == (lo + 1 if exact - lo > Fraction(1, 2) else lo)


def test_binary_encoder_special_cases():
    rng = np.random.default_rng(7)
    x = rng.integers(0, 256, size=(50, 13), dtype=np.uint8)
    # b = 8 is the pixel's own binary expansion
    e8 = oracle.encode_binary(x, 8).reshape(50, 13, 8)
    assert np.array_equal((e8.astype(np.int64) << np.arange(8)).sum(axis=2), x)
    # b = 1 is the thermometer bit x > 127
    assert np.array_equal(oracle.encode_binary(x, 1),
                          oracle.encode(x, np.full((13, 1), 127, np.uint8)))


def test_forward_binary_equals_staged():
    rng = np.random.default_rng(8)
    n, d, b, c = 300, 20, 3, 4
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    layers, w_in = [], d * b
    for w in (40, 24):
        conn = np.stack([rng.choice(w_in, 6, replace=False) for _ in range(w)]).astype(np.int32)
        layers.append((conn, rng.integers(0, 2**63, size=w).astype(np.uint64)))
        w_in = w
    s, p = oracle.forward(x, None, layers, c, binary_bits=b)
    v = oracle.encode_binary(x, b)
    for conn, tab in layers:
        v = oracle.lut_layer(v, conn, tab)
    s2, p2 = oracle.groupsum(v, c)
    assert np.array_equal(s, s2) and np.array_equal(p, p2)


@pytest.mark.parametrize("b", [1, 3, 4, 7, 8, 15])
def test_fit_quantiles_uniform_closed_form(b):
    # every pixel value equally often: the smallest v with (v+1)/256 >= i/(b+1)
    x = np.tile(np.arange(256, dtype=np.uint8), 12).reshape(-1, 4)    # 768 x 4
    th = oracle.fit_quantiles(x, b)
    want = [-(-256 * i // (b + 1)) - 1 for i in range(1, b + 1)]
    assert (th == np.array(want, np.uint8)).all()


def test_fit_quantiles_mnist_collapse():
    # App. B: on MNIST's pixels a point mass at 0 exceeds the 88 % quantile; at
    # b = 4 all thresholds are 0, at b = 8 seven are 0 and the last ~0.706
    # (180 on the 0..255 scale).  Synthetic data with that shape: 88.5 % zeros,
    # the rest at 180.
    n = 2000
    x = np.zeros((n, 100), np.uint8)
    flat = x.reshape(-1)
    flat[: int(0.115 * flat.size)] = 180
    np.random.default_rng(0).shuffle(flat)
    assert (oracle.fit_quantiles(x, 4) == 0).all()
    th8 = oracle.fit_quantiles(x, 8)
    assert (th8[:, :7] == 0).all() and (th8[:, 7] == 180).all()


@pytest.mark.parametrize("seed", range(4))
def test_fit_quantiles_order_statistics(seed):
    rng = np.random.default_rng(seed)
    n, d, groups, b = 37, 12, 3, 5
    x = rng.integers(0, 256, size=(n, d), dtype=np.uint8)
    th = oracle.fit_quantiles(x, b, groups)
    per = d // groups
    for g in range(groups):
        vals = np.sort(x[:, g * per:(g + 1) * per].ravel())
        for i in range(1, b + 1):
            k = -(-i * vals.size // (b + 1))                  # ceil(i * total / (b+1))
            assert (th[g * per:(g + 1) * per, i - 1] == vals[k - 1]).all()
    assert (np.diff(th.astype(int), axis=1) >= 0).all()
