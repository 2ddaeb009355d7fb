"""Pins for the CPU oracle: hand-worked examples, brute force, closed forms and invariants.

None of these re-types the oracle's formula: each compares it with something
the mathematics fixes independently (a worked example, a dense brute-force
loop, a library matmul in an exact or linear regime, a structural invariant).
"""

import json
import math
import os

import numpy as np
import pytest

import oracle
from tests import brute
from workloads import Layer, dense_to_csr, integer_shadow, make_config, tiny_random

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _layers_from_dense(Ws, bs):
    out = []
    for W, b in zip(Ws, bs):
        W = np.asarray(W, dtype=np.float32)
        rp, c, v = dense_to_csr(W)
        out.append(Layer(rp, c, v, np.asarray(b, dtype=np.float32)))
    return out


def _run(n, layers, ymax, Y0, **kw):
    return oracle.csr_to_dense(oracle.forward(n, layers, ymax, dense_to_csr(np.asarray(Y0, np.float32)), **kw), n)


# --------------------------------------------------------------------------- worked examples


def test_hand_example_two_layers():
    g = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    n = g["n"]
    layers = _layers_from_dense([g["W"]] * 2, [g["b"]] * 2)
    y1 = _run(n, layers[:1], math.inf, g["Y0"])
    assert np.array_equal(y1, np.array(g["Y1"], np.float32))
    y2 = _run(n, layers, math.inf, g["Y0"])
    assert np.array_equal(y2, np.array(g["Y2"], np.float32))


def test_hand_example_csr_and_zero_pruning():
    g = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    layers = _layers_from_dense([g["W"]], [g["b"]])
    rp, c, v = oracle.forward(g["n"], layers, math.inf, dense_to_csr(np.array(g["Y0"], np.float32)))
    assert rp.tolist() == g["Y1_csr"]["row_ptr"]
    assert c.tolist() == g["Y1_csr"]["col"]
    assert v.tolist() == g["Y1_csr"]["val"]


def test_hand_example_clamp():
    g = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    layers = _layers_from_dense([g["W"]] * 2, [g["b"]] * 2)
    assert np.array_equal(_run(3, layers[:1], 8.0, g["Y0"]), np.array(g["ymax8_Y1"], np.float32))
    assert np.array_equal(_run(3, layers, 8.0, g["Y0"]), np.array(g["ymax8_Y2"], np.float32))


def test_hand_example_intermediates_by_brute_force():
    """The companion loops reproduce the hand-worked intermediate products too."""
    g = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    z = brute.mxm(g["Y0"], g["W"], brute.S1)
    assert z == [[float(x) for x in r] for r in g["Y0W"]]
    zb = [[a + b for a, b in zip(r, g["b"])] for r in z]
    assert zb == [[float(x) for x in r] for r in g["Y0W_plus_b"]]


def test_maxplus_example():
    g = json.load(open(os.path.join(GOLDEN, "maxplus_example.json")))
    f = lambda M: [[-math.inf if v is None else float(v) for v in r] for r in M]
    assert brute.mxm(f(g["A"]), f(g["B"]), brute.S2) == f(g["C"])


def test_semiring_zero_is_identity_and_annihilator():
    """Sec. II.E: a (+) 0 = a and a (x) 0 = 0 for S1 (0) and S2 (-inf)."""
    for sr in (brute.S1, brute.S2):
        for a in (-3.5, 0.0, 2.25, 7.0):
            assert sr.add(a, sr.zero) == a
            assert sr.mul(a, sr.zero) == sr.zero
            assert sr.mul(a, sr.one) == a


# --------------------------------------------------------------------------- brute force


@pytest.mark.parametrize("seed", range(8))
def test_oracle_equals_dense_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 24))
    L = int(rng.integers(1, 4))
    batch = int(rng.integers(1, 6))
    ymax = [math.inf, 0.75, 3.0][seed % 3]
    p = tiny_random(seed, n, L, batch, w_density=float(rng.uniform(0.05, 0.9)),
                    y_density=float(rng.uniform(0.1, 1.0)), explicit_zeros=bool(seed % 2), ymax=ymax)
    got = oracle.csr_to_dense(oracle.forward(n, p.layers, ymax, p.y0_csr), n)
    want = brute.dense_forward(oracle.csr_to_dense(p.y0_csr, n), [l.to_dense(n) for l in p.layers],
                               [l.bias for l in p.layers], ymax)
    assert got.tobytes() == want.tobytes()


@pytest.mark.parametrize("seed", range(4))
def test_fig4_listing_equals_brute_force(seed):
    """The two-semiring rewrite (Sec. III) in the paper's orientation equals the plain definition."""
    rng = np.random.default_rng(100 + seed)
    n, L, batch = int(rng.integers(2, 12)), int(rng.integers(1, 4)), int(rng.integers(1, 5))
    p = tiny_random(100 + seed, n, L, batch, w_density=0.5, y_density=0.7)
    Y0 = oracle.csr_to_dense(p.y0_csr, n)
    Ws = [l.to_dense(n) for l in p.layers]
    bs = [l.bias for l in p.layers]
    lit = brute.fig4_forward(Y0.tolist(), [w.tolist() for w in Ws], [b.tolist() for b in bs])
    assert lit.tobytes() == brute.dense_forward(Y0, Ws, bs).tobytes()
    got = oracle.csr_to_dense(oracle.forward(n, p.layers, math.inf, p.y0_csr), n)
    assert got.tobytes() == lit.tobytes()


def test_layer_ranges_compose():
    p = tiny_random(7, 20, 4, 5, w_density=0.4)
    full = oracle.forward(20, p.layers, math.inf, p.y0_csr)
    mid = oracle.forward(20, p.layers, math.inf, p.y0_csr, k0=0, k1=2)
    rest = oracle.forward(20, p.layers, math.inf, mid, k0=2, k1=4)
    for a, b in zip(full, rest):
        assert np.array_equal(a, b)
    same = oracle.forward(20, p.layers, math.inf, p.y0_csr, k0=1, k1=1)
    for a, b in zip(same, p.y0_csr):
        assert np.array_equal(a, b)


# --------------------------------------------------------------------------- closed forms


def test_linear_regime_is_chain_product():
    """b = 0, W >= 0, Y >= 0: h is the identity, so Y_L = Y_0 W_0 ... W_{L-1} (Sec. III remark on linear h)."""
    rng = np.random.default_rng(5)
    n, L, batch = 40, 4, 6
    layers, dense = [], []
    for k in range(L):
        W = (rng.random((n, n)) < 0.2) * rng.uniform(0.0, 0.6, (n, n))
        W = W.astype(np.float32)
        dense.append(W.astype(np.float64))
        rp, c, v = dense_to_csr(W)
        layers.append(Layer(rp, c, v, np.zeros(n, np.float32)))
    Y0 = rng.random((batch, n)).astype(np.float32)
    got = _run(n, layers, math.inf, Y0).astype(np.float64)
    want = Y0.astype(np.float64)
    for W in dense:
        want = want @ W
    # one fp32 rounding per layer: relative error below L * 2^-24 up to the condition (all terms >= 0)
    np.testing.assert_allclose(got, want, rtol=L * 2.0 ** -23, atol=0)


def test_affine_regime_is_matmul_plus_bias():
    """b >= max |Y W|: nothing is clipped, so Y_1 = Y W + b exactly up to the final fp32 rounding."""
    rng = np.random.default_rng(6)
    n, batch = 32, 8
    W = ((rng.random((n, n)) < 0.3) * rng.uniform(-1, 1, (n, n))).astype(np.float32)
    Y0 = rng.uniform(-1, 1, (batch, n)).astype(np.float32)
    z = Y0.astype(np.float64) @ W.astype(np.float64)
    b = np.full(n, np.abs(z).max() + 1.0, np.float32)
    rp, c, v = dense_to_csr(W)
    got = _run(n, [Layer(rp, c, v, b)], math.inf, Y0)
    want = (z + b.astype(np.float64)).astype(np.float32)
    assert np.max(np.abs(got.view(np.int32) - want.view(np.int32))) <= 1  # at most one ulp (summation order)


def test_identity_input_reads_back_weights():
    """Y_0 = I (batch = n) gives row i of Y_1 = h(W(i,:) + b): pins the orientation Y W (not W Y)."""
    p = tiny_random(11, 30, 1, 1, w_density=0.3)
    n = 30
    l = p.layers[0]
    got = _run(n, p.layers, math.inf, np.eye(n, dtype=np.float32))
    Wd = l.to_dense(n).astype(np.float64)
    want = np.maximum(Wd + l.bias.astype(np.float64), 0.0).astype(np.float32)
    assert got.tobytes() == want.tobytes()


def test_permutation_weights_permute_columns():
    rng = np.random.default_rng(12)
    n, batch = 25, 4
    perm = rng.permutation(n)
    W = np.zeros((n, n), np.float32)
    W[np.arange(n), perm] = 1.0
    rp, c, v = dense_to_csr(W)
    Y0 = rng.random((batch, n)).astype(np.float32)
    got = _run(n, [Layer(rp, c, v, np.zeros(n, np.float32))], math.inf, Y0)
    want = np.zeros_like(Y0)
    want[:, perm] = Y0
    assert got.tobytes() == want.tobytes()


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_integer_shadow_matches_exact_integer_arithmetic(cfg):
    """Integer-valued inputs: every partial sum is exact, so numpy int64 matmul + bias + clip is the answer."""
    small = {1: dict(n=96, L=3, batch=7), 2: dict(n=128, L=3, batch=9), 3: dict(n=256, L=3, batch=11),
             4: dict(n=2048, L=3, batch=13, window=256), 5: dict(n=1024, L=3, batch=5, block=256)}[cfg]
    p = make_config(cfg, 0.1 if cfg == 2 else None, **small)
    q = integer_shadow(p)
    n = q.n
    Y = q.y0_dense if q.y0_dense is not None else oracle.csr_to_dense(q.y0_csr, n)
    Yi = Y.astype(np.int64)
    for l in q.layers:
        Yi = np.clip(Yi @ l.to_dense(n).astype(np.int64) + l.bias.astype(np.int64), 0, int(q.ymax))
    got = oracle.csr_to_dense(oracle.forward(n, q.layers, q.ymax, q.y0_as_csr()), n)
    assert np.array_equal(got, Yi.astype(np.float32))


def test_deep_sparse_layer0_closed_form():
    """All weights 1/16 and binary inputs: z = c/16 + b with c an integer count (one rounding only)."""
    p = make_config(4, n=4096, L=1, batch=64, window=512)
    n = p.n
    l = p.layers[0]
    Y = oracle.csr_to_dense(p.y0_csr, n)
    c = (Y.astype(np.int64) @ (l.to_dense(n) != 0).astype(np.int64)).astype(np.float64)
    want = np.minimum(np.maximum(c / 16.0 + np.float64(np.float32(-0.3)), 0.0), 32.0).astype(np.float32)
    got = oracle.csr_to_dense(oracle.forward(n, p.layers, p.ymax, p.y0_csr), n)
    assert got.tobytes() == want.tobytes()
    # c = 5 is the first survivor: 5/16 - 0.3 rounds to the same fp32 whichever way it is evaluated
    assert np.float32(5 / 16 + np.float64(np.float32(-0.3))) == np.float32(np.float32(5 / 16) + np.float32(-0.3))


# --------------------------------------------------------------------------- invariants


@pytest.mark.parametrize("seed", range(5))
def test_invariants(seed):
    n, L, batch = 60, 5, 10
    ymax = 2.0 if seed % 2 else math.inf
    p = tiny_random(200 + seed, n, L, batch, w_density=0.15, y_density=0.3, bias_lo=-0.4, bias_hi=0.0,
                    ymax=ymax)
    # zero rows
    rp, c, v = p.y0_csr
    keep = np.ones(batch, bool)
    keep[::3] = False  # make every third sample an all-zero row
    Y0 = oracle.csr_to_dense(p.y0_csr, n) * keep[:, None]
    csr = dense_to_csr(Y0)
    out, trace = oracle.forward(n, p.layers, ymax, csr, trace=True)
    Y = oracle.csr_to_dense(out, n)
    assert np.all(Y >= 0) and np.all(Y <= ymax)
    assert np.all(out[2] != 0)  # no stored zeros
    assert np.all(Y[~keep] == 0)  # b <= 0: zero rows stay zero
    assert trace[-1] == out[0][-1]
    # b <= 0: every stored entry has a structural product path
    struct = (Y0 != 0).astype(np.int64)
    for l in p.layers:
        struct = ((struct @ (l.to_dense(n) != 0).astype(np.int64)) > 0).astype(np.int64)
    assert np.all(struct[Y != 0] == 1)
    # sorted, unique columns per row
    for r in range(batch):
        cols = out[1][out[0][r]:out[0][r + 1]]
        assert np.all(np.diff(cols) > 0)


def test_preact_consistent_with_forward():
    p = tiny_random(31, 50, 1, 6, w_density=0.3)
    z, s = oracle.preact(50, p.layers[0], p.y0_csr)
    out = oracle.csr_to_dense(oracle.forward(50, p.layers, math.inf, p.y0_csr), 50)
    assert out.tobytes() == np.maximum(z, 0.0).astype(np.float32).tobytes()
    assert np.all(s >= np.abs(z) - 1e-12)


def test_preact_scale_hand_example():
    """The condition scale s = sum_i |Y(r,i) W(i,j)| + |b_j| of the worked example, computed by hand (the
    fixture's S_scale), and z = Y W + b beside it."""
    g = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    layers = _layers_from_dense([g["W"]], [g["b"]])
    z, s = oracle.preact(3, layers[0], dense_to_csr(np.array(g["Y0"], np.float32)))
    assert np.array_equal(z, np.array(g["Y0W_plus_b"], np.float64))
    assert np.array_equal(s, np.array(g["S_scale"], np.float64))


def test_preact_scale_integer_and_sign_invariance():
    """Integer-valued inputs make every sum exact: s equals |Y| |W| + |b| from a library matmul of the
    absolute values; flipping the sign of W or b changes z but leaves s unchanged; with nonnegative operands
    there is no cancellation, so s equals z."""
    q = integer_shadow(make_config(3, n=300, L=1, batch=9))
    l = q.layers[0]
    z, s = oracle.preact(300, l, q.y0_csr)
    Y = oracle.csr_to_dense(q.y0_csr, 300).astype(np.int64)
    W = l.to_dense(300).astype(np.int64)
    b = l.bias.astype(np.int64)
    assert np.array_equal(z, (Y @ W + b).astype(np.float64))
    assert np.array_equal(s, (np.abs(Y) @ np.abs(W) + np.abs(b)).astype(np.float64))
    neg = Layer(l.row_ptr, l.col, -l.val, -l.bias)
    z2, s2 = oracle.preact(300, neg, q.y0_csr)
    assert np.array_equal(z2, -z) and np.array_equal(s2, s)
    pos = Layer(l.row_ptr, l.col, np.abs(l.val), np.abs(l.bias))
    z3, s3 = oracle.preact(300, pos, q.y0_csr)
    assert np.array_equal(z3, s3)


def test_rejects_bad_input():
    p = tiny_random(3, 10, 1, 2)
    l = p.layers[0]
    bad = Layer(l.row_ptr, np.where(l.col == l.col.max(), 10, l.col).astype(np.int32), l.val, l.bias)
    with pytest.raises(ValueError):
        oracle.forward(10, [bad], math.inf, p.y0_csr)
    rp, c, v = p.y0_csr
    if len(c) >= 2 and rp[1] - rp[0] >= 2:
        c2 = c.copy()
        c2[0], c2[1] = c2[1], c2[0]
        with pytest.raises(ValueError):
            oracle.forward(10, [l], math.inf, (rp, c2, v))


# --------------------------------------------------------------------------- bias on the structural pattern


def test_pattern_bias_hand_example():
    """Reading (B) of the bias (Fig. 4 pattern semantics) on the worked example, two layers."""
    g = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    layers = _layers_from_dense([g["W"]] * 2, [g["b"]] * 2)
    pb = g["pattern_bias"]
    assert np.array_equal(_run(3, layers[:1], math.inf, g["Y0"], bias_mode=1), np.array(pb["Y1"], np.float32))
    assert np.array_equal(_run(3, layers, math.inf, g["Y0"], bias_mode=1), np.array(pb["Y2"], np.float32))


@pytest.mark.parametrize("seed", [5, 6, 7, 8])
def test_pattern_bias_equals_pattern_listing(seed):
    """The oracle's pattern mode equals the listing run on dictionaries of stored entries, bit for bit,
    with positive biases, explicit zeros in W and Y_0, and a clamp."""
    n = 23
    ymax = [math.inf, 1.25][seed % 2]
    p = tiny_random(seed, n, 3, 6, w_density=0.12, y_density=0.3, bias_lo=-0.3, bias_hi=0.8,
                    explicit_zeros=True, ymax=ymax)
    y0d = oracle.csr_to_dense(p.y0_csr, n)
    got = oracle.csr_to_dense(oracle.forward(n, p.layers, ymax, p.y0_csr, bias_mode=1), n)
    want = brute.fig4_forward_pattern(y0d, [l.entries() for l in p.layers], [l.bias for l in p.layers], ymax)
    assert got.tobytes() == want.tobytes()


@pytest.mark.parametrize("seed", [9, 10])
def test_pattern_bias_invariants(seed):
    """With every b <= 0 the two readings agree; otherwise the pattern reading stores a subset of the
    structural product pattern, and a row with nothing stored stays empty."""
    n = 40
    p = tiny_random(seed, n, 3, 8, w_density=0.06, y_density=0.1, bias_lo=-0.5, bias_hi=0.0)
    a = oracle.forward(n, p.layers, math.inf, p.y0_csr)
    b = oracle.forward(n, p.layers, math.inf, p.y0_csr, bias_mode=1)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    q = tiny_random(seed, n, 1, 8, w_density=0.06, y_density=0.1, bias_lo=0.1, bias_hi=0.5)
    y0d = oracle.csr_to_dense(q.y0_csr, n)
    y0d[0] = 0.0  # an empty sample
    out = oracle.csr_to_dense(oracle.forward(n, q.layers, math.inf, dense_to_csr(y0d), bias_mode=1), n)
    struct = ((y0d != 0).astype(np.int64) @ (q.layers[0].to_dense(n) != 0).astype(np.int64)) > 0
    assert np.all(out[~struct] == 0)
    assert np.all(out[0] == 0)
    dense_a = oracle.csr_to_dense(oracle.forward(n, q.layers, math.inf, dense_to_csr(y0d)), n)
    assert np.array_equal(out[struct], dense_a[struct])  # on the pattern both readings agree


# --------------------------------------------------------------------------- semiring mxm (Sec. II)

_SR = {
    "plus_times": brute.S1,
    "max_plus": brute.S2,
    "max_min": brute.Semiring("max.min", max, min, -math.inf, math.inf),
    "min_max": brute.Semiring("min.max", min, max, math.inf, -math.inf),
    "xor_and": brute.Semiring("xor.and", lambda a, b: float((a != 0) != (b != 0)),
                              lambda a, b: float(a != 0 and b != 0), 0.0, 1.0),
}


def _stored_dense(layer, n, fill):
    """W with its unstored entries set to `fill` (the semiring's 0-element)."""
    w = np.full((n, n), fill, dtype=np.float64)
    rows = np.repeat(np.arange(n), np.diff(layer.row_ptr))
    w[rows, layer.col] = layer.val
    return w


def test_semiring_mxm_maxplus_hand_example():
    """The worked max.+ product (Sec. II.D over S2): null entries of B are unstored (the 0-element)."""
    g = json.load(open(os.path.join(GOLDEN, "maxplus_example.json")))
    A = np.array([[(-math.inf if v is None else v) for v in row] for row in g["A"]], np.float32)
    B = np.array([[(0.0 if v is None else v) for v in row] for row in g["B"]], np.float32)
    mask = np.array([[v is not None for v in row] for row in g["B"]])
    rows, cols = np.nonzero(mask)
    rp = np.zeros(4, np.int64)
    np.cumsum(np.bincount(rows, minlength=3), out=rp[1:])
    lay = Layer(rp, cols.astype(np.int32), B[mask].astype(np.float32), np.zeros(3, np.float32))
    assert np.array_equal(oracle.mxm("max_plus", 3, lay, A), np.array(g["C"], np.float32))


@pytest.mark.parametrize("name", sorted(_SR))
@pytest.mark.parametrize("seed", [1, 2])
def test_semiring_mxm_equals_generic_listing(name, seed):
    """The oracle's mxm equals the semiring-generic dense mxm (unstored W entries are the 0-element), bit
    for bit, with explicit zeros stored in W."""
    n = 13
    p = tiny_random(70 + seed, n, 1, 5, w_density=0.3, dense_input=True, y_density=0.7, explicit_zeros=True)
    l = p.layers[0]
    y = p.y0_dense
    if name == "xor_and":
        y = (y != 0).astype(np.float32)
        l = Layer(l.row_ptr, l.col, (l.val > 0).astype(np.float32), l.bias)
    sr = _SR[name]
    Wd = _stored_dense(l, n, sr.zero).tolist()
    want = np.array(brute.mxm(y.astype(np.float64).tolist(), Wd, sr), dtype=np.float64).astype(np.float32)
    assert oracle.mxm(name, n, l, y).tobytes() == want.tobytes()


def test_semiring_mxm_against_numpy():
    """Special cases that reduce to library routines: +.x to a matmul (integer values, exact), GF(2) to a
    matmul mod 2, max.+ / max.min / min.max to broadcast reductions."""
    n = 40
    p = tiny_random(77, n, 1, 7, w_density=0.2, dense_input=True, y_density=0.6, integer=True)
    l = p.layers[0]
    y = p.y0_dense
    w0 = _stored_dense(l, n, 0.0)
    assert np.array_equal(oracle.mxm("plus_times", n, l, y), (y.astype(np.float64) @ w0).astype(np.float32))
    yb = (y != 0).astype(np.int64)
    wb = (w0 != 0).astype(np.int64)
    assert np.array_equal(oracle.mxm("xor_and", n, l, y), ((yb @ wb) % 2).astype(np.float32))
    wm = _stored_dense(l, n, -math.inf)
    assert np.array_equal(oracle.mxm("max_plus", n, l, y), np.max(y[:, :, None] + wm[None], axis=1).astype(np.float32))
    assert np.array_equal(oracle.mxm("max_min", n, l, y),
                          np.max(np.minimum(y[:, :, None], wm[None]), axis=1).astype(np.float32))
    wp = _stored_dense(l, n, math.inf)
    assert np.array_equal(oracle.mxm("min_max", n, l, y),
                          np.min(np.maximum(y[:, :, None], wp[None]), axis=1).astype(np.float32))


def test_semiring_zero_rows_give_zero_element():
    """A row of Y holding only the 0-element yields the 0-element everywhere (additive identity and
    multiplicative annihilator, Sec. II.E)."""
    n = 9
    l = tiny_random(78, n, 1, 1, w_density=0.5).layers[0]
    for name, zero in (("max_plus", -math.inf), ("max_min", -math.inf), ("min_max", math.inf),
                       ("plus_times", 0.0), ("xor_and", 0.0)):
        z = oracle.mxm(name, n, l, np.full((1, n), zero, np.float32))
        assert np.all(z == zero), name
