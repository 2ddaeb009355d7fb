"""Seeded generators: determinism and the structure each workload recipe promises."""

import math

import numpy as np
import pytest

from workloads import csr_rows, dense_to_csr, integer_shadow, make_config, paper_grid, tiny_random


def _same(p, q):
    assert p.n == q.n and p.L == q.L and p.batch == q.batch
    for a, b in zip(p.layers, q.layers):
        for x, y in ((a.row_ptr, b.row_ptr), (a.col, b.col), (a.val, b.val), (a.bias, b.bias)):
            assert x.tobytes() == y.tobytes()
    if p.y0_dense is not None:
        assert p.y0_dense.tobytes() == q.y0_dense.tobytes()
    else:
        for x, y in zip(p.y0_csr, q.y0_csr):
            assert x.tobytes() == y.tobytes()


def _check_csr(row_ptr, col, n):
    assert row_ptr[0] == 0 and np.all(np.diff(row_ptr) >= 0)
    assert col.dtype == np.int32 and np.all((col >= 0) & (col < n))
    for r in range(len(row_ptr) - 1):
        c = col[row_ptr[r]:row_ptr[r + 1]]
        assert np.all(np.diff(c) > 0)


@pytest.mark.parametrize("cfg,kw", [(1, {}), (2, dict(n=512, L=2, batch=16)), (3, dict(n=1024, L=2, batch=32)),
                                    (4, dict(n=4096, L=2, batch=32)), (5, dict(n=8192, L=2, batch=8))])
def test_deterministic(cfg, kw):
    _same(make_config(cfg, **kw), make_config(cfg, **kw))


def test_config1_structure():
    p = make_config(1)
    assert (p.n, p.L, p.batch, p.ymax) == (1024, 4, 64, math.inf)
    for l in p.layers:
        assert np.all(np.diff(l.row_ptr) == 16)
        _check_csr(l.row_ptr, l.col, p.n)
        assert np.all(l.bias == np.float32(0.01))
        assert abs(np.var(l.val.astype(np.float64)) - 2 / 16) < 0.01
    assert p.y0_dense.shape == (64, 1024) and p.y0_dense.min() >= 0 and p.y0_dense.max() < 1
    assert p.edges() == 64 * 1024 * 16 * 4


@pytest.mark.parametrize("d", [0.5, 0.1, 0.01, 0.001])
def test_config2_density(d):
    p = make_config(2, d, L=1)
    l = p.layers[0]
    nnz = l.nnz
    expect = d * p.n * p.n
    assert abs(nnz - expect) < 6 * math.sqrt(expect)
    assert abs(np.var(l.val.astype(np.float64)) - 2 / (d * p.n)) < 0.1 * 2 / (d * p.n)
    _check_csr(l.row_ptr[:65], l.col, p.n)


def test_config3_structure():
    p = make_config(3, L=2)
    assert (p.n, p.batch) == (16384, 4096)
    for l in p.layers:
        assert np.all(np.diff(l.row_ptr) == 32) and np.all(l.bias == 0)
    rp, c, v = p.y0_csr
    assert abs(len(c) / (p.batch * p.n) - 0.10) < 0.002
    assert v.min() > 0 and v.max() <= 1


def test_config4_windows_and_values():
    p = make_config(4, n=8192, L=2, batch=100, window=1024)
    for l in p.layers:
        assert np.all(np.diff(l.row_ptr) == 32)
        assert np.all(l.val == np.float32(1 / 16)) and np.all(l.bias == np.float32(-0.3))
        _check_csr(l.row_ptr[:200], l.col, p.n)
    assert p.ymax == 32.0
    assert np.all(p.y0_csr[2] == 1)


def test_config5_block_structure():
    p = make_config(5, n=16384, L=1, batch=8, block=4096)
    l = p.layers[0]
    assert np.all(np.diff(l.row_ptr) == 32)
    rows = np.repeat(np.arange(p.n), 32)
    in_block = (l.col // 4096) == (rows // 4096)
    per_row = in_block.reshape(p.n, 32).sum(axis=1)
    assert np.all(per_row >= 24)  # 8 of 32 rewired, a rewired column may land in the block again
    _check_csr(l.row_ptr[:300], l.col, p.n)


def test_integer_shadow_keeps_pattern():
    p = make_config(3, n=512, L=2, batch=8)
    q = integer_shadow(p)
    for a, b in zip(p.layers, q.layers):
        assert a.col.tobytes() == b.col.tobytes()
        assert set(np.unique(b.val)) <= {-2, -1, 1, 2}
    assert set(np.unique(q.y0_csr[2])) <= {1, 2, 3}


def test_csr_helpers():
    p = tiny_random(1, 20, 1, 9, y_density=0.4)
    sub = csr_rows(p.y0_csr, [3, 0, 8])
    dense = np.zeros((9, 20), np.float32)
    rp, c, v = p.y0_csr
    for r in range(9):
        dense[r, c[rp[r]:rp[r + 1]]] = v[rp[r]:rp[r + 1]]
    back = dense_to_csr(dense[[3, 0, 8]])
    for a, b in zip(sub, back):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("m,S", [(256, 1), (512, 2), (1024, 4), (2048, 64), (512, 262144), (4096, 262144)])
def test_paper_grid_recipe(m, S):
    """The paper's matrices (Sec. V.B): Bernoulli(1/S) pattern over m x m, values U[-1,3), Y U[0,1),
    64 samples; the nonzero count lies within 5 standard deviations of m^2 / S."""
    p = paper_grid(m, S, L=2)
    q = paper_grid(m, S, L=2)
    _same(p, q)
    assert p.n == m and p.batch == 64 and p.L == 2 and p.layers[0] is p.layers[1]
    l = p.layers[0]
    _check_csr(l.row_ptr, l.col, m)
    mean = m * m / S
    sd = math.sqrt(m * m * (1.0 / S) * (1.0 - 1.0 / S))
    assert abs(l.nnz - mean) <= 5 * sd + 1
    if S == 1:
        assert l.nnz == m * m
    if l.nnz:
        assert l.val.dtype == np.float32 and l.val.min() >= -1.0 and l.val.max() < 3.0
    assert np.all(l.bias == 0)
    y = p.y0_dense
    assert y.shape == (64, m) and y.min() >= 0.0 and y.max() < 1.0
    assert paper_grid(m, S).layers[0].col.tobytes() == l.col.tobytes()  # L does not change the draw
