"""Comparison of GPU results with the oracle.

Rule (fp32 outputs): on the common pattern every value must satisfy
|gpu - oracle| <= ATOL + RTOL * |oracle| with ATOL = 1e-6, RTOL = 1e-5.  The patterns
must be equal, except that an entry may be present on one side only when the oracle's
fp64 pre-activation z of that entry lies within tau = ATOL + RTOL * s of the ReLU
threshold (s = sum |y w| + |b|, the condition scale), and the value kept there is at
most tau: rounding may legitimately decide such entries either way.  Integer-valued
problems are exact, so there the results must be identical bit for bit.
"""

from __future__ import annotations

import numpy as np

import oracle
from workloads import csr_rows

ATOL = 1e-6
RTOL = 1e-5


def to_dense(csr, n):
    return oracle.csr_to_dense(csr, n)


def dense_to_csr_keep_all(d):
    from workloads import dense_to_csr

    return dense_to_csr(d)


def oracle_rows(problem, rows=None, k0=0, k1=None, threads=None, bias_mode=0):
    y = problem.y0_as_csr()
    if rows is not None:
        y = csr_rows(y, rows)
    return oracle.forward(problem.n, problem.layers, problem.ymax, y, k0=k0, k1=k1, threads=threads,
                          bias_mode=bias_mode)


def fp32_sum_scale(terms: int) -> float:
    """gamma_{terms+2} = (terms + 2) u / (1 - (terms + 2) u), u = 2^-24: the bound on the relative (to
    sum |y w| + |b|) error of a pre-activation whose products and sums over `terms` entries, and the bias add,
    are each rounded to fp32, in any order (the fp32 dense arm)."""
    u = 2.0 ** -24
    return (terms + 2) * u / (1 - (terms + 2) * u)


def compare(problem, got_csr, rows=None, exact=False, k1=None, bias_mode=0, scale_tol=0.0):
    """Compare GPU output rows (CSR, in the order of `rows`) with the oracle; returns a stats dict.
    bias_mode 1 compares against the oracle's bias-on-the-structural-pattern reading.  scale_tol > 0 widens
    the value tolerance and the threshold allowance by scale_tol * s (s = sum |y w| + |b| of the entry) for
    arithmetic that rounds its sums to fp32 (only meaningful for one layer on oracle inputs)."""
    n = problem.n
    k1 = problem.L if k1 is None else k1
    want_csr = oracle_rows(problem, rows, k1=k1, bias_mode=bias_mode)
    got = to_dense(got_csr, n)
    want = to_dense(want_csr, n)
    assert got.shape == want.shape
    stats = {"entries": int(want_csr[0][-1]), "ambiguous": 0, "max_abs": 0.0, "max_rel": 0.0}
    if exact:
        assert got.tobytes() == want.tobytes(), "integer-valued problem must match bit for bit"
        assert np.array_equal(got_csr[0], want_csr[0]) and np.array_equal(got_csr[1], want_csr[1])
        return stats
    gp, wp = got != 0, want != 0
    both = gp & wp
    diff = np.abs(got.astype(np.float64) - want.astype(np.float64))
    if both.any():
        stats["max_abs"] = float(diff[both].max())
        stats["max_rel"] = float((diff[both] / np.maximum(np.abs(want[both]), 1e-30)).max())
    tol = ATOL + RTOL * np.abs(want.astype(np.float64))
    s_all = None
    if scale_tol:
        prev_all = oracle_rows(problem, rows, k1=k1 - 1, bias_mode=bias_mode)
        _, s_all = oracle.preact(n, problem.layers[k1 - 1], prev_all)
        tol = tol + scale_tol * s_all
        if both.any():
            stats["max_scaled"] = float((diff[both] / np.maximum(s_all[both], 1e-300)).max())
    bad = both & (diff > tol)
    assert not bad.any(), f"{int(bad.sum())} values outside tolerance; worst abs {diff[bad].max()}"
    odd = gp ^ wp
    if odd.any():
        r_idx = np.unique(np.nonzero(odd)[0])
        sub_rows = r_idx if rows is None else np.asarray(rows)[r_idx]
        prev = oracle_rows(problem, sub_rows, k1=k1 - 1, bias_mode=bias_mode)
        z, s = oracle.preact(n, problem.layers[k1 - 1], prev)
        for t, r in enumerate(r_idx):
            cols = np.nonzero(odd[r])[0]
            tau = ATOL + RTOL * s[t, cols] + scale_tol * s[t, cols]
            kept = np.maximum(got[r, cols], want[r, cols]).astype(np.float64)
            assert np.all(np.abs(z[t, cols]) <= tau) and np.all(kept <= tau), (
                f"pattern differs at row {r} cols {cols[:8]} beyond the ReLU-threshold allowance")
        stats["ambiguous"] = int(odd.sum())
    # canonical form: ascending columns, no stored zeros
    check_canonical(got_csr)
    return stats


def check_canonical(csr):
    """Strictly ascending columns within each row and no stored zeros."""
    rp, col, val = csr
    assert rp[0] == 0 and np.all(np.diff(rp) >= 0) and rp[-1] == len(col) == len(val)
    assert np.all(val != 0)
    if len(col) > 1:
        starts = np.zeros(len(col), bool)
        inner = rp[1:-1]
        starts[inner[inner < len(col)]] = True
        assert np.all((np.diff(col) > 0) | starts[1:])


def compare_in_chunks(problem, got_csr, rows=None, chunk=512, **kw):
    """compare() over blocks of `chunk` rows (the oracle and the dense views are built per block, so
    memory stays bounded at full size).  got_csr holds the rows in the order of `rows` (all rows when
    None).  Returns the summed entry and ambiguous-entry counts."""
    nrows = len(got_csr[0]) - 1
    rows = np.arange(nrows) if rows is None else np.asarray(rows)
    assert len(rows) == nrows
    tot = {"entries": 0, "ambiguous": 0}
    for a in range(0, nrows, chunk):
        idx = np.arange(a, min(nrows, a + chunk))
        st = compare(problem, csr_rows(got_csr, idx), rows=rows[idx], **kw)
        tot["entries"] += st["entries"]
        tot["ambiguous"] += st["ambiguous"]
    return tot


def compare_exact_csr(problem, got_csr, k0=0, k1=None, chunk=4096, y_in=None):
    """Bit-for-bit comparison of CSR arrays (row extents, columns, value bits) with the oracle over all
    rows, in blocks of `chunk` rows, without dense views.  y_in: the CSR taken as Y_{k0} (default Y_0)."""
    y = problem.y0_as_csr() if y_in is None else y_in
    nrows = len(y[0]) - 1
    assert len(got_csr[0]) == nrows + 1
    total = 0
    for a in range(0, nrows, chunk):
        idx = np.arange(a, min(nrows, a + chunk))
        want = oracle.forward(problem.n, problem.layers, problem.ymax, csr_rows(y, idx), k0=k0, k1=k1)
        got = csr_rows(got_csr, idx)
        assert np.array_equal(np.diff(got[0]), np.diff(want[0])), f"row lengths differ in rows {a}.."
        assert np.array_equal(got[1], want[1]), f"columns differ in rows {a}.."
        assert got[2].tobytes() == want[2].tobytes(), f"values differ in rows {a}.."
        total += len(want[1])
    check_canonical(got_csr)
    return total
