"""Seeded generators for the five synthetic workloads and for small test problems.

Orientation: a layer computes Y_{k+1} = h(Y_k W_k + 1 b_k^T) with Y batch x n
(one sample per row) and W_k stored n_in x n_out in CSR, so row i of W_k lists
the fan-out of input neuron i.  The paper writes the same product as W_k Y_k
with Y neurons x batch (Sec. III, batched inference equation); the two differ
by a transpose only.

Recipes (all draws from numpy's PCG64 seeded with
``SeedSequence([SEED_ROOT, config_id, stream, variant])``; stream k draws layer
k, stream L draws Y_0):

* Bernoulli(p) patterns are drawn as the exact Bernoulli process over the
  flattened matrix (positions are cumulative sums of Geometric(p) gaps), the
  paper's independent Bernoulli selection of nonzero locations (Sec. V.B).
* "exactly k distinct uniform columns" draws k columns uniformly with
  replacement and redraws any row that holds a duplicate, which is uniform over
  k-subsets.
* Normal(0, v) means variance v (He scaling), standard deviation sqrt(v).
* "uniform (0,1]" is 1 - U[0,1) in float32, which is exact and never zero.

None of this code performs the method's arithmetic.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

SEED_ROOT = 20170802937

CONFIG_NAMES = {
    1: "tiny-mlp",
    2: "density-sweep",
    3: "sparse-activation-spgemm",
    4: "deep-sparse",
    5: "very-wide",
    6: "paper-grid",
}

# The paper's own experiment (Sec. V.B-C): square m x m weights over a range of sizes and inverse
# sparsities (total entries / nonzeros) from 1 to 262144, dense Y with 64 samples.
PAPER_GRID_SIZES = (256, 512, 1024, 2048, 4096, 8192, 16384, 32768)
PAPER_GRID_INV_SPARSITY = (1, 2, 4, 16, 64, 256, 1024, 4096, 16384, 65536, 262144)

CONFIG2_DENSITIES = (0.5, 0.1, 0.01, 0.001)


def _rng(config_id: int, stream: int, variant: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([SEED_ROOT, config_id, stream, variant]))


@dataclass
class Layer:
    """One weight layer: CSR W (n_in x n_out, int64 row_ptr, int32 col, fp32 val) and fp32 bias[n]."""

    row_ptr: np.ndarray
    col: np.ndarray
    val: np.ndarray
    bias: np.ndarray

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])

    def to_dense(self, n: int) -> np.ndarray:
        w = np.zeros((n, n), dtype=np.float32)
        rows = np.repeat(np.arange(n), np.diff(self.row_ptr))
        w[rows, self.col] = self.val
        return w

    def entries(self):
        """Stored entries as (i, j, w) triples (explicit zeros included)."""
        rows = np.repeat(np.arange(len(self.row_ptr) - 1), np.diff(self.row_ptr))
        return [(int(i), int(j), float(w)) for i, j, w in zip(rows, self.col, self.val)]


@dataclass
class Problem:
    name: str
    n: int
    L: int
    batch: int
    ymax: float
    layers: list
    y0_dense: np.ndarray | None = None  # (batch, n) float32, row-major
    y0_csr: tuple | None = None  # (row_ptr int64[batch+1], col int32, val float32)
    meta: dict = field(default_factory=dict)

    def y0_as_csr(self):
        if self.y0_csr is not None:
            return self.y0_csr
        return dense_to_csr(self.y0_dense)

    def edges(self) -> int:
        """batch * sum_k nnz(W_k): the edge count behind the edges/s metric."""
        return self.batch * sum(l.nnz for l in self.layers)


# ----------------------------------------------------------------------------- helpers


def dense_to_csr(y: np.ndarray):
    """Dense (rows x n) -> CSR keeping only nonzero entries (columns ascending)."""
    y = np.ascontiguousarray(y, dtype=np.float32)
    mask = y != 0
    counts = mask.sum(axis=1, dtype=np.int64)
    row_ptr = np.zeros(y.shape[0] + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    r, c = np.nonzero(mask)
    return row_ptr, c.astype(np.int32), y[r, c].astype(np.float32)


def csr_rows(csr, rows):
    """Sub-CSR made of the given rows (in the given order)."""
    row_ptr, col, val = csr
    rows = np.asarray(rows, dtype=np.int64)
    starts = row_ptr[rows]
    counts = row_ptr[rows + 1] - starts
    out_ptr = np.zeros(len(rows) + 1, dtype=np.int64)
    np.cumsum(counts, out=out_ptr[1:])
    idx = np.repeat(starts - out_ptr[:-1], counts) + np.arange(out_ptr[-1], dtype=np.int64)
    return out_ptr, col[idx].copy(), val[idx].copy()


def _bernoulli_positions(rng: np.random.Generator, total: int, p: float) -> np.ndarray:
    """Sorted positions of the successes among `total` independent Bernoulli(p) trials."""
    if p >= 1.0:
        return np.arange(total, dtype=np.int64)
    if p <= 0.0 or total == 0:
        return np.zeros(0, dtype=np.int64)
    if p >= 0.05:
        # dense enough that one uniform per trial is cheaper than geometric gaps
        step = 1 << 24
        out = []
        for s in range(0, total, step):
            u = rng.random(min(step, total - s), dtype=np.float32)
            out.append(np.flatnonzero(u < np.float32(p)).astype(np.int64) + s)
        return np.concatenate(out)
    chunks = []
    last = -1
    expect = total * p
    while True:
        m = int(max(1024, (total - 1 - last) * p + 8.0 * math.sqrt(expect) + 64))
        gaps = rng.geometric(p, size=m).astype(np.int64)
        pos = last + np.cumsum(gaps)
        keep = pos[pos < total]
        chunks.append(keep)
        if len(keep) < m:
            break
        last = int(pos[-1])
    return np.concatenate(chunks) if chunks else np.zeros(0, dtype=np.int64)


def _bernoulli_csr(rng, rows: int, cols: int, p: float):
    """CSR pattern of a rows x cols Bernoulli(p) matrix, drawn in blocks of rows (about 4M trials each,
    which keeps the temporaries small; a Bernoulli process restarted at block boundaries is still one)."""
    block = max(1, min(rows, (1 << 22) // max(1, cols)))
    cols_out, counts = [], np.zeros(rows, dtype=np.int64)
    for r0 in range(0, rows, block):
        nr = min(block, rows - r0)
        if p >= 1.0:
            cols_out.append(np.tile(np.arange(cols, dtype=np.int32), nr))
            counts[r0:r0 + nr] = cols
        elif p >= 0.05:
            # the same uniforms as _bernoulli_positions draws, read as a 2-D mask
            mask = (rng.random(nr * cols, dtype=np.float32) < np.float32(p)).reshape(nr, cols)
            cols_out.append(np.nonzero(mask)[1].astype(np.int32))
            counts[r0:r0 + nr] = mask.sum(axis=1)
        else:
            pos = _bernoulli_positions(rng, nr * cols, p)
            r = pos // cols
            cols_out.append((pos - r * cols).astype(np.int32))
            counts[r0:r0 + nr] = np.bincount(r, minlength=nr)
    row_ptr = np.zeros(rows + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    return row_ptr, (np.concatenate(cols_out) if cols_out else np.zeros(0, np.int32))


def _distinct_per_row(rng, rows: int, k: int, width: int) -> np.ndarray:
    """(rows, k) int64 offsets in [0, width), distinct within a row, sorted ascending."""
    if k > width:
        raise ValueError("k > width")
    a = rng.integers(0, width, size=(rows, k), dtype=np.int64)
    a.sort(axis=1)
    bad = np.nonzero(np.any(a[:, 1:] == a[:, :-1], axis=1))[0] if k > 1 else np.zeros(0, np.int64)
    while len(bad):
        b = rng.integers(0, width, size=(len(bad), k), dtype=np.int64)
        b.sort(axis=1)
        a[bad] = b
        still = np.any(b[:, 1:] == b[:, :-1], axis=1)
        bad = bad[still]
    return a


def _fixed_rows_csr(cols2d: np.ndarray):
    rows, k = cols2d.shape
    row_ptr = np.arange(0, rows * k + 1, k, dtype=np.int64)
    return row_ptr, cols2d.reshape(-1).astype(np.int32)


def _normal(rng, size: int, var: float) -> np.ndarray:
    return (rng.standard_normal(size) * math.sqrt(var)).astype(np.float32)


def _unit_open_closed(rng, size: int) -> np.ndarray:
    return (np.float32(1.0) - rng.random(size, dtype=np.float32)).astype(np.float32)


# ----------------------------------------------------------------------------- configs


def make_config(config_id: int, density: float | None = None, *, n: int | None = None,
                L: int | None = None, batch: int | None = None, window: int | None = None,
                block: int | None = None) -> Problem:
    """Build workload `config_id` (1..5) at its stated sizes, or scaled down via keyword overrides.

    Scaling keeps the recipe (nonzeros per row, value laws, bias, input density) and only changes
    the sizes, so a scaled problem exercises the same code paths at a size the oracle finishes fast.
    """
    if config_id == 1:
        n_, L_, b_ = n or 1024, L or 4, batch or 64
        layers = []
        for k in range(L_):
            rng = _rng(1, k)
            row_ptr, col = _fixed_rows_csr(_distinct_per_row(rng, n_, 16, n_))
            layers.append(Layer(row_ptr, col, _normal(rng, len(col), 2.0 / 16), np.full(n_, 0.01, np.float32)))
        y0 = _rng(1, L_).random((b_, n_), dtype=np.float32)
        return Problem("tiny-mlp", n_, L_, b_, math.inf, layers, y0_dense=y0,
                       meta={"config": 1})

    if config_id == 2:
        d = 0.01 if density is None else float(density)
        n_, L_, b_ = n or 4096, L or 16, batch or 1024
        variant = int(round(d * 1e6))
        layers = []
        for k in range(L_):
            rng = _rng(2, k, variant)
            row_ptr, col = _bernoulli_csr(rng, n_, n_, d)
            layers.append(Layer(row_ptr, col, _normal(rng, len(col), 2.0 / (d * n_)),
                                np.full(n_, 0.01, np.float32)))
        y0 = _rng(2, L_, variant).random((b_, n_), dtype=np.float32)
        return Problem(f"density-sweep-d{d:g}", n_, L_, b_, math.inf, layers, y0_dense=y0,
                       meta={"config": 2, "density": d})

    if config_id == 3:
        n_, L_, b_ = n or 16384, L or 32, batch or 4096
        layers = []
        for k in range(L_):
            rng = _rng(3, k)
            row_ptr, col = _fixed_rows_csr(_distinct_per_row(rng, n_, 32, n_))
            layers.append(Layer(row_ptr, col, _normal(rng, len(col), 2.0 / 32), np.zeros(n_, np.float32)))
        rng = _rng(3, L_)
        rp, c = _bernoulli_csr(rng, b_, n_, 0.10)
        y0 = (rp, c, _unit_open_closed(rng, len(c)))
        return Problem("sparse-activation-spgemm", n_, L_, b_, math.inf, layers, y0_csr=y0,
                       meta={"config": 3})

    if config_id == 4:
        n_, L_, b_ = n or 65536, L or 120, batch or 60000
        w_ = window or 1024
        layers = []
        for k in range(L_):
            rng = _rng(4, k)
            start = rng.integers(0, n_ - w_ + 1, size=(n_, 1), dtype=np.int64)
            cols = start + _distinct_per_row(rng, n_, 32, w_)
            perm = rng.permutation(n_).astype(np.int64)
            cols = np.sort(perm[cols], axis=1)
            row_ptr, col = _fixed_rows_csr(cols)
            layers.append(Layer(row_ptr, col, np.full(len(col), 1.0 / 16, np.float32),
                                np.full(n_, -0.3, np.float32)))
        rng = _rng(4, L_)
        rp, c = _bernoulli_csr(rng, b_, n_, 0.015)
        y0 = (rp, c, np.ones(len(c), np.float32))
        return Problem("deep-sparse", n_, L_, b_, 32.0, layers, y0_csr=y0,
                       meta={"config": 4, "window": w_})

    if config_id == 5:
        n_, L_, b_ = n or (1 << 20), L or 8, batch or 8192
        blk = block or 4096
        if n_ % blk:
            raise ValueError("n must be a multiple of the block width")
        layers = []
        for k in range(L_):
            rng = _rng(5, k)
            base = (np.arange(n_, dtype=np.int64)[:, None] // blk) * blk + _distinct_per_row(rng, n_, 32, blk)
            which = np.argsort(rng.random((n_, 32)), axis=1)[:, :8]
            todo = np.arange(n_, dtype=np.int64)
            cols = base.copy()
            while len(todo):
                cand = base[todo].copy()
                np.put_along_axis(cand, which[todo], rng.integers(0, n_, size=(len(todo), 8), dtype=np.int64), axis=1)
                srt = np.sort(cand, axis=1)
                dup = np.any(srt[:, 1:] == srt[:, :-1], axis=1)
                ok = ~dup
                cols[todo[ok]] = srt[ok]
                todo = todo[dup]
            row_ptr, col = _fixed_rows_csr(cols)
            layers.append(Layer(row_ptr, col, _normal(rng, len(col), 2.0 / 32), np.full(n_, 0.01, np.float32)))
        rng = _rng(5, L_)
        rp, c = _bernoulli_csr(rng, b_, n_, 0.02)
        y0 = (rp, c, _unit_open_closed(rng, len(c)))
        return Problem("very-wide", n_, L_, b_, math.inf, layers, y0_csr=y0,
                       meta={"config": 5, "block": blk})

    raise ValueError(f"unknown config {config_id}")


def paper_grid(m: int, inv_sparsity: int, *, batch: int = 64, L: int = 1) -> Problem:
    """One point of the paper's experiment (Sec. V.B): W is m x m with an independent Bernoulli pattern of
    density 1 / inv_sparsity and values U[-1, 3); Y_0 is batch x m with values U[0, 1); batch 64.

    The paper does not state the bias of its timing runs; b = 0 here.  All L layers share one W (the paper
    times one iteration of the layer loop; identical layers let a benchmark difference out the fixed cost
    of entering and leaving the loop).  Values grow layer by layer, as the paper notes for this matrix
    family, so only the first layer is meaningful numerically.
    """
    if m < 1 or inv_sparsity < 1:
        raise ValueError("m and inv_sparsity must be >= 1")
    variant = m * 1000003 + inv_sparsity
    rng = _rng(6, 0, variant)
    row_ptr, col = _bernoulli_csr(rng, m, m, 1.0 / inv_sparsity)
    # U[-1, 3) exactly in float32: 4 * U[0, 1) - 1 is exact and at most 3 - 2^-22
    val = rng.random(len(col), dtype=np.float32) * np.float32(4.0) - np.float32(1.0)
    layer = Layer(row_ptr, col, val, np.zeros(m, np.float32))
    y = _rng(6, 1, variant).random((batch, m), dtype=np.float32)
    return Problem(f"paper-grid-m{m}-S{inv_sparsity}", m, L, batch, math.inf, [layer] * L, y0_dense=y,
                   meta={"config": 6, "m": m, "inv_sparsity": inv_sparsity})


def integer_shadow(p: Problem, seed_variant: int = 7) -> Problem:
    """Same sparsity patterns as `p`, integer values: W in {-2,-1,1,2}, Y_0 in {1,2,3}, b in {-3..1}.

    With ymax = 1000 every partial sum stays far below 2**24, so fp32 and fp64 accumulation are both
    exact in any order and two correct implementations must agree bit for bit.
    """
    cid = int(p.meta.get("config", 0))
    choices_w = np.array([-2, -1, 1, 2], dtype=np.float32)
    layers = []
    for k, l in enumerate(p.layers):
        rng = _rng(1000 + cid, k, seed_variant)
        w = choices_w[rng.integers(0, 4, size=l.nnz)]
        b = rng.integers(-3, 2, size=len(l.bias)).astype(np.float32)
        layers.append(Layer(l.row_ptr, l.col, w, b))
    rng = _rng(1000 + cid, p.L, seed_variant)
    if p.y0_dense is not None:
        y0 = rng.integers(1, 4, size=p.y0_dense.shape).astype(np.float32)
        return Problem(p.name + "-int", p.n, p.L, p.batch, 1000.0, layers, y0_dense=y0,
                       meta=dict(p.meta, shadow=True))
    rp, c, v = p.y0_csr
    y0 = (rp, c, rng.integers(1, 4, size=len(v)).astype(np.float32))
    return Problem(p.name + "-int", p.n, p.L, p.batch, 1000.0, layers, y0_csr=y0,
                   meta=dict(p.meta, shadow=True))


def tiny_random(seed: int, n: int, L: int, batch: int, *, w_density: float = 0.3,
                y_density: float = 0.5, bias_lo: float = -0.5, bias_hi: float = 0.5,
                ymax: float = math.inf, explicit_zeros: bool = False, dense_input: bool = False,
                integer: bool = False) -> Problem:
    """Small random problem for oracle pins and parity tests (empty rows and columns occur)."""
    layers = []
    for k in range(L):
        rng = _rng(9000 + seed, k)
        row_ptr, col = _bernoulli_csr(rng, n, n, w_density)
        if integer:
            val = np.array([-2, -1, 1, 2], np.float32)[rng.integers(0, 4, size=len(col))]
            bias = rng.integers(-3, 2, size=n).astype(np.float32)
        else:
            val = rng.uniform(-1.0, 1.0, size=len(col)).astype(np.float32)
            bias = rng.uniform(bias_lo, bias_hi, size=n).astype(np.float32)
        if explicit_zeros and len(val):
            val[rng.random(len(val)) < 0.1] = 0.0
        layers.append(Layer(row_ptr, col, val, bias))
    rng = _rng(9000 + seed, L)
    if dense_input:
        y = rng.random((batch, n), dtype=np.float32)
        y[rng.random((batch, n)) >= y_density] = 0.0
        if integer:
            y = np.where(y != 0, rng.integers(1, 4, size=y.shape), 0).astype(np.float32)
        return Problem(f"tiny-{seed}", n, L, batch, ymax, layers, y0_dense=y, meta={"config": 0})
    rp, c = _bernoulli_csr(rng, batch, n, y_density)
    if integer:
        v = rng.integers(1, 4, size=len(c)).astype(np.float32)
    else:
        v = _unit_open_closed(rng, len(c))
    if explicit_zeros and len(v):
        v[rng.random(len(v)) < 0.1] = 0.0
    return Problem(f"tiny-{seed}", n, L, batch, ymax, layers, y0_csr=(rp, c, v), meta={"config": 0})
