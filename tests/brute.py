"""Independent brute-force forms of the forward pass, used only to pin the oracle.

* `dense_forward` is the plain definition written as a dense (r, j, i) triple
  loop over Python floats (fp64), every entry including explicit zeros, one
  rounding to fp32 per layer.
* `fig4_forward` follows the structure of the paper's GraphBLAS listing (Fig. 4,
  Sec. IV): per layer an mxm over the +.x semiring S1, an element-wise multiply
  over the max.+ semiring S2 (whose multiply is +) with the replicated bias
  matrix B_k, and an element-wise add over S2 (whose add is max) with an
  all-zero matrix.  It works in the paper's orientation (Y neurons x batch,
  product W_k Y_k) on generic semiring objects, so it checks both the
  two-semiring rewrite (Sec. III) and our transposed orientation.

* `fig4_forward_pattern` is the same listing with GraphBLAS pattern semantics:
  matrices are dictionaries of stored entries, mxm stores an entry only where
  some stored W entry meets a stored Y entry, eWiseMult with the (full) bias
  matrix is an intersection and eWiseAdd with the (full) zero matrix a union;
  activations are stored as their nonzeros.  It pins the oracle's
  bias-on-the-pattern mode.

All run in fp64 and round to fp32 once per layer, like the oracle, so on the
same inputs they must agree with it bit for bit.
"""

from __future__ import annotations

import math

import numpy as np


class Semiring:
    def __init__(self, name, add, mul, zero, one):
        self.name, self.add, self.mul, self.zero, self.one = name, add, mul, zero, one


S1 = Semiring("plus.times", lambda a, b: a + b, lambda a, b: a * b, 0.0, 1.0)
S2 = Semiring("max.plus", max, lambda a, b: a + b, -math.inf, 0.0)


def mxm(A, B, sr: Semiring):
    """C(i,j) = (+)_k A(i,k) (x) B(k,j) for dense list-of-list matrices (Sec. II.D)."""
    m, l = len(A), len(A[0])
    n = len(B[0])
    assert len(B) == l
    C = [[sr.zero] * n for _ in range(m)]
    for i in range(m):
        for j in range(n):
            acc = sr.zero
            for k in range(l):
                acc = sr.add(acc, sr.mul(A[i][k], B[k][j]))
            C[i][j] = acc
    return C


def ewise(A, B, op):
    return [[op(a, b) for a, b in zip(ra, rb)] for ra, rb in zip(A, B)]


def _to_f32(x: float) -> float:
    return float(np.float32(x))


def dense_forward(Y0, Ws, bs, ymax=math.inf):
    """Y_L by the dense triple loop. Y0: batch x n, Ws: list of n x n (W(i,j) = weight i -> j)."""
    Y = [[float(v) for v in row] for row in Y0]
    n = len(Y[0]) if Y else 0
    for W, b in zip(Ws, bs):
        W = [[float(v) for v in row] for row in W]
        out = []
        for r in range(len(Y)):
            row = []
            for j in range(n):
                z = 0.0
                for i in range(n):
                    z += Y[r][i] * W[i][j]
                z += float(b[j])
                z = max(z, 0.0)
                z = min(z, ymax)
                row.append(_to_f32(z))
            out.append(row)
        Y = out
    return np.array(Y, dtype=np.float32).reshape(len(Y0), n)


def fig4_forward(Y0, Ws, bs):
    """Y_L via the listing's three GraphBLAS steps per layer, in the paper's orientation."""
    Yp = [list(map(float, col)) for col in zip(*Y0)]  # neurons x batch
    m, nb = len(Yp), len(Yp[0])
    zero = [[0.0] * nb for _ in range(m)]
    for W, b in zip(Ws, bs):
        Wp = [list(map(float, col)) for col in zip(*W)]  # paper's W_k is our W_k transposed
        Bk = [[float(b[i])] * nb for i in range(m)]  # b_k replicated along columns
        Z = mxm(Wp, Yp, S1)  # Y[k+1] = W[k] * Y[k]
        Z = ewise(Z, Bk, S2.mul)  # ... + B[k]   (S2's multiply is +)
        Z = ewise(Z, zero, S2.add)  # max(..., 0) (S2's add is max)
        Yp = [[_to_f32(v) for v in row] for row in Z]
    return np.array([list(col) for col in zip(*Yp)], dtype=np.float32)


def fig4_forward_pattern(Y0, W_entries, bs, ymax=math.inf):
    """Y_L via the listing with pattern semantics, in the paper's orientation (neurons x batch).

    Y0: batch x n dense (its nonzeros are the stored entries); W_entries[k]: list of stored (i, j, w)
    of W_k (input i -> output j, explicit zeros allowed); bs[k]: bias vector.
    """
    nb, n = len(Y0), len(Y0[0])
    Y = {(i, r): float(Y0[r][i]) for r in range(nb) for i in range(n) if Y0[r][i] != 0}
    for Wl, b in zip(W_entries, bs):
        # paper's W_k is our W transposed: Wp(j, i) = W(i, j); mxm over S1 stores (j, r) when some
        # stored Wp(j, i) meets a stored Y(i, r)
        by_input = {}
        for i, j, w in Wl:
            by_input.setdefault(i, []).append((j, float(w)))
        Z = {}
        for (i, r), y in sorted(Y.items()):
            for j, w in by_input.get(i, ()):
                Z[(j, r)] = S1.add(Z.get((j, r), S1.zero), S1.mul(w, y))
        # eWiseMult over S2 with the full bias matrix: intersection keeps Z's pattern, value z + b_j
        Z = {(j, r): S2.mul(z, float(b[j])) for (j, r), z in Z.items()}
        # eWiseAdd over S2 with the full zero matrix: union; on Z's pattern max(z, 0), elsewhere 0
        Y = {}
        for (j, r), z in Z.items():
            v = _to_f32(min(S2.add(z, 0.0), ymax))
            if v != 0.0:
                Y[(j, r)] = v  # stored as nonzeros
    out = np.zeros((nb, n), dtype=np.float32)
    for (j, r), v in Y.items():
        out[r, j] = v
    return out
