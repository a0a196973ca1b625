"""Packed ternary linear — oracle definition (test infrastructure only).

Paper: section 3, eq. 3 gives the representation W^ = (mu + a0*T0 + a1*T1) (.) M
with T_i in {-1, 0, +1}; the footnote to section 3 places per-group offsets
and scales on a salience-selected subset that carries the second plane;
section 3 also keeps activations in FP16 (A16).  Readings where the paper is
silent:

* Every group g (128 consecutive inputs of row r) has one plane T0 with an
  fp16 scale s0[r, g].  A chosen subset of (r, g) also carries a second plane
  T1 with an fp16 offset mu and an fp16 scale s1 (one record each, stored in
  CSR order by row, then group).  On such a group every weight is
  mu + s0*t0 + s1*t1 (the offset applies to all 128 positions); elsewhere it
  is s0*t0.
* Optionally (the paper's own representation, eq. 3, gives every masked
  block an offset) every group also carries an fp16 offset mu0[r, g]; its
  weights are then mu0 + s0*t0 (+ mu + s1*t1 on two-plane groups).
* x is fp16 and converted exactly.  In fp64 every dequantised weight is exact
  (a sum of up to four fp16 values needs at most 42 significant bits) and every
  product w*x is exact, so ``gemv`` and ``gemm`` differ from the exact result
  only by the rounding of the final dot-product sums (about K * 2**-53).

Functions take plain numpy arrays, in the storage layout of ``codec``.
"""

import numpy as np

from . import codec

G = codec.GROUP


def _two_plane_rows(rowptr1):
    rowptr1 = np.asarray(rowptr1, dtype=np.int64)
    return np.repeat(np.arange(rowptr1.size - 1), np.diff(rowptr1))


def dequantize(n_out, n_in, codes0, scale0, rowptr1=None, gidx1=None,
               codes1=None, offset1=None, scale1=None, offset0=None):
    """Dense fp64 W^ [n_out, n_in] (eq. 3, with the readings above)."""
    assert n_in % G == 0
    ng = n_in // G
    t0, _ = codec.unpack(codes0, n_out * ng)
    s0 = np.asarray(scale0, dtype=np.float16).astype(np.float64)
    w = t0.reshape(n_out, ng, G).astype(np.float64) * s0.reshape(n_out, ng, 1)
    if offset0 is not None:
        w += np.asarray(offset0, dtype=np.float16).astype(np.float64).reshape(n_out, ng, 1)
    nnz = 0 if gidx1 is None else int(np.asarray(gidx1).size)
    if nnz:
        rows = _two_plane_rows(rowptr1)
        g = np.asarray(gidx1).astype(np.int64)
        t1, _ = codec.unpack(codes1, nnz)
        mu = np.asarray(offset1, dtype=np.float16).astype(np.float64)
        s1 = np.asarray(scale1, dtype=np.float16).astype(np.float64)
        # (row, group) pairs are distinct, so this fancy-indexed add is safe.
        w[rows, g] += mu[:, None] + s1[:, None] * t1.astype(np.float64)
    return w.reshape(n_out, n_in)


def gemv(n_out, n_in, codes0, scale0, rowptr1, gidx1, codes1, offset1,
         scale1, x, offset0=None):
    """y = W^ x in fp64 for one fp16 activation vector x [n_in]."""
    w = dequantize(n_out, n_in, codes0, scale0, rowptr1, gidx1, codes1,
                   offset1, scale1, offset0)
    xv = np.asarray(x, dtype=np.float16).astype(np.float64).reshape(n_in)
    return w @ xv


def gemm(n_out, n_in, codes0, scale0, rowptr1, gidx1, codes1, offset1,
         scale1, X, offset0=None):
    """Y = X W^T in fp64 for fp16 activations X [B, n_in] -> [B, n_out]."""
    w = dequantize(n_out, n_in, codes0, scale0, rowptr1, gidx1, codes1,
                   offset1, scale1, offset0)
    xm = np.asarray(X, dtype=np.float16).astype(np.float64).reshape(-1, n_in)
    return xm @ w.T


def dequantize_fp16(n_out, n_in, codes0, scale0, rowptr1=None, gidx1=None,
                    codes1=None, offset1=None, scale1=None, offset0=None):
    """Dense fp16 W^ with the fixed fp32 evaluation order, rounded once.

    Each weight is evaluated in float32 as  a = +0;  a = a + mu0;
    a = a + mu;  a = a + s0*t0;  a = a + s1*t1  (the mu0 step only with
    per-group offsets, the mu and s1 steps only on two-plane groups; every
    product s*t is exact), then rounded to fp16 to nearest-even.
    """
    assert n_in % G == 0
    ng = n_in // G
    t0, _ = codec.unpack(codes0, n_out * ng)
    t0 = t0.reshape(n_out, ng, G).astype(np.float32)
    s0 = np.asarray(scale0, dtype=np.float16).astype(np.float32).reshape(n_out, ng, 1)
    a = np.zeros((n_out, ng, G), dtype=np.float32)
    if offset0 is not None:
        a = a + np.asarray(offset0, dtype=np.float16).astype(np.float32).reshape(n_out, ng, 1)
    nnz = 0 if gidx1 is None else int(np.asarray(gidx1).size)
    if nnz:
        rows = _two_plane_rows(rowptr1)
        g = np.asarray(gidx1).astype(np.int64)
        mu = np.asarray(offset1, dtype=np.float16).astype(np.float32)
        a[rows, g] = a[rows, g] + mu[:, None]
    a = a + s0 * t0
    if nnz:
        t1, _ = codec.unpack(codes1, nnz)
        s1 = np.asarray(scale1, dtype=np.float16).astype(np.float32)
        a[rows, g] = a[rows, g] + s1[:, None] * t1.astype(np.float32)
    return a.astype(np.float16).reshape(n_out, n_in)


def error_bound(n_out, n_in, scale0, rowptr1, gidx1, offset1, scale1, X,
                rel=2e-3, offset0=None):
    """Acceptance bound per output: rel * sum_g coef[r, g] * ||x_g||_1.

    coef[r, g] = |s0| (+ |mu0| with per-group offsets) (+ |mu| + |s1| on
    two-plane groups): the sum of the magnitudes of the group's affine
    coefficients, so the bound dominates rel * sum_k |w_k x_k|.  Returns
    [n_out] for a vector x and [B, n_out] for a matrix X.
    """
    ng = n_in // G
    coef = np.abs(np.asarray(scale0, dtype=np.float16).astype(np.float64)).reshape(n_out, ng)
    if offset0 is not None:
        coef = coef + np.abs(np.asarray(offset0, dtype=np.float16).astype(np.float64)).reshape(n_out, ng)
    nnz = 0 if gidx1 is None else int(np.asarray(gidx1).size)
    if nnz:
        rows = _two_plane_rows(rowptr1)
        g = np.asarray(gidx1).astype(np.int64)
        coef[rows, g] += (np.abs(np.asarray(offset1, dtype=np.float16).astype(np.float64))
                          + np.abs(np.asarray(scale1, dtype=np.float16).astype(np.float64)))
    xa = np.abs(np.asarray(X, dtype=np.float16).astype(np.float64))
    vec = xa.ndim == 1
    xa = xa.reshape(-1, ng, G).sum(axis=2)           # [B, ng]
    out = rel * (xa @ coef.T)                        # [B, n_out]
    return out[0] if vec else out
