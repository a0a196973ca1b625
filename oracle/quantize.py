"""E2M-ATQ group ternarisation — oracle definition (test infrastructure only).

Paper: section 4.2 (E2M-ATQ), eqs. 4-6, and section 3, eq. 3.  For each
block the paper takes the block mean as the offset (eq. 4), thresholds the
centred weights at 0.75 times their mean magnitude (eqs. 5, 6), fits a
least-squares scale to that first support, quantises the residual into a
second support the same way, and then refines the offset and the two scales
with the supports held fixed.

Readings where the paper is silent (the packed format fixes the first two):

* A block is one 128-weight group of a row.
* One-plane groups store no offset (the packed format carries mu only on
  two-plane groups), so they are fitted with mu = 0: T0 from the raw
  weights, s0 the least-squares scale.
* Two-plane groups follow the paper: mu = mean(w), T0 and s0 on w - mu, the
  residual r = w - mu - s0*T0 thresholded the same way into T1 with its
  least-squares scale s1, then ``iters`` sweeps of block coordinate descent
  on the squared error with T0 and T1 fixed, in the order
      mu <- mean(w - s0*T0 - s1*T1)
      s0 <- <T0, w - mu - s1*T1> / <T0, T0>
      s1 <- <T1, w - mu - s0*T0> / <T1, T1>
  (a scale whose support is empty is 0).  The sweeps converge to the joint
  least-squares fit of (mu, s0, s1) for the fixed supports.
* With an offset on every group (the paper's own representation): a
  one-plane group is fitted like the first plane of a two-plane group,
  mu = mean(w), T0 and s0 on w - mu, then ``iters`` sweeps
      mu <- mean(w - s0*T0);   s0 <- <T0, w - mu> / <T0, T0>;
  a two-plane group is fitted as above and its mu becomes the group offset
  (the record's own offset is then 0).  Groups are ranked by the residual
  energy ||w - mu - s0*T0||^2 of this one-plane fit.
* The least-squares scale of a support T for a target v is <T, v> / <T, T>,
  i.e. the mean of |v| over the support.
* Which groups get two planes (the paper's salience masks need calibration
  data that is not here): the fraction f2 of groups with the largest
  one-plane residual energy ||w - s0*T0||^2, ties broken by the lower flat
  index (row-major group order).
* Arithmetic is fp64 with every sum taken in index order 0..127 (the same
  order as the kernel), so every threshold decision is taken in the same
  precision with the same operands on both sides; the stored mu, s0, s1 are
  the fp64 values rounded to fp16 (nearest even).

Functions take numpy arrays of shape [n_groups, 128].
"""

import numpy as np

G = 128
THRESHOLD = 0.75


def _sum(v):
    """Sum over the last axis in index order (float64)."""
    acc = np.zeros(v.shape[:-1], dtype=np.float64)
    for i in range(v.shape[-1]):
        acc = acc + v[..., i]
    return acc


def threshold_support(v):
    """Eqs. 5-6: +1 above 0.75 mean|v|, -1 below its negation, else 0."""
    delta = THRESHOLD * (_sum(np.abs(v)) / v.shape[-1])
    d = delta[..., None]
    return np.where(v > d, 1, np.where(v < -d, -1, 0)).astype(np.int8)


def ls_scale(t, v):
    """Least-squares scale of support t for target v: <t, v> / <t, t> (0 on
    an empty support)."""
    tf = t.astype(np.float64)
    num = _sum(tf * v)
    den = _sum(tf * tf)
    safe = np.where(den > 0, den, 1.0)
    return np.where(den > 0, num / safe, 0.0)


def fit_one_plane(w):
    """One-plane groups: mu = 0, T0 = threshold(w), s0 = LS scale.
    Returns (t0, s0) in fp64."""
    w = np.asarray(w, dtype=np.float64)
    t0 = threshold_support(w)
    return t0, ls_scale(t0, w)


def fit_two_plane(w, iters):
    """Two-plane groups (eqs. 4-6, then the refinement of section 4.2).
    Returns (t0, t1, mu, s0, s1) in fp64."""
    w = np.asarray(w, dtype=np.float64)
    mu = _sum(w) / w.shape[-1]
    wc = w - mu[..., None]
    t0 = threshold_support(wc)
    s0 = ls_scale(t0, wc)
    r = wc - s0[..., None] * t0
    t1 = threshold_support(r)
    s1 = ls_scale(t1, r)
    f0, f1 = t0.astype(np.float64), t1.astype(np.float64)
    for _ in range(iters):
        mu = _sum(w - s0[..., None] * f0 - s1[..., None] * f1) / w.shape[-1]
        s0 = ls_scale(t0, w - mu[..., None] - s1[..., None] * f1)
        s1 = ls_scale(t1, w - mu[..., None] - s0[..., None] * f0)
    return t0, t1, mu, s0, s1


def fit_one_plane_offset(w, iters):
    """One plane with an offset (eqs. 4-6, then the refinement with T0
    fixed).  Returns (t0, mu, s0) in fp64."""
    w = np.asarray(w, dtype=np.float64)
    mu = _sum(w) / w.shape[-1]
    wc = w - mu[..., None]
    t0 = threshold_support(wc)
    s0 = ls_scale(t0, wc)
    f0 = t0.astype(np.float64)
    for _ in range(iters):
        mu = _sum(w - s0[..., None] * f0) / w.shape[-1]
        s0 = ls_scale(t0, w - mu[..., None])
    return t0, mu, s0


def residual_energy_offset(w, t0, mu, s0):
    """||w - mu - s0*T0||^2 per group (fp64, index order)."""
    w = np.asarray(w, dtype=np.float64)
    d = (w - mu[..., None]) - s0[..., None] * t0.astype(np.float64)
    return _sum(d * d)


def residual_energy(w, t0, s0):
    """||w - s0*T0||^2 per group (fp64, index order): the salience used to
    choose two-plane groups."""
    w = np.asarray(w, dtype=np.float64)
    d = w - s0[..., None] * t0.astype(np.float64)
    return _sum(d * d)


def select_two_plane(energy, f2):
    """Indices of the floor(f2 * n) groups with the largest energy (ties: the
    lower index first), sorted ascending."""
    energy = np.asarray(energy, dtype=np.float64)
    n = energy.size
    k = int(np.floor(f2 * n))
    order = np.lexsort((np.arange(n), -energy))   # energy descending, index ascending
    return np.sort(order[:k])


def to_fp16(v):
    return np.asarray(v, dtype=np.float64).astype(np.float16)


def ternarize(w, two_plane, iters):
    """Per-group result for groups w [n, 128] (fp16 values) with a boolean
    two-plane flag per group: (t0, t1, s0, mu, s1) with t1, mu, s1 zero on
    one-plane groups; scales rounded to fp16."""
    w = np.asarray(w, dtype=np.float64)
    two = np.asarray(two_plane, dtype=bool)
    n = w.shape[0]
    t0 = np.zeros((n, G), np.int8)
    t1 = np.zeros((n, G), np.int8)
    s0 = np.zeros(n, np.float64)
    mu = np.zeros(n, np.float64)
    s1 = np.zeros(n, np.float64)
    one = ~two
    if one.any():
        t0[one], s0[one] = fit_one_plane(w[one])
    if two.any():
        a, b, c, d, e = fit_two_plane(w[two], iters)
        t0[two], t1[two], mu[two], s0[two], s1[two] = a, b, c, d, e
    return t0, t1, to_fp16(s0), to_fp16(mu), to_fp16(s1)


def ternarize_with_offsets(w, two_plane, iters):
    """Per-group result with an offset on every group: (t0, t1, s0, mu0,
    s1) with mu0 per group, t1 and s1 zero on one-plane groups; scales and
    offsets rounded to fp16."""
    w = np.asarray(w, dtype=np.float64)
    two = np.asarray(two_plane, dtype=bool)
    n = w.shape[0]
    t0 = np.zeros((n, G), np.int8)
    t1 = np.zeros((n, G), np.int8)
    s0 = np.zeros(n, np.float64)
    mu0 = np.zeros(n, np.float64)
    s1 = np.zeros(n, np.float64)
    one = ~two
    if one.any():
        t0[one], mu0[one], s0[one] = fit_one_plane_offset(w[one], iters)
    if two.any():
        a, b, c, d, e = fit_two_plane(w[two], iters)
        t0[two], t1[two], mu0[two], s0[two], s1[two] = a, b, c, d, e
    return t0, t1, to_fp16(s0), to_fp16(mu0), to_fp16(s1)


def quantize_linear(W, f2, iters, group_offsets=False):
    """A packed linear's unpacked inputs from a dense fp16 W [N, K]:
    returns (t0 [N*G', 128], s0 [N, G'], rowptr1, gidx1, t1 [nnz, 128],
    mu1 [nnz], s1 [nnz]) with G' = K / 128, records in CSR order, and with
    ``group_offsets`` also mu0 [N, G'] (the records' mu1 are then 0)."""
    W = np.asarray(W, dtype=np.float16)
    N, K = W.shape
    assert K % G == 0
    ng = K // G
    groups = W.astype(np.float64).reshape(N * ng, G)
    if group_offsets:
        t0_1, mu_1, s0_1 = fit_one_plane_offset(groups, iters)
        energy = residual_energy_offset(groups, t0_1, mu_1, s0_1)
    else:
        t0_1, s0_1 = fit_one_plane(groups)
        energy = residual_energy(groups, t0_1, s0_1)
    sel = select_two_plane(energy, f2)
    flags = np.zeros(N * ng, dtype=bool)
    flags[sel] = True
    rows, gidx = sel // ng, sel % ng
    rowptr1 = np.zeros(N + 1, dtype=np.int32)
    np.add.at(rowptr1, rows + 1, 1)
    rowptr1 = np.cumsum(rowptr1).astype(np.int32)
    if group_offsets:
        t0, t1, s0, mu0, s1 = ternarize_with_offsets(groups, flags, iters)
        mu1 = np.zeros(sel.size, np.float16)
        return (t0, s0.reshape(N, ng), rowptr1, gidx.astype(np.uint16), t1[sel], mu1, s1[sel],
                mu0.reshape(N, ng))
    t0, t1, s0, mu, s1 = ternarize(groups, flags, iters)
    return (t0, s0.reshape(N, ng), rowptr1, gidx.astype(np.uint16), t1[sel], mu[sel], s1[sel])
