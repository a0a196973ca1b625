"""Pins of the E2M-ATQ oracle (oracle/quantize.py) against closed forms,
hand-worked blocks and an independent least-squares solver.

``test_pins_catch_planted_mistakes`` plants plausible mistakes into patched
copies of the oracle (threshold constant, a non-strict threshold, no
centring, the scale averaged over the whole block, a sign error in the
offset update, an uncentred residual, ties broken the other way) and checks
that each fails at least one pin."""

import numpy as np
import pytest

from oracle import codec, packed, quantize


def rng(seed):
    return np.random.default_rng(seed)


def fp16_groups(r, n, scale=0.02):
    return (r.standard_normal((n, 128)) * scale).astype(np.float16).astype(np.float64)


def test_scaled_ternary_block_is_recovered_exactly():
    # w = c * t: the threshold 0.75 * c * nnz/128 is below c, so T0 = t and
    # the least-squares scale is c, with zero residual.
    r = rng(1)
    t = r.integers(-1, 2, size=(50, 128)).astype(np.int8)
    t[:, 0] = 1                                  # at least one nonzero
    c = r.uniform(0.01, 0.1, 50).astype(np.float16).astype(np.float64)
    w = c[:, None] * t
    t0, s0 = quantize.fit_one_plane(w)
    assert np.array_equal(t0, t)
    assert np.array_equal(s0, c)
    assert np.all(quantize.residual_energy(w, t0, s0) == 0)


def test_threshold_is_strict_at_three_quarters_of_the_mean_magnitude():
    # 64 weights of 5 and 64 of 3: mean |w| = 4, threshold exactly 3, so the
    # 3s stay 0 (strict inequality) and the 5s become +1; negated, -1.
    w = np.array([[5.0] * 64 + [3.0] * 64, [-5.0] * 64 + [-3.0] * 64])
    t = quantize.threshold_support(w)
    assert np.array_equal(t[0], np.array([1] * 64 + [0] * 64, np.int8))
    assert np.array_equal(t[1], np.array([-1] * 64 + [0] * 64, np.int8))
    # Raising the 3s by e moves the threshold by only 3e/8, so they join.
    w2 = np.array([[5.0] * 64 + [3.0 + 2 ** -20] * 64])
    assert np.all(quantize.threshold_support(w2)[0] == 1)


def test_hand_worked_block():
    # [4, -4, 1, -1, 0 x 124]: mean |w| = 10/128, threshold 0.05859375.
    w = np.zeros((1, 128))
    w[0, :4] = [4, -4, 1, -1]
    t0, s0 = quantize.fit_one_plane(w)
    assert list(t0[0, :5]) == [1, -1, 1, -1, 0] and not t0[0, 4:].any()
    assert s0[0] == 2.5                          # (4 + 4 + 1 + 1) / 4


def test_least_squares_scale_is_the_mean_magnitude_over_the_support():
    r = rng(2)
    v = r.standard_normal((40, 128))
    t = quantize.threshold_support(v)
    want = np.array([np.mean(np.abs(v[i][t[i] != 0])) for i in range(40)])
    assert np.allclose(quantize.ls_scale(t, v), want, rtol=1e-14, atol=0)
    assert np.array_equal(quantize.ls_scale(np.zeros((1, 128), np.int8), v[:1]), np.zeros(1))


def test_constant_block_is_its_offset():
    w = np.full((3, 128), 0.015625)
    t0, t1, mu, s0, s1 = quantize.fit_two_plane(w, iters=3)
    assert not t0.any() and not t1.any()
    assert np.all(mu == 0.015625) and np.all(s0 == 0) and np.all(s1 == 0)


def test_first_plane_uses_the_centred_weights():
    # An offset block: w = 0.5 + 0.1*t.  Centring removes the offset, so T0 is
    # t's pattern (t balanced: mean of t is 0) and mu is 0.5.
    t = np.tile(np.array([1, -1, 0, 0], np.int8), 32)[None, :]
    w = 0.5 + 0.1 * t.astype(np.float64)
    t0, t1, mu, s0, s1 = quantize.fit_two_plane(w, iters=0)
    assert np.array_equal(t0, t)
    assert mu[0] == 0.5 and abs(s0[0] - 0.1) < 1e-15


def test_refinement_converges_to_the_joint_least_squares_fit():
    r = rng(3)
    w = fp16_groups(r, 30)
    t0, t1, mu, s0, s1 = quantize.fit_two_plane(w, iters=400)
    for i in range(30):
        A = np.stack([np.ones(128), t0[i].astype(float), t1[i].astype(float)], axis=1)
        sol, *_ = np.linalg.lstsq(A, w[i], rcond=None)
        assert np.allclose([mu[i], s0[i], s1[i]], sol, rtol=1e-9, atol=1e-12)


def test_refinement_never_increases_the_error():
    r = rng(4)
    w = fp16_groups(r, 60)

    def err(k):
        t0, t1, mu, s0, s1 = quantize.fit_two_plane(w, iters=k)
        rec = mu[:, None] + s0[:, None] * t0 + s1[:, None] * t1
        return ((w - rec) ** 2).sum(axis=1)

    prev = err(0)
    for k in range(1, 6):
        cur = err(k)
        assert np.all(cur <= prev * (1 + 1e-12))
        prev = cur


def test_second_plane_reduces_the_error():
    r = rng(5)
    w = fp16_groups(r, 80)
    t0, s0 = quantize.fit_one_plane(w)
    e1 = quantize.residual_energy(w, t0, s0)
    a, b, mu, c, d = quantize.fit_two_plane(w, iters=2)
    rec = mu[:, None] + c[:, None] * a + d[:, None] * b
    e2 = ((w - rec) ** 2).sum(axis=1)
    assert np.all(e2 < e1)


def test_selection_takes_the_largest_energies_with_index_ties():
    e = np.array([0.5, 2.0, 2.0, 0.1, 3.0, 2.0])
    assert list(quantize.select_two_plane(e, 0.5)) == [1, 2, 4]     # 3 of 6: 3.0, then 2.0 at 1 and 2
    assert list(quantize.select_two_plane(e, 0.0)) == []
    assert list(quantize.select_two_plane(e, 1.0)) == [0, 1, 2, 3, 4, 5]


@pytest.mark.parametrize("f2", [0.0, 0.1, 1.0])
def test_quantize_linear_builds_a_valid_packed_linear(f2):
    r = rng(6)
    N, K = 24, 512
    W = (r.standard_normal((N, K)) * 0.02).astype(np.float16)
    t0, s0, rowptr1, gidx1, t1, mu1, s1 = quantize.quantize_linear(W, f2, iters=3)
    nnz = int(np.floor(f2 * N * K / 128))
    assert rowptr1[0] == 0 and rowptr1[-1] == nnz == t1.shape[0]
    for row in range(N):
        g = gidx1[rowptr1[row]:rowptr1[row + 1]]
        assert np.all(np.diff(g.astype(int)) > 0)
    c0, bad0 = codec.pack(t0)
    c1, bad1 = codec.pack(t1) if nnz else (np.zeros(0, np.uint8), 0)
    assert bad0 == 0 and bad1 == 0
    What = packed.dequantize(N, K, c0, s0, rowptr1, gidx1, c1, mu1, s1)
    # The representation tracks W: relative Frobenius error of a 1.6-2 bit fit.
    rel = np.linalg.norm(What - W.astype(np.float64)) / np.linalg.norm(W.astype(np.float64))
    assert rel < 0.6
    if f2 == 1.0:
        e_one = quantize_linear_error(W, 0.0)
        assert rel < e_one


def quantize_linear_error(W, f2):
    N, K = W.shape
    t0, s0, rowptr1, gidx1, t1, mu1, s1 = quantize.quantize_linear(W, f2, iters=3)
    c0, _ = codec.pack(t0)
    c1 = codec.pack(t1)[0] if t1.shape[0] else np.zeros(0, np.uint8)
    What = packed.dequantize(N, K, c0, s0, rowptr1, gidx1, c1, mu1, s1)
    return np.linalg.norm(What - W.astype(np.float64)) / np.linalg.norm(W.astype(np.float64))


def test_offset_block_is_recovered_by_the_one_plane_offset_fit():
    # w = m + c*t with t balanced (mean 0): centring leaves c*t, so T0 = t,
    # s0 = c and mu = m, a fixed point of the refinement.
    t = np.tile(np.array([1, -1, 0, 1, -1, 0, 0, 0], np.int8), 16)[None, :]
    w = 0.25 + 0.0625 * t.astype(np.float64)
    for iters in (0, 3):
        t0, mu, s0 = quantize.fit_one_plane_offset(w, iters)
        assert np.array_equal(t0, t) and mu[0] == 0.25 and s0[0] == 0.0625


def test_one_plane_offset_refinement_converges_to_least_squares():
    r = rng(7)
    w = fp16_groups(r, 25) + 0.01
    t0, mu, s0 = quantize.fit_one_plane_offset(w, iters=300)
    for i in range(25):
        A = np.stack([np.ones(128), t0[i].astype(float)], axis=1)
        sol, *_ = np.linalg.lstsq(A, w[i], rcond=None)
        assert np.allclose([mu[i], s0[i]], sol, rtol=1e-9, atol=1e-12)


def test_quantize_linear_with_group_offsets():
    r = rng(8)
    N, K = 16, 512
    W = (r.standard_normal((N, K)) * 0.02 + 0.005).astype(np.float16)
    t0, s0, rowptr1, gidx1, t1, mu1, s1, mu0 = quantize.quantize_linear(W, 0.036, 3, group_offsets=True)
    assert np.all(mu1 == 0) and mu0.shape == (N, K // 128)
    c0 = codec.pack(t0)[0]
    c1 = codec.pack(t1)[0] if t1.shape[0] else np.zeros(0, np.uint8)
    What = packed.dequantize(N, K, c0, s0, rowptr1, gidx1, c1, mu1, s1, offset0=mu0)
    rel_off = np.linalg.norm(What - W.astype(np.float64)) / np.linalg.norm(W.astype(np.float64))
    assert rel_off < quantize_linear_error(W, 0.036)     # the offsets help on an offset matrix


# --------------------------------------------------- planted mistakes (oracle copies)

PINS = [
    test_scaled_ternary_block_is_recovered_exactly,
    test_threshold_is_strict_at_three_quarters_of_the_mean_magnitude,
    test_hand_worked_block,
    test_least_squares_scale_is_the_mean_magnitude_over_the_support,
    test_constant_block_is_its_offset,
    test_first_plane_uses_the_centred_weights,
    test_refinement_converges_to_the_joint_least_squares_fit,
    test_refinement_never_increases_the_error,
    test_second_plane_reduces_the_error,
    test_selection_takes_the_largest_energies_with_index_ties,
    test_offset_block_is_recovered_by_the_one_plane_offset_fit,
    test_one_plane_offset_refinement_converges_to_least_squares,
]


def _fit_two_plane_mutant(kind):
    sumf = quantize._sum

    def fit(w, iters):
        w = np.asarray(w, dtype=np.float64)
        mu = sumf(w) / 128
        wc = w if kind == "no_centring" else w - mu[..., None]
        t0 = quantize.threshold_support(wc)
        s0 = quantize.ls_scale(t0, wc)
        base = w if kind == "uncentred_residual" else wc
        r = base - s0[..., None] * t0
        t1 = quantize.threshold_support(r)
        s1 = quantize.ls_scale(t1, r)
        f0, f1 = t0.astype(np.float64), t1.astype(np.float64)
        for _ in range(iters):
            sign = 1.0 if kind == "offset_sign" else -1.0
            mu = sumf(w + sign * (s0[..., None] * f0) + sign * (s1[..., None] * f1)) / 128
            s0 = quantize.ls_scale(t0, w - mu[..., None] - s1[..., None] * f1)
            s1 = quantize.ls_scale(t1, w - mu[..., None] - s0[..., None] * f0)
        return t0, t1, mu, s0, s1
    return fit


def _apply_mutant(kind, monkeypatch):
    if kind == "threshold_0.7":
        monkeypatch.setattr(quantize, "THRESHOLD", 0.7)
    elif kind == "non_strict_threshold":
        def thr(v):
            d = (0.75 * (quantize._sum(np.abs(v)) / v.shape[-1]))[..., None]
            return np.where(v >= d, 1, np.where(v <= -d, -1, 0)).astype(np.int8)
        monkeypatch.setattr(quantize, "threshold_support", thr)
    elif kind == "scale_over_block":
        def ls(t, v):
            return quantize._sum(t.astype(np.float64) * v) / v.shape[-1]
        monkeypatch.setattr(quantize, "ls_scale", ls)
    elif kind in ("no_centring", "uncentred_residual", "offset_sign"):
        monkeypatch.setattr(quantize, "fit_two_plane", _fit_two_plane_mutant(kind))
    elif kind == "ties_high_index":
        def sel(energy, f2):
            energy = np.asarray(energy, dtype=np.float64)
            n = energy.size
            order = np.lexsort((-np.arange(n), -energy))
            return np.sort(order[:int(np.floor(f2 * n))])
        monkeypatch.setattr(quantize, "select_two_plane", sel)


@pytest.mark.parametrize("kind", ["threshold_0.7", "non_strict_threshold", "scale_over_block", "no_centring",
                                  "uncentred_residual", "offset_sign", "ties_high_index"])
def test_pins_catch_planted_mistakes(kind, monkeypatch):
    _apply_mutant(kind, monkeypatch)
    failed = 0
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            failed += 1
    assert failed > 0, kind
