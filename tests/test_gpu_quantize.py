"""GPU parity of tq_ternarize (E2M-ATQ group ternarisation) against the
oracle: trits, fp16 scales and fp64 residual energies bit-exact."""

import numpy as np
import pytest
import torch

from gpu_helpers import log
from oracle import codec, packed, quantize
from paper_2609_09240_amd import tq

pytestmark = pytest.mark.gpu


def groups(seed, n, scale=0.02):
    r = np.random.default_rng(seed)
    return (r.standard_normal((n, 128)) * scale).astype(np.float16)


def run(w16, flags, iters, group_offsets=False):
    n = w16.shape[0]
    nnz = int(flags.sum())
    rec = np.full(n, -1, np.int32)
    rec[np.flatnonzero(flags)] = np.arange(nnz, dtype=np.int32)
    t0, s0, t1, mu, s1, e, mu0 = tq.tq_ternarize(torch.from_numpy(w16).cuda(),
                                                 rec_index=torch.from_numpy(rec).cuda() if nnz else None,
                                                 nnz=nnz, iters=iters, group_offsets=group_offsets)
    torch.cuda.synchronize()
    out = [t0.cpu().numpy(), s0.cpu().numpy(), e.cpu().numpy()]
    if nnz:
        out += [t1.cpu().numpy(), mu.cpu().numpy(), s1.cpu().numpy()]
    if group_offsets:
        out.append(mu0.cpu().numpy())
    return out


def check(w16, flags, iters, what):
    got = run(w16, flags, iters)
    w = w16.astype(np.float64)
    t0, t1, s0, mu, s1 = quantize.ternarize(w, flags, iters)
    t0_1, s0_1 = quantize.fit_one_plane(w)
    e = quantize.residual_energy(w, t0_1, s0_1)
    np.testing.assert_array_equal(got[0], t0, err_msg=what + " t0")
    np.testing.assert_array_equal(got[1].view(np.uint16), s0.view(np.uint16), err_msg=what + " s0")
    np.testing.assert_array_equal(got[2].view(np.uint64), e.view(np.uint64), err_msg=what + " energy")
    if flags.any():
        sel = np.flatnonzero(flags)
        np.testing.assert_array_equal(got[3], t1[sel], err_msg=what + " t1")
        np.testing.assert_array_equal(got[4].view(np.uint16), mu[sel].view(np.uint16), err_msg=what + " mu")
        np.testing.assert_array_equal(got[5].view(np.uint16), s1[sel].view(np.uint16), err_msg=what + " s1")


def check_offsets(w16, flags, iters, what):
    """Every group with an offset: the one-plane offset fit (and its energy)
    on one-plane groups, the two-plane fit with mu moved to the group."""
    got = run(w16, flags, iters, group_offsets=True)
    w = w16.astype(np.float64)
    t0, t1, s0, mu0, s1 = quantize.ternarize_with_offsets(w, flags, iters)
    a, m, b = quantize.fit_one_plane_offset(w, iters)
    e = quantize.residual_energy_offset(w, a, m, b)
    np.testing.assert_array_equal(got[0], t0, err_msg=what + " t0")
    np.testing.assert_array_equal(got[1].view(np.uint16), s0.view(np.uint16), err_msg=what + " s0")
    np.testing.assert_array_equal(got[2].view(np.uint64), e.view(np.uint64), err_msg=what + " energy")
    np.testing.assert_array_equal(got[-1].view(np.uint16), mu0.view(np.uint16), err_msg=what + " mu0")
    if flags.any():
        sel = np.flatnonzero(flags)
        np.testing.assert_array_equal(got[3], t1[sel], err_msg=what + " t1")
        assert np.all(got[4].view(np.uint16) == 0), what + " record offsets must be +0"
        np.testing.assert_array_equal(got[5].view(np.uint16), s1[sel].view(np.uint16), err_msg=what + " s1")


@pytest.mark.parametrize("iters", [0, 1, 4])
@pytest.mark.parametrize("frac", [0.0, 0.1, 1.0])
def test_ternarize_matches_oracle(frac, iters):
    n = 777
    w16 = groups(10 + iters, n)
    r = np.random.default_rng(20)
    flags = np.zeros(n, bool)
    flags[r.choice(n, int(frac * n), replace=False)] = True
    log(f"ternarize frac={frac} iters={iters}")
    check(w16, flags, iters, f"frac={frac} iters={iters}")


@pytest.mark.parametrize("iters", [0, 3])
@pytest.mark.parametrize("frac", [0.0, 0.036, 1.0])
def test_ternarize_with_group_offsets_matches_oracle(frac, iters):
    n = 1000
    r = np.random.default_rng(40 + iters)
    # Groups with offsets of their own (a shifted normal per group) so the
    # offset fit is exercised away from mu = 0.
    shift = r.standard_normal((n, 1)) * 0.01
    w16 = (r.standard_normal((n, 128)) * 0.02 + shift).astype(np.float16)
    flags = np.zeros(n, bool)
    flags[r.choice(n, int(frac * n), replace=False)] = True
    log(f"ternarize offsets frac={frac} iters={iters}")
    check_offsets(w16, flags, iters, f"offsets frac={frac} iters={iters}")


def test_special_groups():
    w = np.zeros((8, 128), np.float16)
    w[1] = 0.015625                                              # constant
    w[2] = (np.tile([1, -1, 0, 0], 32) * 0.03125).astype(np.float16)  # scaled ternary
    w[3, :4] = [4, -4, 1, -1]                                    # hand-worked block
    w[4] = np.concatenate([np.full(64, 5.0), np.full(64, 3.0)]).astype(np.float16)   # on the threshold
    w[5] = (np.random.default_rng(3).standard_normal(128) * 1e-6).astype(np.float16)  # subnormal scales
    w[6] = (np.random.default_rng(4).standard_normal(128) * 1000).astype(np.float16)  # large values
    w[7] = np.float16(-0.0)
    for flags in (np.zeros(8, bool), np.ones(8, bool)):
        check(w, flags, 3, f"special two_plane={flags[0]}")
        check_offsets(w, flags, 3, f"special offsets two_plane={flags[0]}")


def test_quantize_linear_matches_the_oracle_and_packs():
    r = np.random.default_rng(30)
    N, K = 96, 1024
    W = (r.standard_normal((N, K)) * 0.02).astype(np.float16)
    mat = tq.quantize_linear(torch.from_numpy(W).cuda(), f2=0.1, iters=4)
    torch.cuda.synchronize()
    t0, s0, rowptr1, gidx1, t1, mu1, s1 = quantize.quantize_linear(W, 0.1, 4)
    c0, _ = codec.pack(t0)
    c1, _ = codec.pack(t1)
    np.testing.assert_array_equal(mat.codes0.cpu().numpy(), c0)
    np.testing.assert_array_equal(mat.scale0.cpu().numpy().view(np.uint16), s0.view(np.uint16))
    np.testing.assert_array_equal(mat.rowptr1.cpu().numpy(), rowptr1)
    np.testing.assert_array_equal(mat.gidx1.cpu().numpy().view(np.uint16), gidx1)
    np.testing.assert_array_equal(mat.codes1.cpu().numpy(), c1)
    np.testing.assert_array_equal(mat.offset1.cpu().numpy().view(np.uint16), mu1.view(np.uint16))
    np.testing.assert_array_equal(mat.scale1.cpu().numpy().view(np.uint16), s1.view(np.uint16))
    # The quantised linear runs through the GEMV like any packed linear.
    x = r.standard_normal(K).astype(np.float16)
    y = tq.tq_gemv(mat, torch.from_numpy(x).cuda(), out_f32=True).cpu().numpy()
    want = packed.gemv(N, K, c0, s0, rowptr1, gidx1, c1, mu1, s1, x)
    bound = packed.error_bound(N, K, s0, rowptr1, gidx1, mu1, s1, x)
    assert np.all(np.abs(y - want) <= bound)


def test_quantize_linear_with_group_offsets_matches_the_oracle():
    """The paper's representation end to end: quantise with an offset on
    every group (the paper's two-plane share), pack, run the GEMV."""
    r = np.random.default_rng(31)
    N, K = 80, 1280
    W = (r.standard_normal((N, K)) * 0.02 + r.standard_normal((N, 1)) * 0.01).astype(np.float16)
    mat = tq.quantize_linear(torch.from_numpy(W).cuda(), f2=0.036, iters=3, group_offsets=True)
    torch.cuda.synchronize()
    t0, s0, rowptr1, gidx1, t1, mu1, s1, mu0 = quantize.quantize_linear(W, 0.036, 3, group_offsets=True)
    assert gidx1.size > 0
    c0, _ = codec.pack(t0)
    c1, _ = codec.pack(t1)
    np.testing.assert_array_equal(mat.codes0.cpu().numpy(), c0)
    np.testing.assert_array_equal(mat.scale0.cpu().numpy().view(np.uint16), s0.view(np.uint16))
    np.testing.assert_array_equal(mat.offset0.cpu().numpy().view(np.uint16), mu0.view(np.uint16))
    np.testing.assert_array_equal(mat.rowptr1.cpu().numpy(), rowptr1)
    np.testing.assert_array_equal(mat.gidx1.cpu().numpy().view(np.uint16), gidx1)
    np.testing.assert_array_equal(mat.codes1.cpu().numpy(), c1)
    np.testing.assert_array_equal(mat.offset1.cpu().numpy().view(np.uint16), mu1.view(np.uint16))
    np.testing.assert_array_equal(mat.scale1.cpu().numpy().view(np.uint16), s1.view(np.uint16))
    x = r.standard_normal(K).astype(np.float16)
    y = tq.tq_gemv(mat, torch.from_numpy(x).cuda(), out_f32=True).cpu().numpy()
    want = packed.gemv(N, K, c0, s0, rowptr1, gidx1, c1, mu1, s1, x, offset0=mu0)
    bound = packed.error_bound(N, K, s0, rowptr1, gidx1, mu1, s1, x, offset0=mu0)
    assert np.all(np.abs(y - want) <= bound)
