"""GPU parity of tq_select_two_plane (the choice of two-plane groups and the
plane-1 CSR) against the oracle's rule (oracle.quantize.select_two_plane):
rec_index, rowptr1 and gidx1 bit-exact.  Energies are seeded numpy arrays,
with ties across the cut, NaN, signed zeros and infinities."""

import math

import numpy as np
import pytest
import torch

from gpu_helpers import log
from oracle import quantize
from paper_2609_09240_amd import tq

pytestmark = pytest.mark.gpu


def expected(energy, n_out, G, nnz):
    """CSR of the oracle's selection (records in flat order)."""
    n = n_out * G
    f2 = nnz / n if n else 0.0
    sel = quantize.select_two_plane(energy, f2)
    assert sel.size == nnz, (sel.size, nnz)
    rec = np.full(n, -1, np.int32)
    rec[sel] = np.arange(nnz, dtype=np.int32)
    rowptr = np.zeros(n_out + 1, np.int64)
    np.add.at(rowptr, sel // G + 1, 1)
    return rec, np.cumsum(rowptr).astype(np.int32), (sel % G).astype(np.uint16)


def check(energy, n_out, G, nnz, what):
    # nnz such that the oracle's floor(f2 * n) reproduces it exactly
    got = tq.tq_select_two_plane(torch.from_numpy(energy).cuda(), n_out, G, nnz)
    torch.cuda.synchronize()
    rec, rowptr, gidx = expected(energy, n_out, G, nnz)
    np.testing.assert_array_equal(got[0].cpu().numpy(), rec, err_msg=f"{what}: rec_index")
    np.testing.assert_array_equal(got[1].cpu().numpy(), rowptr, err_msg=f"{what}: rowptr1")
    np.testing.assert_array_equal(got[2].cpu().numpy().view(np.uint16), gidx, err_msg=f"{what}: gidx1")
    log(f"select {what}: n={n_out * G} nnz={nnz} ok")


def nnz_of(f2, n):
    return int(math.floor(f2 * n))


@pytest.mark.parametrize("f2", [0.0, 0.036, 0.1, 0.5, 1.0])
def test_random_ragged_tiles(f2):
    n_out, G = 1000, 13          # 13000 groups: four tiles, the last ragged
    e = np.random.default_rng(1).exponential(1.0, n_out * G)
    check(e, n_out, G, nnz_of(f2, n_out * G), f"random f2={f2}")


@pytest.mark.parametrize("levels,f2", [(3, 0.1), (5, 0.37), (1, 0.25), (2, 0.5)])
def test_ties_across_the_cut(levels, f2):
    """Few distinct energies, so the cut falls inside a run of equal keys:
    the lower flat indices among them are taken."""
    n_out, G = 777, 32
    e = np.random.default_rng(levels).integers(0, levels, n_out * G).astype(np.float64) * 0.5
    check(e, n_out, G, nnz_of(f2, n_out * G), f"ties levels={levels} f2={f2}")


def test_special_values():
    n_out, G = 300, 17
    r = np.random.default_rng(7)
    e = r.exponential(1.0, n_out * G)
    idx = r.permutation(n_out * G)
    e[idx[:40]] = np.nan
    e[idx[40:80]] = 0.0
    e[idx[80:120]] = -0.0
    e[idx[120:130]] = np.inf
    e[idx[130:140]] = 5e-324                 # smallest subnormal
    e[idx[140:150]] = 1e300
    for f2 in (0.001, 0.05, 0.99, 1.0):
        check(e, n_out, G, nnz_of(f2, n_out * G), f"special f2={f2}")
    # the cut inside the zeros (the NaNs go last)
    nz = int(np.sum(e > 0))
    check(e, n_out, G, nz + 50, "cut among the signed zeros")


def test_single_group_and_row():
    for nnz in (0, 1):
        check(np.array([2.5]), 1, 1, nnz, f"one group nnz={nnz}")
    e = np.array([1.0, 3.0, 3.0, 2.0, 3.0])
    check(e, 1, 5, 2, "one row with a tie")


def test_gate_sized_and_many_tiles():
    """A gate projection's 393216 groups at the benchmark's and the paper's
    shares, and 4.2 M groups (over 1024 tiles: the offsets pass runs in
    chunks)."""
    r = np.random.default_rng(9)
    n_out, G = 12288, 32
    e = np.round(r.chisquare(128, n_out * G) * 4) / 4          # many ties
    for f2 in (0.1, 0.036):
        check(e, n_out, G, nnz_of(f2, n_out * G), f"gate f2={f2}")
    n_out, G = 33000, 128
    e = r.exponential(1.0, n_out * G)
    check(e, n_out, G, nnz_of(0.1, n_out * G), "4.2 M groups")


def test_workspace_reuse_and_explicit_buffers():
    """Repeated calls on one workspace (its contents on entry do not
    matter) give the same result."""
    n_out, G = 513, 32
    e = np.random.default_rng(11).exponential(1.0, n_out * G)
    ed = torch.from_numpy(e).cuda()
    nnz = nnz_of(0.1, n_out * G)
    ws = torch.full((tq.tq_select_workspace_bytes(n_out * G),), 0xAB, dtype=torch.uint8, device="cuda")
    first = [t.cpu().numpy() for t in tq.tq_select_two_plane(ed, n_out, G, nnz, workspace=ws)]
    second = [t.cpu().numpy() for t in tq.tq_select_two_plane(ed, n_out, G, nnz, workspace=ws)]
    for a, b in zip(first, second):
        np.testing.assert_array_equal(a, b)
    rec, rowptr, gidx = expected(e, n_out, G, nnz)
    np.testing.assert_array_equal(first[0], rec)
