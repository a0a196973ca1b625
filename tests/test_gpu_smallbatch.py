"""GPU parity of tq_gemm_smallbatch (B = 1: the GEMV; 2..4: the GEMV's decode
per batch row; larger: the MFMA kernel over quads of groups, or the
per-group fallback) against the fp64 oracle, per (batch row, output) within
the same bound as the GEMV."""

import numpy as np
import pytest
import torch

from gpu_helpers import Case, assert_within_bound, log
from paper_2609_09240_amd import synth, tq

pytestmark = pytest.mark.gpu


def run(case, X, out_f32=False):
    Y = tq.tq_gemm_smallbatch(case.gpu, torch.from_numpy(X).cuda(), out_f32=out_f32)
    torch.cuda.synchronize()
    return Y.cpu().numpy()


@pytest.mark.parametrize("B", [1, 2, 4, 15, 16, 17, 33, 64])
@pytest.mark.parametrize("n_out,n_in,f2", [(100, 512, 0.2), (64, 2560, 0.1), (1, 128, 1.0)])
def test_small_shapes(B, n_out, n_in, f2):
    case = Case(synth.linear(n_out, n_in, f2, (11, n_out, n_in, B)))
    X = synth.activations(n_in, (11, n_out, n_in, 99), batch=B, outlier_frac=0.01)
    got = run(case, X)
    want = case.oracle_gemm(X)
    r = assert_within_bound(got, want, case.bound(X), f"B={B} {n_out}x{n_in}")
    log(f"smallbatch B={B} {n_out}x{n_in}: max err/bound {r:.3g}")


@pytest.mark.parametrize("B", [1, 4, 16, 64])
@pytest.mark.parametrize("name", ["gate", "down"])
def test_mlp_shapes(B, name):
    case = Case(synth.projection(name, layer=0, cfg=4))
    X = synth.stage_activations(synth.STAGE_OF[name], layer=0, cfg=4, batch=B)
    got = run(case, X, out_f32=True)
    want = case.oracle_gemm(X)
    r = assert_within_bound(got, want, case.bound(X), f"{name} B={B}")
    log(f"smallbatch {name} B={B}: max err/bound {r:.3g}")


def test_batch_rows_match_gemv():
    case = Case(synth.projection("k", layer=2, cfg=4))
    X = synth.stage_activations(0, layer=2, cfg=4, batch=8)
    Y = run(case, X, out_f32=True)
    for b in range(8):
        y = tq.tq_gemv(case.gpu, torch.from_numpy(X[b].copy()).cuda(), out_f32=True)
        torch.cuda.synchronize()
        want = case.oracle_gemm(X[b:b + 1])[0]
        bound = case.bound(X[b])
        assert_within_bound(Y[b], want, bound, f"row {b}")
        assert_within_bound(y.cpu().numpy(), want, bound, f"gemv row {b}")


def test_deterministic():
    case = Case(synth.linear(300, 1024, 0.1, (12, 0, 0, 0)))
    X = synth.activations(1024, (12, 0, 0, 1), batch=24)
    a, b = run(case, X, True), run(case, X, True)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("name,B", [("gate", 64), ("down", 16), ("down", 40)])
def test_deterministic_mlp_shapes(name, B):
    """The eight waves' partial sums over K are added in a fixed order, so
    repeated calls give the same bits (fp32 output) at the MLP shapes."""
    case = Case(synth.projection(name, layer=3, cfg=4))
    X = synth.stage_activations(synth.STAGE_OF[name], layer=3, cfg=4, batch=B)
    first = run(case, X, True)
    for _ in range(2):
        assert np.array_equal(first.view(np.uint32), run(case, X, True).view(np.uint32))


@pytest.mark.parametrize("B", [3, 16, 40, 64])
@pytest.mark.parametrize("n_out,n_in,f2", [
    (5000, 512, 0.1),      # one quad of groups (seven of eight waves get none), two row tiles per workgroup
    (13000, 256, 0.1),     # half a quad; four row tiles (three with four column tiles), ragged last workgroup
    (16400, 256, 0.05),    # four row tiles with up to three column tiles
    (300, 10240, 0.1),     # three quads per wave, the last waves' quads past the end of K
    (40, 16384, 0.1),      # four quads per wave, the most the registers allow
    (40, 16896, 0.1),      # more quads per wave than that: the per-group fallback kernel
    (100, 8192, 1.0),      # every group two-plane: over 512 records per workgroup, staged in several batches
])
def test_workgroup_layouts(B, n_out, n_in, f2):
    log(f"smallbatch layout B={B} {n_out}x{n_in} f2={f2}")
    case = Case(synth.linear(n_out, n_in, f2, (13, n_out, n_in, B)))
    X = synth.activations(n_in, (13, n_out, n_in, 98), batch=B, outlier_frac=0.01)
    got = run(case, X, out_f32=(B % 2 == 0))
    want = case.oracle_gemm(X)
    r = assert_within_bound(got, want, case.bound(X), f"B={B} {n_out}x{n_in}")
    log(f"  max err/bound {r:.3g}")


@pytest.mark.parametrize("B", [17, 40, 64])
@pytest.mark.parametrize("n_out,n_in,f2", [(5000, 512, 0.1), (300, 10240, 0.1), (100, 8192, 1.0)])
def test_without_host_row_pointers(B, n_out, n_in, f2):
    """Without the host row pointers the MFMA kernel reads each workgroup's
    record range from the device row pointers (after the codes): same
    results within the bound, for several column tiles and more than 512
    records per workgroup."""
    log(f"smallbatch device ranges B={B} {n_out}x{n_in} f2={f2}")
    inp = synth.linear(n_out, n_in, f2, (23, n_out, n_in, B))
    X = synth.activations(n_in, (23, n_out, n_in, 96), batch=B, outlier_frac=0.01)
    case = Case(inp, host_rowptr=False)
    got = run(case, X, out_f32=True)
    r = assert_within_bound(got, case.oracle_gemm(X), case.bound(X), f"device ranges B={B} {n_out}x{n_in}")
    log(f"  max err/bound {r:.3g}")


@pytest.mark.parametrize("B", [4, 16, 64])
@pytest.mark.parametrize("n_out,n_in,f2", [
    (12288, 4096, 0.036), (4096, 12288, 0.1), (5000, 512, 0.1), (40, 16384, 0.1), (40, 16896, 0.1),
    (100, 1024, 1.0),
])
def test_group_offsets(B, n_out, n_in, f2):
    """Per-group offsets on every group, through every workgroup layout and
    the fallback kernel."""
    log(f"smallbatch offsets B={B} {n_out}x{n_in} f2={f2}")
    case = Case(synth.linear(n_out, n_in, f2, (19, n_out, n_in, B), offset0=True))
    X = synth.activations(n_in, (19, n_out, n_in, 97), batch=B, outlier_frac=0.01)
    got = run(case, X, out_f32=True)
    r = assert_within_bound(got, case.oracle_gemm(X), case.bound(X), f"offsets B={B} {n_out}x{n_in}")
    log(f"  max err/bound {r:.3g}")


# --------------------------------------- B = 2..4: the GEMV decode per row

@pytest.mark.parametrize("B", [2, 3, 4])
@pytest.mark.parametrize("n_out,n_in,f2", [
    (12288, 4096, 0.1), (4096, 12288, 0.1), (1024, 4096, 0.1), (3000, 640, 0.1), (65, 384, 0.5),
    (1, 128, 1.0), (257, 128, 0.0), (100, 32768, 0.05),
])
def test_few_rows_match_oracle_and_mfma_path(B, n_out, n_in, f2):
    """B = 2..4 decode each code byte once for every row (the GEMV's table
    and layout) where the launch fits, the MFMA path otherwise (K = 32768 at
    B = 3, 4, or no host row pointers): both within the bound everywhere."""
    inp = synth.linear(n_out, n_in, f2, (21, n_out, n_in, B))
    X = synth.activations(n_in, (21, n_out, n_in, 98), batch=B, outlier_frac=0.01)
    case = Case(inp)
    got = run(case, X, out_f32=True)
    want = case.oracle_gemm(X)
    r = assert_within_bound(got, want, case.bound(X), f"few rows B={B} {n_out}x{n_in}")
    mfma = run(Case(inp, host_rowptr=False), X, out_f32=True)
    r2 = assert_within_bound(mfma, want, case.bound(X), f"mfma B={B} {n_out}x{n_in}")
    log(f"few rows B={B} {n_out}x{n_in}: max err/bound {r:.3g} (mfma path {r2:.3g})")


@pytest.mark.parametrize("name,B", [
    ("q", 2), ("q", 3), ("q", 4), ("k", 2), ("k", 4), ("gate", 2), ("gate", 3), ("gate", 4), ("down", 2), ("down", 3),
])
def test_few_rows_equal_gemv_per_row(name, B):
    """Each row of a B = 2..4 batch goes through the same arithmetic, in the
    same order, as the GEMV of that row alone: equal values (+0 and -0
    compare equal), fp16 and fp32 outputs.  (down at B = 4 takes the MFMA
    kernel: four staged rows of x do not fit in LDS beside the table; its
    parity is in test_mlp_shapes.)"""
    case = Case(synth.projection(name, layer=1, cfg=4))
    X = synth.stage_activations(synth.STAGE_OF[name], layer=1, cfg=4, batch=B)
    for out_f32 in (False, True):
        Y = run(case, X, out_f32=out_f32)
        for b in range(B):
            y = tq.tq_gemv(case.gpu, torch.from_numpy(X[b].copy()).cuda(), out_f32=out_f32)
            torch.cuda.synchronize()
            assert np.array_equal(Y[b], y.cpu().numpy()), f"{name} B={B} row {b} f32={out_f32}"
    want = case.oracle_gemm(X)
    r = assert_within_bound(run(case, X, True), want, case.bound(X), f"{name} B={B}")
    log(f"few rows {name} B={B}: equal to the GEMV per row, max err/bound {r:.3g}")


@pytest.mark.parametrize("B", [2, 3, 4])
@pytest.mark.parametrize("n_out,n_in,f2", [(4096, 4096, synth.PAPER_TWO_PLANE), (300, 1024, 0.1)])
def test_few_rows_group_offsets(B, n_out, n_in, f2):
    inp = synth.linear(n_out, n_in, f2, (23, n_out, n_in, B), offset0=True)
    X = synth.activations(n_in, (23, n_out, n_in, 97), batch=B, outlier_frac=0.01)
    case = Case(inp)
    got = run(case, X, out_f32=True)
    r = assert_within_bound(got, case.oracle_gemm(X), case.bound(X), f"few rows offsets B={B}")
    for b in range(B):
        y = tq.tq_gemv(case.gpu, torch.from_numpy(X[b].copy()).cuda(), out_f32=True)
        torch.cuda.synchronize()
        assert np.array_equal(got[b], y.cpu().numpy())
    log(f"few rows offsets B={B} {n_out}x{n_in}: max err/bound {r:.3g}")


@pytest.mark.parametrize("B,shift", [(5, 7), (16, -5), (40, 10 ** 6), (3, 10 ** 6)])
def test_bad_host_rowptr_stays_in_bounds(B, shift):
    """A host copy of the row pointers that differs from the device copy
    (shifted, or far past nnz1) gives unspecified values but every access
    stays in bounds: the call completes and the output is finite."""
    case = Case(synth.linear(700, 1024, 0.1, (13, B, 0, 0)))
    good = case.gpu.rowptr1_host.clone()
    case.gpu.rowptr1_host = (good.to(torch.int64) + shift).clamp(-(2 ** 31), 2 ** 31 - 1).to(torch.int32)
    X = synth.activations(1024, (13, B, 0, 1), batch=B)
    got = run(case, X, out_f32=True)
    assert np.all(np.isfinite(got))
    case.gpu.rowptr1_host = good
    want = case.oracle_gemm(X)
    assert_within_bound(run(case, X, out_f32=True), want, case.bound(X), f"B={B} after restoring rowptr")
