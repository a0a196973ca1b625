"""GPU parity of tq_gemv / tq_gemv_grouped against the fp64 oracle.

Every output must satisfy |y - y_oracle| <= 2e-3 * sum_g coef_g * ||x_g||_1
(coef = |s0| + [two-plane](|mu| + |s1|)), computed per output element.
Shapes: the 1024 x 4096 single linear, every Qwen3-8B projection shape
(attention and MLP, 10% two-plane groups, MLP inputs with outlier
channels), a sample of the 36-layer stack run through the grouped launch
the benchmark times, and ragged shapes that leave partial passes, idle lanes
and one-row matrices.
"""

import numpy as np
import pytest
import torch

from gpu_helpers import Case, assert_within_bound, log
from paper_2609_09240_amd import synth, tq

pytestmark = pytest.mark.gpu


def run_gemv(case, x, out_f32=False):
    y = tq.tq_gemv(case.gpu, torch.from_numpy(x).cuda(), out_f32=out_f32)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def check(case, x, what, out_f32=False):
    case.check_codes()
    got = run_gemv(case, x, out_f32)
    want = case.oracle_gemm(x[None])[0]
    r = assert_within_bound(got, want, case.bound(x), what)
    log(f"{what}: max err/bound {r:.3g}")
    return got


def test_single_linear_1024x4096():
    inp, x = synth.single_linear()
    check(Case(inp), x, "cfg0 1024x4096")


@pytest.mark.parametrize("name", ["q", "k", "v", "o"])
def test_attention_projections(name):
    inp = synth.projection(name, layer=0, cfg=1)
    x = synth.stage_activations(synth.STAGE_OF[name], layer=0, cfg=1)
    check(Case(inp), x, f"cfg1 {name}")


@pytest.mark.parametrize("name", ["gate", "up", "down"])
def test_mlp_projections(name):
    inp = synth.projection(name, layer=0, cfg=2)
    x = synth.stage_activations(synth.STAGE_OF[name], layer=0, cfg=2)
    check(Case(inp), x, f"cfg2 {name}")


@pytest.mark.parametrize("n_out,n_in,f2", [
    (1, 128, 0.0), (1, 128, 1.0), (63, 256, 0.1), (65, 384, 0.5), (257, 4096, 0.1),
    (33, 2560, 0.2), (7, 12288, 0.3), (100, 32768, 0.05), (3000, 640, 0.1),
])
def test_ragged_shapes(n_out, n_in, f2):
    inp = synth.linear(n_out, n_in, f2, (7, n_out, n_in, 0))
    x = synth.activations(n_in, (7, n_out, n_in, 1), outlier_frac=0.01)
    check(Case(inp), x, f"ragged {n_out}x{n_in} f2={f2}")


def test_fp32_output_and_determinism():
    inp = synth.projection("q", layer=3, cfg=1)
    x = synth.stage_activations(0, layer=3, cfg=1)
    case = Case(inp)
    y32 = check(case, x, "q fp32", out_f32=True)
    again = run_gemv(case, x, out_f32=True)
    assert np.array_equal(y32.view(np.uint32), again.view(np.uint32))
    y16 = run_gemv(case, x)
    assert np.array_equal(y16.view(np.uint16), y32.astype(np.float16).view(np.uint16))


def test_zero_planes_give_positive_zero():
    inp = synth.linear(64, 512, 0.0, (8, 0, 0, 0))
    inp.t0[:] = 0
    x = synth.activations(512, (8, 0, 0, 1))
    got = run_gemv(Case(inp), x)
    assert np.all(got.view(np.uint16) == 0)


def test_unit_vector_reads_a_column():
    inp = synth.linear(40, 384, 0.5, (9, 0, 0, 0))
    case = Case(inp)
    for col in (0, 127, 128 + 64, 383):
        x = np.zeros(384, np.float16)
        x[col] = 1.0
        got = run_gemv(case, x, out_f32=True)
        want = case.oracle_gemm(x[None])[0]
        np.testing.assert_array_equal(got.astype(np.float64), want)


def test_grouped_matches_single_bitwise():
    layer = 1
    x = synth.stage_activations(0, layer=layer, cfg=1)
    cases = [Case(synth.projection(n, layer=layer, cfg=1)) for n in ("q", "k", "v")]
    xd = torch.from_numpy(x).cuda()
    ys = tq.tq_gemv_grouped([c.gpu for c in cases], xd)
    singles = [tq.tq_gemv(c.gpu, xd) for c in cases]
    torch.cuda.synchronize()
    for c, yg, ys1 in zip(cases, ys, singles):
        assert torch.equal(yg.view(torch.int16), ys1.view(torch.int16))
        want = c.oracle_gemm(x[None])[0]
        assert_within_bound(yg.cpu().numpy(), want, c.bound(x), "grouped")


@pytest.mark.parametrize("n_out,n_in,f2", [
    (4096, 4096, 0.1), (12288, 4096, 0.1), (4096, 12288, 0.1), (1024, 4096, 0.1),
    (3000, 640, 0.1), (100, 32768, 0.05), (65, 384, 0.5), (1, 128, 1.0),
])
def test_device_row_pointers_match_host_ranges(n_out, n_in, f2):
    """Without the host copy of the row pointers the kernel reads the record
    ranges itself and handles records after plane 0; the bits are the same."""
    inp = synth.linear(n_out, n_in, f2, (11, n_out, n_in, 0))
    x = synth.activations(n_in, (11, n_out, n_in, 1), outlier_frac=0.01)
    with_host = Case(inp)
    device_only = Case(inp, host_rowptr=False)
    assert device_only.gpu.rowptr1_host is None
    got = run_gemv(device_only, x, out_f32=True)
    ref = run_gemv(with_host, x, out_f32=True)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
    want = with_host.oracle_gemm(x[None])[0]
    r = assert_within_bound(got, want, with_host.bound(x), f"device ranges {n_out}x{n_in}")
    log(f"device ranges {n_out}x{n_in} f2={f2}: max err/bound {r:.3g}")


@pytest.mark.parametrize("layer", [0, 35])
def test_decode_step_layers_sampled(layer):
    """Layers of the 36-layer stack, in the grouped stages the benchmark runs."""
    for stage, names in enumerate(synth.STAGES):
        x = synth.stage_activations(stage, layer=layer, cfg=3)
        cases = [Case(synth.projection(n, layer=layer, cfg=3)) for n in names]
        ys = tq.tq_gemv_grouped([c.gpu for c in cases], torch.from_numpy(x).cuda())
        torch.cuda.synchronize()
        for n, c, y in zip(names, cases, ys):
            r = assert_within_bound(y.cpu().numpy(), c.oracle_gemm(x[None])[0], c.bound(x), f"L{layer} {n}")
            log(f"layer {layer} {n}: max err/bound {r:.3g}")


# ------------------------------------------------ per-group offsets (ABI 3)

@pytest.mark.parametrize("n_out,n_in,f2", [
    (1024, 4096, 0.0), (4096, 4096, synth.PAPER_TWO_PLANE), (12288, 4096, synth.PAPER_TWO_PLANE),
    (4096, 12288, 0.1), (3000, 640, 0.1), (65, 384, 0.5), (1, 128, 1.0), (100, 32768, 0.05),
])
def test_group_offsets(n_out, n_in, f2):
    """An offset on every group (the paper's representation): mu0 * sum(x_g)
    joins every group, within the bound with |mu0| in each coefficient."""
    inp = synth.linear(n_out, n_in, f2, (17, n_out, n_in, 0), offset0=True)
    x = synth.activations(n_in, (17, n_out, n_in, 1), outlier_frac=0.01)
    case = Case(inp)
    assert case.gpu.offset0 is not None
    check(case, x, f"offsets {n_out}x{n_in} f2={f2}", out_f32=True)
    device_only = Case(inp, host_rowptr=False)
    assert np.array_equal(run_gemv(device_only, x, True).view(np.uint32), run_gemv(case, x, True).view(np.uint32))


def test_grouped_mixes_matrices_with_and_without_offsets():
    """One launch serves matrices with and without offsets; each output is
    bit for bit what its own launch gives."""
    x = synth.activations(4096, (18, 0, 0, 1))
    cases = [Case(synth.linear(4096, 4096, 0.1, (18, 1, 0, 0), offset0=True)),
             Case(synth.linear(1024, 4096, 0.1, (18, 2, 0, 0))),
             Case(synth.linear(1024, 4096, synth.PAPER_TWO_PLANE, (18, 3, 0, 0), offset0=True))]
    xd = torch.from_numpy(x).cuda()
    ys = tq.tq_gemv_grouped([c.gpu for c in cases], xd, out_f32=True)
    singles = [tq.tq_gemv(c.gpu, xd, out_f32=True) for c in cases]
    torch.cuda.synchronize()
    for c, yg, y1 in zip(cases, ys, singles):
        assert torch.equal(yg.view(torch.int32), y1.view(torch.int32))
        assert_within_bound(yg.cpu().numpy(), c.oracle_gemm(x[None])[0], c.bound(x), "grouped offsets")


def _paper_shape(seed):
    """The paper's microbenchmark shape (section 13.1: one 4096 x 2560
    linear; orientation unstated, read as out 4096, in 2560: a 520-byte row
    of codes, not 16-byte aligned), 10% two-plane groups."""
    inp = synth.linear(4096, 2560, synth.TWO_PLANE, (9, 4096, 2560, seed))
    x = synth.activations(2560, (9, 4096, 2560, seed + 1), outlier_frac=0.01)
    return inp, x


def test_paper_microbenchmark_shape_4096x2560():
    inp, x = _paper_shape(0)
    check(Case(inp), x, "4096x2560 fp16 out")
    check(Case(inp), x, "4096x2560 fp32 out", out_f32=True)


@pytest.mark.parametrize("out_f32", [False, True])
def test_unpack_then_dense_route_within_bound(out_f32):
    """The second GPU route (the paper's chunk-unpack + dense GEMV of
    section 13.1): tq_unpack_fp16 to a dense fp16 W, then torch's fp16
    matrix-vector product; every output within the same bound, and the
    dense W bit-exact with the oracle's fp32-order dequantisation."""
    from oracle import packed
    inp, x = _paper_shape(2)
    case = Case(inp)
    W = tq.tq_unpack_fp16(case.gpu)
    xd = torch.from_numpy(x).cuda()
    y = torch.mv(W.float(), xd.float()) if out_f32 else torch.mv(W, xd)
    torch.cuda.synchronize()
    w_want = packed.dequantize_fp16(*case.oracle_args())
    np.testing.assert_array_equal(W.cpu().numpy().view(np.uint16), w_want.view(np.uint16))
    want = case.oracle_gemm(x[None])[0]
    r = assert_within_bound(y.cpu().numpy(), want, case.bound(x), f"unpack + torch.mv (fp32={out_f32})")
    log(f"4096x2560 unpack + dense mv fp32={out_f32}: max err/bound {r:.3g}")
