"""GPU parity of tq_gemv_chain (a chain of dependent grouped GEMVs in one
launch): every stage's outputs equal tq_gemv_grouped's bit for bit and lie
within the oracle's bound; a stage whose x is the previous stage's output
reads it only after it is complete; repeated calls reuse the sync block."""

import numpy as np
import pytest
import torch

from gpu_helpers import Case, assert_within_bound, log
from paper_2609_09240_amd import synth, tq

pytestmark = pytest.mark.gpu


def grouped(mats, x, out_f32):
    ys = tq.tq_gemv_grouped(mats, x, out_f32=out_f32)
    torch.cuda.synchronize()
    return [y.cpu().numpy() for y in ys]


def test_chain_feeds_outputs_forward():
    """Stage s+1 reads stage s's fp16 output as its x: any stale read would
    change the bits of every later stage."""
    shapes = [(512, 256, 0.1), (640, 512, 0.2), (256, 640, 0.1), (384, 256, 0.0), (128, 384, 0.3)]
    cases = [Case(synth.linear(n, k, f2, (31, n, k, i))) for i, (n, k, f2) in enumerate(shapes)]
    x0 = torch.from_numpy(synth.activations(256, (31, 0, 0, 9))).cuda()
    ys = [torch.empty(n, dtype=torch.float16, device="cuda") for n, _, _ in shapes]
    xs = [x0] + ys[:-1]
    chain = tq.Chain([([c.gpu], x, [y]) for c, x, y in zip(cases, xs, ys)])
    for call in range(3):
        for y in ys:
            y.fill_(float("nan"))
        chain.run()
        torch.cuda.synchronize()
        got = [y.cpu().numpy() for y in ys]
        # the same chain, one tq_gemv_grouped after another
        x = x0
        for i, c in enumerate(cases):
            want = grouped([c.gpu], x, False)[0]
            np.testing.assert_array_equal(got[i].view(np.uint16), want.view(np.uint16),
                                          err_msg=f"call {call} stage {i}")
            xn = x.cpu().numpy()
            assert_within_bound(got[i], c.oracle_gemv(xn), c.bound(xn), f"stage {i} vs oracle")
            x = torch.from_numpy(got[i]).cuda()
    assert chain.error_flag() == 0
    log("chain of 5 dependent stages: bit-exact with sequential grouped GEMVs over 3 calls")


@pytest.mark.parametrize("out_f32", [False, True])
def test_chain_two_decode_layers(out_f32):
    """Two layers of the Qwen3-8B decode step (8 stages: q+k+v, o, gate+up,
    down) against tq_gemv_grouped bit for bit and the oracle on layer 0."""
    names = [n for n, _, _ in synth.PROJECTIONS]
    stages, cases, ys = [], [], []
    for layer in (0, 35):
        inps = {n: synth.projection(n, layer, cfg=3) for n in names}
        cs = {n: Case(inps[n]) for n in names}
        for s, group in enumerate(synth.STAGES):
            x = torch.from_numpy(synth.stage_activations(s, layer, cfg=3)).cuda()
            out = [torch.empty(cs[n].inp.n_out, dtype=torch.float32 if out_f32 else torch.float16, device="cuda")
                   for n in group]
            stages.append(([cs[n].gpu for n in group], x, out))
            cases.append([cs[n] for n in group])
            ys.append(out)
    chain = tq.Chain(stages, out_f32=out_f32)
    chain.run()
    torch.cuda.synchronize()
    for si, ((mats, x, out), cs) in enumerate(zip(stages, cases)):
        want = grouped(mats, x, out_f32)
        for i, (y, w) in enumerate(zip(out, want)):
            a = y.cpu().numpy()
            np.testing.assert_array_equal(a.view(np.uint32 if out_f32 else np.uint16),
                                          w.view(np.uint32 if out_f32 else np.uint16), err_msg=f"stage {si}.{i}")
        if si < 4:
            xn = x.cpu().numpy()
            for c, y in zip(cs, out):
                assert_within_bound(y.cpu().numpy(), c.oracle_gemv(xn), c.bound(xn), f"layer 0 stage {si}")
    assert chain.error_flag() == 0
    log(f"chain of 8 decode-step stages (fp32={out_f32}): bit-exact with grouped GEMVs")


def test_chain_mixed_shapes_offsets_and_idle_workgroups():
    """Stages that leave most workgroups idle (one row), K = 12288 and
    K = 128, per-group offsets, no host row pointers (record ranges read on
    the device), and all-two-plane groups."""
    specs = [
        (dict(n_out=1, n_in=128, f2=1.0), True),
        (dict(n_out=300, n_in=12288, f2=0.1), True),
        (dict(n_out=4100, n_in=1024, f2=0.05), False),
        (dict(n_out=64, n_in=4096, f2=0.5), True),
    ]
    stages, cases = [], []
    for i, (sp, host) in enumerate(specs):
        inp = synth.linear(sp["n_out"], sp["n_in"], sp["f2"], (33, i, 0, 0), offset0=(i % 2 == 1))
        c = Case(inp, host_rowptr=host)
        x = torch.from_numpy(synth.activations(sp["n_in"], (33, i, 0, 1), outlier_frac=0.01)).cuda()
        y = torch.empty(sp["n_out"], dtype=torch.float16, device="cuda")
        stages.append(([c.gpu], x, [y]))
        cases.append(c)
    chain = tq.Chain(stages)
    for _ in range(2):
        chain.run()
    torch.cuda.synchronize()
    for (mats, x, (y,)), c in zip(stages, cases):
        want = grouped(mats, x, False)[0]
        np.testing.assert_array_equal(y.cpu().numpy().view(np.uint16), want.view(np.uint16))
        xn = x.cpu().numpy()
        assert_within_bound(y.cpu().numpy(), c.oracle_gemv(xn), c.bound(xn), f"{c.inp.n_out}x{c.inp.n_in}")
    assert chain.error_flag() == 0
