"""GPU parity of the lattice codec and the dense fp16 dequantisation.

Bit-exact against the oracle: tq_pack, tq_unpack, tq_validate (error
counts) and tq_unpack_fp16 (one correct result: the fixed fp32 order rounded
once).
"""

import numpy as np
import pytest
import torch

from gpu_helpers import Case, log
from oracle import codec, packed
from paper_2609_09240_amd import synth, tq

pytestmark = pytest.mark.gpu


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("n", [1, 2, 3, 63, 1000, 32768])
def test_pack_unpack_bit_exact(n):
    log(f"pack/unpack n={n}")
    t = synth.ternary(synth.generator(1, n), (n, 128))
    want, bad = codec.pack(t)
    assert bad == 0
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    codes = tq.tq_pack(_dev(t), d_err=err)
    back = tq.tq_unpack(codes, n, d_err=err)
    v = tq.tq_validate(codes, n, d_err=err)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(codes.cpu().numpy(), want)
    np.testing.assert_array_equal(back.cpu().numpy(), t)
    assert int(v.item()) == 0


def test_empty_input_is_a_noop():
    codes = torch.empty(0, dtype=torch.uint8, device="cuda")
    tq.tq_pack(torch.empty((0, 128), dtype=torch.int8, device="cuda"), codes=codes)
    tq.tq_unpack(codes, 0)
    torch.cuda.synchronize()


def test_every_code_decodes_like_the_oracle():
    # 243 groups: main byte j of group f holds code (f + 7 j) % 256, so every
    # code 0..255 appears in every main position; tails are valid.
    n = 256
    g = np.zeros((n, 26), dtype=np.uint8)
    for f in range(n):
        for j in range(24):
            g[f, j] = (f + 7 * j) % 256
        g[f, 24] = f % 243
        g[f, 25] = 108 + f % 27
    flat = codec.to_storage(g)
    want, nbad = codec.unpack(flat, n)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    got = tq.tq_unpack(_dev(flat), n, d_err=err)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(got.cpu().numpy(), want)
    assert int(err.item()) == nbad == 13 * 24


def test_invalid_trits_give_sentinel_and_count():
    t = np.zeros((5, 128), dtype=np.int8)
    t[0, 7] = 2
    t[3, 127] = -2
    t[4, 0] = 100
    t[4, 1] = -100       # same byte as t[4, 0]: counted once
    want, nbad = codec.pack(t)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    got = tq.tq_pack(_dev(t), d_err=err)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(got.cpu().numpy(), want)
    assert int(err.item()) == nbad == 3


def test_validate_counts_like_the_oracle():
    rng = np.random.default_rng(5)
    n = 4096
    t = synth.ternary(synth.generator(5), (n, 128))
    flat, _ = codec.pack(t)
    flat = flat.copy()
    pos = rng.choice(flat.size, size=300, replace=False)
    flat[pos] = rng.integers(0, 256, size=300, dtype=np.uint8)
    want = codec.validate(flat, n)
    d_err = tq.tq_validate(_dev(flat), n)
    torch.cuda.synchronize()
    assert int(d_err.item()) == want > 0


@pytest.mark.parametrize("shape,f2", [((64, 256), 0.0), ((96, 512), 0.25), ((1024, 4096), 0.10),
                                      ((63, 2560), 1.0), ((5, 12288), 0.10)])
def test_unpack_fp16_bit_exact(shape, f2):
    n_out, n_in = shape
    log(f"unpack_fp16 {shape} f2={f2}")
    case = Case(synth.linear(n_out, n_in, f2, (3, 4, 5, n_out)))
    case.check_codes()
    want = packed.dequantize_fp16(*case.oracle_args())
    got = tq.tq_unpack_fp16(case.gpu)
    torch.cuda.synchronize()
    assert np.array_equal(got.cpu().numpy().view(np.uint16), want.view(np.uint16))
