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


@pytest.mark.parametrize("shape,f2,offsets", [((8200, 4096), 0.10, False), ((8200, 4096), 0.036, True),
                                              ((8200, 4096), 0.0, False), ((8201, 4096), 0.10, False),
                                              ((16387, 256), 0.25, False), ((1030, 32768), 0.10, False)])
def test_unpack_fp16_more_row_blocks_than_workgroups(shape, f2, offsets):
    # More row blocks than persistent workgroups, so workgroups run several
    # pipelined steps: K = 4096 takes the exact-fit variant (4 rows of 32
    # groups per block; also without records), N = 8201 rows the
    # bounds-checked one (4 does not divide N), K = 256 the bounds-checked one
    # with a ragged last block (8 rows of 2 groups), K = 32768 the
    # bounds-checked one with two passes per block.
    n_out, n_in = shape
    log(f"unpack_fp16 pipelined {shape} f2={f2} offsets={offsets}")
    inp = synth.linear(n_out, n_in, f2, (31, 32, 33, n_out), offset0=offsets)
    case = Case(inp)
    want = packed.dequantize_fp16(*case.oracle_args(), offset0=inp.mu0 if offsets else None)
    got = tq.tq_unpack_fp16(case.gpu)
    torch.cuda.synchronize()
    assert np.array_equal(got.cpu().numpy().view(np.uint16), want.view(np.uint16))


@pytest.mark.parametrize("offset", [1, 3, 8])
def test_pack_unpack_unaligned_trit_buffers(offset):
    # Trit buffers that are not 16-byte aligned take the byte-per-thread path.
    n = 777
    log(f"pack/unpack unaligned offset={offset}")
    t = synth.ternary(synth.generator(9, n), (n, 128))
    want, _ = codec.pack(t)
    buf = torch.zeros(n * 128 + 64, dtype=torch.int8, device="cuda")
    src = buf[offset:offset + n * 128].view(n, 128)
    src.copy_(_dev(t))
    codes = tq.tq_pack(src)
    out = torch.zeros(n * 128 + 64, dtype=torch.int8, device="cuda")
    dst = out[offset:offset + n * 128].view(n, 128)
    tq.tq_unpack(codes, n, trits=dst)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(codes.cpu().numpy(), want)
    np.testing.assert_array_equal(dst.cpu().numpy(), t)
    # nothing written outside the view
    assert int(out[:offset].abs().sum()) == 0 and int(out[offset + n * 128:].abs().sum()) == 0


def test_pack_counts_invalid_trits_in_every_byte_position():
    # One bad trit in each of the 26 code bytes of group 1 (positions 5j), plus
    # a clean group on each side.
    t = np.zeros((3, 128), dtype=np.int8)
    t[1, 0:128:5] = [2 if j % 2 else -3 for j in range(26)]
    want, nbad = codec.pack(t)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    got = tq.tq_pack(_dev(t), d_err=err)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(got.cpu().numpy(), want)
    assert int(err.item()) == nbad == 26


def test_unpack_counts_invalid_tail_codes():
    n = 67
    rng = np.random.default_rng(11)
    t = synth.ternary(synth.generator(11), (n, 128))
    flat, _ = codec.pack(t)
    flat = flat.copy()
    tail = 24 * n + rng.choice(2 * n, size=20, replace=False)
    flat[tail] = rng.integers(243, 256, size=20, dtype=np.uint8)
    want, nbad = codec.unpack(flat, n)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    got = tq.tq_unpack(_dev(flat), n, d_err=err)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(got.cpu().numpy(), want)
    assert int(err.item()) == nbad == 20


@pytest.mark.parametrize("n", [1, 2, 3, 5, 7, 129])
def test_validate_ragged_buffers(n):
    # 26 n is not a multiple of 8 for n % 4 != 0: the last chunk is partial.
    rng = np.random.default_rng(100 + n)
    t = synth.ternary(synth.generator(100 + n), (n, 128))
    flat, _ = codec.pack(t)
    flat = flat.copy()
    k = min(flat.size, 9)
    pos = np.concatenate([rng.choice(flat.size, size=k, replace=False), [flat.size - 1, flat.size - 2]])
    flat[pos] = rng.integers(0, 256, size=pos.size, dtype=np.uint8)
    want = codec.validate(flat, n)
    got = tq.tq_validate(_dev(flat), n)
    torch.cuda.synchronize()
    assert int(got.item()) == want


def test_unpack_fp16_special_scales():
    # Scales +-0, subnormal, largest finite, +-inf and NaN on one- and two-plane
    # groups: the fixed fp32 order decides every result (inf * 0 is NaN).
    n_out, n_in = 8, 1024
    inp = synth.linear(n_out, n_in, 0.25, (21, 22, 23, n_out))
    specials = np.array([0x0000, 0x8000, 0x0001, 0x83FF, 0x7BFF, 0xFBFF, 0x7C00, 0xFC00, 0x7E00],
                        dtype=np.uint16)
    s0 = inp.s0.reshape(-1).view(np.uint16)
    s0[: specials.size * 3] = np.tile(specials, 3)
    if inp.nnz1:
        inp.mu1.view(np.uint16)[: specials.size] = specials
        inp.s1.view(np.uint16)[-specials.size:] = specials[::-1]
    case = Case(inp)
    want = packed.dequantize_fp16(*case.oracle_args())
    got = tq.tq_unpack_fp16(case.gpu).cpu().numpy()
    nan_w, nan_g = np.isnan(want), np.isnan(got)
    assert np.array_equal(nan_w, nan_g)
    assert np.array_equal(got.view(np.uint16)[~nan_g], want.view(np.uint16)[~nan_w])


@pytest.mark.parametrize("shape,f2", [((64, 256), 0.0), ((96, 512), 0.25), ((1024, 4096), 0.036),
                                      ((5, 12288), 1.0)])
def test_unpack_fp16_with_group_offsets(shape, f2):
    n_out, n_in = shape
    inp = synth.linear(n_out, n_in, f2, (7, 8, 9, n_out), offset0=True)
    case = Case(inp)
    want = packed.dequantize_fp16(*case.oracle_args(), offset0=inp.mu0)
    got = tq.tq_unpack_fp16(case.gpu)
    torch.cuda.synchronize()
    assert np.array_equal(got.cpu().numpy().view(np.uint16), want.view(np.uint16))
