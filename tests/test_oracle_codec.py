"""Pins of the oracle's lattice codec (CPU only).

The paper (section 12) requires lossless re-encoding of the discrete supports
and fixes no byte layout; these tests pin the oracle's base-3 code to
independent definitions: Python's own base-3 integer parser and
``numpy.base_repr``, brute force over all 3**5 trit tuples, hand-worked
examples, and the layout rules stated in ``oracle/codec.py``.
"""

import itertools

import numpy as np
import pytest

from oracle import codec


def _base3_reference(trits5):
    # Independent route: the digit string (most significant first) parsed by int().
    return int("".join(str(t + 1) for t in reversed(trits5)), 3)


def test_all_243_tuples_encode_like_base3_integers():
    seen = set()
    for tup in itertools.product((-1, 0, 1), repeat=5):
        c = codec.encode_byte(tup)
        assert c == _base3_reference(tup)
        assert 0 <= c < 243
        seen.add(c)
    assert seen == set(range(243))


def test_all_243_codes_decode_like_base_repr():
    for c in range(243):
        digits = np.base_repr(c, 3).zfill(5)[::-1]          # least significant first
        assert codec.decode_byte(c) == [int(d) - 1 for d in digits]
        assert codec.encode_byte(codec.decode_byte(c)) == c


def test_hand_worked_examples():
    # (-1, 0, +1, +1, -1) -> digits (0, 1, 2, 2, 0) -> 0 + 3 + 18 + 54 + 0 = 75
    assert codec.encode_byte((-1, 0, 1, 1, -1)) == 75
    assert codec.encode_byte((0, 0, 0, 0, 0)) == 121
    assert codec.encode_byte((1, 1, 1, 1, 1)) == 242
    assert codec.encode_byte((-1, -1, -1, -1, -1)) == 0


def test_vectorised_group_codes_match_scalar_definition():
    rng = np.random.default_rng(1)
    t = rng.integers(-1, 2, size=(7, 128)).astype(np.int8)
    g, bad = codec.group_codes(t)
    assert not bad.any()
    for n in range(7):
        padded = list(t[n]) + [0, 0]
        for j in range(26):
            assert g[n, j] == codec.encode_byte(padded[5 * j:5 * j + 5])


def test_last_byte_pad_digits_are_one():
    rng = np.random.default_rng(2)
    t = rng.integers(-1, 2, size=(50, 128)).astype(np.int8)
    g, _ = codec.group_codes(t)
    last = g[:, 25].astype(int)
    assert np.all((last >= 108) & (last <= 134))
    assert np.all(last // 27 == 4)
    # trits 125..127 sit in digits 0..2 of byte 25
    for n in range(50):
        assert codec.decode_byte(int(last[n]))[:3] == list(t[n, 125:128])


def test_split_storage_layout_positions():
    rng = np.random.default_rng(3)
    n = 5
    t = rng.integers(-1, 2, size=(n, 128)).astype(np.int8)
    g, _ = codec.group_codes(t)
    flat, bad = codec.pack(t)
    assert bad == 0 and flat.size == 26 * n
    for f in range(n):
        for j in range(24):
            assert flat[24 * f + j] == g[f, j]
        assert flat[24 * n + 2 * f] == g[f, 24]
        assert flat[24 * n + 2 * f + 1] == g[f, 25]


@pytest.mark.parametrize("n", [1, 2, 3, 31, 257])
def test_pack_unpack_roundtrip_bit_exact(n):
    rng = np.random.default_rng(10 + n)
    t = rng.integers(-1, 2, size=(n, 128)).astype(np.int8)
    flat, bad = codec.pack(t)
    assert bad == 0
    back, bad2 = codec.unpack(flat, n)
    assert bad2 == 0
    np.testing.assert_array_equal(back, t)
    assert codec.validate(flat, n) == 0


def test_pack_flags_invalid_trits_with_sentinel():
    t = np.zeros((3, 128), dtype=np.int8)
    t[0, 7] = 2            # byte 1 of group 0
    t[2, 127] = -2         # byte 25 of group 2
    t[2, 0] = 5            # byte 0 of group 2
    flat, bad = codec.pack(t)
    assert bad == 3
    g = codec.from_storage(flat, 3)
    assert g[0, 1] == 0xFF and g[2, 25] == 0xFF and g[2, 0] == 0xFF
    assert g[0, 0] == 121 and g[1, 5] == 121


@pytest.mark.parametrize("code", list(range(243, 256)))
def test_invalid_codes_rejected(code):
    flat, _ = codec.pack(np.zeros((2, 128), dtype=np.int8))
    flat = flat.copy()
    flat[24 + 3] = code                       # group 1, byte 3
    t, bad = codec.unpack(flat, 2)
    assert bad == 1
    assert np.all(t[1, 15:20] == 0)
    assert codec.validate(flat, 2) == 1


def test_validate_flags_bad_pad_digits():
    flat, _ = codec.pack(np.zeros((4, 128), dtype=np.int8))
    flat = flat.copy()
    # group 2, byte 25 (tail region): 121 has digits (1,1,1,1,1); 121 - 27 = 94
    # has digit 3 = 0, i.e. a non-zero pad trit.
    idx = 24 * 4 + 2 * 2 + 1
    assert flat[idx] == 121
    flat[idx] = 94
    assert codec.validate(flat, 4) == 1
    t, bad = codec.unpack(flat, 4)           # unpack decodes only 128 trits
    assert bad == 0 and np.all(t == 0)
