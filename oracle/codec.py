"""Base-3 lattice codes — oracle definition (test infrastructure only).

Paper: section 12 (the lattice-aware format persists the discrete supports
losslessly) and eq. 3 (every support T_i takes values in {-1, 0, +1}).  The
paper fixes no byte layout; the reading used here is:

* A *group* is 128 consecutive trits (one row, 128 consecutive input indices).
* Byte j of a group (j = 0..25) holds trits 5j .. 5j+4 as the base-3 number
      code = sum_{i=0..4} (t_{5j+i} + 1) * 3**i         (digit i = t + 1),
  so a code lies in 0..242 and 243..255 are invalid.
* 128 = 25*5 + 3, so byte 25 holds trits 125..127 in digits 0..2 and its two
  pad digits (3 and 4) are 1, i.e. t = 0; a valid last byte lies in 108..134.
* Storage of n groups ("split layout"): the first 24 code bytes of every group
  come first, group after group (24*n bytes), then the last two code bytes of
  every group (2*n bytes).  Total 26*n bytes, 1.625 bits per trit.

Invalid data: ``pack`` writes 0xFF for a byte with any trit outside
{-1, 0, +1} and counts such bytes; ``unpack`` writes five zero trits for a
code above 242 and counts such bytes; ``validate`` counts codes above 242 plus
last bytes whose pad digits are not both 1.
"""

import numpy as np

GROUP = 128
TRITS_PER_BYTE = 5
BYTES_PER_GROUP = 26           # ceil(128 / 5)
MAIN_BYTES = 24                # code bytes 0..23 live in the main region
TAIL_BYTES = 2                 # code bytes 24, 25 live in the tail region
N_CODES = 243                  # 3**5
SENTINEL = 0xFF
POW3 = np.array([1, 3, 9, 27, 81], dtype=np.int64)


def encode_byte(trits5):
    """One code from five trits (plain Python; digit i is trit i plus one)."""
    assert len(trits5) == TRITS_PER_BYTE
    code = 0
    for i, t in enumerate(trits5):
        assert t in (-1, 0, 1)
        code += (int(t) + 1) * 3 ** i
    return code


def decode_byte(code):
    """Five trits from one code 0..242 (plain Python, repeated division)."""
    assert 0 <= code < N_CODES
    out = []
    for _ in range(TRITS_PER_BYTE):
        out.append(code % 3 - 1)
        code //= 3
    return out


def group_codes(trits):
    """Logical code sequence of each group: int8 [n, 128] -> (uint8 [n, 26], bad).

    ``bad`` is a bool [n, 26] mask of bytes that held an invalid trit.
    """
    trits = np.asarray(trits)
    assert trits.ndim == 2 and trits.shape[1] == GROUP
    n = trits.shape[0]
    t = np.zeros((n, BYTES_PER_GROUP * TRITS_PER_BYTE), dtype=np.int64)
    t[:, :GROUP] = trits           # the two pad positions stay t = 0
    t = t.reshape(n, BYTES_PER_GROUP, TRITS_PER_BYTE)
    bad = ~np.all((t >= -1) & (t <= 1), axis=2)
    codes = ((t + 1) * POW3).sum(axis=2)
    codes[bad] = SENTINEL
    return codes.astype(np.uint8), bad


def to_storage(gcodes):
    """Split layout: uint8 [n, 26] -> flat uint8 [26 n] (mains, then tails)."""
    gcodes = np.asarray(gcodes, dtype=np.uint8)
    return np.concatenate([gcodes[:, :MAIN_BYTES].ravel(),
                           gcodes[:, MAIN_BYTES:].ravel()])


def from_storage(flat, n_groups):
    """Inverse of ``to_storage``: flat uint8 [26 n] -> uint8 [n, 26]."""
    flat = np.asarray(flat, dtype=np.uint8).ravel()
    assert flat.size == BYTES_PER_GROUP * n_groups
    g = np.empty((n_groups, BYTES_PER_GROUP), dtype=np.uint8)
    g[:, :MAIN_BYTES] = flat[:MAIN_BYTES * n_groups].reshape(n_groups, MAIN_BYTES)
    g[:, MAIN_BYTES:] = flat[MAIN_BYTES * n_groups:].reshape(n_groups, TAIL_BYTES)
    return g


def pack(trits):
    """int8 trits [n, 128] -> (flat codes uint8 [26 n], number of bad bytes)."""
    gcodes, bad = group_codes(trits)
    return to_storage(gcodes), int(bad.sum())


def decode_codes(gcodes):
    """uint8 [n, 26] -> (int8 trits [n, 130] incl. pads, bad mask [n, 26])."""
    c = np.asarray(gcodes).astype(np.int64)
    bad = c >= N_CODES
    c = np.where(bad, 0, c)
    digits = (c[..., None] // POW3) % 3          # [n, 26, 5]
    t = (digits - 1).astype(np.int8)
    t[bad] = 0
    return t.reshape(c.shape[0], BYTES_PER_GROUP * TRITS_PER_BYTE), bad


def unpack(flat, n_groups):
    """Flat codes [26 n] -> (int8 trits [n, 128], number of bad bytes)."""
    t, bad = decode_codes(from_storage(flat, n_groups))
    return t[:, :GROUP].copy(), int(bad.sum())


def validate(flat, n_groups):
    """Count invalid bytes: codes > 242, and last bytes with pad digits != 1."""
    g = from_storage(flat, n_groups).astype(np.int64)
    over = g >= N_CODES
    last = g[:, BYTES_PER_GROUP - 1]
    pad_ok = (last // 27) == 4                   # digits 3 and 4 both equal 1
    bad_pad = ~over[:, BYTES_PER_GROUP - 1] & ~pad_ok
    return int(over.sum() + bad_pad.sum())
