"""Representation accounting — oracle definition (test infrastructure only).

Paper: eq. 1 (information of one ternary symbol, log2 3 bits) and section 11,
eq. 8 (effective bits B_eff ~ (1 + f2) * log2 3 where f2 is the fraction of
weights that carry a second plane).  Stored bytes follow the storage layout of
``codec`` and the record layout of the packed linear (fp16 scale per group;
per two-plane record: int16 group index, 26 code bytes, fp16 offset, fp16
scale; int32 row pointers).
"""

import math

TRIT_BITS = math.log2(3)


def b_eff(f2):
    """Effective weight-information bits per weight, eq. 8."""
    return (1.0 + f2) * TRIT_BITS


def packed_bytes(n_out, n_in, nnz1):
    """Bytes held by one packed linear (plane 0, scales, CSR plane 1)."""
    ng = n_in // 128
    plane0 = 26 * n_out * ng + 2 * n_out * ng
    plane1 = (4 * (n_out + 1) + 32 * nnz1) if nnz1 else 0
    return plane0 + plane1


def stored_bits_per_weight(n_out, n_in, nnz1):
    return 8.0 * packed_bytes(n_out, n_in, nnz1) / (n_out * n_in)


def gemv_bytes(n_out, n_in, nnz1, batch=1):
    """Algorithmic HBM bytes of one product: packed weights + fp16 X and Y."""
    return packed_bytes(n_out, n_in, nnz1) + 2 * n_in * batch + 2 * n_out * batch
