"""CPU oracle for the packed ternary GEMV — TEST INFRASTRUCTURE ONLY.

This package is the plain, slow, obviously-correct reference that the HIP
library is checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it; the product path never
does, and it shares no code with the HIP path (it only reads the same input
arrays).

What it computes (paper: section 3, eq. 3; section 12):

* ``codec``      — the base-3 lattice code: five trits per byte, encode /
                   decode / validate, and the byte layout of a packed group.
* ``packed``     — full fp64 dequantisation of a packed linear and the exact
                   products y = W x and Y = X W^T; the fp32-order dense fp16
                   dequantisation; the per-row acceptance bound.
* ``accounting`` — the information / storage bit accounting of section 11.
* ``quantize``   — E2M-ATQ group ternarisation (section 4.2, eqs. 4-6): the
                   offset, thresholded supports, least-squares scales and
                   their refinement, and the choice of two-plane groups.

Parity status: codec, packed, accounting and quantize are pinned by tests in
``tests/test_oracle_*.py`` (brute force over all codes, exact rational
arithmetic on tiny shapes, closed-form special cases, an independent
least-squares solver, and the paper's printed bit-accounting figures).  The paper prints no worked packing or GEMV example,
so agreement with *the paper's own numbers* is pinned only for accounting.
"""

from . import accounting, codec, packed, quantize  # noqa: F401
