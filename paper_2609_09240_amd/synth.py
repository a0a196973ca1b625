"""Seeded synthetic workloads for the packed ternary linear (inputs only).

This module draws the *inputs* of the packed GEMV — trit planes, fp16 scales
and offsets, the two-plane group selection and fp16 activations — and holds
none of the method's arithmetic (no packing, no dequantisation, no products).
Both the HIP path and the CPU oracle consume what it returns.

The converted Qwen3-8B projections of the paper are not available, so these
arrays stand in for them with the shapes of the paper's model (section 3:
36 layers, hidden 4096, intermediate 12288; attention q, k, v, o and MLP
gate, up, down) and these value distributions:

* trits i.i.d. with P(-1) = 0.3, P(0) = 0.4, P(+1) = 0.3 (both planes);
* scales s0, s1 ~ U(0.01, 0.05) and offsets mu ~ U(-0.01, 0.01), rounded to
  fp16;
* the two-plane subset: exactly floor(f2 * N * K/128) groups drawn uniformly
  without replacement over the flattened (row, group) index, sorted;
* activations ~ N(0, 1) rounded to fp16, with an optional fraction of
  channels (the same channels for every batch row) scaled by 20 before
  rounding.

Every array comes from its own generator,
PCG64(SeedSequence([seed, config, layer, projection, field])).
"""

from dataclasses import dataclass

import numpy as np

GROUP = 128
HIDDEN = 4096
INTERMEDIATE = 12288
LAYERS = 36
KV_DIM = 1024

# Qwen3-8B linear projections as (name, out features, in features).
PROJECTIONS = (
    ("q", HIDDEN, HIDDEN),
    ("k", KV_DIM, HIDDEN),
    ("v", KV_DIM, HIDDEN),
    ("o", HIDDEN, HIDDEN),
    ("gate", INTERMEDIATE, HIDDEN),
    ("up", INTERMEDIATE, HIDDEN),
    ("down", HIDDEN, INTERMEDIATE),
)
PROJ_INDEX = {name: i for i, (name, _, _) in enumerate(PROJECTIONS)}
MLP = ("gate", "up", "down")
# Projections that read the same activation vector in one decode step.
STAGES = (("q", "k", "v"), ("o",), ("gate", "up"), ("down",))
STAGE_OF = {name: s for s, names in enumerate(STAGES) for name in names}

F_T0, F_S0, F_SEL, F_T1, F_MU, F_S1, F_X, F_MU0 = range(8)
_TERNARY = np.array([-1, -1, -1, 0, 0, 0, 0, 1, 1, 1], dtype=np.int8)


def generator(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


def ternary(rng, shape):
    """i.i.d. trits with P(-1) = 0.3, P(0) = 0.4, P(+1) = 0.3 (int8)."""
    return _TERNARY[rng.integers(0, 10, size=shape, dtype=np.uint8)]


def fp16_uniform(rng, lo, hi, size):
    return rng.uniform(lo, hi, size=size).astype(np.float16)


@dataclass
class LinearInputs:
    """Unpacked inputs of one packed linear (trits, not codes)."""
    n_out: int
    n_in: int
    t0: np.ndarray        # int8 [n_out, n_in]
    s0: np.ndarray        # fp16 [n_out, n_in/128]
    rowptr1: np.ndarray   # int32 [n_out + 1]
    gidx1: np.ndarray     # uint16 [nnz1]
    t1: np.ndarray        # int8 [nnz1, 128]
    mu1: np.ndarray       # fp16 [nnz1]
    s1: np.ndarray        # fp16 [nnz1]
    mu0: np.ndarray = None   # fp16 [n_out, n_in/128]: per-group offsets on every group, or None

    @property
    def nnz1(self):
        return int(self.gidx1.size)

    @property
    def n_groups(self):
        return self.n_out * (self.n_in // GROUP)


def selection(n_out, n_in, f2, rng):
    """CSR rows / group indices of the two-plane subset."""
    ng = n_in // GROUP
    nnz = int(np.floor(f2 * n_out * ng))
    flat = np.sort(rng.choice(n_out * ng, size=nnz, replace=False)) if nnz else np.zeros(0, np.int64)
    rows = flat // ng
    counts = np.bincount(rows, minlength=n_out)
    rowptr = np.zeros(n_out + 1, dtype=np.int32)
    rowptr[1:] = np.cumsum(counts)
    return rowptr, (flat % ng).astype(np.uint16)


def linear(n_out, n_in, f2, key, t0=None, offset0=False):
    """Inputs of one packed linear; ``key`` = (seed, config, layer, proj).
    With ``offset0`` every group also gets an offset mu0 ~ U(-0.01, 0.01)."""
    assert n_in % GROUP == 0 and n_out > 0
    ng = n_in // GROUP
    if t0 is None:
        t0 = ternary(generator(*key, F_T0), (n_out, n_in))
    s0 = fp16_uniform(generator(*key, F_S0), 0.01, 0.05, (n_out, ng))
    rowptr, gidx = selection(n_out, n_in, f2, generator(*key, F_SEL))
    nnz = gidx.size
    t1 = ternary(generator(*key, F_T1), (nnz, GROUP))
    mu = fp16_uniform(generator(*key, F_MU), -0.01, 0.01, nnz)
    s1 = fp16_uniform(generator(*key, F_S1), 0.01, 0.05, nnz)
    mu0 = fp16_uniform(generator(*key, F_MU0), -0.01, 0.01, (n_out, ng)) if offset0 else None
    return LinearInputs(n_out, n_in, t0, s0, rowptr, gidx, t1, mu, s1, mu0)


def activations(n_in, key, batch=None, outlier_frac=0.0):
    """fp16 activations [n_in] (batch None) or [batch, n_in]."""
    rng = generator(*key, F_X)
    shape = (n_in,) if batch is None else (batch, n_in)
    x = rng.standard_normal(shape)
    n_out = int(np.floor(outlier_frac * n_in))
    if n_out:
        ch = rng.choice(n_in, size=n_out, replace=False)
        x[..., ch] *= 20.0
    return x.astype(np.float16)


# --------------------------------------------------------------------------
# Named workloads (sizes of the Qwen3-8B decode step at batch 1).
# --------------------------------------------------------------------------

SEED = 0
TWO_PLANE = 0.10
# The paper's recorded mask coverages (section 3): 0.5% + 3.1% of blocks carry
# a second plane.
PAPER_TWO_PLANE = 0.036
OUTLIERS = 0.01


def single_linear(seed=SEED):
    """1024 x 4096, one plane only, x ~ N(0, 1)."""
    key = (seed, 0, 0, 0)
    return linear(1024, 4096, 0.0, key), activations(4096, key)


def projection(name, layer=0, cfg=3, seed=SEED, f2=TWO_PLANE, offset0=False):
    """Packed-linear inputs of one Qwen3-8B projection of ``layer`` (with
    ``offset0``, an offset on every group)."""
    p = PROJ_INDEX[name]
    _, n_out, n_in = PROJECTIONS[p]
    return linear(n_out, n_in, f2, (seed, cfg, layer, p), offset0=offset0)


def stage_activations(stage, layer=0, cfg=3, seed=SEED, batch=None):
    """Activations read by decode stage ``stage`` (q/k/v, o, gate/up, down).

    Projections of one stage share their input, as in a decode step; the MLP
    inputs carry outlier channels.
    """
    name = STAGES[stage][0]
    n_in = PROJECTIONS[PROJ_INDEX[name]][2]
    frac = OUTLIERS if name in MLP else 0.0
    return activations(n_in, (seed, cfg, layer, 100 + stage), batch, frac)
