"""Shared helpers of the GPU parity tests: build the same packed linear on
both sides (oracle packing on the CPU, tq_pack on the GPU) and compare."""

import sys

import numpy as np
import torch

from oracle import codec, packed
from paper_2609_09240_amd import tq


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


class Case:
    """One packed linear on both sides, built from the same unpacked inputs."""

    def __init__(self, inp, device="cuda", host_rowptr=True):
        self.inp = inp
        self.c0, b0 = codec.pack(inp.t0.reshape(-1, 128))
        if inp.nnz1:
            self.c1, b1 = codec.pack(inp.t1.reshape(-1, 128))
        else:
            self.c1, b1 = np.zeros(0, np.uint8), 0
        assert b0 == 0 and b1 == 0
        self.gpu = tq.PackedLinear.from_inputs(inp, device, host_rowptr=host_rowptr)

    def oracle_args(self):
        i = self.inp
        return (i.n_out, i.n_in, self.c0, i.s0, i.rowptr1, i.gidx1, self.c1, i.mu1, i.s1)

    def check_codes(self):
        torch.cuda.synchronize()
        np.testing.assert_array_equal(self.gpu.codes0.cpu().numpy(), self.c0)
        if self.inp.nnz1:
            np.testing.assert_array_equal(self.gpu.codes1.cpu().numpy(), self.c1)

    def oracle_gemm(self, X):
        return packed.gemm(*self.oracle_args(), X, offset0=self.inp.mu0)

    def oracle_gemv(self, x):
        return packed.gemv(*self.oracle_args(), x, offset0=self.inp.mu0)

    def bound(self, X):
        i = self.inp
        return packed.error_bound(i.n_out, i.n_in, i.s0, i.rowptr1, i.gidx1, i.mu1, i.s1, X, offset0=i.mu0)


def assert_within_bound(got, want, bound, what):
    got = np.asarray(got, dtype=np.float64)
    err = np.abs(got - want)
    bad = err > bound
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError(f"{what}: {int(bad.sum())} outputs outside the bound, e.g. at {idx.tolist()}: "
                             f"err {err[bad][:5]} bound {bound[bad][:5]}")
    return float((err / np.maximum(bound, 1e-300)).max())
