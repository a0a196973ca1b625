"""ctypes binding of libtq.so — argument marshalling only.

Each function has the name of the C entry point it calls (include/tq.h) and
takes torch tensors that already live on the GPU; torch provides device
memory and the current HIP stream, every step of the computation runs in the
library's kernels.  There is no fallback: if libtq.so is missing, every call
raises.
"""

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtq.so")

ABI_VERSION = 7
GROUP = 128
GROUP_BYTES = 26
OUT_FP16 = 0
OUT_FP32 = 1
MAX_GROUPED = 8
MAX_BATCH = 64

STATUS = {0: "TQ_OK", 1: "TQ_ERR_NULL", 2: "TQ_ERR_SHAPE", 3: "TQ_ERR_ALIGN",
          4: "TQ_ERR_UNSUPPORTED", 5: "TQ_ERR_HIP"}


class TqError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)}")


class TqMatrix(ctypes.Structure):
    _fields_ = [
        ("n_out", ctypes.c_int64),
        ("n_in", ctypes.c_int64),
        ("group", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
        ("codes0", ctypes.c_void_p),
        ("scale0", ctypes.c_void_p),
        ("nnz1", ctypes.c_int64),
        ("rowptr1", ctypes.c_void_p),
        ("gidx1", ctypes.c_void_p),
        ("codes1", ctypes.c_void_p),
        ("offset1", ctypes.c_void_p),
        ("scale1", ctypes.c_void_p),
        ("rowptr1_host", ctypes.c_void_p),
        ("offset0", ctypes.c_void_p),
    ]


class TqStage(ctypes.Structure):
    _fields_ = [
        ("mats", ctypes.POINTER(TqMatrix)),
        ("n", ctypes.c_int32),
        ("flags", ctypes.c_int32),
        ("x", ctypes.c_void_p),
        ("ys", ctypes.POINTER(ctypes.c_void_p)),
    ]


class TqChainInfo(ctypes.Structure):
    _fields_ = [
        ("n_stages", ctypes.c_int32),
        ("n_workgroups", ctypes.c_int32),
        ("lds_bytes", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
        ("plan_bytes", ctypes.c_int64),
        ("sync_bytes", ctypes.c_int64),
    ]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        mp = ctypes.POINTER(TqMatrix)
        sigs = {
            "tq_abi_version": ([], ctypes.c_int),
            "tq_status_string": ([ctypes.c_int], ctypes.c_char_p),
            "tq_pack": ([vp, i64, i32, vp, vp, vp], ctypes.c_int),
            "tq_unpack": ([vp, i64, i32, vp, vp, vp], ctypes.c_int),
            "tq_validate": ([vp, i64, i32, vp, vp], ctypes.c_int),
            "tq_unpack_fp16": ([mp, vp, vp], ctypes.c_int),
            "tq_gemv": ([mp, vp, vp, i32, vp], ctypes.c_int),
            "tq_gemv_grouped": ([mp, i32, vp, ctypes.POINTER(ctypes.c_void_p), i32, vp], ctypes.c_int),
            "tq_gemm_smallbatch": ([mp, vp, i32, vp, i32, vp], ctypes.c_int),
            "tq_ternarize": ([vp, i64, i32, vp, i64, i32, vp, vp, vp, vp, vp, vp, vp, vp], ctypes.c_int),
            "tq_select_workspace_bytes": ([i64], ctypes.c_size_t),
            "tq_select_two_plane": ([vp, i64, i32, i64, vp, vp, vp, vp, ctypes.c_size_t, vp], ctypes.c_int),
            "tq_select_two_plane_noalloc": ([vp, i64, i32, i64, vp, vp, vp, vp], ctypes.c_int),
            "tq_chain_plan": ([ctypes.POINTER(TqStage), i32, ctypes.POINTER(TqChainInfo), vp, ctypes.c_size_t],
                              ctypes.c_int),
            "tq_chain_sync_init": ([vp, ctypes.POINTER(TqChainInfo), vp], ctypes.c_int),
            "tq_gemv_chain": ([vp, vp, ctypes.POINTER(TqChainInfo), vp], ctypes.c_int),
        }
        for name, (args, res) in sigs.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        if L.tq_abi_version() != ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} implements ABI {L.tq_abi_version()}, the binding expects "
                               f"{ABI_VERSION}: rebuild it with __graft_entry__.build()")
        _lib = L
    return _lib


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _used_on(stream, *tensors):
    """Tensors that a launch on `stream` reads or writes: when that is not the
    current stream, tell the caching allocator not to reuse their memory
    before the stream's work is done."""
    if stream is not None and stream != torch.cuda.current_stream():
        for t in tensors:
            if t is not None:
                t.record_stream(stream)


def _after_current(stream):
    """Order `stream` after the work queued so far on the current stream
    (uploads made with .to(device) run there)."""
    if stream is not None and stream != torch.cuda.current_stream():
        stream.wait_stream(torch.cuda.current_stream())


def _host_copy(t, stream):
    """Host copy of a device tensor written on `stream`."""
    if stream is not None:
        torch.cuda.current_stream().wait_stream(stream)
    return t.cpu()


def _check(status, where):
    if status != 0:
        raise TqError(status, where)


def _cuda(t, dtype, name):
    if not (t.is_cuda and t.dtype == dtype and t.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous {dtype} tensor on the GPU")


# --------------------------------------------------------------------------
# Device-resident packed linear.
# --------------------------------------------------------------------------

@dataclass
class PackedLinear:
    """A packed linear in device memory (the buffers tq_matrix points at)."""
    n_out: int
    n_in: int
    codes0: torch.Tensor          # uint8 [26 * N * G]
    scale0: torch.Tensor          # float16 [N, G]
    rowptr1: torch.Tensor = None  # int32 [N + 1]
    gidx1: torch.Tensor = None    # int16 [nnz1] (uint16 values)
    codes1: torch.Tensor = None   # uint8 [26 * nnz1]
    offset1: torch.Tensor = None  # float16 [nnz1]
    scale1: torch.Tensor = None   # float16 [nnz1]
    rowptr1_host: torch.Tensor = None  # optional host copy of rowptr1 (int32, CPU)
    offset0: torch.Tensor = None  # optional float16 [N, G]: an offset on every group

    @property
    def nnz1(self):
        return 0 if self.gidx1 is None else int(self.gidx1.numel())

    @property
    def n_groups(self):
        return self.n_out * (self.n_in // GROUP)

    def struct(self):
        m = TqMatrix()
        m.n_out, m.n_in, m.group, m.reserved = self.n_out, self.n_in, GROUP, 0
        m.codes0 = self.codes0.data_ptr()
        m.scale0 = self.scale0.data_ptr()
        m.nnz1 = self.nnz1
        if self.nnz1:
            m.rowptr1 = self.rowptr1.data_ptr()
            m.gidx1 = self.gidx1.data_ptr()
            m.codes1 = self.codes1.data_ptr()
            m.offset1 = self.offset1.data_ptr()
            m.scale1 = self.scale1.data_ptr()
            if self.rowptr1_host is not None:
                m.rowptr1_host = self.rowptr1_host.data_ptr()
        if self.offset0 is not None:
            m.offset0 = self.offset0.data_ptr()
        return m

    def nbytes(self):
        """Bytes of the packed weights (codes, scales, plane-1 records, CSR)."""
        ng = self.n_groups
        b = GROUP_BYTES * ng + 2 * ng
        if self.offset0 is not None:
            b += 2 * ng
        if self.nnz1:
            b += 4 * (self.n_out + 1) + 32 * self.nnz1
        return b

    @classmethod
    def from_inputs(cls, inp, device="cuda", stream=None, host_rowptr=True):
        """Upload unpacked inputs (trits, scales, CSR) and pack them on the GPU.
        With host_rowptr the row pointers are also kept in host memory (see
        tq_matrix.rowptr1_host)."""
        dev = torch.device(device)
        t0 = torch.from_numpy(inp.t0.reshape(-1, GROUP)).to(dev)
        _after_current(stream)
        codes0 = tq_pack(t0, stream=stream)
        _used_on(stream, t0)
        del t0
        kw = {}
        if inp.nnz1:
            t1 = torch.from_numpy(inp.t1.reshape(-1, GROUP)).to(dev)
            _after_current(stream)
            _used_on(stream, t1)
            kw = dict(
                rowptr1=torch.from_numpy(inp.rowptr1).to(dev),
                gidx1=torch.from_numpy(inp.gidx1.view("int16")).to(dev),
                codes1=tq_pack(t1, stream=stream),
                offset1=torch.from_numpy(inp.mu1).to(dev),
                scale1=torch.from_numpy(inp.s1).to(dev),
            )
            if host_rowptr:
                kw["rowptr1_host"] = torch.from_numpy(inp.rowptr1.astype("int32")).contiguous()
        if getattr(inp, "mu0", None) is not None:
            kw["offset0"] = torch.from_numpy(inp.mu0).to(dev)
        return cls(inp.n_out, inp.n_in, codes0, torch.from_numpy(inp.s0).to(dev), **kw)


# --------------------------------------------------------------------------
# Entry points (same names as the C ABI).
# --------------------------------------------------------------------------

def tq_abi_version():
    return lib().tq_abi_version()


def tq_status_string(status):
    return lib().tq_status_string(status).decode()


def tq_pack(trits, codes=None, d_err=None, stream=None):
    """int8 trits [n, 128] -> uint8 codes [26 n] (split layout)."""
    _cuda(trits, torch.int8, "trits")
    n = trits.numel() // GROUP
    if codes is None:
        codes = torch.empty(GROUP_BYTES * n, dtype=torch.uint8, device=trits.device)
    _check(lib().tq_pack(_ptr(trits), n, GROUP, _ptr(codes), _ptr(d_err), _stream(stream)), "tq_pack")
    return codes


def tq_unpack(codes, n_groups, trits=None, d_err=None, stream=None):
    """uint8 codes [26 n] -> int8 trits [n, 128]."""
    _cuda(codes, torch.uint8, "codes")
    if trits is None:
        trits = torch.empty((n_groups, GROUP), dtype=torch.int8, device=codes.device)
    _check(lib().tq_unpack(_ptr(codes), n_groups, GROUP, _ptr(trits), _ptr(d_err), _stream(stream)),
           "tq_unpack")
    return trits


def tq_validate(codes, n_groups, d_err=None, stream=None):
    """Adds the number of invalid bytes to d_err (int32 [1]); returns d_err."""
    _cuda(codes, torch.uint8, "codes")
    if d_err is None:
        d_err = torch.zeros(1, dtype=torch.int32, device=codes.device)
    _check(lib().tq_validate(_ptr(codes), n_groups, GROUP, _ptr(d_err), _stream(stream)), "tq_validate")
    return d_err


def tq_unpack_fp16(mat, w=None, stream=None):
    """Dense fp16 W^ [N, K] in the fixed fp32 evaluation order."""
    if w is None:
        w = torch.empty((mat.n_out, mat.n_in), dtype=torch.float16, device=mat.codes0.device)
    m = mat.struct()
    _check(lib().tq_unpack_fp16(ctypes.byref(m), _ptr(w), _stream(stream)), "tq_unpack_fp16")
    return w


def _out(n, shape, out_f32, device):
    return torch.empty(shape, dtype=torch.float32 if out_f32 else torch.float16, device=device)


def tq_gemv(mat, x, y=None, out_f32=False, stream=None):
    """y = W^ x for fp16 x [K]; y fp16 [N] (or fp32)."""
    _cuda(x, torch.float16, "x")
    if y is None:
        y = _out(mat.n_out, (mat.n_out,), out_f32, x.device)
    m = mat.struct()
    _check(lib().tq_gemv(ctypes.byref(m), _ptr(x), _ptr(y), OUT_FP32 if out_f32 else OUT_FP16,
                         _stream(stream)), "tq_gemv")
    return y


def tq_gemv_grouped(mats, x, ys=None, out_f32=False, stream=None):
    """[W_i^ x for each matrix] in one launch (all matrices share K)."""
    _cuda(x, torch.float16, "x")
    n = len(mats)
    if ys is None:
        ys = [_out(m.n_out, (m.n_out,), out_f32, x.device) for m in mats]
    arr = (TqMatrix * n)(*[m.struct() for m in mats])
    yp = (ctypes.c_void_p * n)(*[y.data_ptr() for y in ys])
    _check(lib().tq_gemv_grouped(arr, n, _ptr(x), yp, OUT_FP32 if out_f32 else OUT_FP16,
                                 _stream(stream)), "tq_gemv_grouped")
    return ys


class Chain:
    """A planned chain of dependent grouped GEMVs (tq_chain_plan) with its
    device plan and sync block.  ``stages`` is a list of (matrices, x, ys):
    stage s computes tq_gemv_grouped(matrices, x) into ys and reads x only
    after stage s - 1 has finished.  Every tensor named here must outlive the
    chain."""

    def __init__(self, stages, out_f32=False, stream=None):
        import numpy as np
        self._keep = []
        arr = (TqStage * len(stages))()
        for st, (mats, x, ys) in zip(arr, stages):
            _cuda(x, torch.float16, "x")
            m = (TqMatrix * len(mats))(*[mm.struct() for mm in mats])
            yp = (ctypes.c_void_p * len(ys))(*[y.data_ptr() for y in ys])
            self._keep += [m, yp, x, list(mats), list(ys)]
            st.mats = ctypes.cast(m, ctypes.POINTER(TqMatrix))
            st.n = len(mats)
            st.flags = OUT_FP32 if out_f32 else OUT_FP16
            st.x = x.data_ptr()
            st.ys = ctypes.cast(yp, ctypes.POINTER(ctypes.c_void_p))
        self.info = TqChainInfo()
        _check(lib().tq_chain_plan(arr, len(stages), ctypes.byref(self.info), None, 0), "tq_chain_plan")
        host = np.zeros(self.info.plan_bytes, dtype=np.uint8)
        _check(lib().tq_chain_plan(arr, len(stages), ctypes.byref(self.info), host.ctypes.data_as(ctypes.c_void_p),
                                   host.nbytes), "tq_chain_plan")
        dev = stages[0][1].device
        self.plan = torch.from_numpy(host).to(dev)
        self.sync = torch.empty(self.info.sync_bytes, dtype=torch.uint8, device=dev)
        _check(lib().tq_chain_sync_init(_ptr(self.sync), ctypes.byref(self.info), _stream(stream)),
               "tq_chain_sync_init")

    def run(self, stream=None):
        """tq_gemv_chain: every stage, in order, in one launch."""
        _check(lib().tq_gemv_chain(_ptr(self.plan), _ptr(self.sync), ctypes.byref(self.info), _stream(stream)),
               "tq_gemv_chain")

    def error_flag(self, stream=None):
        """The sync block's sticky error word (nonzero after a call whose
        waits gave up)."""
        return int(_host_copy(self.sync[8:12], stream).view(torch.int32).item())


def tq_gemm_smallbatch(mat, X, Y=None, out_f32=False, stream=None):
    """Y = X W^T for fp16 X [B, K]; Y [B, N]."""
    _cuda(X, torch.float16, "X")
    B = X.shape[0]
    if Y is None:
        Y = _out(mat.n_out, (B, mat.n_out), out_f32, X.device)
    m = mat.struct()
    _check(lib().tq_gemm_smallbatch(ctypes.byref(m), _ptr(X), B, _ptr(Y), OUT_FP32 if out_f32 else OUT_FP16,
                                    _stream(stream)), "tq_gemm_smallbatch")
    return Y


def tq_ternarize(w, rec_index=None, nnz=0, iters=4, t0=None, s0=None, t1=None, offset1=None, scale1=None,
                 energy=None, want_energy=True, offset0=None, group_offsets=False, stream=None):
    """E2M-ATQ ternarisation of fp16 groups w [n, 128] (see include/tq.h).
    Returns (t0, s0, t1, offset1, scale1, energy, offset0); t1/offset1/scale1
    have nnz rows, energy is fp64 [n] (None unless requested), offset0 is
    fp16 [n] with ``group_offsets`` (or when passed in), else None."""
    _cuda(w, torch.float16, "w")
    n = w.numel() // GROUP
    dev = w.device
    if t0 is None:
        t0 = torch.empty((n, GROUP), dtype=torch.int8, device=dev)
    if s0 is None:
        s0 = torch.empty(n, dtype=torch.float16, device=dev)
    if nnz > 0:
        if t1 is None:
            t1 = torch.empty((nnz, GROUP), dtype=torch.int8, device=dev)
        if offset1 is None:
            offset1 = torch.empty(nnz, dtype=torch.float16, device=dev)
        if scale1 is None:
            scale1 = torch.empty(nnz, dtype=torch.float16, device=dev)
    if rec_index is not None:
        _cuda(rec_index, torch.int32, "rec_index")
    if want_energy and energy is None:
        energy = torch.empty(n, dtype=torch.float64, device=dev)
    if group_offsets and offset0 is None:
        offset0 = torch.empty(n, dtype=torch.float16, device=dev)
    _check(lib().tq_ternarize(_ptr(w), n, GROUP, _ptr(rec_index), nnz, iters, _ptr(t0), _ptr(s0), _ptr(t1),
                              _ptr(offset1), _ptr(scale1), _ptr(offset0), _ptr(energy), _stream(stream)),
           "tq_ternarize")
    return t0, s0, t1, offset1, scale1, energy, offset0


def tq_select_workspace_bytes(n_groups):
    return int(lib().tq_select_workspace_bytes(n_groups))


def tq_select_two_plane(energy, n_out, groups_per_row, nnz, rec_index=None, rowptr1=None, gidx1=None,
                        workspace=None, stream=None):
    """The nnz groups with the largest energy (fp64 [n_out * groups_per_row],
    on the GPU), ties to the lower flat index, and their plane-1 CSR: returns
    (rec_index int32 [n], rowptr1 int32 [n_out + 1], gidx1 int16 [nnz] holding
    uint16 group indices)."""
    _cuda(energy, torch.float64, "energy")
    n = n_out * groups_per_row
    dev = energy.device
    if rec_index is None:
        rec_index = torch.empty(n, dtype=torch.int32, device=dev)
    if rowptr1 is None:
        rowptr1 = torch.empty(n_out + 1, dtype=torch.int32, device=dev)
    if gidx1 is None:
        gidx1 = torch.empty(nnz, dtype=torch.int16, device=dev)
    if workspace is None:
        workspace = torch.empty(tq_select_workspace_bytes(n), dtype=torch.uint8, device=dev)
    _check(lib().tq_select_two_plane(_ptr(energy), n_out, groups_per_row, nnz, _ptr(rec_index), _ptr(rowptr1),
                                     _ptr(gidx1) if nnz else None, _ptr(workspace), workspace.numel(),
                                     _stream(stream)), "tq_select_two_plane")
    _used_on(stream, energy, rec_index, rowptr1, gidx1, workspace)
    return rec_index, rowptr1, gidx1


def tq_select_two_plane_noalloc(energy, n_out, groups_per_row, nnz, rec_index, rowptr1, gidx1, stream=None):
    """tq_select_two_plane on the library's static scratch: the caller
    passes every output buffer and nothing is allocated."""
    _cuda(energy, torch.float64, "energy")
    _check(lib().tq_select_two_plane_noalloc(_ptr(energy), n_out, groups_per_row, nnz, _ptr(rec_index),
                                             _ptr(rowptr1), _ptr(gidx1) if nnz else None, _stream(stream)),
           "tq_select_two_plane_noalloc")
    return rec_index, rowptr1, gidx1


def quantize_linear(W, f2=0.1, iters=4, host_rowptr=True, group_offsets=False, stream=None):
    """Packed linear from dense fp16 weights W [N, K] on the GPU: one-plane
    fits rank the groups (tq_ternarize), the top floor(f2 * N * K / 128) get
    two planes (tq_select_two_plane), then tq_ternarize and tq_pack produce
    the stored planes (section 4.2 and section 12).  With ``group_offsets``
    every group carries an offset (offset0), the paper's own representation
    of section 3, eq. 3."""
    import math
    _cuda(W, torch.float16, "W")
    N, K = W.shape
    if K % GROUP:
        raise ValueError("K must be a multiple of 128")
    ng = K // GROUP
    groups = W.reshape(N * ng, GROUP)
    _after_current(stream)
    # The ranking fit: with offsets its refinement decides the energy.
    ranking = tq_ternarize(groups, iters=iters if group_offsets else 0, group_offsets=group_offsets,
                           stream=stream)
    energy = ranking[5]
    nnz = int(math.floor(f2 * N * ng))
    rec, rowptr, gidx = tq_select_two_plane(energy, N, ng, nnz, stream=stream)
    _used_on(stream, groups, *[t for t in ranking if t is not None])
    t0, s0, t1, mu, s1, _, mu0 = tq_ternarize(groups, rec_index=rec, nnz=nnz, iters=iters, want_energy=False,
                                              group_offsets=group_offsets, stream=stream)
    codes0 = tq_pack(t0, stream=stream)
    _used_on(stream, rec, t0, t1, s0, mu, s1, mu0)
    kw = {}
    if nnz:
        kw = dict(rowptr1=rowptr, gidx1=gidx, codes1=tq_pack(t1, stream=stream), offset1=mu, scale1=s1)
        if host_rowptr:
            kw["rowptr1_host"] = _host_copy(rowptr, stream).contiguous()
    if group_offsets:
        kw["offset0"] = mu0.reshape(N, ng)
    return PackedLinear(N, K, codes0, s0.reshape(N, ng), **kw)
