"""ctypes binding of libgcnlayer (include/gcn_layer.h), same names as the C ABI.

Argument marshalling only: torch tensors provide device memory and the current
HIP stream; every step of the computation runs in the library's kernels.  The
library must be built (``paper_1810_11899_amd.build``); without it every call
raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

from .build import LIB_PATH

GCN_OK, GCN_EINVAL, GCN_ESHAPE, GCN_EWORKSPACE, GCN_EHIP, GCN_EUNSUPPORTED = 0, -1, -2, -3, -4, -5
GCN_F32, GCN_BF16 = 0, 1
GCN_AGGREGATE_FIRST, GCN_TRANSFORM_FIRST = 0, 1
GCN_SOFTMAX_CE, GCN_SIGMOID_BCE = 0, 1
LOSS_KIND = {"ce": GCN_SOFTMAX_CE, "bce": GCN_SIGMOID_BCE}
GCN_NOALLOC_SCRATCH_BYTES = 64 << 20      # the static scratch array of gcn_aggregate_noalloc
PREC = {"f32": GCN_F32, "fp32": GCN_F32, "bf16": GCN_BF16}


class GcnError(RuntimeError):
    def __init__(self, code: int, where: str, msg: str):
        super().__init__(f"{where} failed with {code}: {msg}")
        self.code = code


class gcn_csr(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int32), ("n_cols", ctypes.c_int32), ("nnz", ctypes.c_int32),
                ("indptr", ctypes.c_void_p), ("indices", ctypes.c_void_p), ("vals", ctypes.c_void_p),
                ("indices16", ctypes.c_void_p)]


class gcn_sampler_params(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int32), ("n", ctypes.c_int32), ("db_entries", ctypes.c_int32),
                ("ia_slots", ctypes.c_int32), ("cap", ctypes.c_int32), ("seed", ctypes.c_uint64)]


class gcn_layer_args(ctypes.Structure):
    _fields_ = [("f_in", ctypes.c_int32), ("h", ctypes.c_int32), ("order", ctypes.c_int),
                ("W_self", ctypes.c_void_p), ("W_neigh", ctypes.c_void_p), ("bias", ctypes.c_void_p),
                ("Y", ctypes.c_void_p), ("ldy", ctypes.c_int32), ("saved", ctypes.c_void_p),
                ("saved_bytes", ctypes.c_size_t), ("dH", ctypes.c_void_p), ("lddh", ctypes.c_int32),
                ("dW_self", ctypes.c_void_p), ("dW_neigh", ctypes.c_void_p), ("dbias", ctypes.c_void_p)]


class gcn_head_args(ctypes.Structure):
    _fields_ = [("W_pred", ctypes.c_void_p), ("b_pred", ctypes.c_void_p), ("C", ctypes.c_int32),
                ("kind", ctypes.c_int), ("labels", ctypes.c_void_p), ("targets", ctypes.c_void_p),
                ("loss", ctypes.c_void_p), ("dHL", ctypes.c_void_p), ("lddhl", ctypes.c_int32),
                ("dW_pred", ctypes.c_void_p), ("db_pred", ctypes.c_void_p)]


SAMPLE_STATUS = {0: "ok", 1: "exhausted", 2: "overflow", 3: "probe_limit", 4: "root_limit", 5: "bad_graph"}

_lib = None
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_CSRP = ctypes.POINTER(gcn_csr)

_SIGNATURES = {
    "gcn_last_error": (ctypes.c_char_p, []),
    "gcn_version": (ctypes.c_int, []),
    "gcn_csr_validate_host": (ctypes.c_int, [_I32, _I32, _I32, _P, _P, ctypes.c_int]),
    "gcn_csr_validate": (ctypes.c_int, [_CSRP, ctypes.c_int, _P, _P]),
    "gcn_csr_transpose_workspace_bytes": (_SZ, [_I32, _I32, _I32]),
    "gcn_csr_transpose": (ctypes.c_int, [_CSRP, _P, _P, _P, _P, _SZ, _P]),
    "gcn_csr_transpose_symmetric_workspace_bytes": (_SZ, [_I32, _I32]),
    "gcn_csr_transpose_symmetric": (ctypes.c_int, [_CSRP, _P, _P, _SZ, _P]),
    "gcn_aggregate_workspace_bytes": (_SZ, [_I32, _I32, _I32, _I32, ctypes.c_int]),
    "gcn_aggregate": (ctypes.c_int, [_CSRP, _P, _I32, _I32, _P, _I32, ctypes.c_int, _P, _SZ, _P]),
    "gcn_aggregate_noalloc": (ctypes.c_int, [_CSRP, _P, _I32, _I32, _P, _I32, ctypes.c_int, _P]),
    "gcn_layer_pick_order": (ctypes.c_int, [_I32, _I32, ctypes.c_int]),
    "gcn_layer_saved_bytes": (_SZ, [_I32, _I32, _I32, ctypes.c_int, ctypes.c_int]),
    "gcn_layer_workspace_bytes": (_SZ, [_I32, _I32, _I32, _I32, ctypes.c_int, ctypes.c_int]),
    "gcn_layer_fwd": (ctypes.c_int, [_CSRP, _P, _I32, _I32, _P, _P, _P, _I32, _P, _I32, _P, _SZ,
                                     ctypes.c_int, ctypes.c_int, _P, _SZ, _P]),
    "gcn_layer_bwd": (ctypes.c_int, [_CSRP, _CSRP, _P, _I32, _I32, _P, _P, _I32, _P, _I32, _P, _SZ,
                                     _P, _I32, _P, _I32, _P, _P, _P, ctypes.c_int, ctypes.c_int, _P, _SZ,
                                     _P]),
    "gcn_loss_workspace_bytes": (_SZ, [_I32, _I32, _I32, ctypes.c_int]),
    "gcn_loss_grad": (ctypes.c_int, [_P, _I32, _I32, _I32, _P, _P, _I32, ctypes.c_int, _P, _P, _P, _P,
                                     _I32, _P, _P, ctypes.c_int, _P, _SZ, _P]),
    "gcn_model_workspace_bytes": (_SZ, [_I32, _I32, _I32, ctypes.POINTER(gcn_layer_args),
                                        ctypes.POINTER(gcn_head_args), ctypes.c_int]),
    "gcn_model_step": (ctypes.c_int, [_CSRP, _CSRP, _P, _I32, _I32, ctypes.POINTER(gcn_layer_args),
                                      ctypes.POINTER(gcn_head_args), _P, _I32, ctypes.c_int, _P, _SZ, _P]),
    "gcn_f32_to_bf16": (ctypes.c_int, [_P, _P, _I64, _P]),
    "gcn_profile_enable": (ctypes.c_int, [ctypes.c_int]),
    "gcn_profile_reset": (ctypes.c_int, []),
    "gcn_profile_class_count": (ctypes.c_int, []),
    "gcn_profile_class_name": (ctypes.c_char_p, [ctypes.c_int]),
    "gcn_profile_read": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_double)]),
    # gcn_sampler.h
    "gcn_sampler_plan": (ctypes.c_int, [_I32, _P, _I32, _I32, ctypes.c_double, _I32, ctypes.c_uint64,
                                        ctypes.POINTER(gcn_sampler_params)]),
    "gcn_frontier_sample": (ctypes.c_int, [_CSRP, ctypes.POINTER(gcn_sampler_params), _I64, _I32, _P, _P, _P,
                                           _P]),
    "gcn_induce_workspace_bytes": (_SZ, [_I32, _I32, _I32]),
    "gcn_induce_subgraphs": (ctypes.c_int, [_CSRP, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _P,
                                            _P, _SZ, _P]),
    "gcn_csr_pattern_symmetric_host": (ctypes.c_int, [_I32, _P, _P]),
    "gcn_gather_rows": (ctypes.c_int, [_P, _I32, _I32, _I64, _P, _I32, _P, _I64, _P]),
    # gcn_optim.h
    "gcn_adam_update": (ctypes.c_int, [_P, _P, _P, _P, _I64, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                       ctypes.c_double, _I32, _P]),
    # gcn_peaks.h
    "gcn_peak_stream_read": (ctypes.c_int, [_P, _I64, _P, _I32, _P]),
    "gcn_peak_mfma": (ctypes.c_int, [ctypes.c_int, _I32, _I32, _P, ctypes.POINTER(ctypes.c_double), _P]),
    "gcn_peak_chase": (ctypes.c_int, [_P, _I64, _I32, _I32, _P, _P]),
    "gcn_peak_gather": (ctypes.c_int, [_P, _I64, _I32, _I64, _P, _I64, _P, _I32, _P]),
}


def lib():
    """Load libgcnlayer.so; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_1810_11899_amd.build "
                               f"(__graft_entry__.build()); there is no fallback path")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def exported_symbols():
    return list(_SIGNATURES)


def _check(rc: int, where: str):
    if rc != GCN_OK:
        raise GcnError(rc, where, lib().gcn_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ld(t: torch.Tensor) -> int:
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("expected a row-major 2-D tensor with unit column stride")
    return int(t.stride(0)) if t.shape[0] > 1 else max(int(t.stride(0)), int(t.shape[1]))


def _dev_f32(t: torch.Tensor, name: str):
    if not (t.is_cuda and t.dtype == torch.float32):
        raise TypeError(f"{name} must be a float32 CUDA/HIP tensor")


# --------------------------------------------------------------------------
class Workspace:
    """Grow-only device scratch handed to the library."""

    def __init__(self, device="cuda"):
        self.device = torch.device(device)
        self.buf = torch.empty(0, dtype=torch.uint8, device=self.device)

    def get(self, nbytes: int) -> torch.Tensor:
        nbytes = max(int(nbytes), 256)
        if self.buf.numel() < nbytes:
            self.buf = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        return self.buf

    def args(self, nbytes: int):
        b = self.get(nbytes)
        return ctypes.c_void_p(b.data_ptr()), ctypes.c_size_t(b.numel())


class DeviceCSR:
    """CSR arrays resident on the device: int32 indptr, float32 vals, and the
    column indices as int32, or as uint16 (an int16 tensor holding the bits)
    when the columns number at most 65,536."""

    def __init__(self, n_rows, n_cols, indptr, indices, vals):
        self.n_rows, self.n_cols = int(n_rows), int(n_cols)
        self.indptr, self.indices, self.vals = indptr, indices, vals
        self.nnz = int(indices.numel())
        if indices.dtype not in (torch.int32, torch.int16):
            raise TypeError("indices must be int32, or int16 holding uint16 bits")
        if indices.dtype == torch.int16 and self.n_cols > 65536:
            raise ValueError("uint16 indices need n_cols <= 65536")

    @property
    def index_bits(self) -> int:
        return 16 if self.indices.dtype == torch.int16 else 32

    @classmethod
    def from_host(cls, n_rows, n_cols, indptr, indices, vals, device="cuda", index_bits=32):
        import numpy as np
        d = torch.device(device)
        ip = torch.as_tensor(indptr, dtype=torch.int32).to(d)
        if index_bits == 16:
            ix = torch.from_numpy(np.ascontiguousarray(np.asarray(indices, dtype=np.uint16)).view(np.int16)).to(d)
        else:
            ix = torch.as_tensor(indices, dtype=torch.int32).to(d)
        vv = torch.as_tensor(vals, dtype=torch.float32).to(d)
        return cls(n_rows, n_cols, ip, ix, vv)

    def struct(self) -> gcn_csr:
        ix = self.indices.data_ptr() if self.nnz else None
        return gcn_csr(self.n_rows, self.n_cols, self.nnz, self.indptr.data_ptr(),
                       ix if self.index_bits == 32 else None,
                       self.vals.data_ptr() if self.nnz else None,
                       ix if self.index_bits == 16 else None)


# ------------------------------------------------------------------- calls
def gcn_csr_validate_host(n_rows, n_cols, indptr, indices, require_sorted=True) -> int:
    import numpy as np
    ip = np.ascontiguousarray(indptr, dtype=np.int32)
    ix = np.ascontiguousarray(indices, dtype=np.int32)
    return lib().gcn_csr_validate_host(n_rows, n_cols, int(ix.size), ip.ctypes.data,
                                       ix.ctypes.data if ix.size else None, int(require_sorted))


CSR_VIOLATION = {0: "ok", 1: "endpoints", 2: "indptr decreases", 3: "index out of range", 4: "not ascending"}


def gcn_csr_validate(A: DeviceCSR, require_sorted=True, status: Optional[torch.Tensor] = None, stream=None):
    """Enqueue the device-side CSR check; returns the int32[2] status tensor
    (kind of the first violation, its row), valid after synchronization."""
    if status is None:
        status = torch.empty(2, dtype=torch.int32, device=A.indptr.device)
    s = A.struct()
    _check(lib().gcn_csr_validate(ctypes.byref(s), int(bool(require_sorted)), _ptr(status), _stream(stream)),
           "gcn_csr_validate")
    return status


def gcn_csr_transpose(A: DeviceCSR, ws: Workspace, stream=None) -> DeviceCSR:
    d = A.indptr.device
    t_indptr = torch.empty(A.n_cols + 1, dtype=torch.int32, device=d)
    t_indices = torch.empty(max(A.nnz, 1), dtype=torch.int32, device=d)[:A.nnz]
    t_vals = torch.empty(max(A.nnz, 1), dtype=torch.float32, device=d)[:A.nnz]
    gcn_csr_transpose_into(A, t_indptr, t_indices, t_vals, ws, stream)
    return DeviceCSR(A.n_cols, A.n_rows, t_indptr, t_indices, t_vals)


def gcn_csr_transpose_into(A: DeviceCSR, t_indptr, t_indices, t_vals, ws: Workspace, stream=None):
    L = lib()
    need = L.gcn_csr_transpose_workspace_bytes(A.n_rows, A.n_cols, A.nnz)
    w, wb = ws.args(need)
    s = A.struct()
    _check(L.gcn_csr_transpose(ctypes.byref(s), _ptr(t_indptr), _ptr(t_indices), _ptr(t_vals), w, wb,
                               _stream(stream)), "gcn_csr_transpose")


def gcn_csr_transpose_symmetric(A: DeviceCSR, ws: Workspace, t_vals=None, stream=None) -> DeviceCSR:
    """A^T of a symmetric-pattern A: A's indptr / indices with the transposed values."""
    if t_vals is None:
        t_vals = torch.empty(max(A.nnz, 1), dtype=torch.float32, device=A.indptr.device)[:A.nnz]
    L = lib()
    w, wb = ws.args(L.gcn_csr_transpose_symmetric_workspace_bytes(A.n_rows, A.nnz))
    s = A.struct()
    _check(L.gcn_csr_transpose_symmetric(ctypes.byref(s), _ptr(t_vals), w, wb, _stream(stream)),
           "gcn_csr_transpose_symmetric")
    return DeviceCSR(A.n_cols, A.n_rows, A.indptr, A.indices, t_vals[:A.nnz])


def gcn_aggregate(A: DeviceCSR, X: torch.Tensor, out: torch.Tensor, ws: Workspace, prec=GCN_F32, stream=None):
    _dev_f32(X, "X")
    _dev_f32(out, "out")
    L = lib()
    k = int(X.shape[1])
    need = L.gcn_aggregate_workspace_bytes(A.n_rows, A.n_cols, A.nnz, k, prec)
    w, wb = ws.args(need)
    s = A.struct()
    _check(L.gcn_aggregate(ctypes.byref(s), _ptr(X), k, _ld(X), _ptr(out), _ld(out), prec, w, wb,
                           _stream(stream)), "gcn_aggregate")
    return out


def gcn_aggregate_noalloc(A: DeviceCSR, X: torch.Tensor, out: torch.Tensor, prec=GCN_F32, stream=None):
    """gcn_aggregate with the library's own static scratch (no workspace)."""
    _dev_f32(X, "X")
    _dev_f32(out, "out")
    s = A.struct()
    _check(lib().gcn_aggregate_noalloc(ctypes.byref(s), _ptr(X), int(X.shape[1]), _ld(X), _ptr(out), _ld(out),
                                       prec, _stream(stream)), "gcn_aggregate_noalloc")
    return out


def gcn_layer_pick_order(f_in, h, need_dH) -> int:
    return lib().gcn_layer_pick_order(f_in, h, int(bool(need_dH)))


def gcn_layer_saved_bytes(n, f_in, h, order, prec=GCN_F32) -> int:
    return int(lib().gcn_layer_saved_bytes(n, f_in, h, order, prec))


def gcn_layer_workspace_bytes(n, nnz, f_in, h, order, prec=GCN_F32) -> int:
    return int(lib().gcn_layer_workspace_bytes(n, nnz, f_in, h, order, prec))


def gcn_layer_fwd(A: DeviceCSR, H, W_self, W_neigh, bias, Y, saved, order, ws: Workspace, prec=GCN_F32,
                  stream=None):
    for t, nm in ((H, "H"), (W_self, "W_self"), (W_neigh, "W_neigh"), (bias, "bias"), (Y, "Y")):
        _dev_f32(t, nm)
    L = lib()
    f_in, h = int(W_self.shape[0]), int(W_self.shape[1])
    need = L.gcn_layer_workspace_bytes(A.n_rows, A.nnz, f_in, h, order, prec)
    w, wb = ws.args(need)
    s = A.struct()
    sv = saved.numel() * saved.element_size() if saved is not None else 0
    _check(L.gcn_layer_fwd(ctypes.byref(s), _ptr(H), f_in, _ld(H), _ptr(W_self), _ptr(W_neigh), _ptr(bias), h,
                           _ptr(Y), _ld(Y), _ptr(saved), sv, order, prec, w, wb, _stream(stream)),
           "gcn_layer_fwd")
    return Y


def gcn_layer_bwd(A: DeviceCSR, AT: DeviceCSR, H, W_self, W_neigh, Y, saved, dY, dH, dW_self, dW_neigh, dbias,
                  order, ws: Workspace, prec=GCN_F32, stream=None):
    L = lib()
    f_in, h = int(W_self.shape[0]), int(W_self.shape[1])
    need = L.gcn_layer_workspace_bytes(A.n_rows, A.nnz, f_in, h, order, prec)
    w, wb = ws.args(need)
    s, st = A.struct(), AT.struct()
    sv = saved.numel() * saved.element_size() if saved is not None else 0
    _check(L.gcn_layer_bwd(ctypes.byref(s), ctypes.byref(st), _ptr(H), f_in, _ld(H), _ptr(W_self),
                           _ptr(W_neigh), h, _ptr(Y), _ld(Y), _ptr(saved), sv, _ptr(dY), _ld(dY), _ptr(dH),
                           _ld(dH) if dH is not None else 0, _ptr(dW_self), _ptr(dW_neigh), _ptr(dbias), order,
                           prec, w, wb, _stream(stream)), "gcn_layer_bwd")


def gcn_loss_grad(HL, W_pred, b_pred, kind, labels, targets, loss, dHL, dW_pred, db_pred, ws: Workspace,
                  prec=GCN_F32, stream=None):
    L = lib()
    n, f = int(HL.shape[0]), int(HL.shape[1])
    C = int(W_pred.shape[1])
    need = L.gcn_loss_workspace_bytes(n, f, C, prec)
    w, wb = ws.args(need)
    _check(L.gcn_loss_grad(_ptr(HL), n, f, _ld(HL), _ptr(W_pred), _ptr(b_pred), C, kind, _ptr(labels),
                           _ptr(targets), _ptr(loss), _ptr(dHL), _ld(dHL), _ptr(dW_pred), _ptr(db_pred), prec,
                           w, wb, _stream(stream)), "gcn_loss_grad")


class ModelStep:
    """gcn_model_step with the per-layer descriptors built once.

    layers: one dict per layer with the tensors W_self, W_neigh, bias, Y,
    saved (uint8 or None), dH (or None), dW_self, dW_neigh, dbias and the int
    order; head: None or a dict with W_pred, b_pred, kind, labels, targets,
    loss, dHL, dW_pred, db_pred.  Buffers may hold more rows than a call's
    subgraph (the row count is A's); they must stay alive and in place."""

    def __init__(self, layers, head=None, prec=GCN_F32):
        self.L = len(layers)
        self.prec = prec
        self.arr = (gcn_layer_args * self.L)()
        self._keep = [layers, head]
        for i, d in enumerate(layers):
            for nm in ("W_self", "W_neigh", "bias", "dW_self", "dW_neigh", "dbias"):
                _dev_f32(d[nm], nm)
            Y = d.get("Y")      # None: no float32 copy of the output (bfloat16 steps only)
            if Y is not None:
                _dev_f32(Y, "Y")
            f_in, h = int(d["W_self"].shape[0]), int(d["W_self"].shape[1])
            sv, dH = d.get("saved"), d.get("dH")
            self.arr[i] = gcn_layer_args(
                f_in, h, int(d["order"]), d["W_self"].data_ptr(), d["W_neigh"].data_ptr(), d["bias"].data_ptr(),
                None if Y is None else Y.data_ptr(), 2 * h if Y is None else _ld(Y),
                None if sv is None else sv.data_ptr(),
                0 if sv is None else sv.numel() * sv.element_size(), None if dH is None else dH.data_ptr(),
                0 if dH is None else _ld(dH), d["dW_self"].data_ptr(), d["dW_neigh"].data_ptr(),
                d["dbias"].data_ptr())
        if head is None:
            self.head = None
        else:
            p = lambda t: None if t is None else t.data_ptr()
            self.head = gcn_head_args(p(head["W_pred"]), p(head["b_pred"]), int(head["W_pred"].shape[1]),
                                      int(head["kind"]), p(head.get("labels")), p(head.get("targets")),
                                      p(head["loss"]), p(head["dHL"]), _ld(head["dHL"]), p(head["dW_pred"]),
                                      p(head["db_pred"]))
        self._head_ref = None if self.head is None else ctypes.byref(self.head)

    def set_loss(self, loss: torch.Tensor):
        """Where the next call writes its loss (a 1-element float32 device tensor)."""
        self.head.loss = loss.data_ptr()

    def set_labels(self, labels: Optional[torch.Tensor] = None, targets: Optional[torch.Tensor] = None):
        """Where the next call reads its labels (int32, CE) or targets
        (float32 n x C, BCE): the head of a subgraph in another input buffer."""
        self._labels_ref = (labels, targets)
        self.head.labels = None if labels is None else labels.data_ptr()
        self.head.targets = None if targets is None else targets.data_ptr()

    def workspace_bytes(self, n: int, nnz: int) -> int:
        return int(lib().gcn_model_workspace_bytes(n, nnz, self.L, self.arr, self._head_ref, self.prec))

    def __call__(self, A: DeviceCSR, AT: DeviceCSR, H0: torch.Tensor, ws: Workspace, dY=None, stream=None):
        L = lib()
        w, wb = ws.args(self.workspace_bytes(A.n_rows, A.nnz))
        s, st = A.struct(), AT.struct()
        _check(L.gcn_model_step(ctypes.byref(s), ctypes.byref(st), H0.data_ptr(), _ld(H0), self.L, self.arr,
                                self._head_ref, _ptr(dY), 0 if dY is None else _ld(dY), self.prec, w, wb,
                                _stream(stream)), "gcn_model_step")


def gcn_f32_to_bf16(x: torch.Tensor, stream=None) -> torch.Tensor:
    _dev_f32(x, "x")
    x = x.contiguous()
    y = torch.empty(x.shape, dtype=torch.int16, device=x.device)
    _check(lib().gcn_f32_to_bf16(_ptr(x), _ptr(y), x.numel(), _stream(stream)), "gcn_f32_to_bf16")
    return y


# ----------------------------------------------------------------- sampling
def gcn_sampler_plan(indptr_host, m: int, n: int, eta: float = 2.0, cap: int = 0,
                     seed: int = 0) -> gcn_sampler_params:
    """Dashboard / Index-Array sizes for G's row pointer (host array)."""
    import numpy as np
    ip = np.ascontiguousarray(indptr_host, dtype=np.int32)
    p = gcn_sampler_params()
    _check(lib().gcn_sampler_plan(int(ip.size - 1), ip.ctypes.data, m, n, float(eta), cap,
                                  seed & (2 ** 64 - 1), ctypes.byref(p)), "gcn_sampler_plan")
    return p


def gcn_frontier_sample(G: DeviceCSR, params: gcn_sampler_params, first_sampler: int, S: int,
                        vertices=None, counts=None, status=None, stream=None):
    """S frontier-sampling runs; returns (vertices [S x n], counts [S], status [S]) device tensors."""
    d = G.indptr.device
    n = params.n
    if vertices is None:
        vertices = torch.empty((max(S, 1), n), dtype=torch.int32, device=d)
    if counts is None:
        counts = torch.empty(max(S, 1), dtype=torch.int32, device=d)
    if status is None:
        status = torch.empty(max(S, 1), dtype=torch.int32, device=d)
    if vertices.dtype != torch.int32 or vertices.numel() < S * n or counts.numel() < S or status.numel() < S:
        raise ValueError("vertices [S x n], counts [S] and status [S] int32 tensors are needed")
    g = G.struct()
    _check(lib().gcn_frontier_sample(ctypes.byref(g), ctypes.byref(params), int(first_sampler), int(S),
                                     _ptr(vertices), _ptr(counts), _ptr(status), _stream(stream)),
           "gcn_frontier_sample")
    return vertices, counts, status


class InducedBatch:
    """Device outputs of gcn_induce_subgraphs for S vertex lists of length n."""

    def __init__(self, S: int, n: int, edge_capacity: int, device, with_transpose: bool = False):
        self.S, self.n = S, n
        d = torch.device(device)
        self.n_sub = torch.empty(max(S, 1), dtype=torch.int32, device=d)
        self.vsub = torch.empty((max(S, 1), max(n, 1)), dtype=torch.int32, device=d)
        self.indptr = torch.empty((max(S, 1), n + 1), dtype=torch.int32, device=d)
        self.edge_offsets = torch.empty(S + 1, dtype=torch.int64, device=d)
        self.edge_capacity = int(edge_capacity)
        self.indices = torch.empty(max(self.edge_capacity, 1), dtype=torch.int32, device=d)
        self.vals = torch.empty(max(self.edge_capacity, 1), dtype=torch.float32, device=d)
        self.vals_t = (torch.empty(max(self.edge_capacity, 1), dtype=torch.float32, device=d)
                       if with_transpose else None)
        self.status = torch.empty(1, dtype=torch.int32, device=d)

    def csr(self, s: int, n_sub: int, e0: int, e1: int) -> DeviceCSR:
        """Subgraph s as a DeviceCSR (host copies of n_sub / edge offsets given)."""
        return DeviceCSR(n_sub, n_sub, self.indptr[s, :n_sub + 1], self.indices[e0:e1], self.vals[e0:e1])

    def csr_t(self, s: int, n_sub: int, e0: int, e1: int) -> DeviceCSR:
        """The transposed aggregation matrix of subgraph s (symmetric G only)."""
        if self.vals_t is None:
            raise ValueError("built without the transposed values")
        return DeviceCSR(n_sub, n_sub, self.indptr[s, :n_sub + 1], self.indices[e0:e1], self.vals_t[e0:e1])


def gcn_induce_subgraphs(G: DeviceCSR, vertices: torch.Tensor, counts: torch.Tensor, out: InducedBatch,
                         ws: Workspace, stream=None):
    L = lib()
    S, n = out.S, out.n
    need = L.gcn_induce_workspace_bytes(G.n_rows, n, S)
    w, wb = ws.args(need)
    g = G.struct()
    _check(L.gcn_induce_subgraphs(ctypes.byref(g), S, n, _ptr(vertices), _ptr(counts), _ptr(out.n_sub),
                                  _ptr(out.vsub), _ptr(out.indptr), _ptr(out.edge_offsets), _ptr(out.indices),
                                  _ptr(out.vals), _ptr(out.vals_t), out.edge_capacity, _ptr(out.status), w, wb,
                                  _stream(stream)),
           "gcn_induce_subgraphs")
    return out


def gcn_csr_pattern_symmetric_host(indptr, indices) -> bool:
    import numpy as np
    ip = np.ascontiguousarray(indptr, dtype=np.int32)
    ix = np.ascontiguousarray(indices, dtype=np.int32)
    r = lib().gcn_csr_pattern_symmetric_host(int(ip.size - 1), ip.ctypes.data, ix.ctypes.data if ix.size else None)
    if r < 0:
        _check(r, "gcn_csr_pattern_symmetric_host")
    return bool(r)


def gcn_gather_rows(X: torch.Tensor, rows: torch.Tensor, count: int, out: torch.Tensor, stream=None):
    """out[:count] = X[rows[:count]] for 4-byte tensors (float32 rows or int32 labels)."""
    if X.element_size() != 4 or out.element_size() != 4 or rows.dtype != torch.int32:
        raise TypeError("4-byte X / out and int32 rows are needed")
    X2 = X if X.dim() == 2 else X.view(-1, 1)
    o2 = out if out.dim() == 2 else out.view(-1, 1)
    width = int(X2.shape[1])
    if int(o2.shape[1]) != width or o2.shape[0] < count or rows.numel() < count:
        raise ValueError("shape mismatch")
    _check(lib().gcn_gather_rows(_ptr(X2), int(X2.shape[0]), width, _ld(X2), _ptr(rows), int(count), _ptr(o2),
                                 _ld(o2), _stream(stream)), "gcn_gather_rows")
    return out


# ---------------------------------------------------------------- optimiser
def gcn_adam_update(params, grads, m, v, lr: float, step: int, beta1: float = 0.9, beta2: float = 0.999,
                    eps: float = 1e-8, stream=None):
    """One Adam step over flat float32 tensors of equal length, in place."""
    for t, nm in ((params, "params"), (grads, "grads"), (m, "m"), (v, "v")):
        _dev_f32(t, nm)
        if not t.is_contiguous() or t.numel() != params.numel():
            raise ValueError(f"{nm} must be contiguous with as many elements as params")
    _check(lib().gcn_adam_update(_ptr(params), _ptr(grads), _ptr(m), _ptr(v), params.numel(), lr, beta1, beta2,
                                 eps, int(step), _stream(stream)), "gcn_adam_update")


# ---------------------------------------------------------------- profiling
def gcn_profile_enable(on: bool):
    _check(lib().gcn_profile_enable(int(bool(on))), "gcn_profile_enable")


def gcn_profile_reset():
    _check(lib().gcn_profile_reset(), "gcn_profile_reset")


def gcn_profile_read_all():
    """{class name: (ms, launches, flops, bytes)} since the last reset."""
    L = lib()
    out = {}
    for c in range(L.gcn_profile_class_count()):
        ms, n = ctypes.c_double(), ctypes.c_int64()
        fl, by = ctypes.c_double(), ctypes.c_double()
        _check(L.gcn_profile_read(c, ctypes.byref(ms), ctypes.byref(n), ctypes.byref(fl), ctypes.byref(by)),
               "gcn_profile_read")
        out[L.gcn_profile_class_name(c).decode()] = (ms.value, n.value, fl.value, by.value)
    return out


# ------------------------------------------------------------ peak probes
def gcn_peak_stream_read(x: torch.Tensor, sink: torch.Tensor, blocks: int, stream=None):
    """Enqueue one streaming read of every element of the float32 tensor x."""
    _dev_f32(x, "x")
    _dev_f32(sink, "sink")
    if sink.numel() < blocks * 256:
        raise ValueError("sink needs blocks * 256 floats")
    _check(lib().gcn_peak_stream_read(_ptr(x), x.numel(), _ptr(sink), blocks, _stream(stream)),
           "gcn_peak_stream_read")


def gcn_peak_mfma(prec: int, blocks: int, iters: int, sink: torch.Tensor, stream=None) -> float:
    """Enqueue the matrix-core probe; returns the floating-point operations it issues."""
    _dev_f32(sink, "sink")
    if sink.numel() < blocks * 256:
        raise ValueError("sink needs blocks * 256 floats")
    fl = ctypes.c_double(0.0)
    _check(lib().gcn_peak_mfma(prec, blocks, iters, _ptr(sink), ctypes.byref(fl), _stream(stream)),
           "gcn_peak_mfma")
    return fl.value


def gcn_peak_gather(X: torch.Tensor, row_bytes: int, idx: torch.Tensor, sink: torch.Tensor, blocks: int,
                    stream=None):
    """Enqueue the gather of the first row_bytes of rows idx of the 2-D tensor X
    (one row per index, rows X.stride(0) elements apart)."""
    if X.dim() != 2 or X.stride(1) != 1 or idx.dtype != torch.int32 or sink.dtype != torch.float32 \
            or sink.numel() < blocks * 256 or row_bytes > X.shape[1] * X.element_size():
        raise TypeError("a row-major 2-D X wide enough, int32 indices and a float32 sink of blocks*256")
    _check(lib().gcn_peak_gather(_ptr(X), X.shape[0], int(row_bytes), X.stride(0) * X.element_size(), _ptr(idx),
                                 idx.numel(), _ptr(sink), int(blocks), _stream(stream)), "gcn_peak_gather")


def gcn_peak_chase(next_idx: torch.Tensor, steps: int, chains: int, sink: torch.Tensor, stream=None):
    """Enqueue `chains` dependent-load walks of `steps` hops over next_idx (int32)."""
    if next_idx.dtype != torch.int32 or sink.dtype != torch.int32 or sink.numel() < chains:
        raise TypeError("int32 next_idx and an int32 sink of >= chains elements are needed")
    _check(lib().gcn_peak_chase(_ptr(next_idx), next_idx.numel(), int(steps), int(chains), _ptr(sink),
                                _stream(stream)), "gcn_peak_chase")
