"""CPU oracle for the graph-sampling GCN layer of arXiv 1810.11899.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package; the HIP library never does, and this
package imports nothing from it.

It computes, plainly and slowly, in float64 from the float32 inputs, what the
hot path computes (the layer of Sec. II and Alg. 1, forward and backward, and
the loss head of Alg. 1).  The method reaches exactly (up to rounding order)
the plain matrix expressions below, so the oracle *is* those expressions:
the feature-partitioned propagation of Alg. 6 computes the same sums in another
order.  Library routines serve as steps: numpy's float64 matmul for the dense
products (the paper uses a BLAS ``dgemm``, Sec. V-A / VI-C-4) and numpy's stable
sort for the transpose; the sparse aggregation is a plain C loop
(``gcnref_aggregate.c``).

Readings of points the paper leaves open:
  * concat order self-first: ``[H W_self || A H W_neigh]``;
  * no self-loops are added to A (the self term is W_self's);
  * A is row-normalised (the mean of Sec. II): ``A[i, j] = 1/deg(i)``;
  * sigma = ReLU on every layer, derivative 0 at 0;
  * a bias of width 2h is added after the concat, before the ReLU;
  * PREDICT is linear, ``X = H_L W_pred + b_pred``;
  * LOSS is the mean softmax cross-entropy over all n nodes, or the mean sigmoid
    binary cross-entropy over all n*C entries.

ReLU kinks.  The derivative of max(z, 0) switches at z = 0, so an output
computed in float32 may take the other branch wherever z lies within float32
rounding of zero; both branches are then correct results of a float32
computation.  With ``envelope=True`` the oracle marks every pre-activation with
|z| < C_AMB * u32 * (the sum of the magnitudes of its terms) as ambiguous and
propagates, with absolute values through the backward pass, a per-entry bound
on how far any choice of those branches can move each gradient.  Comparisons
allow that bound on top of the float32 tolerance; everywhere else they are
strict.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRCS = [os.path.join(_HERE, "gcnref_aggregate.c"), os.path.join(_HERE, "gcnref_sampler.c")]
_LIB_PATH = os.path.join(_HERE, "libgcnref.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the C part of the oracle (plain gcc, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-o", tmp] + _SRCS)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        lib = ctypes.CDLL(_LIB_PATH)
        i64, p = ctypes.c_int64, ctypes.c_void_p
        lib.gcnref_aggregate.argtypes = [i64, i64, p, p, p, p, i64, p, i64]
        lib.gcnref_aggregate.restype = None
        lib.gcnref_num_threads.restype = ctypes.c_int
        lib.gcnref_set_num_threads.argtypes = [ctypes.c_int]
        lib.gcnref_set_num_threads.restype = None
        _lib = lib
    return _lib


def num_threads() -> int:
    return int(_load().gcnref_num_threads())


def set_num_threads(n: int) -> None:
    """OpenMP threads of the C aggregation (for timing a serial run)."""
    _load().gcnref_set_num_threads(int(n))


U32 = 2.0 ** -24      # unit roundoff of float32
C_AMB = 16.0          # safety factor on u32 * sum|terms| (covers upstream float32 error too)


def f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


# --------------------------------------------------------------------------
# sparse pieces
# --------------------------------------------------------------------------
def aggregate(indptr, indices, vals, X) -> np.ndarray:
    """out = A X for CSR A (row = destination), Sec. II step 1, in float64."""
    indptr = np.ascontiguousarray(indptr, dtype=np.int32)
    indices = np.ascontiguousarray(indices, dtype=np.int32)
    v = f64(vals)
    X = f64(X)
    n_rows = indptr.shape[0] - 1
    k = X.shape[1] if X.ndim == 2 else 0
    out = np.empty((n_rows, k), dtype=np.float64)
    if n_rows and k:
        _load().gcnref_aggregate(n_rows, k, indptr.ctypes.data, indices.ctypes.data,
                                 v.ctypes.data, X.ctypes.data, k, out.ctypes.data, k)
    return out


def csr_transpose(n_rows: int, n_cols: int, indptr, indices, vals):
    """CSR of A^T (the transpose appearing in Alg. 1's propagation step).

    Row j of A^T lists the rows i of A holding column j, i ascending (entries
    with equal (i, j) keep their order), values carried bit for bit.  Done as a
    stable sort of the entries, which are already in row-major order, by column.
    """
    indptr = np.asarray(indptr, dtype=np.int64)
    indices = np.asarray(indices, dtype=np.int64)
    rows = np.repeat(np.arange(n_rows, dtype=np.int64), np.diff(indptr))
    order = np.argsort(indices, kind="stable")
    t_indices = rows[order].astype(np.int32)
    t_vals = np.asarray(vals)[order]
    counts = np.bincount(indices, minlength=n_cols) if indices.size else np.zeros(n_cols, np.int64)
    t_indptr = np.zeros(n_cols + 1, dtype=np.int64)
    np.cumsum(counts, out=t_indptr[1:])
    return t_indptr.astype(np.int32), t_indices, t_vals


# --------------------------------------------------------------------------
# one layer
# --------------------------------------------------------------------------
@dataclass
class LayerCache:
    H: np.ndarray     # layer input, float64
    AGG: np.ndarray   # A H
    Z: np.ndarray     # pre-activation [S || N] + b
    amb: Optional[np.ndarray] = None     # |Z| within float32 rounding of 0
    absAGG: Optional[np.ndarray] = None  # |A| |H|


def layer_fwd(g, H, W_self, W_neigh, bias, ambiguity: bool = False):
    """Forward of one layer (Sec. II; Alg. 1 forward loop), float64.

    S = H W_self, N = (A H) W_neigh, Z = [S || N] + b, Y = max(Z, 0).
    With ``ambiguity`` the cache also marks the ReLU kinks that float32 cannot
    resolve: |Z| < C_AMB u32 (|b| + |H| |W_self|) on the self half and
    |Z| < C_AMB u32 (|b| + |A| |H| |W_neigh|) on the neighbour half.
    """
    H = f64(H)
    AGG = aggregate(g.indptr, g.indices, g.vals, H)
    S = H @ f64(W_self)
    N = AGG @ f64(W_neigh)
    b = f64(bias)
    Z = np.concatenate([S, N], axis=1) + b[None, :]
    Y = np.maximum(Z, 0.0)
    cache = LayerCache(H, AGG, Z)
    if ambiguity:
        absAGG = aggregate(g.indptr, g.indices, np.abs(f64(g.vals)), np.abs(H))
        mag = np.concatenate([np.abs(H) @ np.abs(f64(W_self)), absAGG @ np.abs(f64(W_neigh))], axis=1)
        mag += np.abs(b)[None, :]
        cache.amb = np.abs(Z) < C_AMB * U32 * mag
        cache.absAGG = absAGG
    return Y, cache


def layer_bwd(gT, cache: LayerCache, W_self, W_neigh, dY, need_dH: bool, mask=None):
    """Backward of one layer: the same two kernels, transposed (Sec. III-B).

    dZ = dY * [Z > 0]; db = sum_i dZ; dW_self = H^T dZ_s; dW_neigh = (A H)^T dZ_n;
    dH = dZ_s W_self^T + A^T (dZ_n W_neigh^T).  ``gT`` is the CSR of A^T.
    ``mask`` overrides [Z > 0] (used to enumerate kink choices).
    """
    Ws, Wn = f64(W_self), f64(W_neigh)
    h = Ws.shape[1]
    m = (cache.Z > 0.0) if mask is None else mask
    dZ = f64(dY) * m
    db = dZ.sum(axis=0)
    dZs, dZn = dZ[:, :h], dZ[:, h:]
    dWs = cache.H.T @ dZs
    dWn = cache.AGG.T @ dZn
    dH = None
    if need_dH:
        dH = dZs @ Ws.T + aggregate(gT.indptr, gT.indices, gT.vals, dZn @ Wn.T)
    return dWs, dWn, db, dH


def layer_bwd_envelope(gT, cache: LayerCache, W_self, W_neigh, dY, E_dY, need_dH: bool):
    """Bound on how far the layer's gradients can move over the ReLU kinks.

    An ambiguous entry of dZ may be 0 or dY (plus the upstream bound E_dY);
    any other entry is dY * [Z > 0] up to E_dY.  The bound is carried through
    the same products with absolute values: |H|^T, (|A||H|)^T, |W|^T, |A^T|.
    """
    Ws, Wn = np.abs(f64(W_self)), np.abs(f64(W_neigh))
    h = Ws.shape[1]
    E_dY = np.zeros_like(cache.Z) if E_dY is None else E_dY
    E = np.where(cache.amb, np.abs(f64(dY)) + E_dY, (cache.Z > 0.0) * E_dY)
    Es, En = E[:, :h], E[:, h:]
    E_db = E.sum(axis=0)
    E_dWs = np.abs(cache.H).T @ Es
    E_dWn = cache.absAGG.T @ En
    E_dH = None
    if need_dH:
        E_dH = Es @ Ws.T + aggregate(gT.indptr, gT.indices, np.abs(f64(gT.vals)), En @ Wn.T)
    return E_dWs, E_dWn, E_db, E_dH


# --------------------------------------------------------------------------
# PREDICT + LOSS (Alg. 1) and their gradient
# --------------------------------------------------------------------------
def loss_grad(kind: str, HL, W_pred, b_pred, labels=None, targets=None):
    """Linear PREDICT, mean loss, and the gradients of the loss.

    ce : loss = mean_i (logsumexp(X_i) - X[i, y_i]);  G = (softmax(X) - onehot(y)) / n
    bce: loss = mean_{i,c} (max(x,0) - x t + log(1 + exp(-|x|)));  G = (sigmoid(X) - t) / (n C)
    then dW_pred = HL^T G, db_pred = sum_i G, dHL = G W_pred^T.
    """
    HL, Wp = f64(HL), f64(W_pred)
    X = HL @ Wp + f64(b_pred)[None, :]
    n, C = X.shape
    if kind == "ce":
        lab = np.asarray(labels, dtype=np.int64)
        m = X.max(axis=1, keepdims=True)
        lse = m[:, 0] + np.log(np.exp(X - m).sum(axis=1))
        loss = float(np.mean(lse - X[np.arange(n), lab])) if n else 0.0
        G = np.exp(X - lse[:, None])
        G[np.arange(n), lab] -= 1.0
        G /= max(n, 1)
    elif kind == "bce":
        t = f64(targets)
        loss = float(np.mean(np.maximum(X, 0.0) - X * t + np.log1p(np.exp(-np.abs(X))))) if n else 0.0
        G = (1.0 / (1.0 + np.exp(-X)) - t) / max(n * C, 1)
    else:
        raise ValueError(kind)
    return loss, HL.T @ G, G.sum(axis=0), G @ Wp.T, X


# --------------------------------------------------------------------------
# a whole fwd+bwd step on one subgraph
# --------------------------------------------------------------------------
@dataclass
class StepResult:
    Y: List[np.ndarray]
    dW_self: List[np.ndarray]
    dW_neigh: List[np.ndarray]
    db: List[np.ndarray]
    dH: List[Optional[np.ndarray]]
    loss: Optional[float] = None
    dW_pred: Optional[np.ndarray] = None
    db_pred: Optional[np.ndarray] = None
    dHL: Optional[np.ndarray] = None
    t_indptr: Optional[np.ndarray] = None
    t_indices: Optional[np.ndarray] = None
    t_vals: Optional[np.ndarray] = None
    # per-entry kink envelopes of the gradients (envelope=True), same shapes
    E_dW_self: Optional[List[np.ndarray]] = None
    E_dW_neigh: Optional[List[np.ndarray]] = None
    E_db: Optional[List[np.ndarray]] = None
    E_dH: Optional[List[Optional[np.ndarray]]] = None
    ambiguous: Optional[List[int]] = None


class _CSR:
    def __init__(self, indptr, indices, vals):
        self.indptr, self.indices, self.vals = indptr, indices, vals


def step(wl, first_layer_dH: Optional[bool] = None, envelope: bool = False, masks=None) -> StepResult:
    """Forward through every layer, PREDICT/LOSS (or the given dY), backward.

    The layer-1 input gradient is computed only for single-layer workloads
    unless ``first_layer_dH`` says otherwise (training never needs it).
    ``envelope`` adds the ReLU-kink bounds of every gradient.

    ``masks`` (one 0/1 array of Z's shape per layer) fixes the branch of every
    activation: layer l outputs Y = Z * m_l and passes dZ = dY * m_l back,
    the network in which each ReLU is replaced by the gate its branch choice
    gives (exactly the ReLU network where m_l = [Z_l > 0]).  A computation
    whose rounding decides some near-zero branches the other way computes
    this network for its own choices; comparing on the same choices leaves
    only the arithmetic to compare.
    """
    g = wl.graph
    L = len(wl.layers)
    if first_layer_dH is None:
        first_layer_dH = (L == 1)
    t_indptr, t_indices, t_vals = csr_transpose(g.n, g.n, g.indptr, g.indices, g.vals)
    gT = _CSR(t_indptr, t_indices, t_vals)
    H = wl.H
    caches, Ys = [], []
    if masks is not None and (envelope or len(masks) != L):
        raise ValueError("masks: one per layer, and not together with the kink envelope")
    for li, lay in enumerate(wl.layers):
        Y, cache = layer_fwd(g, H, lay.W_self, lay.W_neigh, lay.bias, ambiguity=envelope)
        if masks is not None:
            Y = cache.Z * np.asarray(masks[li], dtype=np.float64)
        caches.append(cache)
        Ys.append(Y)
        H = Y
    res = StepResult(Ys, [None] * L, [None] * L, [None] * L, [None] * L,
                     t_indptr=t_indptr, t_indices=t_indices, t_vals=t_vals)
    if wl.spec.head is None:
        dY = f64(wl.dY)
    else:
        loss, dWp, dbp, dHL, _ = loss_grad(wl.spec.head, Ys[-1], wl.W_pred, wl.b_pred,
                                           labels=wl.labels, targets=wl.targets)
        res.loss, res.dW_pred, res.db_pred, res.dHL = loss, dWp, dbp, dHL
        dY = dHL
    if envelope:
        res.E_dW_self, res.E_dW_neigh, res.E_db, res.E_dH = [None] * L, [None] * L, [None] * L, [None] * L
        res.ambiguous = [int(c.amb.sum()) for c in caches]
    E_dY = None
    for li in range(L - 1, -1, -1):
        lay = wl.layers[li]
        need = li > 0 or first_layer_dH
        dWs, dWn, db, dH = layer_bwd(gT, caches[li], lay.W_self, lay.W_neigh, dY, need,
                                     mask=None if masks is None else np.asarray(masks[li], dtype=np.float64))
        res.dW_self[li], res.dW_neigh[li], res.db[li], res.dH[li] = dWs, dWn, db, dH
        if envelope:
            e = layer_bwd_envelope(gT, caches[li], lay.W_self, lay.W_neigh, dY, E_dY, need)
            res.E_dW_self[li], res.E_dW_neigh[li], res.E_db[li], res.E_dH[li] = e
            E_dY = e[3]
        dY = dH
    return res
