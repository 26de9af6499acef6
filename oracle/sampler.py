"""CPU oracle of the subgraph sampler and of GCN construction on a sample.

TEST INFRASTRUCTURE ONLY, like the rest of this package: only the tests, the
smoke check and the benchmark's CPU-baseline leg may use it.

  frontier_sample  frontier sampling with the Dashboard (Sec. IV-A, Alg. 2;
                   Sec. IV-B/IV-C, Alg. 3 and Alg. 4), sequential, in plain C
                   (``gcnref_sampler.c``, whose header lists the readings taken)
  philox4x64       the counter-based generator both sides draw from
  induce           the subgraph of G induced by the sampled vertices (last step
                   of Alg. 2 and Alg. 3) as a mean-normalised CSR: the plain
                   definition, with numpy set operations
  gather_rows      the feature rows of the sampled vertices, H^(0)[V_sub]
                   (GCN construction on the subgraph, Alg. 1 / Alg. 5)
"""
from __future__ import annotations

import ctypes
from typing import Tuple

import numpy as np

from . import gcnref

STATUS = {0: "ok", 1: "exhausted", 2: "overflow", 3: "probe_limit", 4: "root_limit", -1: "einval"}


def _lib():
    lib = gcnref._load()
    if not getattr(lib, "_sampler_ready", False):
        u64p = ctypes.POINTER(ctypes.c_uint64)
        lib.gcnref_philox4x64.argtypes = [u64p, u64p, u64p]
        lib.gcnref_philox4x64.restype = None
        i64, i32, p = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
        lib.gcnref_frontier_sample.argtypes = [i64, p, p, i32, i32, i64, i32, i32, i32,
                                               ctypes.c_uint64, ctypes.c_uint64, p, ctypes.POINTER(i32)]
        lib.gcnref_frontier_sample.restype = ctypes.c_int
        lib._sampler_ready = True
    return lib


def philox4x64(counter, key) -> np.ndarray:
    """One block of Philox4x64-10: four 64-bit words for a 256-bit counter and a
    128-bit key (each given as a sequence of 64-bit words, low word first)."""
    c = (ctypes.c_uint64 * 4)(*[int(x) & (2 ** 64 - 1) for x in counter])
    k = (ctypes.c_uint64 * 2)(*[int(x) & (2 ** 64 - 1) for x in key])
    o = (ctypes.c_uint64 * 4)()
    _lib().gcnref_philox4x64(c, k, o)
    return np.array(list(o), dtype=np.uint64)


def frontier_sample(indptr, indices, m: int, n: int, db_cap: int, ia_cap: int, cap: int = 0,
                    p: int = 64, seed: int = 0, sampler_id: int = 0) -> Tuple[np.ndarray, str]:
    """Vertex list of one frontier-sampling run on the graph G = (indptr, indices).

    Returns (vertices, status): the m roots followed by the vertex added at each
    of the following steps (length n unless the status is not "ok"), and the
    status name (see ``gcnref_sampler.c``).  db_cap / ia_cap are the Dashboard
    and Index-Array capacities, cap the per-vertex entry limit (0 = none), p the
    number of probes per round.
    """
    indptr = np.ascontiguousarray(indptr, dtype=np.int32)
    indices = np.ascontiguousarray(indices, dtype=np.int32)
    nV = indptr.shape[0] - 1
    out = np.zeros(max(n, 1), dtype=np.int32)
    cnt = ctypes.c_int32(0)
    st = _lib().gcnref_frontier_sample(nV, indptr.ctypes.data, indices.ctypes.data, m, n, db_cap, ia_cap, cap,
                                       p, seed & (2 ** 64 - 1), sampler_id & (2 ** 64 - 1), out.ctypes.data,
                                       ctypes.byref(cnt))
    return out[:cnt.value].copy(), STATUS[st]


def induce(indptr, indices, vertices):
    """Subgraph of G induced by the set of `vertices` (duplicates ignored).

    Returns (vsub, sub_indptr, sub_indices, sub_vals): vsub = the distinct
    vertices in ascending order (local id = position); row i of the CSR lists
    the local ids of the neighbours of vsub[i] that are in the set, in
    ascending order; vals are the mean weights float32(1) / float32(row
    length), the row normalisation of Sec. II.
    """
    indptr = np.asarray(indptr, dtype=np.int64)
    indices = np.asarray(indices, dtype=np.int64)
    vsub = np.unique(np.asarray(vertices, dtype=np.int64))
    rows, lens = [], []
    for u in vsub:
        nb = indices[indptr[u]:indptr[u + 1]]
        keep = nb[np.isin(nb, vsub)]
        loc = np.searchsorted(vsub, keep)
        rows.append(np.sort(loc))
        lens.append(loc.size)
    ns = vsub.size
    sub_indptr = np.zeros(ns + 1, dtype=np.int64)
    np.cumsum(np.asarray(lens, dtype=np.int64), out=sub_indptr[1:])
    sub_indices = np.concatenate(rows) if rows else np.zeros(0, np.int64)
    lens = np.asarray(lens, dtype=np.int64)
    per_row = np.zeros(ns, dtype=np.float32)
    nz = lens > 0
    per_row[nz] = np.float32(1.0) / lens[nz].astype(np.float32)
    sub_vals = np.repeat(per_row, lens)
    return (vsub.astype(np.int32), sub_indptr.astype(np.int32), sub_indices.astype(np.int32),
            sub_vals.astype(np.float32))


def gather_rows(X, rows) -> np.ndarray:
    """X[rows]: the input features of the sampled vertices, copied as they are."""
    return np.asarray(X)[np.asarray(rows, dtype=np.int64)]
