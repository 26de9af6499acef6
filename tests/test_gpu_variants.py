"""The scope table's variants on the GPU: uint16 column indices (half the
index bytes; the paper's subgraphs use 16-bit indices, Sec. V-B) and
self-loop aggregation (a self-connection on every vertex, Sec. V-B), each
against the oracle and, for the index width, bit for bit against int32."""
import numpy as np
import pytest
import torch

import oracle
from paper_1810_11899_amd import binding as B
from paper_1810_11899_amd import synth
from paper_1810_11899_amd.runner import StepRunner

from gpu_util import dev, require_gpu
from test_gpu_layer import compare_bf16_chain, compare_step

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def _bits(results):
    out = {}
    for k, v in results.items():
        if isinstance(v, list):
            out[k] = [None if x is None else x.view(np.uint32) if x.dtype == np.float32 else x for x in v]
        elif isinstance(v, np.ndarray):
            out[k] = v.view(np.uint32) if v.dtype == np.float32 else v
        else:
            out[k] = v
    return out


def _same(a, b):
    a, b = _bits(a), _bits(b)
    for k in a:
        x, y = a[k], b[k]
        if isinstance(x, list):
            for i, (p, q) in enumerate(zip(x, y)):
                assert (p is None and q is None) or np.array_equal(p, q), (k, i)
        elif isinstance(x, np.ndarray):
            assert np.array_equal(x, y), k
        else:
            assert x == y, k


@pytest.mark.parametrize("case", ["cfg1-f32", "cfg2-f32", "cfg1-bf16", "directed-f32"])
def test_uint16_indices_step_bitwise_equal_to_int32(case):
    """The whole model step with A's indices as uint16 equals the int32 run
    bit for bit (integer handling is exact: same kernels, same order), and
    matches the oracle.  'directed' has a non-symmetric pattern, so A^T comes
    from the general transpose (int32 output) while A stays uint16."""
    if case.startswith("cfg"):
        wl = synth.config(int(case[3]))
        kw = {}
    else:
        wl = synth.custom(6000, "rmat", 12, [(64, 48), (96, 40)], head="ce", classes=17, seed=3)
        g = wl.graph
        rows = np.repeat(np.arange(g.n), g.degrees())
        keep = (rows + g.indices) % 3 != 0               # drop a third of the entries: directed
        import dataclasses
        wl = dataclasses.replace(wl, graph=synth.csr_from_pairs(g.n, rows[keep], g.indices[keep]))
        kw = {"first_layer_dH": True}
    prec = B.GCN_BF16 if case.endswith("bf16") else B.GCN_F32
    print(f"uint16 vs int32 indices: {case} n={wl.n} nnz={wl.graph.nnz}", flush=True)
    r32 = StepRunner(wl, prec=prec, **kw)
    r16 = StepRunner(wl, prec=prec, index_bits=16, **kw)
    assert r16.A.index_bits == 16 and r16.csr_bytes() < r32.csr_bytes()
    r32.step()
    r16.step()
    torch.cuda.synchronize()
    a, b = r32.results(), r16.results()
    _same(a, b)
    if prec == B.GCN_F32:
        compare_step(b, oracle.step(wl, envelope=True, **kw))
    else:
        compare_bf16_chain(r16, wl)


def test_uint16_indices_reach_the_last_vertex():
    """n = 65,536: indices up to 65,535 (the top of the uint16 range) gather
    the right rows, bit for bit, through a permutation graph (every row one
    entry of weight 1.0: A X is a row permutation of X, exactly) in both
    precisions and through the no-allocation entry point."""
    n, k = 65536, 48
    rng = np.random.default_rng(5)
    g = synth.permutation_graph(n, rng)
    assert g.indices.max() == n - 1
    X = rng.standard_normal((n, k)).astype(np.float32)
    A16 = B.DeviceCSR.from_host(n, n, g.indptr, g.indices, g.vals, index_bits=16)
    ws = B.Workspace("cuda")
    out = torch.empty((n, k), device="cuda")
    B.gcn_aggregate(A16, dev(X), out, ws)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().view(np.uint32), X[g.indices].view(np.uint32))
    B.gcn_aggregate_noalloc(A16, dev(X), out)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().view(np.uint32), X[g.indices].view(np.uint32))
    from oracle import bf16 as obf16
    B.gcn_aggregate(A16, dev(X), out, ws, B.GCN_BF16)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().view(np.uint32), obf16.round_bf16(X[g.indices]).view(np.uint32))


def test_uint16_transposes_and_validation():
    """The general transpose (int32 output) and the symmetric-pattern values
    from a uint16 A equal those from an int32 A bit for bit; the device
    validator reads uint16 indices (an index past n_cols and an unsorted row
    are found)."""
    wl = synth.custom(30000, "rmat", 14, [(4, 4)], seed=7)
    g = wl.graph
    ws = B.Workspace("cuda")
    A32 = B.DeviceCSR.from_host(g.n, g.n, g.indptr, g.indices, g.vals)
    A16 = B.DeviceCSR.from_host(g.n, g.n, g.indptr, g.indices, g.vals, index_bits=16)
    T32, T16 = B.gcn_csr_transpose(A32, ws), B.gcn_csr_transpose(A16, ws)
    S32, S16 = B.gcn_csr_transpose_symmetric(A32, ws), B.gcn_csr_transpose_symmetric(A16, ws)
    torch.cuda.synchronize()
    for x, y in ((T32.indptr, T16.indptr), (T32.indices, T16.indices), (T32.vals, T16.vals),
                 (S32.vals, S16.vals)):
        assert torch.equal(x, y)
    ti, tj, tv = oracle.csr_transpose(g.n, g.n, g.indptr, g.indices, g.vals)
    assert np.array_equal(T16.indices.cpu().numpy(), tj)
    st = B.gcn_csr_validate(A16)
    torch.cuda.synchronize()
    assert st.cpu().tolist() == [0, 0]
    bad = g.indices.copy()
    r = int(np.flatnonzero(np.diff(g.indptr) >= 2)[0])
    bad[g.indptr[r]], bad[g.indptr[r] + 1] = bad[g.indptr[r] + 1], bad[g.indptr[r]]
    Ab = B.DeviceCSR.from_host(g.n, g.n, g.indptr, bad, g.vals, index_bits=16)
    st = B.gcn_csr_validate(Ab)
    torch.cuda.synchronize()
    assert st.cpu().tolist() == [4, r]
    Ac = B.DeviceCSR.from_host(g.n, 20000, g.indptr, g.indices, g.vals, index_bits=16)
    st = B.gcn_csr_validate(Ac)
    torch.cuda.synchronize()
    row_of_big = int(np.searchsorted(g.indptr, np.flatnonzero(g.indices >= 20000)[0], side="right") - 1)
    assert st.cpu().tolist() == [3, row_of_big]


@pytest.mark.parametrize("prec", [B.GCN_F32, B.GCN_BF16])
@pytest.mark.parametrize("cfg", [1, 2])
def test_self_loop_aggregation_step(prec, cfg):
    """The model step on the workload's graph with a self-connection on every
    vertex (mean over the row, the vertex included): the symmetric-pattern
    transpose with diagonal entries, then every output against the oracle."""
    wl = synth.config(cfg, self_loops=True)
    assert wl.graph.nnz == synth.config(cfg).graph.nnz + wl.n
    r = StepRunner(wl, prec=prec)
    assert r.symmetric
    print(f"self-loop step: workload {cfg} prec={prec}", flush=True)
    r.step()
    torch.cuda.synchronize()
    if prec == B.GCN_F32:
        compare_step(r.results(), oracle.step(wl, envelope=True))
    else:
        compare_bf16_chain(r, wl)


def test_measured_order_choice():
    """orders="tuned": every grouping combination is timed on the workload and
    the fastest is kept; the tuned step still matches the oracle."""
    wl = synth.config(1)
    r = StepRunner(wl, orders="tuned")
    t = r.order_timings
    assert len(t) == 4 and tuple(r.orders) == min(t, key=t.get)
    assert all(v > 0 for v in t.values())
    print("order step times (ms):", t, "chosen:", r.orders, flush=True)
    r.step()
    torch.cuda.synchronize()
    compare_step(r.results(), oracle.step(wl, envelope=True))
