"""The seeded input generator: determinism and well-formed mean-normalised CSR."""
from fractions import Fraction

import numpy as np
import pytest

from paper_1810_11899_amd import synth


def _check_csr(g: synth.Graph, symmetric=True):
    n = g.n
    ip = g.indptr.astype(np.int64)
    assert g.indptr.dtype == np.int32 and g.indices.dtype == np.int32 and g.vals.dtype == np.float32
    assert ip[0] == 0 and ip[-1] == g.nnz and np.all(np.diff(ip) >= 0)
    assert g.nnz == 0 or (g.indices.min() >= 0 and g.indices.max() < n)
    rows = np.repeat(np.arange(n), np.diff(ip))
    # strictly ascending within each row: no duplicates, sorted
    same_row = rows[1:] == rows[:-1]
    assert np.all(g.indices[1:][same_row] > g.indices[:-1][same_row])
    assert not np.any(rows == g.indices), "self-loop"
    if symmetric:
        a = set(zip(rows.tolist(), g.indices.tolist()))
        b = set(zip(g.indices.tolist(), rows.tolist()))
        assert a == b


@pytest.mark.parametrize("cfg", [0, 1])
def test_config_graph_well_formed(cfg):
    wl = synth.config(cfg)
    spec = synth.WORKLOADS[cfg]
    _check_csr(wl.graph)
    assert wl.graph.nnz == spec.n * spec.d
    assert wl.H.shape == (spec.n, spec.layers[0][0]) and wl.H.dtype == np.float32


def test_mean_values_are_correctly_rounded_reciprocals():
    wl = synth.custom(500, "rmat", 12, [(8, 4)])
    deg = wl.graph.degrees()
    rows = np.repeat(np.arange(wl.n), deg)
    for p in range(0, wl.graph.nnz, 37):
        d = int(deg[rows[p]])
        v = Fraction(float(wl.graph.vals[p]))
        # nearest float32 to 1/d: error at most half an ulp of v
        ulp = Fraction(2) ** (int(np.floor(np.log2(float(v)))) - 23)
        assert abs(v - Fraction(1, d)) <= ulp / 2


def test_determinism_same_seed_bitwise():
    a = synth.config(1)
    b = synth.config(1)
    for x, y in [(a.graph.indptr, b.graph.indptr), (a.graph.indices, b.graph.indices),
                 (a.graph.vals, b.graph.vals), (a.H, b.H), (a.W_pred, b.W_pred),
                 (a.labels, b.labels)]:
        assert np.array_equal(x, y)
    for la, lb in zip(a.layers, b.layers):
        assert np.array_equal(la.W_self, lb.W_self) and np.array_equal(la.W_neigh, lb.W_neigh)
    c = synth.config(4, s=1)
    d = synth.config(4, s=2)
    assert c.graph.nnz != d.graph.nnz or not np.array_equal(c.graph.indices, d.graph.indices)


def test_rmat_is_skewed_and_er_is_not():
    r = synth.custom(4096, "rmat", 20, [(4, 4)])
    e = synth.custom(4096, "er", 20, [(4, 4)])
    _check_csr(r.graph)
    _check_csr(e.graph)
    assert r.graph.degrees().max() > 10 * 20
    assert e.graph.degrees().max() < 3 * 20


def test_glorot_range_and_labels():
    wl = synth.config(1)
    for lay in wl.layers:
        f_in, h = lay.W_self.shape
        a = np.sqrt(6.0 / (f_in + h))
        assert np.abs(lay.W_self).max() <= a and np.abs(lay.W_neigh).max() <= a
        assert not np.any(lay.bias)
    assert wl.labels.min() >= 0 and wl.labels.max() < 41
    w2 = synth.custom(300, "er", 6, [(5, 4)], head="bce", classes=30)
    assert set(np.unique(w2.targets).tolist()) <= {0.0, 1.0}


def test_special_graphs():
    rng = np.random.default_rng(0)
    p = synth.permutation_graph(50, rng)
    assert np.all(p.degrees() == 1) and np.all(p.vals == 1.0)
    k = synth.complete_graph(7)
    _check_csr(k)
    assert np.all(k.degrees() == 6)
    s = synth.star_graph(100)
    _check_csr(s)
    assert s.degrees()[0] == 99
    e = synth.empty_graph(5)
    assert e.nnz == 0 and e.indptr.shape == (6,)


def test_epoch_stream_shares_model_weights():
    a = synth.config(4, s=0)
    b = synth.config(4, s=7)
    for la, lb in zip(a.layers, b.layers):
        assert np.array_equal(la.W_self, lb.W_self) and np.array_equal(la.W_neigh, lb.W_neigh)
    assert np.array_equal(a.W_pred, b.W_pred)
    assert not np.array_equal(a.H, b.H)


def test_with_self_loops_structure():
    g0 = synth.custom(300, "rmat", 6, [(4, 4)], seed=2).graph
    g1 = synth.with_self_loops(g0)
    assert g1.nnz == g0.nnz + g0.n
    rows = np.repeat(np.arange(g1.n), g1.degrees())
    assert np.count_nonzero(rows == g1.indices) == g1.n            # one diagonal entry per row
    assert np.array_equal(g1.degrees(), g0.degrees() + 1)
    assert np.all(g1.vals == np.float32(1) / (g0.degrees() + 1).astype(np.float32)[rows])
    ok = np.all(np.diff(g1.indices)[np.diff(rows) == 0] > 0)
    assert ok
    assert B_symmetric(g1)
    with pytest.raises(ValueError):
        synth.with_self_loops(g1)
    wl = synth.config(1, self_loops=True, n=500)
    assert wl.spec.self_loops and wl.graph.nnz == synth.config(1, n=500).graph.nnz + 500


def B_symmetric(g):
    rows = np.repeat(np.arange(g.n), g.degrees())
    a = set(zip(rows.tolist(), g.indices.tolist()))
    return all((j, i) in a for i, j in a)
