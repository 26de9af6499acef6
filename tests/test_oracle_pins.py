"""Pins for the CPU oracle against what the paper and the mathematics fix.

None of these re-types the oracle's own expressions: each checks a value that
is fixed independently (exact rational brute force, closed forms, invariants,
special cases that reduce to a library routine, finite differences), chosen so
that a plausible slip in the oracle (a dropped term, a wrong sign or index, a
transposed operand, a swapped concat half) fails at least one of them.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import scipy.sparse as sp

import oracle
from oracle import bf16 as obf16
from paper_1810_11899_amd import synth


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = max(np.abs(b).max(), 1e-300) if b.size else 1.0
    return float(np.abs(a - b).max() / den) if b.size else 0.0


# ---------------------------------------------------------------- forward ----
def test_exact_rational_layer_forward():
    """Tiny graph, small-integer inputs: the layer of Sec. II in exact rationals."""
    rng = np.random.default_rng(3)
    n, f, h = 7, 3, 2
    # a small directed pattern with varied degrees and one empty row
    pairs = [(0, 1), (0, 2), (0, 5), (1, 0), (2, 3), (2, 4), (2, 6), (2, 1), (3, 2),
             (5, 6), (5, 0), (6, 4)]
    rows, cols = zip(*pairs)
    g = synth.csr_from_pairs(n, np.array(rows), np.array(cols))
    H = rng.integers(-4, 5, size=(n, f)).astype(np.float32)
    Ws = rng.integers(-3, 4, size=(f, h)).astype(np.float32)
    Wn = rng.integers(-3, 4, size=(f, h)).astype(np.float32)
    b = np.array([1, -2, 0, 3], np.float32)
    Y, cache = oracle.layer_fwd(g, H, Ws, Wn, b)
    # the stored weights are float32(1/deg); the layer applies exactly those values
    ent = {i: [(int(g.indices[p]), Fraction(float(g.vals[p])))
               for p in range(g.indptr[i], g.indptr[i + 1])] for i in range(n)}
    for i in range(n):
        assert sorted(j for j, _ in ent[i]) == sorted(c for (r, c) in pairs if r == i)
        agg = [sum((w * int(H[j, c]) for j, w in ent[i]), Fraction(0)) for c in range(f)]
        for o in range(h):
            s = sum(Fraction(int(H[i, c])) * int(Ws[c, o]) for c in range(f)) + int(b[o])
            nn = sum(agg[c] * int(Wn[c, o]) for c in range(f)) + int(b[h + o])
            assert abs(Y[i, o] - float(max(s, 0))) <= 1e-12 * (1 + abs(float(s)))
            assert abs(Y[i, h + o] - float(max(nn, 0))) <= 1e-12 * (1 + abs(float(nn)))
            assert abs(cache.AGG[i, 0] - float(agg[0])) <= 1e-12 * (1 + abs(float(agg[0])))


def test_constant_features_mean_invariant():
    """Mean aggregation of constant features returns the constant (0 on empty rows)."""
    wl = synth.custom(3000, "rmat", 16, [(4, 4)])
    g = wl.graph
    c = np.array([1.5, -2.25, 1e3, 7.0])
    X = np.tile(c, (g.n, 1))
    out = oracle.aggregate(g.indptr, g.indices, g.vals, X)
    deg = g.degrees()
    assert np.all(out[deg == 0] == 0.0)
    nz = deg > 0
    err = np.abs(out[nz] - c[None, :]) / np.abs(c)[None, :]
    # float32(1/d) carries a relative error <= 2^-24; d of them add up to within ~d 2^-24
    assert np.all(err <= (deg[nz, None] + 4) * 2.0 ** -23)


def test_permutation_graph_is_exact_gather():
    rng = np.random.default_rng(5)
    g = synth.permutation_graph(257, rng)
    X = rng.standard_normal((257, 9))
    out = oracle.aggregate(g.indptr, g.indices, g.vals, X)
    assert np.array_equal(out, X[g.indices])


def test_complete_graph_closed_form():
    n = 23
    g = synth.complete_graph(n)
    X = np.random.default_rng(2).standard_normal((n, 5))
    out = oracle.aggregate(g.indptr, g.indices, g.vals, X)
    expect = (X.sum(axis=0)[None, :] - X) / (n - 1)
    assert rel(out, expect) < 1e-6  # vals are float32(1/(n-1))


def test_empty_graph_reduces_to_dense_layer():
    rng = np.random.default_rng(7)
    n, f, h = 40, 6, 5
    g = synth.empty_graph(n)
    H = rng.standard_normal((n, f)).astype(np.float32)
    Ws = rng.standard_normal((f, h)).astype(np.float32)
    Wn = rng.standard_normal((f, h)).astype(np.float32)
    b = rng.standard_normal(2 * h).astype(np.float32)
    Y, _ = oracle.layer_fwd(g, H, Ws, Wn, b)
    import torch  # a library linear layer as the independent reference
    lin = torch.nn.functional.linear(torch.tensor(H, dtype=torch.float64),
                                     torch.tensor(Ws.T, dtype=torch.float64),
                                     torch.tensor(b[:h], dtype=torch.float64))
    assert rel(Y[:, :h], torch.relu(lin).numpy()) < 1e-14
    assert np.array_equal(Y[:, h:], np.tile(np.maximum(b[h:], 0), (n, 1)).astype(np.float64))


def test_dense_brute_force_small_graphs():
    """Against a scipy dense product of the densified matrix, n <= 64."""
    for seed in range(3):
        wl = synth.custom(61, "rmat", 6, [(7, 5)], seed=seed)
        g = wl.graph
        A = sp.csr_matrix((g.vals.astype(np.float64), g.indices, g.indptr), shape=(g.n, g.n)).toarray()
        lay = wl.layers[0]
        b = np.random.default_rng(seed).standard_normal(10).astype(np.float32)
        Y, cache = oracle.layer_fwd(g, wl.H, lay.W_self, lay.W_neigh, b)
        N = np.linalg.multi_dot([A, wl.H.astype(np.float64), lay.W_neigh.astype(np.float64)])
        S = wl.H.astype(np.float64) @ lay.W_self.astype(np.float64)
        assert rel(Y[:, 5:], np.maximum(N + b[5:], 0)) < 1e-12
        assert rel(Y[:, :5], np.maximum(S + b[:5], 0)) < 1e-12


def test_linearity_of_aggregation():
    wl = synth.custom(500, "rmat", 10, [(3, 3)])
    g = wl.graph
    rng = np.random.default_rng(1)
    X, Z = rng.standard_normal((500, 6)), rng.standard_normal((500, 6))
    lhs = oracle.aggregate(g.indptr, g.indices, g.vals, 2.5 * X - 0.75 * Z)
    rhs = 2.5 * oracle.aggregate(g.indptr, g.indices, g.vals, X) - 0.75 * oracle.aggregate(
        g.indptr, g.indices, g.vals, Z)
    assert rel(lhs, rhs) < 1e-13


def test_permutation_equivariance_of_step():
    wl = synth.custom(120, "rmat", 8, [(6, 4), (8, 3)], head="ce", classes=5, seed=4)
    base = oracle.step(wl, first_layer_dH=True)
    rng = np.random.default_rng(11)
    P = rng.permutation(wl.n)          # new id of old vertex v is P[v]
    inv = np.argsort(P)
    g = wl.graph
    rows = np.repeat(np.arange(wl.n), g.degrees())
    g2 = synth.csr_from_pairs(wl.n, P[rows], P[g.indices], g.vals)
    import copy
    wl2 = copy.deepcopy(wl)
    wl2.graph = g2
    wl2.H = wl.H[inv]
    wl2.labels = wl.labels[inv]
    r2 = oracle.step(wl2, first_layer_dH=True)
    for a, b in zip(base.Y, r2.Y):
        assert rel(b, a[inv]) < 1e-12
    for li in range(2):
        assert rel(r2.dW_self[li], base.dW_self[li]) < 1e-11
        assert rel(r2.dW_neigh[li], base.dW_neigh[li]) < 1e-11
        assert rel(r2.dH[li], base.dH[li][inv]) < 1e-11
    assert abs(r2.loss - base.loss) < 1e-12


# -------------------------------------------------------------- transpose ----
def test_transpose_matches_scipy_and_is_an_involution():
    wl = synth.custom(700, "rmat", 9, [(2, 2)])
    g = wl.graph
    # non-symmetric values (row-normalised) make the value check meaningful
    ti, tj, tv = oracle.csr_transpose(g.n, g.n, g.indptr, g.indices, g.vals)
    ref = sp.csr_matrix((g.vals, g.indices, g.indptr), shape=(g.n, g.n)).T.tocsr()
    assert np.array_equal(ti, ref.indptr) and np.array_equal(tj, ref.indices)
    assert np.array_equal(tv.view(np.uint32), ref.data.astype(np.float32).view(np.uint32))
    bi, bj, bv = oracle.csr_transpose(g.n, g.n, ti, tj, tv)
    assert np.array_equal(bi, g.indptr) and np.array_equal(bj, g.indices)
    assert np.array_equal(bv.view(np.uint32), g.vals.view(np.uint32))
    # undirected graph: same pattern; row lengths of A^T are column counts of A
    assert np.array_equal(ti, g.indptr) and np.array_equal(tj, g.indices)
    assert np.array_equal(np.diff(ti), np.bincount(g.indices, minlength=g.n))


def test_transpose_rectangular_and_empty():
    rows = np.array([0, 0, 2, 2, 2])
    cols = np.array([4, 1, 0, 1, 3])
    g = synth.csr_from_pairs(3, rows, cols, np.arange(5, dtype=np.float32))
    ti, tj, tv = oracle.csr_transpose(3, 6, g.indptr, g.indices, g.vals)
    assert ti.tolist() == [0, 1, 3, 3, 4, 5, 5]
    assert tj.tolist() == [2, 0, 2, 2, 0]
    # values: original order after (row, col) sort is (0,1)=1 (0,4)=0 (2,0)=2 (2,1)=3 (2,3)=4
    assert tv.tolist() == [2.0, 1.0, 3.0, 4.0, 0.0]
    e = synth.empty_graph(4)
    ti, tj, tv = oracle.csr_transpose(4, 4, e.indptr, e.indices, e.vals)
    assert ti.tolist() == [0] * 5 and tj.size == 0


def test_adjoint_identity():
    wl = synth.custom(900, "rmat", 12, [(2, 2)], seed=1)
    g = wl.graph
    ti, tj, tv = oracle.csr_transpose(g.n, g.n, g.indptr, g.indices, g.vals)
    rng = np.random.default_rng(9)
    X, Y = rng.standard_normal((g.n, 4)), rng.standard_normal((g.n, 4))
    lhs = np.sum(oracle.aggregate(g.indptr, g.indices, g.vals, X) * Y)
    rhs = np.sum(X * oracle.aggregate(ti, tj, tv, Y))
    assert abs(lhs - rhs) <= 1e-12 * (abs(lhs) + 1)


# ------------------------------------------------------------------- head ----
def test_ce_closed_forms():
    n, f, C = 50, 6, 7
    rng = np.random.default_rng(0)
    HL = rng.standard_normal((n, f))
    lab = rng.integers(0, C, n)
    loss, dWp, dbp, dHL, _ = oracle.loss_grad("ce", HL, np.zeros((f, C)), np.zeros(C), labels=lab)
    assert abs(loss - math.log(C)) < 1e-14
    G = np.full((n, C), 1.0 / C)
    G[np.arange(n), lab] -= 1.0
    G /= n
    assert rel(dbp, G.sum(axis=0)) < 1e-13
    assert np.all(dHL == 0.0)
    # a row whose logit for the true class dominates has ~zero loss
    Wp = np.zeros((f, C))
    bp = np.zeros(C)
    bp[3] = 60.0
    loss2, *_ = oracle.loss_grad("ce", HL, Wp, bp, labels=np.full(n, 3))
    assert loss2 < 1e-20
    loss3, *_ = oracle.loss_grad("ce", HL, Wp, bp, labels=np.full(n, 0))
    assert abs(loss3 - 60.0) < 1e-12


def test_ce_gradient_rows_sum_to_zero_and_bce_closed_form():
    rng = np.random.default_rng(1)
    HL = rng.standard_normal((30, 5))
    Wp = rng.standard_normal((5, 4))
    _, _, dbp, _, X = oracle.loss_grad("ce", HL, Wp, np.zeros(4), labels=rng.integers(0, 4, 30))
    assert abs(dbp.sum()) < 1e-15
    t = (rng.random((30, 4)) < 0.3).astype(np.float64)
    loss, _, dbp, dHL, _ = oracle.loss_grad("bce", HL, np.zeros((5, 4)), np.zeros(4), targets=t)
    assert abs(loss - math.log(2.0)) < 1e-15
    assert rel(dbp, (0.5 - t).sum(axis=0) / 120) < 1e-14
    # large |x| stays finite (the log1p(exp(-|x|)) form)
    big = np.full((2, 1), 800.0)
    loss_big, *_ = oracle.loss_grad("bce", big, np.ones((1, 1)), np.zeros(1), targets=np.zeros((2, 1)))
    assert abs(loss_big - 800.0) < 1e-9


# ---------------------------------------------------- finite differences ----
def _fd_workload(head, seed):
    """A 2-layer float64 workload whose pre-activations keep away from the ReLU kink."""
    for s in range(seed, seed + 50):
        wl = synth.custom(14, "er", 4, [(5, 4), (8, 3)], head=head, classes=4, seed=s)
        for lay in wl.layers:
            lay.W_self = lay.W_self.astype(np.float64)
            lay.W_neigh = lay.W_neigh.astype(np.float64)
            lay.bias = np.random.default_rng(s).standard_normal(lay.bias.shape) * 0.1
        wl.H = wl.H.astype(np.float64)
        if wl.W_pred is not None:
            wl.W_pred = wl.W_pred.astype(np.float64)
            wl.b_pred = np.random.default_rng(s + 1).standard_normal(wl.b_pred.shape) * 0.1
        else:
            wl.dY = wl.dY.astype(np.float64)
        H = wl.H
        ok = True
        for lay in wl.layers:
            Y, c = oracle.layer_fwd(wl.graph, H, lay.W_self, lay.W_neigh, lay.bias)
            ok &= np.abs(c.Z).min() > 1e-3
            H = Y
        if ok:
            return wl
    raise RuntimeError("no kink-free seed")


def _objective(wl):
    H = wl.H
    for lay in wl.layers:
        H, _ = oracle.layer_fwd(wl.graph, H, lay.W_self, lay.W_neigh, lay.bias)
    if wl.spec.head is None:
        return float(np.sum(H * wl.dY))
    loss, *_ = oracle.loss_grad(wl.spec.head, H, wl.W_pred, wl.b_pred, labels=wl.labels,
                                targets=wl.targets)
    return loss


@pytest.mark.parametrize("head", ["ce", "bce", None])
def test_finite_difference_gradients(head):
    wl = _fd_workload(head, 100)
    r = oracle.step(wl, first_layer_dH=True)
    eps = 1e-6
    rng = np.random.default_rng(0)
    checks = []
    for li, lay in enumerate(wl.layers):
        checks += [(lay.W_self, r.dW_self[li]), (lay.W_neigh, r.dW_neigh[li]), (lay.bias, r.db[li])]
    checks.append((wl.H, r.dH[0]))
    if head is not None:
        checks += [(wl.W_pred, r.dW_pred), (wl.b_pred, r.db_pred)]
    for arr, grad in checks:
        flat = arr.reshape(-1)
        gflat = np.asarray(grad).reshape(-1)
        for idx in rng.choice(flat.size, size=min(8, flat.size), replace=False):
            old = flat[idx]
            flat[idx] = old + eps
            jp = _objective(wl)
            flat[idx] = old - eps
            jm = _objective(wl)
            flat[idx] = old
            fd = (jp - jm) / (2 * eps)
            scale = max(np.abs(gflat).max(), 1e-12)
            assert abs(fd - gflat[idx]) <= 1e-6 * scale + 1e-9, (arr.shape, idx, fd, gflat[idx])


def test_relu_derivative_at_zero_is_zero():
    """An isolated vertex with zero bias has Z == 0 exactly on its neighbour half."""
    g = synth.csr_from_undirected(3, np.array([0]), np.array([1]))  # vertex 2 isolated
    H = np.ones((3, 2))
    Y, cache = oracle.layer_fwd(g, H, np.ones((2, 1)), np.ones((2, 1)), np.zeros(2))
    assert cache.Z[2, 1] == 0.0
    gT = type("T", (), {})()
    gT.indptr, gT.indices, gT.vals = oracle.csr_transpose(3, 3, g.indptr, g.indices, g.vals)
    _, _, db, _ = oracle.layer_bwd(gT, cache, np.ones((2, 1)), np.ones((2, 1)), np.ones((3, 2)), False)
    assert db[1] == 2.0  # only the two connected vertices pass gradient


# ------------------------------------------------------------------- bf16 ----
def test_bf16_rounding_against_torch_and_special_values():
    import torch
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(10000).astype(np.float32),
        np.array([0.0, -0.0, 1.0, np.inf, -np.inf, 3.4e38, 1e-40, -1e-45], np.float32),
        # exact ties: 1 + 2^-8 (ties down to even), 1 + 3*2^-8 (ties up to even)
        np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8], np.float32),
    ])
    ours = obf16.f32_to_bf16_bits(x)
    ref = torch.tensor(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert obf16.round_bf16(np.float32(1.0 + 2.0 ** -8))[()] == 1.0
    assert obf16.round_bf16(np.float32(1.0 + 3 * 2.0 ** -8))[()] == np.float32(1.0 + 2 ** -6)
    nan = obf16.round_bf16(np.array([np.nan], np.float32))
    assert np.isnan(nan[0])


# ------------------------------------------------------------ kink envelope ----
def test_kink_envelope_bounds_every_branch_choice(monkeypatch):
    """Brute force: with an enlarged ambiguity band, every assignment of the
    ambiguous ReLU branches moves each gradient by at most the envelope."""
    import itertools
    from oracle import gcnref
    monkeypatch.setattr(gcnref, "C_AMB", 1.0e6)   # widen the band to a handful of entries
    checked = 0
    for seed in range(8):
        wl = synth.custom(9, "er", 4, [(4, 3), (6, 2)], head="ce", classes=3, seed=seed)
        for lay in wl.layers:
            lay.bias = np.random.default_rng(seed).standard_normal(lay.bias.shape).astype(np.float32) * 0.05
        res = oracle.step(wl, first_layer_dH=True, envelope=True)
        g = wl.graph
        gT = synth.Graph(g.n, res.t_indptr, res.t_indices, res.t_vals)
        H = wl.H
        caches = []
        for lay in wl.layers:
            H, c = oracle.layer_fwd(g, H, lay.W_self, lay.W_neigh, lay.bias, ambiguity=True)
            caches.append(c)
        amb = [np.argwhere(c.amb) for c in caches]
        total = sum(a.shape[0] for a in amb)
        if total == 0 or total > 10:
            continue
        attained = 0.0
        for bits in itertools.product([0, 1], repeat=total):
            masks = [(c.Z > 0).astype(np.float64) for c in caches]
            k = 0
            for li, a in enumerate(amb):
                for (i, j) in a:
                    masks[li][i, j] = bits[k]
                    k += 1
            dY = res.dHL
            for li in range(1, -1, -1):
                lay = wl.layers[li]
                dWs, dWn, db, dH = oracle.layer_bwd(gT, caches[li], lay.W_self, lay.W_neigh, dY, True,
                                                    mask=masks[li])
                for got, ref, E in ((dWs, res.dW_self[li], res.E_dW_self[li]),
                                    (dWn, res.dW_neigh[li], res.E_dW_neigh[li]),
                                    (db, res.db[li], res.E_db[li]), (dH, res.dH[li], res.E_dH[li])):
                    dev_ = np.abs(got - ref)
                    assert np.all(dev_ <= E + 1e-12), (seed, li, (dev_ - E).max())
                    attained = max(attained, float(dev_.max()))
                dY = dH
        assert attained > 0.0  # some branch choice really moves a gradient
        checked += 1
    assert checked >= 2, "too few seeds with a small ambiguous set"


def test_kink_envelope_is_zero_without_ambiguity():
    wl = synth.custom(40, "er", 5, [(6, 4)], head="bce", classes=3, seed=1)
    res = oracle.step(wl, first_layer_dH=True, envelope=True)
    if res.ambiguous == [0]:
        for E in res.E_dW_self + res.E_dW_neigh + res.E_db + res.E_dH:
            assert not np.any(E)


# ----------------------------------------------------------------- Adam ----
def test_adam_matches_torch_optim_adam_float64():
    """Adam of Alg. 1 against torch.optim.Adam (an independent implementation),
    both in float64, over several steps with changing gradients."""
    import torch
    from oracle import optim
    rng = np.random.default_rng(0)
    p0 = rng.standard_normal(1000)
    tp = torch.tensor(p0.copy(), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([tp], lr=0.01, betas=(0.9, 0.999), eps=1e-8)
    p, m, v = p0.copy(), np.zeros(1000), np.zeros(1000)
    for t in range(1, 8):
        g = rng.standard_normal(1000) * (10.0 ** rng.integers(-6, 2))
        tp.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        p, m, v = optim.adam(p, g, m, v, t, 0.01)
        assert np.max(np.abs(p - tp.detach().numpy())) <= 1e-12 * np.max(np.abs(p))


def test_adam_closed_forms():
    from oracle import optim
    g = np.array([3.0, -2e-3, 0.0, 1e-12])
    # first step from zero moments: lr * g / (|g| + eps)
    p, m, v = optim.adam(np.zeros(4), g, np.zeros(4), np.zeros(4), 1, 0.1)
    assert np.allclose(p, -0.1 * g / (np.abs(g) + 1e-8), rtol=1e-14, atol=0)
    # a constant gradient keeps the bias-corrected moments equal to g and g^2
    p, m, v = np.zeros(4), np.zeros(4), np.zeros(4)
    for t in range(1, 6):
        p, m, v = optim.adam(p, g, m, v, t, 0.1)
    assert np.allclose(p, -5 * 0.1 * g / (np.abs(g) + 1e-8), rtol=1e-12, atol=1e-15)


def test_bf16_relu_threshold_is_the_rounding_rule():
    """The bfloat16 path's ReLU derivative [bf16(y) > 0] equals [y > 2^-134]
    (half the smallest bfloat16 subnormal; the tie rounds to even, i.e. 0)."""
    import numpy as np
    from oracle.bf16 import f32_to_bf16_bits
    t = np.float32(2.0 ** -134)
    ys = [0.0, -0.0, 2.0 ** -149, 2.0 ** -135, 2.0 ** -134, 2.0 ** -133, 2.0 ** -126, 1e-30, 1.0,
          -(2.0 ** -133), float("inf"), float("-inf")]
    ys = np.array(ys, dtype=np.float32)
    ys = np.concatenate([ys, np.nextafter(t, np.float32(1)), np.nextafter(t, np.float32(0))], axis=None)
    bits = f32_to_bf16_bits(ys).astype(np.uint32)
    positive = ((bits & 0x8000) == 0) & (bits != 0) & ((bits & 0x7FFF) <= 0x7F80)
    assert np.array_equal(positive, ys > t)


# ------------------------------------------------- given branch masks ----
def _gated_objective(wl, masks):
    """The network with every ReLU replaced by the fixed gate m (Y = Z * m),
    evaluated through the oracle's forward pre-activations."""
    H = wl.H
    for lay, m in zip(wl.layers, masks):
        _, c = oracle.layer_fwd(wl.graph, H, lay.W_self, lay.W_neigh, lay.bias)
        H = c.Z * m
    if wl.spec.head is None:
        return float(np.sum(H * wl.dY))
    loss, *_ = oracle.loss_grad(wl.spec.head, H, wl.W_pred, wl.b_pred, labels=wl.labels, targets=wl.targets)
    return loss


@pytest.mark.parametrize("head", ["ce", "bce", None])
def test_step_with_masks_is_the_gradient_of_the_gated_network(head):
    """With branch masks given, the step returns the gradient of the gated
    network: central finite differences of that network's objective, with
    random masks that differ from [Z > 0] in about half of the entries."""
    wl = synth.custom(40, "er", 5, [(5, 4), (8, 3)], head=head, classes=4, seed=7)
    rng = np.random.default_rng(3)
    for lay in wl.layers:            # float64 parameters: the perturbations are exact
        lay.W_self = lay.W_self.astype(np.float64)
        lay.W_neigh = lay.W_neigh.astype(np.float64)
        lay.bias = rng.standard_normal(lay.bias.shape) * 0.2
    wl.H = wl.H.astype(np.float64)
    if head is None:
        wl.dY = rng.standard_normal((wl.n, 6))
    else:
        wl.W_pred = wl.W_pred.astype(np.float64)
        wl.b_pred = rng.standard_normal(wl.b_pred.shape) * 0.1
    masks = [(rng.random((wl.n, 2 * lay.h)) < 0.5).astype(np.float64) for lay in wl.layers]
    r = oracle.step(wl, first_layer_dH=True, masks=masks)
    H = wl.H
    for li, (lay, m) in enumerate(zip(wl.layers, masks)):
        _, c = oracle.layer_fwd(wl.graph, H, lay.W_self, lay.W_neigh, lay.bias)
        H = c.Z * m
        assert np.array_equal(r.Y[li], H)                     # the forward is gated too
    checks = []
    for li, lay in enumerate(wl.layers):
        checks += [(lay.W_self, r.dW_self[li]), (lay.W_neigh, r.dW_neigh[li]), (lay.bias, r.db[li])]
    checks.append((wl.H, r.dH[0]))
    if head is not None:
        checks += [(wl.W_pred, r.dW_pred), (wl.b_pred, r.db_pred)]
    eps = 1e-6
    for arr, grad in checks:
        flat = arr.reshape(-1)
        gflat = np.asarray(grad).reshape(-1)
        for idx in rng.choice(flat.size, size=min(8, flat.size), replace=False):
            old = flat[idx]
            flat[idx] = old + eps
            jp = _gated_objective(wl, masks)
            flat[idx] = old - eps
            jm = _gated_objective(wl, masks)
            flat[idx] = old
            fd = (jp - jm) / (2 * eps)
            assert abs(fd - gflat[idx]) <= 1e-6 * max(np.abs(gflat).max(), 1e-12) + 1e-9, (arr.shape, idx)


def test_step_with_its_own_masks_is_the_relu_step():
    """m_l = [Z_l > 0] reproduces the ReLU step exactly."""
    wl = synth.custom(300, "rmat", 7, [(9, 6), (12, 5)], head="ce", classes=6, seed=8)
    base = oracle.step(wl, first_layer_dH=True)
    H, masks = wl.H, []
    for lay in wl.layers:
        H, c = oracle.layer_fwd(wl.graph, H, lay.W_self, lay.W_neigh, lay.bias)
        masks.append(c.Z > 0)
    r = oracle.step(wl, first_layer_dH=True, masks=masks)
    for a, b in [(base.Y, r.Y), (base.dW_self, r.dW_self), (base.dW_neigh, r.dW_neigh), (base.db, r.db),
                 (base.dH, r.dH)]:
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
    assert base.loss == r.loss and np.array_equal(base.dW_pred, r.dW_pred)


# ----------------------------------------------------------- self-loops ----
def test_self_loop_aggregation_closed_form():
    """Sec. V-B's self-connection: with a self-loop added to every vertex the
    mean aggregation is (H[i] + sum of the neighbours' H) / (deg(i) + 1),
    written here from the loop-free neighbour lists; an isolated vertex keeps
    its own row."""
    wl0 = synth.custom(90, "rmat", 5, [(6, 3)], seed=4)
    g0 = wl0.graph
    g1 = synth.with_self_loops(g0)
    H = wl0.H.astype(np.float64)
    got = oracle.aggregate(g1.indptr, g1.indices, g1.vals, H)
    for i in range(g0.n):
        nb = g0.indices[g0.indptr[i]:g0.indptr[i + 1]]
        want = (H[i] + H[nb].sum(axis=0)) / (len(nb) + 1)
        assert np.allclose(got[i], want, rtol=1e-6, atol=1e-12), i   # vals are float32(1/(deg+1))
    iso = np.flatnonzero(np.diff(g0.indptr) == 0)
    assert iso.size > 0 and np.array_equal(got[iso], H[iso])
    c = oracle.aggregate(g1.indptr, g1.indices, g1.vals, np.full((g0.n, 3), 2.5))
    assert np.abs(c - 2.5).max() < 1e-6        # no empty rows: the constant comes back everywhere


def test_self_loop_step_against_dense_brute_force():
    wl = synth.custom(40, "er", 4, [(5, 3), (6, 2)], head="ce", classes=3, seed=9, self_loops=True)
    g = wl.graph
    A = sp.csr_matrix((g.vals.astype(np.float64), g.indices, g.indptr), shape=(g.n, g.n)).toarray()
    assert np.allclose(np.diag(A), 1.0 / (np.count_nonzero(A, axis=1)))
    H = wl.H.astype(np.float64)
    r = oracle.step(wl, first_layer_dH=True)
    for li, lay in enumerate(wl.layers):
        Ws, Wn = lay.W_self.astype(np.float64), lay.W_neigh.astype(np.float64)
        Z = np.concatenate([H @ Ws, A @ H @ Wn], axis=1) + lay.bias
        H = np.maximum(Z, 0)
        assert rel(r.Y[li], H) < 1e-12
