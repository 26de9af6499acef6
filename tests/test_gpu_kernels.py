"""Kernel-level parity on the GPU, through the C ABI, against the CPU oracle.

Sizes span several tiles / wavefront work units and leave ragged tails.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import bf16 as obf16
from paper_1810_11899_amd import binding as B
from paper_1810_11899_amd import synth

from gpu_util import TOL_F32, dev, rel_inf, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


@pytest.fixture(scope="module")
def ws():
    return B.Workspace("cuda")


def dcsr(g, n_cols=None):
    return B.DeviceCSR.from_host(g.n, g.n if n_cols is None else n_cols, g.indptr, g.indices, g.vals)


# ------------------------------------------------------------- transpose ----
@pytest.mark.parametrize("case", ["cfg1", "rmat3000", "star", "empty", "dup", "rect"])
def test_transpose_bit_exact(case, ws):
    n_cols = None
    if case == "cfg1":
        g = synth.config(1).graph
    elif case == "rmat3000":
        g = synth.custom(3001, "rmat", 13, [(2, 2)], seed=5).graph
    elif case == "star":
        g = synth.star_graph(70000)
    elif case == "empty":
        g = synth.empty_graph(333)
    elif case == "dup":   # duplicated entries must keep their CSR order
        rows = np.array([0, 0, 0, 1, 2, 2, 3, 3, 3, 3])
        cols = np.array([2, 2, 1, 2, 0, 2, 3, 3, 2, 0])
        g = synth.csr_from_pairs(4, rows, cols, np.arange(10, dtype=np.float32))
    else:                 # rectangular: 500 rows, 1300 columns
        rng = np.random.default_rng(0)
        rows = rng.integers(0, 500, 4000)
        cols = rng.integers(0, 1300, 4000)
        key = np.unique(rows * 1300 + cols)
        g = synth.csr_from_pairs(500, key // 1300, key % 1300)
        n_cols = 1300
    nc = g.n if n_cols is None else n_cols
    A = dcsr(g, nc)
    AT = B.gcn_csr_transpose(A, ws)
    ti, tj, tv = oracle.csr_transpose(g.n, nc, g.indptr, g.indices, g.vals)
    torch.cuda.synchronize()
    assert np.array_equal(AT.indptr.cpu().numpy(), ti)
    assert np.array_equal(AT.indices.cpu().numpy(), tj)
    assert np.array_equal(AT.vals.cpu().numpy().view(np.uint32), np.asarray(tv, np.float32).view(np.uint32))


@pytest.mark.parametrize("case", ["cfg1", "rmat3000_random_vals", "star", "complete", "empty"])
def test_transpose_symmetric_pattern_bit_exact(case, ws):
    """A symmetric pattern's transpose: A's indptr / indices with values found
    in the partner rows, equal bit for bit to the general transpose."""
    rng = np.random.default_rng(3)
    if case == "cfg1":
        g = synth.config(1).graph
    elif case == "rmat3000_random_vals":      # values that are not constant along rows
        g0 = synth.custom(3001, "rmat", 13, [(2, 2)], seed=5).graph
        g = synth.Graph(g0.n, g0.indptr, g0.indices, rng.standard_normal(g0.nnz).astype(np.float32))
    elif case == "star":
        g = synth.star_graph(70000)
    elif case == "complete":
        g = synth.complete_graph(300)
    else:
        g = synth.empty_graph(333)
    assert B.gcn_csr_pattern_symmetric_host(g.indptr, g.indices)
    A = dcsr(g)
    AT = B.gcn_csr_transpose(A, ws)
    ATs = B.gcn_csr_transpose_symmetric(A, ws)
    ti, tj, tv = oracle.csr_transpose(g.n, g.n, g.indptr, g.indices, g.vals)
    torch.cuda.synchronize()
    assert np.array_equal(ATs.indptr.cpu().numpy(), ti) and np.array_equal(ATs.indices.cpu().numpy(), tj)
    assert np.array_equal(ATs.vals.cpu().numpy().view(np.uint32), np.asarray(tv, np.float32).view(np.uint32))
    assert torch.equal(ATs.vals.view(torch.int32), AT.vals.view(torch.int32))


def test_transpose_symmetric_marks_missing_partners_nan(ws):
    """Outside the contract (pattern not symmetric): a missing partner in a row
    whose values differ, and an index out of range, give NaN."""
    # entries (0,1) (1,1) (1,2) (2,1) (2,7); (1,0) is missing, 7 is out of range
    ip = np.array([0, 1, 3, 5], np.int32)
    ix = np.array([1, 1, 2, 1, 7], np.int32)
    vals = np.array([1.0, 5.0, 6.0, 3.0, 4.0], np.float32)
    A = B.DeviceCSR.from_host(3, 3, ip, ix, vals)
    t = B.gcn_csr_transpose_symmetric(A, ws).vals.cpu().numpy()
    assert np.isnan(t[0]) and np.isnan(t[4])
    assert t[1] == 5.0 and t[2] == 3.0 and t[3] == 6.0


# ------------------------------------------------------------- aggregate ----
@pytest.mark.parametrize("k", [1, 50, 64, 100, 128, 130, 192, 200, 256, 300, 512, 602, 1024])
def test_aggregate_parity_widths(k, ws):
    wl = synth.custom(3001, "rmat", 13, [(2, 2)], seed=k)
    g = wl.graph
    X = np.random.default_rng(k).standard_normal((g.n, k)).astype(np.float32)
    out = torch.empty((g.n, k), dtype=torch.float32, device="cuda")
    B.gcn_aggregate(dcsr(g), dev(X), out, ws)
    ref = oracle.aggregate(g.indptr, g.indices, g.vals, X)
    assert rel_inf(out.cpu().numpy(), ref) <= TOL_F32 / 10


def test_aggregate_leading_dimensions(ws):
    g = synth.custom(2000, "rmat", 9, [(2, 2)], seed=3).graph
    Xbig = np.random.default_rng(1).standard_normal((g.n, 200)).astype(np.float32)
    X = dev(Xbig)[:, 10:138]                    # k = 128 inside a 200-wide buffer
    outbuf = torch.full((g.n, 300), 7.0, device="cuda")
    out = outbuf[:, 50:178]
    B.gcn_aggregate(dcsr(g), X, out, ws)
    ref = oracle.aggregate(g.indptr, g.indices, g.vals, Xbig[:, 10:138])
    o = outbuf.cpu().numpy()
    assert rel_inf(o[:, 50:178], ref) <= TOL_F32 / 10
    assert np.all(o[:, :50] == 7.0) and np.all(o[:, 178:] == 7.0)  # nothing outside the view


def test_aggregate_permutation_is_bit_exact(ws):
    rng = np.random.default_rng(2)
    g = synth.permutation_graph(5001, rng)
    X = rng.standard_normal((g.n, 512)).astype(np.float32)
    out = torch.empty((g.n, 512), dtype=torch.float32, device="cuda")
    B.gcn_aggregate(dcsr(g), dev(X), out, ws)
    assert np.array_equal(out.cpu().numpy().view(np.uint32), X[g.indices].view(np.uint32))


def test_aggregate_constant_features_mean(ws):
    g = synth.custom(4000, "rmat", 20, [(2, 2)], seed=9).graph
    c = np.array([1.5, -3.25, 1000.0, 0.1], np.float32)
    X = np.tile(np.tile(c, 64), (g.n, 1))   # k = 256
    out = torch.empty((g.n, 256), dtype=torch.float32, device="cuda")
    B.gcn_aggregate(dcsr(g), dev(X), out, ws)
    o = out.cpu().numpy()
    deg = g.degrees()
    assert np.all(o[deg == 0] == 0.0)
    nz = deg > 0
    err = np.abs(o[nz] - X[nz]) / np.abs(X[nz])
    assert np.all(err <= (2.0 * deg[nz, None] + 4) * 2.0 ** -23)


@pytest.mark.parametrize("n, k", [(70000, 96), (5, 96), (70000, 512), (3, 512)])
def test_aggregate_long_row_split_over_wavefronts(n, k, ws):
    g = synth.star_graph(n)
    X = np.random.default_rng(4).standard_normal((g.n, k)).astype(np.float32)
    out = torch.empty((g.n, k), dtype=torch.float32, device="cuda")
    B.gcn_aggregate(dcsr(g), dev(X), out, ws)
    ref = oracle.aggregate(g.indptr, g.indices, g.vals, X)
    assert rel_inf(out.cpu().numpy(), ref) <= TOL_F32 / 10


def test_aggregate_empty_graph_and_zero_rows(ws):
    g = synth.empty_graph(1000)
    out = torch.full((1000, 64), 3.0, device="cuda")
    B.gcn_aggregate(dcsr(g), torch.ones((1000, 64), device="cuda"), out, ws)
    assert torch.count_nonzero(out).item() == 0
    g0 = synth.empty_graph(0)
    A0 = B.DeviceCSR(0, 0, torch.zeros(1, dtype=torch.int32, device="cuda"),
                     torch.zeros(0, dtype=torch.int32, device="cuda"),
                     torch.zeros(0, dtype=torch.float32, device="cuda"))
    B.gcn_aggregate(A0, torch.ones((0, 8), device="cuda"), torch.ones((0, 8), device="cuda"), ws)


def test_aggregate_is_deterministic(ws):
    g = synth.custom(20000, "rmat", 30, [(2, 2)], seed=1).graph
    X = dev(np.random.default_rng(0).standard_normal((g.n, 256)).astype(np.float32))
    A = dcsr(g)
    o1 = torch.empty((g.n, 256), device="cuda")
    o2 = torch.empty((g.n, 256), device="cuda")
    B.gcn_aggregate(A, X, o1, ws)
    B.gcn_aggregate(A, X, o2, ws)
    assert torch.equal(o1.view(torch.int32), o2.view(torch.int32))


# ------------------------------------------------------------------ bf16 ----
@pytest.mark.parametrize("k", [64, 128, 200, 256, 264, 384, 512, 602, 1024])
def test_aggregate_bf16(k, ws):
    """Against the oracle on the unrounded inputs (the 2e-2 gate) and, tighter,
    on the bfloat16-rounded inputs (float32 accumulation only)."""
    wl = synth.custom(3001, "rmat", 13, [(2, 2)], seed=k + 7)
    g = wl.graph
    X = np.random.default_rng(k).standard_normal((g.n, k)).astype(np.float32)
    out = torch.empty((g.n, k), dtype=torch.float32, device="cuda")
    B.gcn_aggregate(dcsr(g), dev(X), out, ws, prec=B.GCN_BF16)
    o = out.cpu().numpy()
    assert rel_inf(o, oracle.aggregate(g.indptr, g.indices, g.vals, X)) <= 2e-2
    assert rel_inf(o, oracle.aggregate(g.indptr, g.indices, g.vals, obf16.round_bf16(X))) <= 1e-5


@pytest.mark.parametrize("n, k", [(70000, 96), (70000, 512), (3, 512)])
def test_aggregate_bf16_long_row_split_over_wavefronts(n, k, ws):
    """A 70,000-entry hub row cut over ~270 wavefronts with bfloat16 rows: the
    sliced schedule (512 columns) and the unsliced one (96), each against the
    oracle on the bfloat16-rounded inputs (float32 accumulation only)."""
    g = synth.star_graph(n)
    X = np.random.default_rng(5).standard_normal((g.n, k)).astype(np.float32)
    out = torch.empty((g.n, k), dtype=torch.float32, device="cuda")
    B.gcn_aggregate(dcsr(g), dev(X), out, ws, prec=B.GCN_BF16)
    ref = oracle.aggregate(g.indptr, g.indices, g.vals, obf16.round_bf16(X))
    assert rel_inf(out.cpu().numpy(), ref) <= TOL_F32 / 10


def test_bf16_conversion_bit_exact():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100003).astype(np.float32) * 1e3,
                        np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 3.4e38, 1e-40, -1e-45,
                                  1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8], np.float32)])
    y = B.gcn_f32_to_bf16(dev(x)).cpu().numpy().view(np.uint16)
    assert np.array_equal(y, obf16.f32_to_bf16_bits(x))


# ----------------------------------------------------- device CSR check ----
def first_violation(n_rows, n_cols, nnz, indptr, indices, sorted_):
    """The documented result of gcn_csr_validate, written out row by row."""
    if indptr[0] != 0:
        return 1, 0
    if indptr[n_rows] != nnz:
        return 1, n_rows
    for r in range(n_rows):
        b, e = int(indptr[r]), int(indptr[r + 1])
        if e < b:
            return 2, r
        if b < 0 or e > nnz:
            continue
        for p in range(b, e):
            if not 0 <= indices[p] < n_cols:
                return 3, r
            if sorted_ and p > b and indices[p - 1] >= indices[p]:
                return 4, r
    return 0, 0


@pytest.mark.parametrize("case", ["valid", "unsorted", "duplicate_unsorted_ok", "out_of_range", "negative",
                                  "decreasing", "bad_start", "bad_end", "empty", "no_rows", "two_faults"])
def test_device_validate_matches_row_order_semantics(case):
    g = synth.custom(3000, "rmat", 12, [(4, 4)], seed=5).graph
    n, ip, ix = g.n, g.indptr.copy(), g.indices.copy()
    sorted_ = True
    hub = int(np.argmax(np.diff(ip)))                     # the longest row: many wavefront strides
    if case == "unsorted":
        b = ip[hub]
        ix[b + 100], ix[b + 101] = ix[b + 101], ix[b + 100]
    elif case == "duplicate_unsorted_ok":
        b = ip[hub]
        ix[b + 1] = ix[b]
        sorted_ = False
    elif case == "out_of_range":
        ix[ip[hub] + 70] = n
    elif case == "negative":
        ix[ip[7] if ip[8] > ip[7] else 0] = -3
    elif case == "decreasing":
        ip[1234] = ip[1235] + 1
    elif case == "bad_start":
        ip[0] = 1
    elif case == "bad_end":
        ip[-1] -= 1
    elif case == "empty":
        ip = np.zeros(n + 1, np.int32)
        ix = np.zeros(0, np.int32)
    elif case == "no_rows":
        n, ip, ix = 0, np.zeros(1, np.int32), np.zeros(0, np.int32)
    elif case == "two_faults":                             # the earlier row wins
        ix[ip[hub] + 5] = n + 7
        r = max(0, hub - 3)
        while r > 0 and ip[r + 1] - ip[r] < 2:
            r -= 1
        ix[ip[r] + 1] = ix[ip[r]]
    nnz = int(ix.size)
    want = first_violation(n, max(n, 1) if case == "no_rows" else n, nnz, ip, ix, sorted_)
    A = B.DeviceCSR(n, n, torch.from_numpy(ip).cuda(), torch.from_numpy(ix).cuda(),
                    torch.ones(nnz, dtype=torch.float32, device="cuda"))
    print(f"validate: {case}", flush=True)
    st = B.gcn_csr_validate(A, require_sorted=sorted_)
    got = tuple(int(x) for x in st.cpu())
    assert got == want, (case, got, want)
    if case not in ("decreasing",):   # the host check reads out of range on a decreasing indptr
        host_ok = B.gcn_csr_validate_host(n, n, ip, ix, require_sorted=sorted_) == B.GCN_OK
        assert host_ok == (want[0] == 0)
