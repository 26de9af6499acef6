"""Sampler, induced-subgraph and gather kernels on the GPU, through the C ABI,
against the CPU oracle.  Integer outputs must match bit for bit: both sides
draw the same Philox4x64-10 numbers and take the same decisions."""
import numpy as np
import pytest
import torch

from oracle import sampler as OS
from paper_1810_11899_amd import binding as B
from paper_1810_11899_amd import synth

from gpu_util import require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


@pytest.fixture(scope="module")
def ws():
    return B.Workspace("cuda")


def dcsr(g):
    return B.DeviceCSR.from_host(g.n, g.n, g.indptr, g.indices, g.vals)


def run_and_compare(g, params, S, first=0):
    """GPU runs first .. first+S-1 against the oracle, run by run."""
    G = dcsr(g)
    print(f"sampler: n_vertices={g.n} nnz={g.nnz} m={params.m} n={params.n} db={params.db_entries} "
          f"ia={params.ia_slots} cap={params.cap} S={S}", flush=True)
    v, c, st = B.gcn_frontier_sample(G, params, first, S)
    torch.cuda.synchronize()
    v, c, st = v.cpu().numpy(), c.cpu().numpy(), st.cpu().numpy()
    outs = []
    for r in range(S):
        ov, ost = OS.frontier_sample(g.indptr, g.indices, params.m, params.n, params.db_entries, params.ia_slots,
                                     cap=params.cap, p=64, seed=params.seed, sampler_id=first + r)
        assert B.SAMPLE_STATUS[int(st[r])] == ost, (r, st[r], ost)
        assert int(c[r]) == ov.size, (r, c[r], ov.size)
        assert np.array_equal(v[r, :c[r]], ov), f"run {r}: first difference at {np.argmax(v[r, :c[r]] != ov)}"
        outs.append(ov)
    return v, c, st, outs


def params_for(g, m, n, eta=2.0, cap=0, seed=1, db=None, ia=None):
    p = B.gcn_sampler_plan(g.indptr, m, n, eta=eta, cap=cap, seed=seed)
    if db is not None:
        p.db_entries = db
    if ia is not None:
        p.ia_slots = ia
    return p


# ------------------------------------------------------------- sampling ----
@pytest.mark.parametrize("cap", [30, 0])
def test_frontier_rmat_matches_oracle(cap):
    g = synth.training_graph(20000, 30, 4, 3, seed=1).graph
    p = params_for(g, 300, 2500, cap=cap, seed=7)
    _, c, st, _ = run_and_compare(g, p, 6, first=11)
    assert np.all(st == 0) and np.all(c == 2500)


def test_frontier_paper_scale_matches_oracle():
    """m = 1000 roots, budget 8000 (the paper's frontier size and subgraph scale)."""
    g = synth.training_graph(100000, 40, 4, 3, seed=2).graph
    p = params_for(g, 1000, 8000, eta=2.0, cap=30, seed=3)
    _, c, st, _ = run_and_compare(g, p, 4)
    assert np.all(st == 0)


def test_frontier_constant_cleanups_match_oracle():
    """Dashboard and Index Array barely larger than a frontier: a cleanup
    before nearly every append."""
    g = synth.custom(2000, "rmat", 12, [(4, 4)], seed=4).graph
    m = 50
    wmax = int(np.minimum(g.degrees(), 20).max())
    p = params_for(g, m, 1200, cap=20, seed=9, db=m * wmax, ia=m + 1)
    run_and_compare(g, p, 5)


def test_frontier_directed_graph_runs_dry():
    # a directed cycle 0 -> 1 -> ... -> 99 -> 0 plus sinks 100..149 reached from even vertices
    src = list(range(100)) + list(range(0, 100, 2))
    dst = [(i + 1) % 100 for i in range(100)] + list(range(100, 150))
    g = synth.csr_from_pairs(150, np.array(src), np.array(dst))
    p = params_for(g, 5, 400, seed=5, db=64, ia=16)
    _, _, st, _ = run_and_compare(g, p, 16)
    assert np.any(st == 1)     # some runs end with every frontier vertex a sink


def test_frontier_degenerate_cases():
    e = synth.empty_graph(500)
    _, c, st, _ = run_and_compare(e, params_for(e, 40, 100, seed=1, db=8, ia=64), 3)
    assert np.all(st == 1) and np.all(c == 40)
    k = synth.complete_graph(64)
    run_and_compare(k, params_for(k, 64, 300, seed=2, db=64 * 63, ia=65), 2)      # every vertex a root
    _, c, st, _ = run_and_compare(k, params_for(k, 8, 300, seed=2, db=8 * 63 - 1, ia=64), 2)
    assert np.all(st == 2) and np.all(c == 8)                                     # roots overflow
    _, c, st, _ = run_and_compare(k, params_for(k, 8, 8, seed=2), 2)              # no steps
    assert np.all(st == 0) and np.all(c == 8)
    s = synth.star_graph(3000)                                                     # one hub
    run_and_compare(s, params_for(s, 100, 900, seed=4), 3)


def test_frontier_is_deterministic_and_run_id_keyed():
    g = synth.custom(3000, "rmat", 16, [(4, 4)], seed=6).graph
    p = params_for(g, 100, 700, cap=16, seed=1)
    G = dcsr(g)
    a = B.gcn_frontier_sample(G, p, 0, 6)[0].cpu()
    b = B.gcn_frontier_sample(G, p, 0, 6)[0].cpu()
    c = B.gcn_frontier_sample(G, p, 3, 3)[0].cpu()
    assert torch.equal(a, b) and torch.equal(a[3:], c)


# ------------------------------------------------------ induced subgraphs ----
def check_induced(g, verts, counts, ib):
    n_sub = ib.n_sub.cpu().numpy()
    off = ib.edge_offsets.cpu().numpy()
    vsub = ib.vsub.cpu().numpy()
    ip = ib.indptr.cpu().numpy()
    ix = ib.indices.cpu().numpy()
    vv = ib.vals.cpu().numpy()
    for s in range(ib.S):
        v = verts[s, :counts[s]]
        v = v[(v >= 0) & (v < g.n)]                 # ids outside G are skipped (gcn_sampler.h)
        ov, oip, oix, ovals = OS.induce(g.indptr, g.indices, v)
        ns = int(n_sub[s])
        assert ns == ov.size
        assert np.array_equal(vsub[s, :ns], ov)
        assert np.array_equal(ip[s, :ns + 1], oip)
        assert np.all(ip[s, ns:] == oip[-1])
        e0, e1 = int(off[s]), int(off[s + 1])
        assert e1 - e0 == oix.size
        assert np.array_equal(ix[e0:e1], oix)
        assert np.array_equal(vv[e0:e1].view(np.uint32), ovals.view(np.uint32))


def test_induce_sampled_subgraphs_bit_exact(ws):
    g = synth.training_graph(20000, 30, 4, 3, seed=1).graph
    p = params_for(g, 300, 2500, cap=30, seed=7)
    S = 5
    v, c, st = B.gcn_frontier_sample(dcsr(g), p, 0, S)
    ib = B.InducedBatch(S, p.n, 4_000_000, "cuda", with_transpose=True)
    print("induce: S=5 n=2500", flush=True)
    B.gcn_induce_subgraphs(dcsr(g), v, c, ib, ws)
    torch.cuda.synchronize()
    assert int(ib.status.item()) == 0
    check_induced(g, v.cpu().numpy(), c.cpu().numpy(), ib)
    # G is symmetric, so the transposed values make the transpose of each
    # subgraph's aggregation matrix: the same as the CSR transpose, bit for bit
    assert B.gcn_csr_pattern_symmetric_host(g.indptr, g.indices)
    n_sub = ib.n_sub.cpu().numpy()
    off = ib.edge_offsets.cpu().numpy()
    for s in range(S):
        A = ib.csr(s, int(n_sub[s]), int(off[s]), int(off[s + 1]))
        AT = B.gcn_csr_transpose(A, ws)
        ATs = ib.csr_t(s, int(n_sub[s]), int(off[s]), int(off[s + 1]))
        torch.cuda.synchronize()
        assert torch.equal(AT.indptr, ATs.indptr) and torch.equal(AT.indices, ATs.indices)
        assert torch.equal(AT.vals.view(torch.int32), ATs.vals.view(torch.int32))


def test_induce_edge_cases_and_capacity(ws):
    g = synth.custom(3000, "rmat", 10, [(4, 4)], seed=3).graph
    rng = np.random.default_rng(0)
    S, n = 4, 700
    verts = rng.integers(0, g.n, (S, n)).astype(np.int32)   # duplicates on purpose
    verts[1, :] = 17                                          # one vertex only
    counts = np.array([n, n, 0, 333], np.int32)               # an empty list, a short one
    V, C = torch.from_numpy(verts).cuda(), torch.from_numpy(counts).cuda()
    small = B.InducedBatch(S, n, 10, "cuda")
    B.gcn_induce_subgraphs(dcsr(g), V, C, small, ws)
    torch.cuda.synchronize()
    assert int(small.status.item()) == 1                     # too small: nothing written
    need = int(small.edge_offsets[-1].item())
    ib = B.InducedBatch(S, n, need, "cuda")
    B.gcn_induce_subgraphs(dcsr(g), V, C, ib, ws)
    torch.cuda.synchronize()
    assert int(ib.status.item()) == 0
    check_induced(g, verts, counts, ib)


def test_induce_large_graph_table_outside_lds(ws):
    """G of 600,000 vertices: a list's bitmap and prefix (8 bytes per 32
    vertices, 150 KB) exceed what the row kernels hold in LDS, so they read
    them from memory.  Lists: a contiguous range, one wrapping the end of the
    vertex range, a random one with duplicates, one with out-of-range ids."""
    nV = 600_000
    g = synth.circulant_graph(nV, [1, 2, 3, 1000])
    rng = np.random.default_rng(5)
    S, n = 4, 3000
    verts = np.empty((S, n), np.int32)
    verts[0] = np.arange(n)
    verts[1] = (nV - 1500 + np.arange(n)) % nV
    verts[2] = rng.integers(nV - 40_000, nV, n)
    verts[3] = rng.integers(0, 5000, n)
    verts[3, ::7] = -5
    verts[3, 3::7] = nV
    counts = np.array([n, n, n, 2500], np.int32)
    V, C = torch.from_numpy(verts).cuda(), torch.from_numpy(counts).cuda()
    ib = B.InducedBatch(S, n, 200_000, "cuda", with_transpose=True)
    print("induce: nV=600000 S=4 n=3000", flush=True)
    B.gcn_induce_subgraphs(dcsr(g), V, C, ib, ws)
    torch.cuda.synchronize()
    assert int(ib.status.item()) == 0
    check_induced(g, verts, counts, ib)
    assert int(ib.edge_offsets[1].item()) > 0


# ----------------------------------------------------------------- gather ----
@pytest.mark.parametrize("width", [602, 512, 1])
def test_gather_rows_bit_exact(width):
    rng = np.random.default_rng(width)
    X = rng.standard_normal((5000, width)).astype(np.float32)
    rows = rng.integers(0, 5000, 3001).astype(np.int32)
    rows[7] = -1
    rows[8] = 5000                                            # out of range: zero rows
    Xd, Rd = torch.from_numpy(X).cuda(), torch.from_numpy(rows).cuda()
    out = torch.full((3001, width), 9.0, device="cuda")
    B.gcn_gather_rows(Xd, Rd, 3001, out)
    o = out.cpu().numpy()
    ok = (rows >= 0) & (rows < 5000)
    assert np.array_equal(o[ok].view(np.uint32), OS.gather_rows(X, rows[ok]).view(np.uint32))
    assert np.all(o[~ok] == 0.0)


def test_gather_labels_int32():
    labels = np.arange(1000, dtype=np.int32) * 7 % 41
    rows = np.array([5, 999, 0, 5, 123], np.int32)
    out = torch.empty(5, dtype=torch.int32, device="cuda")
    B.gcn_gather_rows(torch.from_numpy(labels).cuda(), torch.from_numpy(rows).cuda(), 5, out)
    assert np.array_equal(out.cpu().numpy(), labels[rows])
