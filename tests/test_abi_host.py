"""The C-ABI library on the host: it loads, exports every declared symbol, and
rejects malformed arguments before launching anything (no GPU needed)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_1810_11899_amd import binding as B
from paper_1810_11899_amd import build as pkg_build
from paper_1810_11899_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(pkg_build.LIB_PATH):
        pkg_build.build_library()
    return B.lib()


def declared_functions():
    names = set()
    inc = os.path.join(ROOT, "include")
    for h in sorted(os.listdir(inc)):
        if h.endswith(".h"):
            text = re.sub(r"/\*.*?\*/", "", open(os.path.join(inc, h)).read(), flags=re.S)
            names |= set(re.findall(r"\b(gcn_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) >= 18
    for nm in names:
        assert hasattr(L, nm), nm
    assert set(names) == set(B.exported_symbols())


def test_version(L):
    assert L.gcn_version() >= 100


def test_validate_host_accepts_generated_graph(L):
    g = synth.config(0).graph
    assert B.gcn_csr_validate_host(g.n, g.n, g.indptr, g.indices) == B.GCN_OK


@pytest.mark.parametrize("mutate, msg", [
    (lambda ip, ix: (ip, np.where(np.arange(ix.size) == 3, 10 ** 6, ix)), "outside"),
    (lambda ip, ix: (np.where(np.arange(ip.size) == 5, ip[4] - 1, ip), ix), "decreases"),
    (lambda ip, ix: (ip, np.concatenate([ix[:1], ix[:1], ix[2:]])), "ascending"),
])
def test_validate_host_rejects(L, mutate, msg):
    g = synth.custom(50, "er", 6, [(2, 2)]).graph
    ip, ix = mutate(g.indptr.copy(), g.indices.copy())
    rc = B.gcn_csr_validate_host(g.n, g.n, ip, ix)
    assert rc == B.GCN_EINVAL
    assert msg in L.gcn_last_error().decode()


def test_validate_host_bad_endpoints(L):
    ip = np.array([1, 2, 3], np.int32)
    assert B.gcn_csr_validate_host(2, 2, ip, np.array([0, 1], np.int32)) == B.GCN_EINVAL
    ip = np.array([0, 1, 1], np.int32)
    assert B.gcn_csr_validate_host(2, 2, ip, np.array([0, 1], np.int32)) == B.GCN_EINVAL  # nnz mismatch


def _fake_csr(n, nnz):
    # non-null placeholder addresses: validation must fail before they are used
    return B.gcn_csr(n, n, nnz, 0x1000, 0x2000 if nnz else None, 0x3000 if nnz else None)


def test_layer_fwd_argument_errors(L):
    A = _fake_csr(100, 400)
    P = ctypes.c_void_p
    fake = P(0x4000)

    def fwd(f_in=8, ldh=8, h=4, ldy=8, order=0, prec=0, ws_bytes=1 << 30, saved_bytes=1 << 30, A=A):
        return L.gcn_layer_fwd(ctypes.byref(A), fake, f_in, ldh, fake, fake, fake, h, fake, ldy, fake,
                               saved_bytes, order, prec, fake, ws_bytes, None)

    assert fwd(ldh=7) == B.GCN_ESHAPE
    assert fwd(ldy=7) == B.GCN_ESHAPE
    assert fwd(h=0) == B.GCN_ESHAPE
    assert fwd(order=7) == B.GCN_EINVAL
    assert fwd(prec=9) == B.GCN_EINVAL
    assert fwd(ws_bytes=16) == B.GCN_EWORKSPACE
    assert fwd(saved_bytes=16) == B.GCN_EWORKSPACE
    rect = B.gcn_csr(100, 90, 400, 0x1000, 0x2000, 0x3000)
    assert fwd(A=rect) == B.GCN_ESHAPE
    nullcsr = B.gcn_csr(100, 100, 400, 0x1000, None, 0x3000)
    assert fwd(A=nullcsr) == B.GCN_EINVAL
    assert "null" in L.gcn_last_error().decode()


def test_layer_bwd_transpose_mismatch(L):
    A = _fake_csr(100, 400)
    AT = _fake_csr(100, 399)
    fake = ctypes.c_void_p(0x4000)
    rc = L.gcn_layer_bwd(ctypes.byref(A), ctypes.byref(AT), fake, 8, 8, fake, fake, 4, fake, 8, fake,
                         1 << 30, fake, 8, None, 0, fake, fake, fake, 0, 0, fake, 1 << 30, None)
    assert rc == B.GCN_ESHAPE


def test_loss_argument_errors(L):
    fake = ctypes.c_void_p(0x4000)

    def loss(n=10, f=8, ld=8, C=5, kind=0, labels=fake, targets=None, ws=1 << 30):
        return L.gcn_loss_grad(fake, n, f, ld, fake, fake, C, kind, labels, targets, fake, fake, ld, fake,
                               fake, 0, fake, ws, None)

    assert loss(ld=7) == B.GCN_ESHAPE
    assert loss(kind=5) == B.GCN_EINVAL
    assert loss(labels=None) == B.GCN_EINVAL
    assert loss(kind=1, targets=None) == B.GCN_EINVAL
    assert loss(ws=8) == B.GCN_EWORKSPACE


def test_workspace_queries_are_monotone(L):
    a = L.gcn_layer_workspace_bytes(1000, 10000, 64, 64, 0, 0)
    b = L.gcn_layer_workspace_bytes(2000, 20000, 64, 64, 0, 0)
    assert 0 < a < b
    assert L.gcn_layer_saved_bytes(1000, 64, 32, B.GCN_AGGREGATE_FIRST, 0) >= 1000 * 64 * 4
    assert L.gcn_layer_saved_bytes(1000, 64, 32, B.GCN_TRANSFORM_FIRST, 0) == 0
    assert L.gcn_csr_transpose_workspace_bytes(1000, 1000, 5000) >= 4 * 5000 * 4


def test_pick_order_minimises_aggregation_width(L):
    # first layer (no input gradient): aggregate at f_in when f_in <= 2h
    assert L.gcn_layer_pick_order(512, 512, 0) == B.GCN_AGGREGATE_FIRST
    assert L.gcn_layer_pick_order(602, 128, 0) == B.GCN_TRANSFORM_FIRST
    # with the input gradient: aggregate-first only when f_in < h
    assert L.gcn_layer_pick_order(1024, 512, 1) == B.GCN_TRANSFORM_FIRST
    assert L.gcn_layer_pick_order(50, 64, 1) == B.GCN_AGGREGATE_FIRST


def test_profile_classes(L):
    n = L.gcn_profile_class_count()
    names = [L.gcn_profile_class_name(i).decode() for i in range(n)]
    assert "spmm" in names and "gemm_nn" in names and "gemm_tn" in names
    assert L.gcn_profile_read(n, None, None, None, None) == B.GCN_EINVAL


# ------------------------------------------------------------ sampler ABI ----
def test_sampler_plan_sizes_fit_lds(L):
    g = synth.custom(5000, "rmat", 20, [(4, 4)], seed=1).graph
    for m, cap in [(1000, 30), (200, 0), (64, 5)]:
        p = B.gcn_sampler_plan(g.indptr, m, 4 * m, eta=2.0, cap=cap, seed=3)
        w = np.minimum(g.degrees(), cap) if cap else g.degrees()
        clamped = 12 * p.ia_slots + 2 * p.db_entries > 160 * 1024 - 4
        assert clamped or p.db_entries >= max(int(np.ceil(2.0 * m * w.mean())), m * int(w.max()))
        assert 12 * p.ia_slots + 2 * p.db_entries <= 160 * 1024
        assert m < p.ia_slots <= 65535 and p.m == m and p.n == 4 * m and p.cap == cap and p.seed == 3


def test_sampler_plan_rejects_bad_arguments(L):
    g = synth.custom(500, "rmat", 8, [(4, 4)], seed=1).graph
    with pytest.raises(B.GcnError) as e:
        B.gcn_sampler_plan(g.indptr, 501, 600)
    assert e.value.code == B.GCN_EINVAL
    with pytest.raises(B.GcnError) as e:
        B.gcn_sampler_plan(g.indptr, 10, 100, eta=1.0)
    assert e.value.code == B.GCN_EINVAL
    big = synth.custom(40000, "er", 2, [(4, 4)], seed=1).graph
    with pytest.raises(B.GcnError) as e:
        B.gcn_sampler_plan(big.indptr, 30000, 30000)
    assert e.value.code == B.GCN_EUNSUPPORTED


def test_sampler_entry_points_check_arguments_before_launch(L):
    p = B.gcn_sampler_params(10, 20, 100, 32, 0, 1)
    csr = B.gcn_csr(100, 100, 0, None, None, None)
    assert L.gcn_frontier_sample(ctypes.byref(csr), ctypes.byref(p), 0, 1, None, None, None, None) == B.GCN_EINVAL
    fake = ctypes.c_void_p(256)   # never dereferenced: the shape check fails first
    csr2 = B.gcn_csr(100, 90, 0, fake, None, None)
    assert L.gcn_frontier_sample(ctypes.byref(csr2), ctypes.byref(p), 0, 1, fake, fake, fake, None) == B.GCN_ESHAPE
    p_bad = B.gcn_sampler_params(10, 20, 100, 10, 0, 1)   # ia_slots must exceed m
    csr3 = B.gcn_csr(100, 100, 0, fake, None, None)
    assert L.gcn_frontier_sample(ctypes.byref(csr3), ctypes.byref(p_bad), 0, 1, fake, fake, fake, None) == B.GCN_EINVAL
    assert L.gcn_induce_subgraphs(ctypes.byref(csr3), 1, 10, None, None, None, None, None, None, None, None, None,
                                  0, None, None, 0, None) == B.GCN_EINVAL
    assert L.gcn_gather_rows(fake, 10, 8, 4, fake, 3, fake, 8, None) == B.GCN_ESHAPE
    assert L.gcn_gather_rows(None, 10, 8, 8, None, 0, None, 8, None) == B.GCN_OK   # nothing to do
    assert L.gcn_induce_workspace_bytes(1000, 100, 4) >= 4 * ((1000 + 31) // 32) * 8   # bitmap + prefix per list


def test_pattern_symmetry_check(L):
    g = synth.custom(800, "rmat", 10, [(4, 4)], seed=2).graph
    assert B.gcn_csr_pattern_symmetric_host(g.indptr, g.indices) is True
    d = synth.csr_from_pairs(5, np.array([0, 1, 2]), np.array([1, 2, 0]))   # a directed cycle
    assert B.gcn_csr_pattern_symmetric_host(d.indptr, d.indices) is False
    assert B.gcn_csr_pattern_symmetric_host(synth.empty_graph(4).indptr, np.zeros(0, np.int32)) is True
    with pytest.raises(B.GcnError):
        B.gcn_csr_pattern_symmetric_host(np.array([0, 2], np.int32), np.array([0, 0], np.int32))


def test_transpose_symmetric_checks_arguments(L):
    csr = B.gcn_csr(10, 12, 0, ctypes.c_void_p(256), None, None)
    assert L.gcn_csr_transpose_symmetric(ctypes.byref(csr), None, None, 0, None) == B.GCN_ESHAPE
    assert L.gcn_csr_transpose_symmetric(None, None, None, 0, None) == B.GCN_EINVAL
    sq = B.gcn_csr(10, 10, 5, ctypes.c_void_p(256), ctypes.c_void_p(256), ctypes.c_void_p(256))
    assert L.gcn_csr_transpose_symmetric(ctypes.byref(sq), ctypes.c_void_p(256), None, 0, None) == B.GCN_EWORKSPACE


def _layer_args(f_in, h, ld_extra=0, dH=True):
    f = 0x4000
    return B.gcn_layer_args(f_in, h, B.GCN_AGGREGATE_FIRST, f, f, f, f, 2 * h + ld_extra, f, 1 << 30,
                            f if dH else None, f_in, f, f, f)


def test_model_step_checks_every_call_before_launch(L):
    A = _fake_csr(100, 400)
    fake = ctypes.c_void_p(0x4000)
    head = B.gcn_head_args(0x4000, 0x4000, 5, B.GCN_SOFTMAX_CE, 0x4000, None, 0x4000, 0x4000, 16, 0x4000,
                           0x4000)

    def step(layers, head=head, dY=None, lddy=0, ws=1 << 30):
        arr = (B.gcn_layer_args * len(layers))(*layers)
        hp = None if head is None else ctypes.byref(head)
        return L.gcn_model_step(ctypes.byref(A), ctypes.byref(A), fake, 8, len(layers), arr, hp, dY, lddy, 0,
                                fake, ws, None)

    ok = [_layer_args(8, 4, dH=False), _layer_args(8, 8)]
    assert step([_layer_args(8, 4, dH=False), _layer_args(6, 8)]) == B.GCN_ESHAPE      # 2h != next f_in
    assert "layer 1" in L.gcn_last_error().decode()
    assert step([ok[0], _layer_args(8, 8, dH=False)]) == B.GCN_EINVAL                 # no dH for layer 0
    assert step(ok, head=None) == B.GCN_EINVAL                                         # no head, no dY
    assert step([ok[0], _layer_args(8, 8, ld_extra=-1)]) == B.GCN_ESHAPE               # layer 1's ldy
    assert "gcn_layer_fwd" in L.gcn_last_error().decode()
    bad_head = B.gcn_head_args(0x4000, 0x4000, 5, 7, 0x4000, None, 0x4000, 0x4000, 16, 0x4000, 0x4000)
    assert step(ok, head=bad_head) == B.GCN_EINVAL                                     # the head's kind
    assert step(ok, head=None, dY=fake, lddy=15) == B.GCN_ESHAPE                       # dY narrower than 2h
    assert "gcn_layer_bwd" in L.gcn_last_error().decode()
    assert step(ok, ws=4096) == B.GCN_EWORKSPACE
    assert L.gcn_model_step(ctypes.byref(A), ctypes.byref(A), fake, 8, 0, (B.gcn_layer_args * 1)(), None, fake,
                            8, 0, fake, 1 << 30, None) == B.GCN_EINVAL                # L = 0


def test_model_workspace_is_the_largest_call(L):
    """The model step's workspace is its largest call's, plus the merge-path
    row ranges of A and A^T that it computes once for all of its SpMMs (one
    int32 per wavefront of at least 32 merge items, plus one), plus with
    bfloat16 operands the last layer's output as bfloat16 rows and transposed
    rows for the head (2 x n x 2h bfloat16, each region 256-byte aligned) and
    the step's weights converted up front: W_self^T and W_neigh^T of every
    layer, W_self and W_neigh of a layer with an input gradient, W_pred padded
    to 64 classes and W_pred^T."""
    layers = (B.gcn_layer_args * 2)(_layer_args(602, 128, dH=False), _layer_args(256, 128))
    head = B.gcn_head_args(0x4000, 0x4000, 41, B.GCN_SOFTMAX_CE, 0x4000, None, 0x4000, 0x4000, 256, 0x4000,
                           0x4000)
    n, nnz = 8000, 120000
    ranges = 2 * ((((n + nnz) // 32 + 2) * 4 + 255) // 256 * 256)
    for prec in (B.GCN_F32, B.GCN_BF16):
        need = L.gcn_model_workspace_bytes(n, nnz, 2, layers, ctypes.byref(head), prec)
        parts = [L.gcn_layer_workspace_bytes(n, nnz, 602, 128, B.GCN_AGGREGATE_FIRST, prec),
                 L.gcn_layer_workspace_bytes(n, nnz, 256, 128, B.GCN_AGGREGATE_FIRST, prec),
                 L.gcn_loss_workspace_bytes(n, 256, 41, prec)]
        a256 = lambda b: (b + 255) // 256 * 256
        hl16 = 2 * a256(n * 256 * 2) if prec == B.GCN_BF16 else 0
        w16 = (2 * a256(602 * 128 * 2) + 4 * a256(256 * 128 * 2) + a256(256 * 64 * 2) + a256(256 * 41 * 2)
               if prec == B.GCN_BF16 else 0)
        assert max(parts) + hl16 + w16 < need <= max(parts) + ranges + hl16 + w16


def test_device_validate_checks_arguments_before_launch(L):
    A = _fake_csr(10, 20)
    st = ctypes.c_void_p(0x4000)
    assert L.gcn_csr_validate(None, 1, st, None) == B.GCN_EINVAL
    assert L.gcn_csr_validate(ctypes.byref(A), 1, None, None) == B.GCN_EINVAL
    assert L.gcn_csr_validate(ctypes.byref(A), 1, ctypes.c_void_p(0x4004), None) == B.GCN_EINVAL
    assert "aligned" in L.gcn_last_error().decode()
    bad = B.gcn_csr(10, 10, 20, 0x1000, None, 0x3000)
    assert L.gcn_csr_validate(ctypes.byref(bad), 1, st, None) == B.GCN_EINVAL


def test_uint16_indices_host_checks(L):
    """uint16 indices: only for n_cols <= 65536, never together with int32
    indices, and refused by the sampler (its G is larger); all before any launch."""
    import ctypes
    p = ctypes.c_void_p(256)
    big = B.gcn_csr(70000, 70000, 10, p, None, p, p)
    both = B.gcn_csr(100, 100, 10, p, p, p, p)
    ok16 = B.gcn_csr(100, 100, 10, p, None, p, p)
    X = ctypes.c_void_p(256)
    for csr, code in ((big, B.GCN_ESHAPE), (both, B.GCN_EINVAL)):
        assert L.gcn_aggregate(ctypes.byref(csr), X, 4, 4, X, 4, B.GCN_F32, X, 1 << 30, None) == code
    assert L.gcn_aggregate(ctypes.byref(ok16), X, 4, 4, X, 4, B.GCN_F32, X, 0, None) == B.GCN_EWORKSPACE
    params = B.gcn_sampler_params(2, 4, 64, 8, 0, 1)
    assert L.gcn_frontier_sample(ctypes.byref(ok16), ctypes.byref(params), 0, 1, X, X, X, None) == B.GCN_ESHAPE
