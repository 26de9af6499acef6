"""Layer, loss and whole-step parity on the GPU, through the C ABI, against the
CPU oracle on the same seeded inputs."""
import numpy as np
import pytest
import torch

import oracle
from paper_1810_11899_amd import binding as B
from paper_1810_11899_amd import synth
from paper_1810_11899_amd.runner import StepRunner

from gpu_util import TOL_BF16, TOL_F32, dev, rel_inf, require_gpu

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


def _bias(h, seed):
    return (np.random.default_rng(seed).standard_normal(2 * h) * 0.3).astype(np.float32)


SHAPES = [(777, "rmat", 9, 37, 24), (1500, "er", 12, 64, 48), (2049, "rmat", 15, 130, 100),
          (1000, "rmat", 11, 256, 128), (900, "rmat", 10, 264, 256), (1024, "rmat", 9, 96, 64),
          (2048, "er", 8, 128, 100),
          # bf16 forward products on the large-tile kernel with 1, 2 and 3
          # k-tiles of 32 (the pipeline's prologue and tail without a steady state)
          (1100, "rmat", 9, 32, 160), (700, "er", 8, 64, 200), (600, "rmat", 7, 96, 136)]


PRECS = [(B.GCN_F32, TOL_F32), (B.GCN_BF16, TOL_BF16)]


@pytest.mark.parametrize("prec, tol", PRECS)
@pytest.mark.parametrize("order", [B.GCN_AGGREGATE_FIRST, B.GCN_TRANSFORM_FIRST])
@pytest.mark.parametrize("shape", SHAPES)
def test_layer_forward(prec, tol, order, shape, ws):
    n, kind, d, f_in, h = shape
    wl = synth.custom(n, kind, d, [(f_in, h)], seed=f_in)
    lay = wl.layers[0]
    b = _bias(h, n)
    A = dcsr(wl.graph)
    Y = torch.empty((n, 2 * h), device="cuda")
    nb = B.gcn_layer_saved_bytes(n, f_in, h, order, prec)
    saved = torch.empty(max(nb, 1), dtype=torch.uint8, device="cuda") if nb else None
    B.gcn_layer_fwd(A, dev(wl.H), dev(lay.W_self), dev(lay.W_neigh), dev(b), Y, saved, order, ws, prec)
    Yref, _ = oracle.layer_fwd(wl.graph, wl.H, lay.W_self, lay.W_neigh, b)
    assert rel_inf(Y.cpu().numpy(), Yref) <= tol


@pytest.mark.parametrize("prec, tol", PRECS)
@pytest.mark.parametrize("order", [B.GCN_AGGREGATE_FIRST, B.GCN_TRANSFORM_FIRST])
@pytest.mark.parametrize("want_dH", [True, False])
@pytest.mark.parametrize("shape", SHAPES)
def test_layer_backward(prec, tol, order, want_dH, shape, ws):
    """float32: the backward runs on the GPU's own forward output, with the
    oracle's kink envelope.  bfloat16 (rounding far coarser than any kink
    band worth modelling): the backward receives the oracle's Y, so both sides
    take every ReLU branch on the same sign, and the gate is strict."""
    n, kind, d, f_in, h = shape
    wl = synth.custom(n, kind, d, [(f_in, h)], seed=f_in + 1)
    lay = wl.layers[0]
    b = _bias(h, n + 1)
    g = wl.graph
    A = dcsr(g)
    AT = B.gcn_csr_transpose(A, ws)
    H = dev(wl.H)
    Ws, Wn = dev(lay.W_self), dev(lay.W_neigh)
    Y = torch.empty((n, 2 * h), device="cuda")
    nb = B.gcn_layer_saved_bytes(n, f_in, h, order, prec)
    saved = torch.empty(max(nb, 1), dtype=torch.uint8, device="cuda") if nb else None
    B.gcn_layer_fwd(A, H, Ws, Wn, dev(b), Y, saved, order, ws, prec)
    Yref, cache = oracle.layer_fwd(g, wl.H, lay.W_self, lay.W_neigh, b, ambiguity=True)
    if prec == B.GCN_BF16:
        Y32 = Yref.astype(np.float32)
        assert np.array_equal(Y32 > 0, cache.Z > 0)
        Y = dev(Y32)
    dY = np.random.default_rng(n).standard_normal((n, 2 * h)).astype(np.float32)
    dH = torch.empty((n, f_in), device="cuda") if want_dH else None
    dWs = torch.empty((f_in, h), device="cuda")
    dWn = torch.empty((f_in, h), device="cuda")
    db = torch.empty(2 * h, device="cuda")
    B.gcn_layer_bwd(A, AT, H, Ws, Wn, Y, saved, dev(dY), dH, dWs, dWn, db, order, ws, prec)
    ti, tj, tv = oracle.csr_transpose(g.n, g.n, g.indptr, g.indices, g.vals)
    gT = synth.Graph(g.n, ti, tj, tv)
    rWs, rWn, rdb, rdH = oracle.layer_bwd(gT, cache, lay.W_self, lay.W_neigh, dY, want_dH)
    if prec == B.GCN_BF16:
        eWs = eWn = edb = edH = None
    else:
        eWs, eWn, edb, edH = oracle.layer_bwd_envelope(gT, cache, lay.W_self, lay.W_neigh, dY, None, want_dH)
    assert rel_inf(dWs.cpu().numpy(), rWs, eWs) <= tol
    assert rel_inf(dWn.cpu().numpy(), rWn, eWn) <= tol
    assert rel_inf(db.cpu().numpy(), rdb, edb) <= tol
    if want_dH:
        assert rel_inf(dH.cpu().numpy(), rdH, edH) <= tol


@pytest.mark.parametrize("prec, tol", PRECS)
@pytest.mark.parametrize("kind", ["ce", "bce"])
# (the head's grouped row kernel takes up to 128 classes, 16 rows per block:
# 257 and 5 rows leave part of a block empty, 128 classes fill its lanes,
# 150 classes take the one-wavefront-per-row kernel and the separate sums)
@pytest.mark.parametrize("n, f, C", [(3000, 256, 41), (1001, 130, 100), (257, 64, 7), (513, 96, 128), (700, 64, 150),
                                     (5, 32, 3)])
def test_loss_grad(prec, tol, kind, n, f, C, ws):
    rng = np.random.default_rng(n + C)
    HL = np.maximum(rng.standard_normal((n, f)), 0).astype(np.float32)
    Wp = (rng.standard_normal((f, C)) * 0.2).astype(np.float32)
    bp = (rng.standard_normal(C) * 0.1).astype(np.float32)
    labels = rng.integers(0, C, n).astype(np.int32)
    targets = (rng.random((n, C)) < 0.1).astype(np.float32)
    loss = torch.empty(1, device="cuda")
    dHL = torch.empty((n, f), device="cuda")
    dWp = torch.empty((f, C), device="cuda")
    dbp = torch.empty(C, device="cuda")
    B.gcn_loss_grad(dev(HL), dev(Wp), dev(bp), B.LOSS_KIND[kind], dev(labels, torch.int32),
                    dev(targets) if kind == "bce" else None, loss, dHL, dWp, dbp, ws, prec)
    rl, rdWp, rdbp, rdHL, _ = oracle.loss_grad(kind, HL, Wp, bp, labels=labels, targets=targets)
    assert abs(loss.item() - rl) / abs(rl) <= tol
    assert rel_inf(dWp.cpu().numpy(), rdWp) <= tol
    assert rel_inf(dbp.cpu().numpy(), rdbp) <= tol
    assert rel_inf(dHL.cpu().numpy(), rdHL) <= tol


# ------------------------------------------------------------ whole steps ----
def compare_step(run: dict, ref: oracle.StepResult, tol=TOL_F32):
    """Every output of a step: integer transpose bit-exact; floats within
    ``tol`` (infinity-norm relative), gradients beyond the ReLU-kink envelope
    when the oracle carries one."""
    errs = {}
    assert np.array_equal(run["t_indptr"], ref.t_indptr)
    assert np.array_equal(run["t_indices"], ref.t_indices)
    assert np.array_equal(run["t_vals"].view(np.uint32), np.asarray(ref.t_vals, np.float32).view(np.uint32))
    env = ref.E_dW_self is not None
    for li in range(len(ref.Y)):
        errs[f"Y{li}"] = rel_inf(run["Y"][li], ref.Y[li])
        errs[f"dW_self{li}"] = rel_inf(run["dW_self"][li], ref.dW_self[li], ref.E_dW_self[li] if env else None)
        errs[f"dW_neigh{li}"] = rel_inf(run["dW_neigh"][li], ref.dW_neigh[li],
                                        ref.E_dW_neigh[li] if env else None)
        errs[f"db{li}"] = rel_inf(run["db"][li], ref.db[li], ref.E_db[li] if env else None)
        if ref.dH[li] is not None and run["dH"][li] is not None:
            errs[f"dH{li}"] = rel_inf(run["dH"][li], ref.dH[li], ref.E_dH[li] if env else None)
    if ref.loss is not None:
        errs["loss"] = abs(run["loss"] - ref.loss) / abs(ref.loss)
        errs["dW_pred"] = rel_inf(run["dW_pred"], ref.dW_pred)
        errs["db_pred"] = rel_inf(run["db_pred"], ref.db_pred)
        if run["dHL"] is not None:
            errs["dHL"] = rel_inf(run["dHL"], ref.dHL)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, f"over tolerance {tol}: {bad}"
    return errs


def check_bf16_decisions(Y_gpu, masks, wl):
    """The forward of a bfloat16 chain against the oracle's, entry by entry:
    |Y_gpu - max(Z, 0)| <= 16 * 2^-8 * M and every ReLU decision that differs
    from the oracle's at an entry with |Z| <= 16 * 2^-8 * M, where M is the
    sum of the magnitudes of Z's terms with each layer's input magnitude taken
    as the M of the layer below (|H0| for the first).  Each layer rounds its
    input, both weights and the neighbour operand (at most 3 units of 2^-8 of
    M) and passes on the deviation of its input (at most the lower layer's
    bound, carried through the same magnitudes), so 16 units hold for up to
    five layers.  Returns the largest deviation in units of 2^-8 M and the
    number of decisions per layer that differ from the oracle's."""
    u, C = 2.0 ** -8, 16.0
    g = wl.graph
    absA = np.abs(g.vals.astype(np.float64))
    H, Min, worst, nflip = wl.H, np.abs(wl.H.astype(np.float64)), 0.0, []
    for li, lay in enumerate(wl.layers):
        Yref, c = oracle.layer_fwd(g, H, lay.W_self, lay.W_neigh, lay.bias)
        mag = np.concatenate([Min @ np.abs(lay.W_self.astype(np.float64)),
                              oracle.aggregate(g.indptr, g.indices, absA, Min) @ np.abs(lay.W_neigh.astype(np.float64))],
                             axis=1) + np.abs(lay.bias.astype(np.float64))[None, :]
        band = C * u * mag
        dev_ = np.abs(np.asarray(Y_gpu[li], np.float64) - Yref)
        assert np.all(dev_ <= band), ("forward deviation beyond the rounding bound", li)
        flips = np.asarray(masks[li], bool) != (c.Z > 0)
        assert np.all(np.abs(c.Z[flips]) <= band[flips]), ("a ReLU decision rounding cannot explain", li)
        nflip.append(int(flips.sum()))
        worst = max(worst, float(np.divide(dev_, u * mag, out=np.zeros_like(dev_), where=mag > 0).max()))
        H, Min = Yref, mag
    return worst, nflip


def compare_bf16_chain(r: StepRunner, wl, first_layer_dH=None):
    """The bfloat16 model step as the benchmark runs it (one gcn_model_step:
    fused masked epilogues, dZ kept as bfloat16 rows between layers) against
    the float64 oracle on the unrounded inputs.  The bfloat16 rounding decides
    some near-zero ReLU branches differently from float64; each such decision
    is a correct result of the bfloat16 computation, so (a) every decision is
    checked to be one that rounding explains, entry by entry, and (b) the
    oracle then takes the GPU's decisions (its gated network, Y = Z * m,
    dZ = dY * m, m = [bf16(Y) > 0], the bfloat16 path's ReLU rule) and every
    output -- each layer's Y, the loss, every gradient -- is compared at 2e-2
    with no allowance."""
    from oracle import bf16 as obf16
    got = r.results()
    masks = [obf16.round_bf16(y) > 0 for y in got["Y"]]
    worst, nflip = check_bf16_decisions(got["Y"], masks, wl)
    ref = oracle.step(wl, first_layer_dH=first_layer_dH, masks=masks)
    errs = compare_step(got, ref, tol=TOL_BF16)
    errs["forward_units"] = worst
    errs["decisions_differing_from_float64"] = nflip
    return errs, ref


@pytest.mark.parametrize("cfg", [1, 2])
def test_config_step_parity_bf16_chain(cfg):
    wl = synth.config(cfg)
    r = StepRunner(wl, prec=B.GCN_BF16)
    print(f"bf16 chained step, workload {cfg}", flush=True)
    r.step()
    torch.cuda.synchronize()
    errs, _ = compare_bf16_chain(r, wl)
    print("bf16 chain:", errs)


@pytest.mark.parametrize("order", [B.GCN_AGGREGATE_FIRST, B.GCN_TRANSFORM_FIRST])
def test_bf16_weight_gradients_from_row_major_operands(order):
    """Weight gradients read H, AGG, dZ and G as the layer keeps them (n rows,
    k-major for the product) on the large-tile kernel, both orders, two
    layers; the chained step against the oracle."""
    wl = synth.custom(4096, "rmat", 10, [(256, 256), (512, 192)], head="ce", classes=20, seed=7)
    r = StepRunner(wl, prec=B.GCN_BF16, orders=[order, order], first_layer_dH=True)
    print(f"bf16 row-major weight gradients, order {order}", flush=True)
    B.gcn_profile_reset()
    B.gcn_profile_enable(True)
    r.step()
    torch.cuda.synchronize()
    B.gcn_profile_enable(False)
    prof = B.gcn_profile_read_all()
    assert prof["gemm_tn_bf16_big"][1] == 2, prof
    errs, _ = compare_bf16_chain(r, wl, first_layer_dH=True)
    print("bf16 chain:", errs)


@pytest.mark.parametrize("prec", [B.GCN_F32, B.GCN_BF16])
@pytest.mark.parametrize("order", [B.GCN_AGGREGATE_FIRST, B.GCN_TRANSFORM_FIRST])
def test_zero_vertex_subgraph(prec, order, ws):
    """n = 0: every call succeeds; the gradients and the loss are sums over no
    rows, so they come out as zeros (written over NaN-filled buffers)."""
    f_in, h, C = 48, 32, 9
    rng = np.random.default_rng(5)
    A = B.DeviceCSR.from_host(0, 0, np.zeros(1, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))
    AT = B.gcn_csr_transpose(A, ws)
    assert AT.nnz == 0 and AT.indptr.cpu().tolist() == [0]
    e = lambda *shape: torch.empty(shape, device="cuda")
    nan = lambda *shape: torch.full(shape, float("nan"), device="cuda")
    Ws, Wn = dev(rng.standard_normal((f_in, h)) * 0.1), dev(rng.standard_normal((f_in, h)) * 0.1)
    b = dev(_bias(h, 1))
    H, Y = e(0, f_in), e(0, 2 * h)
    nb = B.gcn_layer_saved_bytes(0, f_in, h, order, prec)
    saved = torch.empty(max(nb, 1), dtype=torch.uint8, device="cuda") if nb else None
    B.gcn_layer_fwd(A, H, Ws, Wn, b, Y, saved, order, ws, prec)
    dWs, dWn, db = nan(f_in, h), nan(f_in, h), nan(2 * h)
    B.gcn_layer_bwd(A, AT, H, Ws, Wn, Y, saved, e(0, 2 * h), e(0, f_in), dWs, dWn, db, order, ws, prec)
    Wp, bp = dev(rng.standard_normal((2 * h, C)) * 0.1), dev(np.zeros(C, np.float32))
    loss, dWp, dbp = nan(1), nan(2 * h, C), nan(C)
    B.gcn_loss_grad(Y, Wp, bp, B.GCN_SOFTMAX_CE, torch.empty(0, dtype=torch.int32, device="cuda"), None, loss,
                    e(0, 2 * h), dWp, dbp, ws, prec)
    torch.cuda.synchronize()
    for name, t in (("dW_self", dWs), ("dW_neigh", dWn), ("dbias", db), ("loss", loss), ("dW_pred", dWp),
                    ("db_pred", dbp)):
        assert torch.count_nonzero(t).item() == 0 and not torch.isnan(t).any().item(), name


@pytest.mark.parametrize("cfg", [0, 1, 2])
def test_config_step_parity(cfg):
    wl = synth.config(cfg)
    r = StepRunner(wl)
    r.step()
    torch.cuda.synchronize()
    compare_step(r.results(), oracle.step(wl, envelope=True))


def test_step_is_deterministic():
    wl = synth.config(1)
    r = StepRunner(wl)
    r.step()
    a = r.results()
    r.step()
    b = r.results()
    for key in ("Y", "dW_self", "dW_neigh", "db"):
        for x, y in zip(a[key], b[key]):
            assert np.array_equal(x.view(np.uint32), y.view(np.uint32)), key
    assert a["loss"] == b["loss"]


@pytest.mark.parametrize("order", [B.GCN_AGGREGATE_FIRST, B.GCN_TRANSFORM_FIRST])
def test_forced_orders_agree_with_oracle(order):
    wl = synth.custom(3000, "rmat", 12, [(96, 64), (128, 64)], head="bce", classes=30, seed=2)
    r = StepRunner(wl, orders=[order, order], first_layer_dH=True)
    r.step()
    torch.cuda.synchronize()
    compare_step(r.results(), oracle.step(wl, first_layer_dH=True, envelope=True))


@pytest.mark.parametrize("case", ["cfg1-f32", "cfg1-bf16", "cfg2-bf16", "dY-f32", "bce-transform-first",
                                  "f32-odd-widths", "bf16-odd-widths", "bf16-odd-wide", "bf16-row-major-dw",
                                  "cfg3-f32", "cfg3-bf16"])
def test_model_step_matches_separate_calls(case):
    """gcn_model_step computes what the separate calls compute: every output
    bit for bit, except that a layer whose dZ arrives from the head or from an
    unsplit input-gradient product (masked in that product's epilogue) has its
    bias gradient summed there, in another order.  The inter-layer gradient
    buffers then hold the separate calls' gradient times [input > 0] (as
    packed bfloat16 rows with bfloat16 operands), or that gradient itself."""
    if case.startswith("cfg"):
        wl = synth.config(int(case[3]))
        orders = [B.GCN_AGGREGATE_FIRST, B.GCN_TRANSFORM_FIRST] if case[3] == "3" else None   # the bench's
        r = StepRunner(wl, prec=B.GCN_BF16 if case.endswith("bf16") else B.GCN_F32, orders=orders)
    elif case == "dY-f32":
        wl = synth.custom(2500, "rmat", 10, [(64, 32), (64, 48)], head=None, seed=4)
        r = StepRunner(wl, first_layer_dH=True)
    elif case.endswith("odd-widths"):   # ragged tiles, widths not a multiple of 4 (scalar mask loads)
        wl = synth.custom(2999, "rmat", 9, [(70, 51), (102, 50)], head="ce", classes=13, seed=5)
        r = StepRunner(wl, prec=B.GCN_BF16 if case.startswith("bf16") else B.GCN_F32,
                       orders=[B.GCN_TRANSFORM_FIRST] * 2, first_layer_dH=True)
    elif case == "bf16-row-major-dw":   # weight gradients on k-major operands, aggregate-first
        wl = synth.custom(4096, "rmat", 10, [(256, 256), (512, 192)], head="ce", classes=20, seed=7)
        r = StepRunner(wl, prec=B.GCN_BF16, orders=[B.GCN_AGGREGATE_FIRST] * 2, first_layer_dH=True)
    elif case == "bf16-odd-wide":   # masked input gradient on the large-tile kernel, 150-wide mask rows
        wl = synth.custom(2999, "rmat", 9, [(300, 75), (150, 64)], head="ce", classes=13, seed=6)
        r = StepRunner(wl, prec=B.GCN_BF16, orders=[B.GCN_TRANSFORM_FIRST] * 2, first_layer_dH=True)
    else:
        wl = synth.custom(3000, "rmat", 12, [(96, 64), (128, 64)], head="bce", classes=30, seed=2)
        r = StepRunner(wl, orders=[B.GCN_TRANSFORM_FIRST] * 2, first_layer_dH=True)
    print(f"model step vs calls: {case}", flush=True)
    r.step_calls()
    a = r.results()
    B.gcn_profile_reset()
    B.gcn_profile_enable(True)
    r.step()
    torch.cuda.synchronize()
    B.gcn_profile_enable(False)
    prof = B.gcn_profile_read_all()
    b = r.results()
    if case == "bf16-odd-wide":   # the masked input gradient really ran on the large-tile kernel
        assert prof["gemm_nt_bf16_big_masked"][1] >= 1, prof
    if case == "bf16-row-major-dw":
        assert prof["gemm_tn_bf16_big"][1] == 2, prof
    inner = [t.detach().cpu().numpy() for t in ([r.dHL] if r.head is not None else []) + r.dH[1:]]
    for key in ("Y", "dW_self", "dW_neigh", "dH"):
        for i, (x, y) in enumerate(zip(a[key], b[key])):
            if x is None or y is None:
                assert y is None and (x is None or key == "dH" and i > 0)
                continue
            assert np.array_equal(x.view(np.uint32), y.view(np.uint32)), (key, i)
    fp32 = r.prec == B.GCN_F32
    for i, (x, y) in enumerate(zip(a["db"], b["db"])):
        assert rel_inf(y, x) <= 1e-6, i
    if "loss" in a:
        assert a["loss"] == b["loss"]
        for key in ("dW_pred", "db_pred"):
            assert np.array_equal(a[key].view(np.uint32), b[key].view(np.uint32)), key
    # the inter-layer buffers: the gradient, or the gradient times [input > 0]
    sep = ([a["dHL"]] if r.head is not None else []) + a["dH"][1:]
    below = [a["Y"][-1]] if r.head is not None else []
    below += [a["Y"][li - 1] for li in range(1, r.L)]
    for i, (g, got, y) in enumerate(zip(sep, inner, below)):
        masked = np.where(y > 0, g, np.float32(0))
        same = np.array_equal(got.view(np.uint32), g.view(np.uint32))
        if fp32:
            fused = np.array_equal(got.view(np.uint32), masked.view(np.uint32))
        else:
            rows, cols = masked.shape
            packed = got.view(np.uint16).reshape(-1)[: rows * cols].reshape(rows, cols)
            bits = torch.from_numpy(np.ascontiguousarray(masked)).to(torch.bfloat16).view(torch.int16).numpy()
            fused = np.array_equal(packed, bits.view(np.uint16))
        assert same or fused, ("inter-layer gradient", i)
        if r.head is not None and i == 0:
            assert fused, "the head writes the last layer's dZ"
        if case in ("bce-transform-first", "f32-odd-widths", "bf16-odd-widths", "bf16-odd-wide"):
            assert fused and not same, ("unsplit input-gradient product writes dZ", i)


def _random_model(seed):
    """A seeded random model and subgraph: 1-3 layers, widths 8-300 (odd ones
    included), random orders, head and precision."""
    r = np.random.default_rng(1000 + seed)
    n = int(r.integers(200, 5000))
    L = int(r.integers(1, 4))
    dims, f = [], int(r.integers(8, 301))
    for _ in range(L):
        h = int(r.integers(4, 151))
        dims.append((f, h))
        f = 2 * h
    head = [None, "ce", "bce"][int(r.integers(0, 3))]
    classes = int(r.integers(2, 120)) if head else 0
    wl = synth.custom(n, ["er", "rmat"][int(r.integers(0, 2))], int(r.integers(2, 30)), dims, head=head,
                      classes=classes, seed=seed)
    orders = [int(r.integers(0, 2)) for _ in range(L)]
    prec = B.GCN_BF16 if r.random() < 0.4 else B.GCN_F32
    return wl, orders, prec


@pytest.mark.parametrize("seed", range(48))
def test_model_step_random_models(seed):
    """Seeded random models through gcn_model_step (fused mask epilogues where
    they apply, split and unsplit products, ragged tiles): both precisions
    against the oracle (float32 at 1e-4, bfloat16 chained at 2e-2, each beyond
    the kink envelope of its unit roundoff) and against the separate calls.
    (Seed 12 found a split-K workspace that the input-gradient plan sized for
    one split too few.)"""
    wl, orders, prec = _random_model(seed)
    r = StepRunner(wl, prec=prec, orders=orders, first_layer_dH=True)
    print(f"seed {seed}: n={wl.n} nnz={wl.graph.nnz} dims={[l for l in wl.spec.layers]} head={wl.spec.head} "
          f"C={wl.spec.classes} orders={orders} prec={prec}", flush=True)
    r.step_calls()
    a = r.results()
    r.step()
    torch.cuda.synchronize()
    b = r.results()
    for key in ("Y", "dW_self", "dW_neigh"):
        for i, (x, y) in enumerate(zip(a[key], b[key])):
            assert np.array_equal(x.view(np.uint32), y.view(np.uint32)), (key, i)
    assert np.array_equal(a["dH"][0].view(np.uint32), b["dH"][0].view(np.uint32))
    for i, (x, y) in enumerate(zip(a["db"], b["db"])):
        assert rel_inf(y, x) <= 1e-6, ("db", i)
    if prec == B.GCN_F32:
        compare_step(b, oracle.step(wl, first_layer_dH=True, envelope=True))
    else:
        compare_bf16_chain(r, wl, first_layer_dH=True)


@pytest.mark.parametrize("graph", ["empty", "star"])
def test_model_step_degenerate_graphs_match_oracle(graph):
    """The whole step through gcn_model_step on a graph without edges (every
    aggregation is zero, so the neighbour halves are ReLU(bias)) and on a star
    (one hub row over every vertex)."""
    import dataclasses
    wl = synth.custom(777, "er", 6, [(48, 32), (64, 40)], head="ce", classes=9, seed=3)
    g = synth.empty_graph(wl.n) if graph == "empty" else synth.star_graph(wl.n)
    wl = dataclasses.replace(wl, graph=g)
    r = StepRunner(wl, first_layer_dH=True)
    print(f"model step on {graph} graph: n={wl.n} nnz={g.nnz}", flush=True)
    r.step()
    torch.cuda.synchronize()
    compare_step(r.results(), oracle.step(wl, first_layer_dH=True, envelope=True))


def test_bf16_step_without_float_outputs_refused_where_needed():
    """At 8,000 vertices layer 2's input-gradient product runs split, so
    layer 1's output gradient arrives unmasked and its float32 Y is needed:
    the step is refused before anything is launched."""
    wl = synth.config(1)
    r = StepRunner(wl, prec=B.GCN_BF16, float_outputs=False)
    for y in r.Y:
        y.fill_(7.0)
    with pytest.raises(B.GcnError) as e:
        r.step()
    assert e.value.code == B.GCN_EINVAL and "masked" in str(e.value)
    torch.cuda.synchronize()
    assert all(bool((y == 7.0).all()) for y in r.Y)


@pytest.mark.parametrize("cfg", [3])
def test_bf16_step_without_float_outputs(cfg):
    """The bfloat16 step with no float32 layer outputs (activations kept only
    as the bfloat16 operand rows the next consumer reads, as the benchmark
    runs it) gives the same loss and gradients bit for bit as the step that
    also writes them, and its kept outputs are the bfloat16 rounding of the
    float32 ones."""
    from oracle import bf16 as obf16
    wl = synth.config(cfg)
    a = StepRunner(wl, prec=B.GCN_BF16)
    b = StepRunner(wl, prec=B.GCN_BF16, float_outputs=False, orders=a.orders)
    print(f"bf16 step without float outputs: workload {cfg}", flush=True)
    a.step()
    b.step()
    torch.cuda.synchronize()
    ra, rb = a.results(), b.results()
    for key in ("dW_self", "dW_neigh", "db"):
        for i, (x, y) in enumerate(zip(ra[key], rb[key])):
            assert np.array_equal(x.view(np.uint32), y.view(np.uint32)), (key, i)
    assert ra["loss"] == rb["loss"]
    for key in ("dW_pred", "db_pred"):
        assert np.array_equal(ra[key].view(np.uint32), rb[key].view(np.uint32)), key
    for li in range(a.L - 1):
        assert np.array_equal(rb["Y"][li].view(np.uint32), obf16.round_bf16(ra["Y"][li]).view(np.uint32)), li
    assert rb["Y"][-1] is None
