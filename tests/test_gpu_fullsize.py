"""Full-size parity: the 65,536-vertex 2-layer workload (float32) and subgraphs
of the 200-subgraph epoch stream, in the launch configuration the benchmark
times, against the complete CPU oracle (tens of seconds each)."""
import numpy as np
import pytest
import torch

import oracle
from paper_1810_11899_amd import synth
from paper_1810_11899_amd.runner import StepRunner

from gpu_util import TOL_F32, rel_inf, require_gpu
from test_gpu_layer import compare_step

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def test_rmat65536_two_layer_f32_step():
    wl = synth.config(3)
    r = StepRunner(wl)
    r.step()
    torch.cuda.synchronize()
    got = r.results()
    ref = oracle.step(wl, envelope=True)
    errs = compare_step(got, ref)
    print("ambiguous ReLU kinks per layer:", ref.ambiguous)
    print("max relative errors beyond the kink envelope:", {k: f"{v:.1e}" for k, v in errs.items()})


def test_rmat65536_two_layer_bf16_chained_step():
    """The bfloat16 step the benchmark times, as one chain (the forward loop,
    PREDICT/LOSS and the backward pass in one gcn_model_step), against the
    float64 oracle on the unrounded inputs."""
    from paper_1810_11899_amd import binding as B
    from test_gpu_layer import compare_bf16_chain
    wl = synth.config(3)
    r = StepRunner(wl, prec=B.GCN_BF16)
    B.gcn_profile_reset()
    B.gcn_profile_enable(True)
    r.step()
    torch.cuda.synchronize()
    B.gcn_profile_enable(False)
    prof = B.gcn_profile_read_all()
    # every weight gradient (both layers' and the head's, K = 65,536) reads
    # its operands as row-major bfloat16 rows on the large-tile kernel
    assert prof["gemm_tn_bf16_big"][1] == 3 and prof["gemm_nt_bf16"][1] == 0, prof
    errs, _ = compare_bf16_chain(r, wl)
    print("bf16 chain:", errs)


def test_epoch_stream_subgraphs_reuse_buffers():
    """The oracle subset of the stream (subgraphs 0, 1, 2, 50, 100, 150, 198,
    199) through the double-buffered upload pipeline of one runner (input
    slots sized for the largest nnz, activations and workspace reused); each
    checked against the oracle."""
    spec = synth.WORKLOADS[4]
    subs = [0, 1, 2, 50, 100, 150, 198, 199]
    wls = [synth.config(4, s=s) for s in subs]
    cap = spec.n * spec.d_range[1]
    r = StepRunner(wls[0], nnz_capacity=cap)
    from paper_1810_11899_amd.runner import EpochPipeline
    pipe = EpochPipeline(r, cap, slots=2)       # as the benchmark streams them
    for s, w in zip(subs, wls):
        print(f"stream subgraph {s}: nnz={w.graph.nnz}", flush=True)
        pipe.submit(w)
        torch.cuda.synchronize()
        compare_step(r.results(), oracle.step(w, envelope=True))
    assert len({w.graph.nnz for w in wls}) > 1  # the stream really varies nnz
    assert spec.subgraphs == 200


@pytest.mark.parametrize("prec", [0, 1])
def test_epoch_pipeline_matches_serial_loads(prec):
    """The double-buffered stream (pinned uploads on a copy stream into two
    input slots, each step behind its upload, each upload behind the release
    of its slot) computes, subgraph by subgraph, bit for bit what loading
    each subgraph synchronously and stepping computes.  The outputs of every
    step are copied on the compute stream behind it and compared at the end,
    so the uploads really overlap the steps.  Subgraphs vary in nnz; one has a
    non-symmetric pattern (general transpose), one is a BCE head's."""
    import dataclasses
    from paper_1810_11899_amd import binding as B
    from paper_1810_11899_amd.runner import EpochPipeline
    wls = [synth.custom(3000, "rmat", d, [(64, 64), (128, 32)], head="ce", classes=10, seed=s)
           for s, d in enumerate([8, 12, 6, 10, 9, 12, 7])]
    g = wls[3].graph
    rows = np.repeat(np.arange(g.n), g.degrees())
    keep = (rows + g.indices) % 3 != 0
    wls[3] = dataclasses.replace(wls[3], graph=synth.csr_from_pairs(g.n, rows[keep], g.indices[keep]))
    cap = max(w.graph.nnz for w in wls)
    ref = StepRunner(wls[0], prec=prec, nnz_capacity=cap)
    want = []
    for w in wls:
        ref.load(w)
        ref.step()
        torch.cuda.synchronize()
        want.append([ref.loss.cpu().numpy()] + [t.cpu().numpy() for t in ref.dWs + ref.dWn + ref.db]
                    + [ref.dW_pred.cpu().numpy(), ref.db_pred.cpu().numpy()])
    run = StepRunner(wls[0], prec=prec, nnz_capacity=cap)
    pipe = EpochPipeline(run, cap, slots=2)
    got = []
    for i, w in enumerate(wls):
        print(f"pipelined subgraph {i} nnz={w.graph.nnz}", flush=True)
        pipe.submit(w)
        got.append([run.loss.clone()] + [t.clone() for t in run.dWs + run.dWn + run.db]
                   + [run.dW_pred.clone(), run.db_pred.clone()])
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(want, got)):
        for x, y in zip(a, b):
            assert np.array_equal(x, y.cpu().numpy()), i
    # a different head kind through the slots: BCE targets
    wb = [synth.custom(2000, "er", d, [(32, 32)], head="bce", classes=6, seed=10 + d) for d in (5, 9, 7)]
    capb = max(w.graph.nnz for w in wb)
    refb = StepRunner(wb[0], prec=prec, nnz_capacity=capb)
    runb = StepRunner(wb[0], prec=prec, nnz_capacity=capb)
    pipeb = EpochPipeline(runb, capb, slots=2)
    outs = []
    for w in wb:
        pipeb.submit(w)
        outs.append((runb.loss.clone(), runb.dWs[0].clone()))
    for w, (l, dw) in zip(wb, outs):
        refb.load(w)
        refb.step()
        torch.cuda.synchronize()
        assert np.array_equal(refb.loss.cpu().numpy(), l.cpu().numpy())
        assert np.array_equal(refb.dWs[0].cpu().numpy(), dw.cpu().numpy())


def _f32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


@pytest.mark.parametrize("cfg, prec", [(2, 0), (3, 0), (4, 0), (2, 1), (3, 1)])
def test_layerwise_strict(cfg, prec):
    """Every layer of the full-size workload on the oracle's own (float32-
    rounded) layer inputs: forward Y, the loss head and every gradient within
    1e-4 (float32) or 2e-2 (bfloat16 operands) with no kink allowance.  The
    backward receives the oracle's Y, so the ReLU branch is decided on the same
    sign on both sides."""
    from paper_1810_11899_amd import binding as B
    from gpu_util import TOL_BF16
    tol = TOL_BF16 if prec == B.GCN_BF16 else TOL_F32
    wl = synth.config(cfg)
    g = wl.graph
    L = len(wl.layers)
    # oracle forward, head and backward (float64)
    ti, tj, tv = oracle.csr_transpose(g.n, g.n, g.indptr, g.indices, g.vals)
    gT = synth.Graph(g.n, ti, tj, tv)
    H = wl.H
    caches, Ys = [], []
    for lay in wl.layers:
        Y, c = oracle.layer_fwd(g, H, lay.W_self, lay.W_neigh, lay.bias)
        caches.append(c)
        Ys.append(Y)
        H = Y
    loss, dWp, dbp, dHL, _ = oracle.loss_grad(wl.spec.head, Ys[-1], wl.W_pred, wl.b_pred,
                                              labels=wl.labels, targets=wl.targets)
    dYs = [None] * L
    dY = dHL
    for li in range(L - 1, -1, -1):
        dYs[li] = dY
        lay = wl.layers[li]
        *_, dY = oracle.layer_bwd(gT, caches[li], lay.W_self, lay.W_neigh, dY, li > 0)

    ws = B.Workspace("cuda")
    A = B.DeviceCSR.from_host(g.n, g.n, g.indptr, g.indices, g.vals)
    AT = B.gcn_csr_transpose(A, ws)
    d = lambda a, dt=torch.float32: torch.as_tensor(_f32(a) if dt == torch.float32 else a).to("cuda")
    errs = {}
    # head
    C = wl.spec.classes
    n = g.n
    l_gpu = torch.empty(1, device="cuda")
    dHL_gpu = torch.empty((n, Ys[-1].shape[1]), device="cuda")
    dWp_gpu = torch.empty((Ys[-1].shape[1], C), device="cuda")
    dbp_gpu = torch.empty(C, device="cuda")
    B.gcn_loss_grad(d(Ys[-1]), d(wl.W_pred), d(wl.b_pred), B.LOSS_KIND[wl.spec.head],
                    d(wl.labels.astype(np.int32), torch.int32) if wl.labels is not None else None,
                    d(wl.targets) if wl.targets is not None else None, l_gpu, dHL_gpu, dWp_gpu, dbp_gpu, ws, prec)
    errs["loss"] = abs(l_gpu.item() - loss) / abs(loss)
    errs["dW_pred"] = rel_inf(dWp_gpu.cpu().numpy(), dWp)
    errs["db_pred"] = rel_inf(dbp_gpu.cpu().numpy(), dbp)
    errs["dHL"] = rel_inf(dHL_gpu.cpu().numpy(), dHL)
    for li, lay in enumerate(wl.layers):
        f_in, h = lay.f_in, lay.h
        need = li > 0
        order = B.gcn_layer_pick_order(f_in, h, need)
        Hin = d(caches[li].H)
        Ws, Wn, b = d(lay.W_self), d(lay.W_neigh), d(lay.bias)
        Y_gpu = torch.empty((n, 2 * h), device="cuda")
        nb = B.gcn_layer_saved_bytes(n, f_in, h, order, prec)
        saved = torch.empty(max(nb, 1), dtype=torch.uint8, device="cuda") if nb else None
        B.gcn_layer_fwd(A, Hin, Ws, Wn, b, Y_gpu, saved, order, ws, prec)
        errs[f"Y{li}"] = rel_inf(Y_gpu.cpu().numpy(), Ys[li])
        Y32 = _f32(Ys[li])
        assert np.array_equal(Y32 > 0, caches[li].Z > 0)  # same ReLU branch on both sides
        dH_gpu = torch.empty((n, f_in), device="cuda") if need else None
        dWs = torch.empty((f_in, h), device="cuda")
        dWn = torch.empty((f_in, h), device="cuda")
        db = torch.empty(2 * h, device="cuda")
        B.gcn_layer_bwd(A, AT, Hin, Ws, Wn, d(Y32), saved, d(dYs[li]), dH_gpu, dWs, dWn, db, order, ws, prec)
        rWs, rWn, rdb, rdH = oracle.layer_bwd(gT, caches[li], lay.W_self, lay.W_neigh, dYs[li], need)
        errs[f"dW_self{li}"] = rel_inf(dWs.cpu().numpy(), rWs)
        errs[f"dW_neigh{li}"] = rel_inf(dWn.cpu().numpy(), rWn)
        errs[f"db{li}"] = rel_inf(db.cpu().numpy(), rdb)
        if need:
            errs[f"dH{li}"] = rel_inf(dH_gpu.cpu().numpy(), rdH)
    print("max relative errors:", {k: f"{v:.1e}" for k, v in errs.items()})
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad
