"""GCN training with the parallel frontier sampler (Alg. 5), on one GPU.

The scheduler keeps a pool of sampled subgraphs.  When the pool runs out it
is refilled by S sampler runs launched at once (inter-subgraph parallelism,
Sec. IV-C), and each training iteration pops one subgraph, builds the GCN on it
and runs forward, loss, backward and the ADAM update (Alg. 1, Alg. 5).

MI355X mapping:
  - two pools are double-buffered: while the compute stream trains on one, a
    second stream (default priority) samples and induces the next, so sampling
    overlaps training;
  - the training graph G, its attributes and labels stay resident in HBM; an
    iteration gathers the subgraph's rows on the device;
  - all trained tensors live in one flat buffer, so one kernel applies ADAM to
    the whole model.
Every step of the computation is a call into libgcnlayer; this module only
sequences the calls and moves pool metadata (vertex and edge counts) to the
host, which the layer calls take as sizes.
"""
from __future__ import annotations

import time

from dataclasses import dataclass
from typing import List, Optional, Tuple

import numpy as np
import torch

from . import binding as B
from . import synth


@dataclass
class SamplerConfig:
    m: int = 1000          # frontier size (Sec. IV-A uses 1000)
    n: int = 8000          # vertex-list length per subgraph
    eta: float = 2.0       # Dashboard enlargement factor
    cap: int = 30          # Dashboard entries per vertex at most (Sec. VI-C-2)
    pool: int = 256        # subgraphs per refill (p_inter)
    seed: int = 1


def pad4(f: int) -> int:
    return (f + 3) // 4 * 4


class FlatModel:
    """Weights, biases and the prediction layer in one flat float32 buffer,
    with gradient, first- and second-moment buffers of the same layout.

    The first layer's weights are stored with pad4(f_in) rows, the rows past
    f_in zero: the features are stored with zero columns to the same width,
    so those rows only ever meet zeros, get zero gradients and stay zero under
    ADAM, and the model is the f_in-wide one exactly.  The padded width lets
    the products take 16-byte loads (a width such as 602 is not a multiple of
    four floats)."""

    def __init__(self, dims: List[Tuple[int, int]], classes: int, device, seed: int = 0):
        self.dims = list(dims)
        self.classes = classes
        self.f0 = dims[0][0]
        shapes = []
        for li, (f_in, h) in enumerate(dims):
            fs = pad4(f_in) if li == 0 else f_in
            shapes += [(fs, h), (fs, h), (2 * h,)]
        shapes += [(2 * dims[-1][1], classes), (classes,)]
        self.shapes = shapes
        offs, o = [], 0
        for sh in shapes:
            offs.append(o)
            o += (int(np.prod(sh)) + 63) // 64 * 64     # 256-byte aligned views
        self.offsets, self.total = offs, o
        d = torch.device(device)
        self.params = torch.zeros(o, dtype=torch.float32, device=d)
        self.grads = torch.zeros(o, dtype=torch.float32, device=d)
        self.m = torch.zeros(o, dtype=torch.float32, device=d)
        self.v = torch.zeros(o, dtype=torch.float32, device=d)
        rg = np.random.Generator(np.random.PCG64(np.random.SeedSequence([synth.SEED_ROOT, 3000, seed])))
        host = np.zeros(o, dtype=np.float32)
        for i, sh in enumerate(shapes):
            if len(sh) == 2:
                rows = self.f0 if i < 2 else sh[0]      # the first layer's real rows
                w = np.zeros(sh, np.float32)
                w[:rows] = synth.glorot(rg, rows, sh[1])
                host[offs[i]:offs[i] + sh[0] * sh[1]] = w.ravel()
        self.params.copy_(torch.from_numpy(host))
        self.step_count = 0

    def _view(self, buf, i):
        sh = self.shapes[i]
        return buf[self.offsets[i]:self.offsets[i] + int(np.prod(sh))].view(*sh)

    def layer(self, li, buf=None):
        buf = self.params if buf is None else buf
        return tuple(self._view(buf, 3 * li + j) for j in range(3))

    def head(self, buf=None):
        buf = self.params if buf is None else buf
        k = 3 * len(self.dims)
        return self._view(buf, k), self._view(buf, k + 1)

    def padding_rows(self):
        """The first layer's padding rows of W_self and W_neigh (host copies)."""
        p = self.params.cpu().numpy()
        return [p[o:o + int(np.prod(sh))].reshape(sh)[self.f0:] for o, sh in zip(self.offsets[:2], self.shapes[:2])]

    def host_tensors(self, buf=None):
        """{name: numpy array} of the current parameters (or of another buffer
        of the same layout, such as the gradients), the first layer's weights
        at their f_in rows (for checks)."""
        p = (self.params if buf is None else buf).cpu().numpy()
        out = {}
        names = []
        for li in range(len(self.dims)):
            names += [f"W_self{li}", f"W_neigh{li}", f"bias{li}"]
        names += ["W_pred", "b_pred"]
        for i, (nm, o, sh) in enumerate(zip(names, self.offsets, self.shapes)):
            a = p[o:o + int(np.prod(sh))].reshape(sh)
            out[nm] = (a[:self.f0] if i < 2 else a).copy()
        return out


class _Pool:
    """Device buffers of S sampled subgraphs and their induced CSRs."""

    def __init__(self, S: int, n: int, nV: int, edge_capacity: int, device, with_transpose: bool):
        d = torch.device(device)
        self.S, self.n = S, n
        self.with_transpose = with_transpose
        self.vertices = torch.empty((S, n), dtype=torch.int32, device=d)
        self.counts = torch.empty(S, dtype=torch.int32, device=d)
        self.status = torch.empty(S, dtype=torch.int32, device=d)
        self.batch = B.InducedBatch(S, n, edge_capacity, d, with_transpose)
        self.ws = B.Workspace(d)
        self.ws.get(B.lib().gcn_induce_workspace_bytes(nV, n, S))
        self.h_nsub = torch.empty(S, dtype=torch.int32).pin_memory()
        self.h_off = torch.empty(S + 1, dtype=torch.int64).pin_memory()
        self.h_status = torch.empty(S, dtype=torch.int32).pin_memory()
        self.h_istatus = torch.empty(1, dtype=torch.int32).pin_memory()
        self.ready = torch.cuda.Event()
        self.released = torch.cuda.Event()
        self.first_id = 0
        self.next = S       # nothing to pop until filled


class Trainer:
    """Alg. 5 on one GPU: pool refills on a side stream, iterations on the
    current stream."""

    def __init__(self, tg: "synth.TrainingGraph", dims: List[Tuple[int, int]], cfg: SamplerConfig,
                 lr: float = 0.01, prec: int = B.GCN_F32, device: str = "cuda", model_seed: int = 0):
        self.dev = torch.device(device)
        self.cfg = cfg
        self.prec = prec
        self.lr = lr
        g = tg.graph
        if dims[0][0] != tg.X.shape[1]:
            raise ValueError("the first layer's width must match the attributes")
        self.G = B.DeviceCSR.from_host(g.n, g.n, g.indptr, g.indices, g.vals, device=self.dev)
        # attributes stored pad4(f_in) wide, the extra columns zero (see FlatModel)
        f0p = pad4(dims[0][0])
        self.X = torch.zeros((g.n, f0p), dtype=torch.float32, device=self.dev)
        self.X[:, :dims[0][0]].copy_(torch.from_numpy(tg.X))
        self.labels_all = torch.from_numpy(tg.labels).to(self.dev)
        self.classes = tg.classes
        self.params = B.gcn_sampler_plan(g.indptr, cfg.m, cfg.n, eta=cfg.eta, cap=cfg.cap, seed=cfg.seed)
        self.model = FlatModel(dims, tg.classes, self.dev, seed=model_seed)
        self.dims = list(dims)
        self.L = len(dims)
        self.orders = [B.gcn_layer_pick_order(f, h, li > 0) for li, (f, h) in enumerate(dims)]
        n = cfg.n
        d = self.dev
        mean_deg = g.nnz / max(g.n, 1)
        self.edge_cap = int(cfg.n * max(mean_deg, 1.0) * 2) + 1024
        # on a symmetric G the induce step also emits the transposed matrix's
        # values, and the per-iteration CSR transpose is not needed
        self.symmetric = B.gcn_csr_pattern_symmetric_host(g.indptr, g.indices)
        self.side = torch.cuda.Stream(device=d)
        self.pools = [_Pool(cfg.pool, n, g.n, cfg.pool * self.edge_cap // 4 + 1024, d, self.symmetric)
                      for _ in range(2)]
        self.cur = 0
        self.next_id = 0
        self.wait_s = 0.0     # host time spent waiting for pool refills
        # iteration buffers, sized for the largest subgraph (n vertices)
        self.ws = B.Workspace(d)
        self.H0 = torch.empty((n, f0p), dtype=torch.float32, device=d)
        self.lab = torch.empty(n, dtype=torch.int32, device=d)
        self.Y = [torch.empty((n, 2 * h), dtype=torch.float32, device=d) for (_, h) in dims]
        self.dH = [None] + [torch.empty((n, f), dtype=torch.float32, device=d) for (f, _) in dims[1:]]
        self.dHL = torch.empty((n, 2 * dims[-1][1]), dtype=torch.float32, device=d)
        self.saved = []
        for li, ((f, h), o) in enumerate(zip(dims, self.orders)):
            nb = B.gcn_layer_saved_bytes(n, f0p if li == 0 else f, h, o, prec)
            self.saved.append(torch.empty(max(nb, 256), dtype=torch.uint8, device=d) if nb else None)
        self._alloc_edges(self.edge_cap)
        self.losses = torch.zeros(1 << 16, dtype=torch.float32, device=d)
        # every step is one gcn_model_step call over these buffers
        mdl = self.model
        layers = []
        for li in range(self.L):
            Ws, Wn, b = mdl.layer(li)
            gWs, gWn, gb = mdl.layer(li, mdl.grads)
            layers.append(dict(W_self=Ws, W_neigh=Wn, bias=b, Y=self.Y[li], saved=self.saved[li], dH=self.dH[li],
                               dW_self=gWs, dW_neigh=gWn, dbias=gb, order=self.orders[li]))
        Wp, bp = mdl.head()
        dWp, dbp = mdl.head(mdl.grads)
        self.fused = B.ModelStep(layers, dict(W_pred=Wp, b_pred=bp, kind=B.GCN_SOFTMAX_CE, labels=self.lab,
                                              targets=None, loss=self.losses[:1], dHL=self.dHL, dW_pred=dWp,
                                              db_pred=dbp), prec)
        self.iteration = 0
        self.subgraph_ids: List[int] = []
        for p in self.pools:
            self._refill(p)

    def _alloc_edges(self, cap):
        d = self.dev
        self.t_indptr = torch.empty(self.cfg.n + 1, dtype=torch.int32, device=d)
        self.t_indices = torch.empty(max(cap, 1), dtype=torch.int32, device=d)
        self.t_vals = torch.empty(max(cap, 1), dtype=torch.float32, device=d)
        self.t_cap = cap

    # ---------------------------------------------------------------- pools
    def _refill(self, p: _Pool):
        """Sample and induce S subgraphs on the side stream (after the compute
        stream has released the pool's buffers)."""
        p.first_id = self.next_id
        self.next_id += p.S
        s = self.side
        s.wait_event(p.released)
        with torch.cuda.stream(s):
            B.gcn_frontier_sample(self.G, self.params, p.first_id, p.S, p.vertices, p.counts, p.status, stream=s)
            B.gcn_induce_subgraphs(self.G, p.vertices, p.counts, p.batch, p.ws, stream=s)
            p.h_status.copy_(p.status, non_blocking=True)
            p.h_nsub.copy_(p.batch.n_sub, non_blocking=True)
            p.h_off.copy_(p.batch.edge_offsets, non_blocking=True)
            p.h_istatus.copy_(p.batch.status, non_blocking=True)
            p.ready.record(s)
        p.next = -1   # filled, metadata not read yet

    def _open(self, p: _Pool):
        """Wait for a refill and read its metadata on the host (the time the
        host spends waiting is added to `wait_s`: with the host ahead of the
        GPU, that is the GPU's backpressure, not issue work)."""
        t0 = time.perf_counter()
        p.ready.synchronize()
        self.wait_s += time.perf_counter() - t0
        if int(p.h_istatus[0]) != 0:       # edge arrays too small: grow and induce again
            need = int(p.h_off[-1])
            s = self.side
            with torch.cuda.stream(s):
                p.batch = B.InducedBatch(p.S, p.n, need + need // 8, self.dev, p.with_transpose)
                B.gcn_induce_subgraphs(self.G, p.vertices, p.counts, p.batch, p.ws, stream=s)
                p.h_nsub.copy_(p.batch.n_sub, non_blocking=True)
                p.h_off.copy_(p.batch.edge_offsets, non_blocking=True)
                p.ready.record(s)
            t0 = time.perf_counter()
            p.ready.synchronize()
            self.wait_s += time.perf_counter() - t0
        bad = [B.SAMPLE_STATUS[int(x)] for x in p.h_status.numpy() if int(x) not in (0, 1)]
        if bad:
            raise RuntimeError(f"sampler runs failed: {sorted(set(bad))}")
        p.nsub = p.h_nsub.numpy().copy()
        p.off = p.h_off.numpy().copy()
        p.next = 0
        torch.cuda.current_stream(self.dev).wait_event(p.ready)

    def _pop(self):
        p = self.pools[self.cur]
        if p.next < 0:
            self._open(p)
        if p.next >= p.S:
            p.released.record(torch.cuda.current_stream(self.dev))
            self._refill(p)
            self.cur ^= 1
            p = self.pools[self.cur]
            if p.next < 0:
                self._open(p)
        s = p.next
        p.next += 1
        return p, s

    # ------------------------------------------------------------ iteration
    def step(self):
        """One training iteration on the next subgraph of the pool."""
        p, s = self._pop()
        ns, e0, e1 = int(p.nsub[s]), int(p.off[s]), int(p.off[s + 1])
        self.subgraph_ids.append(p.first_id + s)
        nnz = e1 - e0
        if nnz > self.t_cap:
            self._alloc_edges(nnz + nnz // 8)
        A = p.batch.csr(s, ns, e0, e1)
        rows = p.batch.vsub[s]
        B.gcn_gather_rows(self.X, rows, ns, self.H0)
        B.gcn_gather_rows(self.labels_all, rows, ns, self.lab)
        if self.symmetric:
            AT = p.batch.csr_t(s, ns, e0, e1)
        else:
            AT = B.DeviceCSR(ns, ns, self.t_indptr[:ns + 1], self.t_indices[:nnz], self.t_vals[:nnz])
            B.gcn_csr_transpose_into(A, AT.indptr, AT.indices, AT.vals, self.ws)
        mdl = self.model
        t = self.iteration % self.losses.numel()
        self.fused.set_loss(self.losses[t:t + 1])
        self.fused(A, AT, self.H0, self.ws)
        mdl.step_count += 1
        B.gcn_adam_update(mdl.params, mdl.grads, mdl.m, mdl.v, self.lr, mdl.step_count)
        self.iteration += 1
        return ns, nnz

    def loss_history(self) -> np.ndarray:
        k = min(self.iteration, self.losses.numel())
        return self.losses[:k].cpu().numpy()
