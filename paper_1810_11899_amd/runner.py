"""One fwd+bwd training step of an L-layer GCN on a sampled subgraph.

Holds the device buffers of a workload (sized once, reused across steps and
across the subgraphs of an epoch stream) and issues the C-ABI calls of one
step on one stream: CSR transpose, the layers' forward, PREDICT/LOSS (or a
given output gradient), the layers' backward (Alg. 1, forward loop, PREDICT,
LOSS and the backward pass that ADAM consumes).  No arithmetic happens here.
"""
from __future__ import annotations

from typing import List, Optional

import numpy as np
import torch

from . import binding as B


class StepRunner:
    def __init__(self, wl, prec: int = B.GCN_F32, device: str = "cuda",
                 first_layer_dH: Optional[bool] = None, nnz_capacity: int = 0,
                 orders: Optional[List[int]] = None, transpose_shortcut: bool = True,
                 index_bits: int = 32, float_outputs: bool = True):
        """index_bits = 16 keeps A's column indices as uint16 (n <= 65,536):
        half the index bytes, the same results bit for bit.  orders: one
        gcn_order per layer, None for gcn_layer_pick_order's width rule, or
        "tuned" for the combination tune_orders measures fastest on this
        workload.  float_outputs=False (bfloat16 only): the model step keeps
        the layers' outputs only as the bfloat16 copies the next consumer
        reads, with no float32 Y (the library refuses where a layer's output
        gradient would not arrive masked)."""
        if not float_outputs and prec != B.GCN_BF16:
            raise ValueError("float32 steps write their float32 outputs")
        self.float_outputs = float_outputs
        if isinstance(orders, str):
            if orders != "tuned":
                raise ValueError(f"orders: a list, None or 'tuned' (got {orders!r})")
            orders, self.order_timings = tune_orders(wl, prec=prec, device=device, first_layer_dH=first_layer_dH,
                                                     index_bits=index_bits, float_outputs=float_outputs)
        self.dev = torch.device(device)
        self.prec = prec
        if index_bits not in (16, 32) or (index_bits == 16 and wl.n > 65536):
            raise ValueError("index_bits: 32, or 16 for at most 65,536 vertices")
        self.index_bits = index_bits
        self.transpose_shortcut = transpose_shortcut
        self.spec = wl.spec
        self.L = len(wl.layers)
        self.first_layer_dH = (self.L == 1) if first_layer_dH is None else bool(first_layer_dH)
        self.ws = B.Workspace(self.dev)
        self.n = wl.n
        self._alloc_graph(max(nnz_capacity, wl.graph.nnz))
        f = lambda a: torch.as_tensor(a, dtype=torch.float32).to(self.dev)
        self.W = [(f(l.W_self), f(l.W_neigh), f(l.bias)) for l in wl.layers]
        self.dims = [(l.f_in, l.h) for l in wl.layers]
        self.orders = []
        for li, (f_in, h) in enumerate(self.dims):
            need = li > 0 or self.first_layer_dH
            self.orders.append(orders[li] if orders is not None else B.gcn_layer_pick_order(f_in, h, need))
        n = self.n
        self.H0 = torch.empty((n, self.dims[0][0]), dtype=torch.float32, device=self.dev)
        self.Y = [torch.empty((n, 2 * h), dtype=torch.float32, device=self.dev) for (_, h) in self.dims]
        self.saved = []
        for (f_in, h), o in zip(self.dims, self.orders):
            nb = B.gcn_layer_saved_bytes(n, f_in, h, o, prec)
            self.saved.append(torch.empty(max(nb, 256), dtype=torch.uint8, device=self.dev) if nb else None)
        self.dH = []
        for li, (f_in, _) in enumerate(self.dims):
            need = li > 0 or self.first_layer_dH
            self.dH.append(torch.empty((n, f_in), dtype=torch.float32, device=self.dev) if need else None)
        self.dWs = [torch.empty((f_in, h), dtype=torch.float32, device=self.dev) for (f_in, h) in self.dims]
        self.dWn = [torch.empty((f_in, h), dtype=torch.float32, device=self.dev) for (f_in, h) in self.dims]
        self.db = [torch.empty(2 * h, dtype=torch.float32, device=self.dev) for (_, h) in self.dims]
        self.head = self.spec.head
        hl2 = 2 * self.dims[-1][1]
        if self.head is None:
            self.dY = torch.empty((n, hl2), dtype=torch.float32, device=self.dev)
        else:
            C = self.spec.classes
            self.W_pred = f(wl.W_pred)
            self.b_pred = f(wl.b_pred)
            self.kind = B.LOSS_KIND[self.head]
            self.labels = torch.empty(n, dtype=torch.int32, device=self.dev) if self.head == "ce" else None
            self.targets = torch.empty((n, C), dtype=torch.float32, device=self.dev) if self.head == "bce" else None
            self.loss = torch.empty(1, dtype=torch.float32, device=self.dev)
            self.dHL = torch.empty((n, hl2), dtype=torch.float32, device=self.dev)
            self.dW_pred = torch.empty((hl2, C), dtype=torch.float32, device=self.dev)
            self.db_pred = torch.empty(C, dtype=torch.float32, device=self.dev)
        self.load(wl)
        layers = [dict(W_self=Ws, W_neigh=Wn, bias=b, Y=self.Y[li] if float_outputs else None, saved=self.saved[li],
                       dH=self.dH[li],
                       dW_self=self.dWs[li], dW_neigh=self.dWn[li], dbias=self.db[li], order=self.orders[li])
                  for li, (Ws, Wn, b) in enumerate(self.W)]
        head = None if self.head is None else dict(
            W_pred=self.W_pred, b_pred=self.b_pred, kind=self.kind, labels=self.labels, targets=self.targets,
            loss=self.loss, dHL=self.dHL, dW_pred=self.dW_pred, db_pred=self.db_pred)
        self.model = B.ModelStep(layers, head, prec)

    # ------------------------------------------------------------ buffers
    def _alloc_graph(self, cap: int):
        n, d = self.n, self.dev
        self.cap = max(int(cap), 1)
        self.indptr = torch.empty(n + 1, dtype=torch.int32, device=d)
        self.indices = torch.empty(self.cap, dtype=torch.int16 if self.index_bits == 16 else torch.int32, device=d)
        self.vals = torch.empty(self.cap, dtype=torch.float32, device=d)
        self.t_indptr = torch.empty(n + 1, dtype=torch.int32, device=d)
        self.t_indices = torch.empty(self.cap, dtype=torch.int32, device=d)
        self.t_vals = torch.empty(self.cap, dtype=torch.float32, device=d)

    def load(self, wl, non_blocking: bool = False):
        """Copy a subgraph's CSR, features and labels into the resident buffers."""
        g = wl.graph
        if g.n != self.n:
            raise ValueError("subgraph size differs from the buffers")
        if g.nnz > self.cap:
            self._alloc_graph(g.nnz)
        self.nnz = g.nnz
        self.indptr.copy_(torch.from_numpy(g.indptr), non_blocking=non_blocking)
        if g.nnz:
            ix = g.indices.astype(np.uint16).view(np.int16) if self.index_bits == 16 else g.indices
            self.indices[:g.nnz].copy_(torch.from_numpy(ix), non_blocking=non_blocking)
            self.vals[:g.nnz].copy_(torch.from_numpy(g.vals), non_blocking=non_blocking)
        self.H0.copy_(torch.from_numpy(wl.H), non_blocking=non_blocking)
        if self.head is None:
            self.dY.copy_(torch.from_numpy(wl.dY), non_blocking=non_blocking)
        else:
            if self.labels is not None:
                self.labels.copy_(torch.from_numpy(wl.labels), non_blocking=non_blocking)
            if self.targets is not None:
                self.targets.copy_(torch.from_numpy(wl.targets), non_blocking=non_blocking)
        self.A = B.DeviceCSR(self.n, self.n, self.indptr, self.indices[:self.nnz], self.vals[:self.nnz])
        # an undirected subgraph's A^T shares A's pattern: only its values are
        # computed (gcn_csr_transpose_symmetric); otherwise the full transpose
        self.symmetric = self.transpose_shortcut and B.gcn_csr_pattern_symmetric_host(g.indptr, g.indices)
        if self.symmetric:
            self.AT = B.DeviceCSR(self.n, self.n, self.indptr, self.indices[:self.nnz], self.t_vals[:self.nnz])
        else:
            self.AT = B.DeviceCSR(self.n, self.n, self.t_indptr, self.t_indices[:self.nnz], self.t_vals[:self.nnz])

    def attach(self, slot: "InputSlot"):
        """Run the next steps on the subgraph held in an input slot (its CSR,
        H0 and labels), in place of the runner's own input buffers."""
        if slot.n != self.n or slot.index_bits != self.index_bits:
            raise ValueError("input slot built for another runner")
        self.nnz = slot.nnz
        self.H0 = slot.H0
        self.A = B.DeviceCSR(self.n, self.n, slot.indptr, slot.indices[:slot.nnz], slot.vals[:slot.nnz])
        self.symmetric = slot.symmetric
        if self.symmetric:
            self.AT = B.DeviceCSR(self.n, self.n, slot.indptr, slot.indices[:slot.nnz], slot.t_vals[:slot.nnz])
        else:
            self.AT = B.DeviceCSR(self.n, self.n, slot.t_indptr, slot.t_indices[:slot.nnz], slot.t_vals[:slot.nnz])
        if self.head is None:
            self.dY = slot.dY
        else:
            self.labels, self.targets = slot.labels, slot.targets
            self.model.set_labels(slot.labels, slot.targets)

    # --------------------------------------------------------------- step
    def _transpose(self, stream):
        if self.symmetric:
            B.gcn_csr_transpose_symmetric(self.A, self.ws, self.AT.vals, stream)
        else:
            B.gcn_csr_transpose_into(self.A, self.AT.indptr, self.AT.indices, self.AT.vals, self.ws, stream)

    def step(self, stream=None):
        """The transpose, then the whole fwd+bwd in one gcn_model_step call."""
        self._transpose(stream)
        self.model(self.A, self.AT, self.H0, self.ws, dY=self.dY if self.head is None else None, stream=stream)
        self._last = "step"

    def step_calls(self, stream=None):
        """The same step as separate gcn_layer_fwd / gcn_loss_grad / gcn_layer_bwd calls."""
        self._transpose(stream)
        H = self.H0
        for li in range(self.L):
            Ws, Wn, b = self.W[li]
            B.gcn_layer_fwd(self.A, H, Ws, Wn, b, self.Y[li], self.saved[li], self.orders[li], self.ws,
                            self.prec, stream)
            H = self.Y[li]
        if self.head is None:
            dY = self.dY
        else:
            B.gcn_loss_grad(self.Y[-1], self.W_pred, self.b_pred, self.kind, self.labels, self.targets,
                            self.loss, self.dHL, self.dW_pred, self.db_pred, self.ws, self.prec, stream)
            dY = self.dHL
        for li in range(self.L - 1, -1, -1):
            Ws, Wn, _ = self.W[li]
            Hin = self.H0 if li == 0 else self.Y[li - 1]
            B.gcn_layer_bwd(self.A, self.AT, Hin, Ws, Wn, self.Y[li], self.saved[li], dY, self.dH[li],
                            self.dWs[li], self.dWn[li], self.db[li], self.orders[li], self.ws, self.prec,
                            stream)
            dY = self.dH[li]
        self._last = "calls"

    # ------------------------------------------------------------ results
    def csr_bytes(self) -> int:
        """Device bytes of A's CSR (row pointers, column indices, values)."""
        return 4 * (self.n + 1) + (2 if self.index_bits == 16 else 4) * self.nnz + 4 * self.nnz

    def results(self) -> dict:
        """Host copies of the last step's outputs.  After ``step()`` the
        inter-layer gradient buffers (dHL, dH of layers 1..L-1) hold
        intermediate values and are reported as None."""
        c = lambda t: None if t is None else t.detach().cpu().numpy()
        inner = getattr(self, "_last", "calls") == "step"
        Ys = [c(y) for y in self.Y]
        if inner and not self.float_outputs:
            # outputs kept as bfloat16 rows at the start of the next layer's
            # saved buffer; the last layer's is not kept
            for li in range(self.L):
                if li + 1 < self.L:
                    nb = self.n * 2 * self.dims[li][1]
                    bits = self.saved[li + 1][:2 * nb].view(torch.int16).cpu().numpy().view(np.uint16)
                    Ys[li] = (bits.astype(np.uint32) << 16).view(np.float32).reshape(self.n, -1)
                else:
                    Ys[li] = None
        r = {"Y": Ys, "dW_self": [c(t) for t in self.dWs],
             "dW_neigh": [c(t) for t in self.dWn], "db": [c(t) for t in self.db],
             "dH": [None if (inner and li > 0) else c(t) for li, t in enumerate(self.dH)],
             "t_indptr": c(self.AT.indptr), "t_indices": _as_int32(c(self.AT.indices)), "t_vals": c(self.AT.vals)}
        if self.head is not None:
            r.update(loss=float(self.loss.item()), dW_pred=c(self.dW_pred), db_pred=c(self.db_pred),
                     dHL=None if inner else c(self.dHL))
        return r

    # ---------------------------------------------------- work accounting
    def work(self) -> dict:
        return step_work(self.n, self.nnz, self.dims, self.orders,
                         [d is not None for d in self.dH],
                         self.spec.classes if self.head is not None else 0)


def tune_orders(wl, prec: int = B.GCN_F32, device: str = "cuda", first_layer_dH: Optional[bool] = None,
                index_bits: int = 32, warmup: int = 2, reps: int = 5, float_outputs: bool = True):
    """Measure the whole model step for every combination of the layers'
    groupings (aggregate-first or transform-first, 2^L combinations) on this
    workload's graph and widths, and return the fastest combination with the
    per-combination median step times (ms).  The two groupings compute the
    same layer (Alg. 1's (A H) W and A (H W)); which is faster depends on the
    widths, the graph and which fused epilogues each grouping allows, so it
    is measured rather than predicted."""
    import itertools
    L = len(wl.layers)
    dev = torch.device(device)
    stream = torch.cuda.current_stream(dev)
    timings = {}
    for combo in itertools.product((B.GCN_AGGREGATE_FIRST, B.GCN_TRANSFORM_FIRST), repeat=L):
        r = StepRunner(wl, prec=prec, device=device, first_layer_dH=first_layer_dH, orders=list(combo),
                       index_bits=index_bits, float_outputs=float_outputs)
        for _ in range(warmup):
            r.step()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        ev[0].record(stream)
        for i in range(reps):
            r.step()
            ev[i + 1].record(stream)
        torch.cuda.synchronize(dev)
        t = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(reps))
        timings[tuple(combo)] = t[reps // 2]
        del r
    best = min(timings, key=timings.get)
    return list(best), timings


def _as_int32(ix: np.ndarray) -> np.ndarray:
    """Column indices as int32 (uint16 indices are held as int16 bits)."""
    return ix.view(np.uint16).astype(np.int32) if ix.dtype == np.int16 else ix


def step_work(n: int, nnz: int, dims, orders, need_dH, classes: int = 0) -> dict:
    """Algorithmic work of one fwd+bwd step.

    edge-features: sum over the aggregation passes of nnz x (aggregated width);
    GEMM flops: 2*M*N*K summed over every dense product of the step.
    Aggregate-first aggregates H at f_in in the forward pass and, for the input
    gradient, A^T at min(f_in, h); transform-first aggregates at h forward and
    h backward (A^T dZ_n, shared by dW_neigh and dH).
    """
    ef = 0
    fl = 0.0
    for (f_in, h), o, dH in zip(dims, orders, need_dH):
        fl += 2.0 * n * f_in * h * 2          # forward: two n x f_in x h products
        fl += 2.0 * n * f_in * h * 2          # weight gradients (K = n)
        if dH:
            fl += 2.0 * n * f_in * h * 2      # input gradient
        if o == B.GCN_AGGREGATE_FIRST:
            ef += nnz * f_in
            if dH:
                ef += nnz * min(f_in, h)
        else:
            ef += nnz * h * 2
    if classes:
        f2 = 2 * dims[-1][1]
        fl += 3 * 2.0 * n * f2 * classes      # logits, dW_pred, dH_L
    return {"edge_features": float(ef), "gemm_flops": fl, "spmm_flops": 2.0 * ef}


class InputSlot:
    """One subgraph's inputs resident on the device (A's CSR with room for
    A^T, H0, and the labels, targets or given output gradient), with pinned
    host buffers of the same sizes from which they are uploaded
    asynchronously.  Two slots double-buffer an epoch stream (EpochPipeline):
    the next subgraph is uploaded into one while the step runs on the other.

    Events order the reuse: `uploaded` is recorded on the copy stream behind
    a slot's uploads (the host refills the pinned buffers only after it, the
    compute stream starts the step only after it); `released` is recorded on
    the compute stream behind the step that read the slot (the next upload
    into the slot waits for it)."""

    def __init__(self, runner: StepRunner, nnz_capacity: int):
        n, dev = runner.n, runner.dev
        self.n, self.index_bits, self.cap = n, runner.index_bits, max(int(nnz_capacity), 1)
        idt = torch.int16 if runner.index_bits == 16 else torch.int32

        def pair(shape, dtype):
            return (torch.empty(shape, dtype=dtype, device=dev),
                    torch.empty(shape, dtype=dtype, pin_memory=True))
        self.indptr, self._h_indptr = pair(n + 1, torch.int32)
        self.indices, self._h_indices = pair(self.cap, idt)
        self.vals, self._h_vals = pair(self.cap, torch.float32)
        self.t_indptr = torch.empty(n + 1, dtype=torch.int32, device=dev)
        self.t_indices = torch.empty(self.cap, dtype=torch.int32, device=dev)
        self.t_vals = torch.empty(self.cap, dtype=torch.float32, device=dev)
        self.H0, self._h_H0 = pair(tuple(runner.H0.shape), torch.float32)
        self.labels = self.targets = self.dY = None
        self._h_labels = self._h_targets = self._h_dY = None
        if runner.head is None:
            self.dY, self._h_dY = pair(tuple(runner.dY.shape), torch.float32)
        elif runner.head == "ce":
            self.labels, self._h_labels = pair(n, torch.int32)
        else:
            self.targets, self._h_targets = pair((n, runner.spec.classes), torch.float32)
        self.uploaded = torch.cuda.Event()
        self.released = torch.cuda.Event()
        self.nnz = 0
        self.symmetric = False
        self.bytes = 0

    def stage(self, wl, symmetric: bool):
        """Host side: copy subgraph `wl` into the pinned buffers, once the
        previous upload from them has finished."""
        g = wl.graph
        if g.n != self.n:
            raise ValueError("subgraph size differs from the slot")
        if g.nnz > self.cap:
            raise ValueError(f"subgraph has {g.nnz} entries, the slot holds {self.cap}")
        self.uploaded.synchronize()
        self.nnz, self.symmetric = int(g.nnz), bool(symmetric)
        self._h_indptr.numpy()[:] = g.indptr
        ix = self._h_indices.numpy()
        ix[:g.nnz] = g.indices.astype(np.uint16).view(np.int16) if self.index_bits == 16 else g.indices
        self._h_vals.numpy()[:g.nnz] = g.vals
        self._h_H0.numpy()[:] = wl.H
        if self._h_dY is not None:
            self._h_dY.numpy()[:] = wl.dY
        if self._h_labels is not None:
            self._h_labels.numpy()[:] = wl.labels
        if self._h_targets is not None:
            self._h_targets.numpy()[:] = wl.targets

    def upload(self, copy_stream, start_event=None):
        """Enqueue the uploads on `copy_stream`, behind the release of the
        slot by the last step that read it (start_event, if given, is
        recorded once that release has been waited for)."""
        nnz = self.nnz
        copy_stream.wait_event(self.released)
        if start_event is not None:
            start_event.record(copy_stream)
        with torch.cuda.stream(copy_stream):
            pairs = [(self.indptr, self._h_indptr), (self.indices[:nnz], self._h_indices[:nnz]),
                     (self.vals[:nnz], self._h_vals[:nnz]), (self.H0, self._h_H0)]
            for d, h in ((self.dY, self._h_dY), (self.labels, self._h_labels), (self.targets, self._h_targets)):
                if d is not None:
                    pairs.append((d, h))
            for d, h in pairs:
                d.copy_(h, non_blocking=True)
            self.uploaded.record(copy_stream)
        self.bytes = sum(h.numel() * h.element_size() for _, h in pairs)


class EpochPipeline:
    """An epoch stream of independent subgraphs of one size (Alg. 5's pool
    of sampled subgraphs, here drawn on the host): each subgraph goes through
    pinned host buffers on a copy stream into one of `slots` device input
    slots, and its step runs on the compute stream once its upload is done,
    so the upload of subgraph s + 1 overlaps the step of subgraph s.  The
    runner's weights, activations, gradients and workspace are shared by the
    stream."""

    def __init__(self, runner: StepRunner, nnz_capacity: int, slots: int = 2, compute_stream=None):
        if slots < 1:
            raise ValueError("at least one input slot")
        self.runner = runner
        self.slots = [InputSlot(runner, nnz_capacity) for _ in range(slots)]
        self.copy_stream = torch.cuda.Stream(device=runner.dev)
        self.compute_stream = compute_stream if compute_stream is not None else torch.cuda.current_stream(runner.dev)
        # the workspace sized for the largest subgraph up front: no
        # reallocation while steps are in flight
        runner.ws.get(runner.model.workspace_bytes(runner.n, int(nnz_capacity)))
        self.count = 0

    def submit(self, wl, symmetric: Optional[bool] = None, events=None):
        """Stage, upload and step subgraph `wl`.  events: None, or four
        timing events (upload start, upload end, step start, step end) to
        record around the upload on the copy stream and the step on the
        compute stream."""
        slot = self.slots[self.count % len(self.slots)]
        self.count += 1
        if symmetric is None:
            g = wl.graph
            symmetric = self.runner.transpose_shortcut and B.gcn_csr_pattern_symmetric_host(g.indptr, g.indices)
        slot.stage(wl, symmetric)
        slot.upload(self.copy_stream, None if events is None else events[0])
        if events is not None:
            events[1].record(self.copy_stream)
        cs = self.compute_stream
        cs.wait_event(slot.uploaded)
        self.runner.attach(slot)
        if events is not None:
            events[2].record(cs)
        self.runner.step(cs)
        if events is not None:
            events[3].record(cs)
        slot.released.record(cs)
        return slot
