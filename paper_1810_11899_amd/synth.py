"""Seeded synthetic inputs for the graph-sampling GCN layer (arXiv 1810.11899).

This module only *draws* inputs: subgraph CSR patterns with their mean weights,
vertex features, Glorot weights, labels.  It holds none of the layer's
arithmetic, and it is the single source of inputs for both the HIP library and
the CPU oracle, which never import each other.

The paper trains on frontier-sampled subgraphs of PPI, Reddit, Yelp and Amazon
(Sec. VI-A, Table I).  Those datasets are not available, so every workload here
is synthetic and stands in for them: Erdos-Renyi or R-MAT subgraphs (R-MAT for
the skewed, power-law degree mix that sampled social/product graphs have), with
the attribute widths and class counts of Table I and the hidden width 512 of
Sec. VI-C.  All graphs are undirected, without self-loops or duplicate edges;
the stored CSR is symmetric in pattern and row-normalised in value
(``vals[p] = 1/deg(row)``, the mean of Sec. II), which is how the per-subgraph
aggregation matrix is handed to the layer.

Random streams: ``np.random.SeedSequence([181011899, cfg, s, ...])`` spawned
into children in a fixed order (graph, relabel, H, unused, labels, degree) for
everything that belongs to subgraph s; the model weights come from
``SeedSequence([181011899, cfg, WEIGHT_KEY])`` so that every subgraph of an
epoch stream trains the same model.  PCG64 output is platform independent, so
the same seed gives bitwise equal arrays on every machine.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

SEED_ROOT = 181011899
WEIGHT_KEY = 0x5EED
RMAT_ABC = (0.57, 0.19, 0.19)  # d = 0.05


# --------------------------------------------------------------------------
# graphs
# --------------------------------------------------------------------------
@dataclass
class Graph:
    """CSR of the aggregation matrix: row i = destination vertex i."""
    n: int
    indptr: np.ndarray   # int32 [n+1]
    indices: np.ndarray  # int32 [nnz], ascending within a row
    vals: np.ndarray     # float32 [nnz]

    @property
    def nnz(self) -> int:
        return int(self.indices.shape[0])

    def degrees(self) -> np.ndarray:
        return np.diff(self.indptr.astype(np.int64))


def _mean_values(indptr: np.ndarray) -> np.ndarray:
    """float32(1/deg(row)) for every stored entry, as an IEEE float32 quotient."""
    deg = np.diff(indptr.astype(np.int64))
    per_row = np.zeros(deg.shape[0], dtype=np.float32)
    nz = deg > 0
    per_row[nz] = np.float32(1.0) / deg[nz].astype(np.float32)
    return np.repeat(per_row, deg)


def csr_from_pairs(n: int, rows: np.ndarray, cols: np.ndarray,
                   vals: Optional[np.ndarray] = None) -> Graph:
    """Directed (row, col) pairs -> CSR sorted by (row, col).

    With ``vals=None`` the values are the mean weights 1/deg(row); otherwise the
    given values travel with their pairs.  Duplicates are kept as given.
    """
    rows = np.asarray(rows, dtype=np.int64)
    cols = np.asarray(cols, dtype=np.int64)
    order = np.lexsort((cols, rows))
    rows, cols = rows[order], cols[order]
    counts = np.bincount(rows, minlength=n) if rows.size else np.zeros(n, np.int64)
    indptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(counts, out=indptr[1:])
    if vals is None:
        v = _mean_values(indptr)
    else:
        v = np.asarray(vals, dtype=np.float32)[order]
    return Graph(n, indptr.astype(np.int32), cols.astype(np.int32), v.astype(np.float32))


def csr_from_undirected(n: int, u: np.ndarray, v: np.ndarray) -> Graph:
    """Undirected edge list (no self-loops, no duplicates) -> symmetric CSR."""
    u = np.asarray(u, dtype=np.int64)
    v = np.asarray(v, dtype=np.int64)
    return csr_from_pairs(n, np.concatenate([u, v]), np.concatenate([v, u]))


def with_self_loops(g: Graph) -> Graph:
    """The same graph with a self-connection added to every vertex (the
    GraphSAGE convention Sec. V-B follows), re-normalised to the mean over
    the row: vals = 1/(deg + 1), the vertex itself included."""
    rows = np.repeat(np.arange(g.n, dtype=np.int64), g.degrees())
    if g.nnz and np.any(rows == g.indices):
        raise ValueError("the graph already has self-loops")
    diag = np.arange(g.n, dtype=np.int64)
    return csr_from_pairs(g.n, np.concatenate([rows, diag]), np.concatenate([g.indices.astype(np.int64), diag]))


def _first_unique(keys: np.ndarray) -> np.ndarray:
    """Distinct keys in order of first appearance."""
    _, first = np.unique(keys, return_index=True)
    return keys[np.sort(first)]


def _fill_edges(draw, n: int, m: int) -> Tuple[np.ndarray, np.ndarray]:
    """Keep drawing canonical (min,max) pairs until m distinct ones exist."""
    keys = np.zeros(0, dtype=np.int64)
    while keys.size < m:
        need = m - keys.size
        u, v = draw(2 * need + 1024)
        ok = (u < n) & (v < n) & (u != v)
        u, v = u[ok], v[ok]
        lo, hi = np.minimum(u, v), np.maximum(u, v)
        keys = _first_unique(np.concatenate([keys, lo * n + hi]))
    keys = keys[:m]
    return keys // n, keys % n


def erdos_renyi(rng: np.random.Generator, n: int, m: int):
    """G(n, m): m distinct unordered pairs drawn uniformly."""
    def draw(k):
        return rng.integers(0, n, size=k), rng.integers(0, n, size=k)
    return _fill_edges(draw, n, m)


def rmat(rng: np.random.Generator, n: int, m: int, abc=RMAT_ABC):
    """R-MAT with quadrant probabilities (a, b, c, 1-a-b-c), no noise."""
    a, b, c = abc
    scale = max(1, int(math.ceil(math.log2(max(n, 2)))))

    def draw(k):
        u = np.zeros(k, dtype=np.int64)
        v = np.zeros(k, dtype=np.int64)
        for _ in range(scale):
            r = rng.random(k)
            bu = (r >= a + b).astype(np.int64)            # quadrants c, d: lower half
            bv = ((r >= a) & (r < a + b)) | (r >= a + b + c)  # quadrants b, d: right half
            u = (u << 1) | bu
            v = (v << 1) | bv.astype(np.int64)
        return u, v
    return _fill_edges(draw, n, m)


def make_graph(kind: str, n: int, d: int, rng_graph: np.random.Generator,
               rng_relabel: np.random.Generator) -> Graph:
    """Undirected graph with exactly n*d/2 edges, vertex ids randomly relabelled."""
    m = (n * d) // 2
    if kind == "er":
        u, v = erdos_renyi(rng_graph, n, m)
    elif kind == "rmat":
        u, v = rmat(rng_graph, n, m)
    else:
        raise ValueError(f"unknown graph kind {kind!r}")
    perm = rng_relabel.permutation(n).astype(np.int64)
    return csr_from_undirected(n, perm[u], perm[v])


# special graphs used by tests --------------------------------------------
def permutation_graph(n: int, rng: np.random.Generator) -> Graph:
    """Each row holds exactly one entry, 1.0, at a random permuted column."""
    p = rng.permutation(n)
    return csr_from_pairs(n, np.arange(n), p, np.ones(n, np.float32))


def circulant_graph(n: int, offsets) -> Graph:
    """Row i holds columns (i + o) mod n and (i - o) mod n for each offset o
    (distinct, 0 < o < n/2): an undirected graph of degree 2 * len(offsets)
    whose rows reach across the whole vertex range."""
    o = np.asarray(offsets, dtype=np.int64)
    i = np.arange(n, dtype=np.int64)[:, None]
    cols = np.sort(np.concatenate([(i + o) % n, (i - o) % n], axis=1), axis=1)
    deg = cols.shape[1]
    indptr = (np.arange(n + 1, dtype=np.int64) * deg).astype(np.int32)
    vals = np.full(n * deg, np.float32(1.0) / np.float32(deg), dtype=np.float32)
    return Graph(n, indptr, cols.reshape(-1).astype(np.int32), vals)


def complete_graph(n: int) -> Graph:
    i, j = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    keep = i != j
    return csr_from_pairs(n, i[keep], j[keep])


def star_graph(n: int) -> Graph:
    """Vertex 0 joined to all others: one row of length n-1, the rest of length 1."""
    leaves = np.arange(1, n)
    return csr_from_undirected(n, np.zeros(n - 1, np.int64), leaves)


def empty_graph(n: int) -> Graph:
    return Graph(n, np.zeros(n + 1, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))


# --------------------------------------------------------------------------
# workloads
# --------------------------------------------------------------------------
@dataclass
class Spec:
    """A GCN fwd+bwd workload on one sampled subgraph."""
    name: str
    n: int
    graph: str                      # "er" | "rmat"
    d: int                          # average degree (nnz = n*d)
    layers: List[Tuple[int, int]]   # (f_in, h) per layer; output width 2h
    head: Optional[str]             # None (dY given) | "ce" | "bce"
    classes: int = 0
    label_p: float = 0.1            # Bernoulli rate for BCE targets
    d_range: Optional[Tuple[int, int]] = None  # per-subgraph degree draw (epoch stream)
    subgraphs: int = 1
    self_loops: bool = False        # add a self-connection to every vertex (Sec. V-B)


@dataclass
class Layer:
    W_self: np.ndarray   # float32 [f_in, h]
    W_neigh: np.ndarray  # float32 [f_in, h]
    bias: np.ndarray     # float32 [2h]

    @property
    def f_in(self) -> int:
        return self.W_self.shape[0]

    @property
    def h(self) -> int:
        return self.W_self.shape[1]


@dataclass
class Workload:
    spec: Spec
    s: int
    graph: Graph
    H: np.ndarray                     # float32 [n, f_in(1)]
    layers: List[Layer]
    W_pred: Optional[np.ndarray] = None   # float32 [2h_L, C]
    b_pred: Optional[np.ndarray] = None   # float32 [C]
    labels: Optional[np.ndarray] = None   # int32 [n]           (ce)
    targets: Optional[np.ndarray] = None  # float32 [n, C] {0,1} (bce)
    dY: Optional[np.ndarray] = None       # float32 [n, 2h_L]    (no head)
    d: int = 0

    @property
    def n(self) -> int:
        return self.graph.n


def periodic_normal(rng: np.random.Generator, n: int, f: int, period: int = 65537):
    """An n x f float32 matrix described by parts, for matrices too large to
    draw entry by entry in seconds (billions of entries): row i is
    2^e_i * R[i mod period] with R ~ N(0, 1) (period x f) and e_i uniform on
    {-1, 0, 1}.  The scaling is exact in float32, and no two rows 2^k rows
    apart are equal (the period is odd).  Returns (R, e); periodic_rows
    gives rows of the matrix."""
    R = rng.standard_normal((min(period, n), f), dtype=np.float32)
    e = rng.integers(-1, 2, size=n).astype(np.int8)
    return R, e


def periodic_rows(R: np.ndarray, e: np.ndarray, rows) -> np.ndarray:
    """Rows `rows` of the matrix described by periodic_normal's parts."""
    rows = np.asarray(rows, dtype=np.int64)
    return np.ldexp(R[rows % R.shape[0]], e[rows].astype(np.int32)[:, None]).astype(np.float32)


def glorot(rng: np.random.Generator, fan_in: int, fan_out: int) -> np.ndarray:
    a = math.sqrt(6.0 / (fan_in + fan_out))
    return rng.uniform(-a, a, size=(fan_in, fan_out)).astype(np.float32)


def build(spec: Spec, s: int = 0, cfg_key: int = 99, n: Optional[int] = None) -> Workload:
    """Draw one seeded workload.  ``n`` overrides the vertex count (same family)."""
    n_eff = spec.n if n is None else int(n)
    key = [SEED_ROOT, cfg_key, s] + ([n_eff] if n is not None else [])
    children = np.random.SeedSequence(key).spawn(6)
    rg_graph, rg_relabel, rg_h, _, rg_lab, rg_deg = (
        np.random.Generator(np.random.PCG64(c)) for c in children)
    rg_w = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, cfg_key, WEIGHT_KEY])))
    d = spec.d
    if spec.d_range is not None:
        d = int(rg_deg.integers(spec.d_range[0], spec.d_range[1] + 1))
    g = make_graph(spec.graph, n_eff, d, rg_graph, rg_relabel)
    if spec.self_loops:
        g = with_self_loops(g)
    f0 = spec.layers[0][0]
    H = rg_h.standard_normal((n_eff, f0), dtype=np.float32)
    layers = []
    for (f_in, h) in spec.layers:
        Ws = glorot(rg_w, f_in, h)
        Wn = glorot(rg_w, f_in, h)
        layers.append(Layer(Ws, Wn, np.zeros(2 * h, np.float32)))
    wl = Workload(spec, s, g, H, layers, d=d)
    hl2 = 2 * spec.layers[-1][1]
    if spec.head is None:
        wl.dY = rg_lab.standard_normal((n_eff, hl2), dtype=np.float32)
    else:
        C = spec.classes
        wl.W_pred = glorot(rg_w, hl2, C)
        wl.b_pred = np.zeros(C, np.float32)
        if spec.head == "ce":
            wl.labels = rg_lab.integers(0, C, size=n_eff).astype(np.int32)
        elif spec.head == "bce":
            wl.targets = (rg_lab.random((n_eff, C)) < spec.label_p).astype(np.float32)
        else:
            raise ValueError(spec.head)
    return wl


# The five workloads.  Attribute widths / class counts follow Table I
# (PPI 50, Reddit 602/41 single-label, Yelp 300/100 multi-label, Amazon 200),
# the hidden width 512 follows Sec. VI-C.
WORKLOADS = {
    0: Spec("er2000_d15_50x64_givendY", 2000, "er", 15, [(50, 64)], None),
    1: Spec("rmat8000_d20_602-128-128_ce41", 8000, "rmat", 20, [(602, 128), (256, 128)], "ce", 41),
    2: Spec("rmat16000_d30_300-256x3_bce100", 16000, "rmat", 30,
            [(300, 256), (512, 256), (512, 256)], "bce", 100),
    3: Spec("rmat65536_d50_512-512-512_ce100", 65536, "rmat", 50, [(512, 512), (1024, 512)], "ce", 100),
    4: Spec("stream200_rmat50000_d30-50_200-512x3_ce50", 50000, "rmat", 40,
            [(200, 512), (1024, 512), (1024, 512)], "ce", 50, d_range=(30, 50), subgraphs=200),
}


def config(cfg: int, s: int = 0, n: Optional[int] = None, self_loops: bool = False) -> Workload:
    """Workload `cfg`; with ``self_loops`` the same draw with a self-connection
    added to every vertex of the graph."""
    spec = WORKLOADS[cfg]
    if self_loops:
        import dataclasses
        spec = dataclasses.replace(spec, name=spec.name + "_selfloops", self_loops=True)
    return build(spec, s=s, cfg_key=cfg, n=n)


def custom(n: int, graph: str, d: int, layers, head=None, classes=0, seed: int = 0,
           self_loops: bool = False) -> Workload:
    """Small workloads for tests (ragged sizes spanning several tiles)."""
    spec = Spec(f"custom_{graph}{n}_d{d}", n, graph, d, list(layers), head, classes, self_loops=self_loops)
    return build(spec, s=seed, cfg_key=1000)


# --------------------------------------------------------------------------
# training graphs for the sampler (the graph G that subgraphs are drawn from)
# --------------------------------------------------------------------------
@dataclass
class TrainingGraph:
    """G with its vertex attributes H^(0) and labels (the input of Alg. 5)."""
    name: str
    graph: Graph
    X: np.ndarray        # float32 [nV, f]
    labels: np.ndarray   # int32 [nV] in [0, classes)
    classes: int


def training_graph(n: int, d: int, f: int, classes: int, seed: int = 0, kind: str = "rmat",
                   name: Optional[str] = None) -> TrainingGraph:
    """Undirected graph with n*d/2 edges (R-MAT by default), N(0,1) attributes,
    uniform single-label classes.  Streams: SeedSequence([181011899, 2000,
    seed, n]) spawned into graph, relabel, attributes, labels."""
    children = np.random.SeedSequence([SEED_ROOT, 2000, seed, n]).spawn(4)
    rg_graph, rg_relabel, rg_x, rg_lab = (np.random.Generator(np.random.PCG64(c)) for c in children)
    g = make_graph(kind, n, d, rg_graph, rg_relabel)
    X = rg_x.standard_normal((n, f), dtype=np.float32)
    labels = rg_lab.integers(0, classes, size=n).astype(np.int32)
    return TrainingGraph(name or f"{kind}{n}_d{d}_f{f}_c{classes}", g, X, labels, classes)


# A Reddit-shaped training graph (Table I: 232,965 vertices, 602 attributes,
# 41 classes), R-MAT with 50 stored edges per vertex on average.
TRAINING_GRAPHS = {
    "reddit_like": dict(n=232965, d=50, f=602, classes=41),
}
