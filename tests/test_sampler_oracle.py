"""Pins of the sampler oracle (CPU only).

The frontier sampler draws random numbers, so the oracle is pinned by:
  * its generator against an independent implementation (numpy's Philox) and
    the generator's published all-zero test vector;
  * the exact distribution of the frontier-sampling Markov chain (Sec. IV-A,
    Alg. 2: pop u with probability w(u) / sum of w over the frontier, step to a
    uniform neighbour), enumerated path by path on tiny graphs, against the
    empirical distribution of the Dashboard implementation over many sampler
    ids -- with and without constant cleanups, for several probe widths p,
    with a degree cap, and on a directed graph whose frontier can run dry;
  * invariants (distinct roots, each added vertex adjacent to an earlier one,
    determinism) and the status of the degenerate cases;
  * the induced subgraph against the dense adjacency submatrix.
"""
import itertools
from collections import Counter, defaultdict
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

from oracle import sampler as S
from paper_1810_11899_amd import synth


# ------------------------------------------------------------- generator ----
def test_philox_matches_numpy_philox():
    rng = np.random.default_rng(7)
    for _ in range(50):
        key = rng.integers(0, 2 ** 63, 2, dtype=np.uint64) * np.uint64(2) + rng.integers(0, 2, 2, dtype=np.uint64)
        ctr = rng.integers(0, 2 ** 63, 4, dtype=np.uint64)
        bg = np.random.Philox(key=key, counter=ctr)
        got_np = bg.random_raw(4)  # numpy advances the counter by one before each block
        nxt = [int(ctr[0]) + 1, int(ctr[1]), int(ctr[2]), int(ctr[3])]
        carry = nxt[0] >> 64
        nxt[0] &= 2 ** 64 - 1
        nxt[1] += carry
        assert np.array_equal(S.philox4x64(nxt, key), got_np)


def test_philox_counter_carry_matches_numpy():
    key = np.array([5, 9], np.uint64)
    ctr = np.array([2 ** 64 - 1, 3, 0, 0], np.uint64)
    got_np = np.random.Philox(key=key, counter=ctr).random_raw(4)
    assert np.array_equal(S.philox4x64([0, 4, 0, 0], key), got_np)


def test_philox_published_zero_vector():
    # Philox4x64-10, counter 0, key 0 (the generator's published known answer)
    want = [0x16554D9ECA36314C, 0xDB20FE9D672D0FDC, 0xD7E772CEE186176B, 0x7E68B68AEC7BA23B]
    assert [int(x) for x in S.philox4x64([0, 0, 0, 0], [0, 0])] == want


# ------------------------------------------------- exact Markov chain pins ----
def _weights(indptr, cap):
    deg = np.diff(indptr)
    return np.minimum(deg, cap) if cap > 0 else deg


def exact_distribution(indptr, indices, m, n, cap=0):
    """Probability of every outcome (sorted roots, added vertices in order) of
    frontier sampling, by enumerating the chain of Alg. 2: roots a uniform
    m-subset; then n - m times pop a frontier entry with probability
    w / (sum of w) and replace it by a uniform neighbour.  A frontier whose
    weights are all zero ends the run early."""
    nV = len(indptr) - 1
    w = _weights(indptr, cap)
    dist = defaultdict(Fraction)

    def walk(fs, added, prob):
        if len(added) == n - m:
            dist[(tuple(sorted(root_set)), tuple(added))] += prob
            return
        tot = sum(int(w[u]) for u in fs)
        if tot == 0:
            dist[(tuple(sorted(root_set)), tuple(added))] += prob
            return
        for e, u in enumerate(fs):
            if w[u] == 0:
                continue
            nb = indices[indptr[u]:indptr[u + 1]]
            for v in nb:
                walk(fs[:e] + fs[e + 1:] + [int(v)], added + [int(v)],
                     prob * Fraction(int(w[u]), tot) / len(nb))

    combos = list(itertools.combinations(range(nV), m))
    for root_set in combos:
        walk(list(root_set), [], Fraction(1, len(combos)))
    return dist


def empirical(indptr, indices, m, n, db_cap, ia_cap, cap, p, runs, seed=11):
    c = Counter()
    statuses = Counter()
    for sid in range(runs):
        v, st = S.frontier_sample(indptr, indices, m, n, db_cap, ia_cap, cap=cap, p=p, seed=seed, sampler_id=sid)
        statuses[st] += 1
        c[(tuple(sorted(v[:m].tolist())), tuple(v[m:].tolist()))] += 1
    return c, statuses


def chi2_pvalue(exact, observed, runs, min_bins=10):
    keys = sorted(exact, key=lambda k: exact[k])
    for k in observed:
        assert k in exact, f"outcome {k} is impossible under Alg. 2"
    exp, obs = [], []
    pool_e = pool_o = 0.0
    for k in keys:
        e = float(exact[k]) * runs
        if e < 5:
            pool_e += e
            pool_o += observed.get(k, 0)
        else:
            exp.append(e)
            obs.append(observed.get(k, 0))
    if pool_e > 0:
        exp.append(pool_e)
        obs.append(pool_o)
    assert len(exp) >= min_bins
    return stats.chisquare(obs, exp).pvalue


def small_graph():
    # 0-1, 0-2, 0-3, 1-2, 3-4, 4-5; vertex 6 isolated
    pairs = [(0, 1), (0, 2), (0, 3), (1, 2), (3, 4), (4, 5)]
    r = [a for a, b in pairs] + [b for a, b in pairs]
    c = [b for a, b in pairs] + [a for a, b in pairs]
    g = synth.csr_from_pairs(7, np.array(r), np.array(c))
    return g.indptr, g.indices


@pytest.mark.parametrize("p, small_db, cap", [(1, False, 0), (3, True, 0), (64, False, 0), (64, True, 0),
                                             (64, True, 2)])
def test_frontier_distribution_matches_alg2(p, small_db, cap):
    ip, ix = small_graph()
    m, n = 2, 4
    w = _weights(ip, cap)
    if small_db:   # Dashboard just large enough: a cleanup before nearly every append
        db_cap, ia_cap = m * int(w.max()), m + 1
    else:
        db_cap, ia_cap = 10 * m * int(w.max()), 64
    exact = exact_distribution(ip, ix, m, n, cap)
    assert abs(sum(exact.values()) - 1) == 0
    runs = 40000
    obs, statuses = empirical(ip, ix, m, n, db_cap, ia_cap, cap, p, runs)
    assert set(statuses) <= {"ok", "exhausted"}
    assert chi2_pvalue(exact, obs, runs) > 1e-4


def test_frontier_distribution_directed_graph_runs_dry():
    # directed: 0->1, 1->2, 2->0, 0->3, 3 has no out-edges (weight 0)
    g = synth.csr_from_pairs(4, np.array([0, 1, 2, 0]), np.array([1, 2, 0, 3]))
    m, n = 1, 5
    exact = exact_distribution(g.indptr, g.indices, m, n)
    runs = 30000
    obs, statuses = empirical(g.indptr, g.indices, m, n, 8, 4, 0, 64, runs)
    assert statuses["exhausted"] > 0 and statuses["ok"] > 0
    assert chi2_pvalue(exact, obs, runs, min_bins=5) > 1e-4


def test_planted_uniform_pop_is_detected():
    """The chi-square pin has the power to see a plausible mistake: popping
    uniformly over the frontier instead of by degree."""
    ip, ix = small_graph()
    m, n = 2, 4
    exact = exact_distribution(ip, ix, m, n)
    nV = len(ip) - 1
    rng = np.random.default_rng(3)
    runs = 40000
    obs = Counter()
    for _ in range(runs):
        roots = rng.choice(nV, m, replace=False).tolist()
        fs, added = list(roots), []
        for _ in range(n - m):
            live = [e for e, u in enumerate(fs) if ip[u + 1] > ip[u]]
            if not live:
                break
            e = live[rng.integers(len(live))]        # the planted mistake
            nb = ix[ip[fs[e]]:ip[fs[e] + 1]]
            v = int(nb[rng.integers(len(nb))])
            fs[e] = v
            added.append(v)
        obs[(tuple(sorted(roots)), tuple(added))] += 1
    assert chi2_pvalue(exact, obs, runs) < 1e-6


# ------------------------------------------------------------ invariants ----
def test_invariants_on_rmat_graph():
    g = synth.custom(3000, "rmat", 20, [(4, 4)], seed=2).graph
    m, n = 200, 1500
    db_cap, ia_cap = int(2 * m * g.nnz / g.n) + 64, 1024
    for sid in range(3):
        v, st = S.frontier_sample(g.indptr, g.indices, m, n, db_cap, ia_cap, cap=30, seed=5, sampler_id=sid)
        assert st == "ok" and v.shape == (n,)
        assert np.unique(v[:m]).size == m
        adj = set(zip(np.repeat(np.arange(g.n), g.degrees()).tolist(), g.indices.tolist()))
        seen = set(v[:m].tolist())
        for x in v[m:].tolist():
            assert any((y, x) in adj for y in seen) or x in seen
            seen.add(x)
    a, _ = S.frontier_sample(g.indptr, g.indices, m, n, db_cap, ia_cap, cap=30, seed=5, sampler_id=1)
    b, _ = S.frontier_sample(g.indptr, g.indices, m, n, db_cap, ia_cap, cap=30, seed=5, sampler_id=1)
    c, _ = S.frontier_sample(g.indptr, g.indices, m, n, db_cap, ia_cap, cap=30, seed=6, sampler_id=1)
    assert np.array_equal(a, b) and not np.array_equal(a, c)


def test_degenerate_cases():
    e = synth.empty_graph(50)
    v, st = S.frontier_sample(e.indptr, e.indices, 10, 30, 16, 32)
    assert st == "exhausted" and v.size == 10 and np.unique(v).size == 10
    v, st = S.frontier_sample(e.indptr, e.indices, 10, 10, 16, 32)
    assert st == "ok" and v.size == 10
    g = synth.complete_graph(12)
    v, st = S.frontier_sample(g.indptr, g.indices, 12, 40, 12 * 11, 13)   # every vertex a root
    assert st == "ok" and sorted(v[:12].tolist()) == list(range(12))
    v, st = S.frontier_sample(g.indptr, g.indices, 4, 40, 4 * 11 - 1, 8)    # roots overflow
    assert st == "overflow" and v.size == 4
    assert S.frontier_sample(g.indptr, g.indices, 13, 40, 1000, 64)[1] == "einval"
    assert S.frontier_sample(g.indptr, g.indices, 4, 3, 1000, 64)[1] == "einval"
    assert S.frontier_sample(g.indptr, g.indices, 4, 10, 1000, 4)[1] == "einval"


# ------------------------------------------------------- induced subgraph ----
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_induce_matches_dense_submatrix(seed):
    g = synth.custom(300, "rmat", 8, [(4, 4)], seed=seed).graph
    rng = np.random.default_rng(seed)
    verts = rng.integers(0, g.n, 120)          # duplicates on purpose
    vsub, ip, ix, vals = S.induce(g.indptr, g.indices, verts)
    assert np.array_equal(vsub, np.unique(verts))
    dense = np.zeros((g.n, g.n), bool)
    dense[np.repeat(np.arange(g.n), g.degrees()), g.indices] = True
    sub = dense[np.ix_(vsub, vsub)]
    rows = np.repeat(np.arange(vsub.size), np.diff(ip))
    got = np.zeros_like(sub)
    got[rows, ix] = True
    assert np.array_equal(got, sub)
    assert np.array_equal(got, got.T)            # G is undirected
    assert np.all(np.diff(ix)[np.diff(rows) == 0] > 0)
    lens = np.diff(ip)
    assert np.all(vals == (np.float32(1) / lens[rows].astype(np.float32)))


def test_gather_rows_pins():
    """The row gather of GCN construction, pinned by what a copy of rows must
    satisfy rather than by re-stating it: rows that carry their own index come
    back carrying the requested index; the identity list gives X; gathering by
    a then by b is gathering by a[b]; a permutation and its inverse cancel;
    integer rows (labels) are copied exactly, int32 extremes included."""
    rng = np.random.default_rng(9)
    nX, w = 500, 7
    X = (np.arange(nX, dtype=np.float32)[:, None] * 16 + np.arange(w, dtype=np.float32)[None, :])
    rows = rng.integers(0, nX, 300)
    out = S.gather_rows(X, rows)
    assert out.shape == (300, w) and out.dtype == np.float32
    assert np.array_equal(out[:, 0] / 16, rows.astype(np.float32))
    assert np.array_equal(out - out[:, :1], np.broadcast_to(np.arange(w, dtype=np.float32), out.shape))
    Y = rng.standard_normal((nX, w)).astype(np.float32)
    assert np.array_equal(S.gather_rows(Y, np.arange(nX)).view(np.uint32), Y.view(np.uint32))
    a, b = rng.integers(0, nX, 400), rng.integers(0, 400, 250)
    assert np.array_equal(S.gather_rows(S.gather_rows(Y, a), b), S.gather_rows(Y, a[b]))
    perm = rng.permutation(nX)
    inv = np.empty_like(perm)
    inv[perm] = np.arange(nX)
    assert np.array_equal(S.gather_rows(S.gather_rows(Y, perm), inv), Y)
    lab = np.array([[2 ** 31 - 1], [-2 ** 31], [0], [41]], np.int32)
    got = S.gather_rows(lab, np.array([3, 0, 1, 1, 2]))
    assert got.dtype == np.int32 and got[:, 0].tolist() == [41, 2 ** 31 - 1, -2 ** 31, -2 ** 31, 0]
    assert S.gather_rows(Y, np.zeros(0, np.int64)).shape == (0, w)


# ------------------------------------------------ draw layout, known answer ----
# The oracle's sampler must take its random numbers exactly where the sampler
# header says they come from (the same stream layout the GPU sampler uses, so
# that both give the same subgraph for the same seed and run id).  The known
# answer below is built WITHOUT the oracle: numpy's own Philox4x64-10 gives
# the blocks, and a short re-statement of the documented run (roots, Dashboard
# probing rounds, neighbour choice, cleanup) turns them into a vertex list.
def _np_block(seed, sid, kind, c0, c2):
    """Philox4x64-10 block at counter (c0, kind, c2, 0), key (seed, sid), from
    numpy (which steps its counter by one before producing a block)."""
    c = (int(c0) | (int(kind) << 64) | (int(c2) << 128)) - 1
    ctr = np.array([(c >> (64 * w)) & (2 ** 64 - 1) for w in range(4)], dtype=np.uint64)
    return np.random.Philox(key=np.array([seed, sid], np.uint64), counter=ctr).random_raw(4)


def _np_below(word, N):
    return (int(word) * int(N)) >> 64


def _documented_run(indptr, indices, m, n, db_cap, ia_cap, cap, p, seed, sid):
    """The vertex list the documented draw layout gives: root candidate t from
    word 0 of counter (t, 1, 0, 0); probe of processor j in the run's r-th
    probing round from word r % 4 of counter (r // 4, 2, j, 0), uniform over
    the used Dashboard, first hitting processor wins; neighbour of step t from
    word t % 4 of counter (t // 4, 3, 0, 0).  Dashboard entries name slots;
    cleanup keeps live slots in order before an overflowing append."""
    deg = np.diff(indptr)
    w = np.minimum(deg, cap) if cap > 0 else deg
    nV = len(deg)
    roots, t = [], 0
    while len(roots) < m:
        v = _np_below(_np_block(seed, sid, 1, t, 0)[0], nV)
        t += 1
        if v not in roots:
            roots.append(v)
    slots, db = [], []                       # slot = [vertex, weight, live]

    def append(v):
        slots.append([v, int(w[v]), True])
        db.extend([len(slots) - 1] * int(w[v]))

    for v in roots:
        append(v)
    out, r = list(roots), 0
    for i in range(m, n):
        if sum(s[1] for s in slots if s[2]) == 0:
            return out, "exhausted"
        k = None
        while k is None:
            for j in range(p):
                e = _np_below(_np_block(seed, sid, 2, r // 4, j)[r % 4], len(db))
                if slots[db[e]][2]:
                    k = db[e]
                    break
            r += 1
        slots[k][2] = False
        u = slots[k][0]
        t = i - m
        pick = _np_below(_np_block(seed, sid, 3, t // 4, 0)[t % 4], deg[u])
        v = int(indices[indptr[u] + pick])
        if len(db) + w[v] > db_cap or len(slots) == ia_cap:
            live = [s for s in slots if s[2]]
            slots.clear()
            db.clear()
            for s in live:
                slots.append(s)
                db.extend([len(slots) - 1] * s[1])
        append(v)
        out.append(v)
    return out, "ok"


@pytest.mark.parametrize("m, n, p, small_db, cap", [(2, 4, 64, False, 0), (2, 4, 1, False, 0),
                                                   (2, 11, 3, False, 0), (2, 11, 1, True, 0),
                                                   (3, 13, 64, True, 2)])
def test_draw_layout_known_answer(m, n, p, small_db, cap):
    """First roots, probes and neighbour picks of tiny runs on the 7-vertex
    graph, from numpy's Philox and the documented layout, against the oracle.
    n = 11 and 13 run past four neighbour steps and (with p <= 3) past four
    probing rounds, so the word index and the counter's first word both move;
    the small Dashboards force cleanups."""
    ip, ix = small_graph()
    deg = np.diff(ip)
    wmax = int((np.minimum(deg, cap) if cap else deg).max())
    db_cap, ia_cap = (m * wmax, m + 1) if small_db else (10 * m * wmax, 64)
    checked = 0
    for seed, sid in [(0, 0), (1, 0), (12345, 7), (2 ** 63 + 5, 2 ** 40 + 3)]:
        want, wst = _documented_run(ip, ix, m, n, db_cap, ia_cap, cap, p, seed, sid)
        got, st = S.frontier_sample(ip, ix, m, n, db_cap, ia_cap, cap=cap, p=p, seed=seed, sampler_id=sid)
        assert st == wst and got.tolist() == want, (seed, sid, got.tolist(), want)
        checked += len(want)
    assert checked >= 4 * n - 4


def test_draw_layout_known_answer_detects_a_swapped_word():
    """The known answer has the power to see a layout mistake: taking the
    neighbour word from word 0 of every block (instead of word t % 4) changes
    some run of the same sizes."""
    ip, ix = small_graph()
    orig = _np_block
    differs = False
    try:
        def word0(seed, sid, kind, c0, c2):
            b = orig(seed, sid, kind, c0, c2)
            return np.array([b[0]] * 4, np.uint64) if kind == 3 else b
        globals()["_np_block"] = word0
        for seed in range(6):
            a, _ = _documented_run(ip, ix, 2, 11, 200, 64, 0, 64, seed, 0)
            b, _ = S.frontier_sample(ip, ix, 2, 11, 200, 64, cap=0, p=64, seed=seed, sampler_id=0)
            differs |= a != b.tolist()
    finally:
        globals()["_np_block"] = orig
    assert differs
