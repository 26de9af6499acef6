"""gcn_aggregate_noalloc (scratch in the library's static device array)
against gcn_aggregate (caller workspace), through the C ABI: bitwise equal
results on consecutive calls, the second smaller than the first, in both
precisions; a size past the array is refused before any launch."""
import numpy as np
import pytest
import torch

from paper_1810_11899_amd import binding as B
from paper_1810_11899_amd import synth

from gpu_util import dev, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def _case(n, d, k, seed):
    g = synth.custom(n, "rmat", d, [(4, 4)], seed=seed).graph
    X = np.random.default_rng(seed).standard_normal((n, k)).astype(np.float32)
    return B.DeviceCSR.from_host(g.n, g.n, g.indptr, g.indices, g.vals), dev(X)


@pytest.mark.parametrize("prec", [B.GCN_F32, B.GCN_BF16])
def test_noalloc_matches_workspace_entry_point(prec):
    ws = B.Workspace("cuda")
    # first a large call (many wavefronts, hub rows cut across wavefronts),
    # then a smaller one that reuses the array the first left behind
    for n, d, k, seed in [(20000, 24, 384 if prec == B.GCN_F32 else 256, 1), (3001, 9, 130, 2)]:
        print(f"noalloc vs workspace: prec={prec} n={n} d={d} k={k}", flush=True)
        A, X = _case(n, d, k, seed)
        ref = torch.full((n, k), float("nan"), device="cuda")
        got = torch.full((n, k), float("nan"), device="cuda")
        B.gcn_aggregate(A, X, ref, ws, prec)
        B.gcn_aggregate_noalloc(A, X, got, prec)
        torch.cuda.synchronize()
        assert torch.equal(ref.view(torch.int32), got.view(torch.int32)), (n, k)


def test_noalloc_rejects_sizes_past_its_array():
    n, k = 65536, 2048
    need = B.lib().gcn_aggregate_workspace_bytes(n, n, n * 50, k, B.GCN_F32)
    assert need > B.GCN_NOALLOC_SCRATCH_BYTES
    ip = np.zeros(n + 1, np.int32)
    ip[1:] = np.minimum(np.arange(1, n + 1) * 50, n * 50)
    A = B.DeviceCSR(n, n, torch.from_numpy(ip).cuda(), torch.zeros(n * 50, dtype=torch.int32, device="cuda"),
                    torch.zeros(n * 50, device="cuda"))
    X = torch.zeros((n, k), device="cuda")
    out = torch.full((n, k), 7.0, device="cuda")
    with pytest.raises(B.GcnError) as e:
        B.gcn_aggregate_noalloc(A, X, out, B.GCN_F32)
    assert e.value.code == B.GCN_EUNSUPPORTED
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())   # nothing was launched
