"""Helpers shared by the GPU tests (comparison metric, device transfer)."""
import numpy as np
import pytest
import torch

# Parity gates (max relative error in the infinity norm, per output tensor).
TOL_F32 = 1e-4
TOL_BF16 = 2e-2


def rel_inf(gpu, ref, env=None) -> float:
    """max_i (|gpu_i - ref_i| - env_i)_+ / max_i |ref_i|.

    ``env`` is the oracle's per-entry ReLU-kink envelope (0 where no kink
    within float32 rounding can reach the entry); without it this is the plain
    infinity-norm relative error.
    """
    g = np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    assert g.shape == r.shape, (g.shape, r.shape)
    if r.size == 0:
        return 0.0
    d = np.abs(g - r)
    if env is not None:
        d = np.maximum(d - np.asarray(env, dtype=np.float64), 0.0)
    den = np.abs(r).max()
    num = d.max()
    if den == 0.0:
        return float(num)
    return float(num / den)


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_1810_11899_amd import binding
    binding.lib()  # raises loudly if the HIP library is missing


def dev(a, dtype=torch.float32):
    return torch.as_tensor(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)
