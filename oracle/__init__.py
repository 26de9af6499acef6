"""CPU oracle (test infrastructure only; see gcnref.py)."""
from .gcnref import (aggregate, build, csr_transpose, layer_bwd, layer_bwd_envelope, layer_fwd,
                     loss_grad, num_threads, step, LayerCache, StepResult)
from . import optim, sampler

__all__ = ["aggregate", "build", "csr_transpose", "layer_bwd", "layer_bwd_envelope", "layer_fwd",
           "loss_grad", "num_threads", "optim", "sampler", "step", "LayerCache", "StepResult"]
