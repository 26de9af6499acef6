"""CPU oracle (test infrastructure only; see gcnref.py)."""
from .gcnref import (aggregate, build, csr_transpose, layer_bwd, layer_bwd_envelope, layer_fwd,
                     loss_grad, num_threads, set_num_threads, step, LayerCache, StepResult, U32, C_AMB)
from . import optim, sampler

__all__ = ["aggregate", "build", "csr_transpose", "layer_bwd", "layer_bwd_envelope", "layer_fwd",
           "loss_grad", "num_threads", "optim", "set_num_threads", "sampler", "step", "LayerCache", "StepResult",
           "U32", "C_AMB"]
