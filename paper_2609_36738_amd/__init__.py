"""MI355X (gfx950) implementation of the per-step hot path of Backpropagated Output Momentum.

The product is ``libbom.so`` (C-ABI in ``include/bom.h``): hand-written HIP kernels for the
residual / batch-mean residual, the task-space EMA, the output-head vector-Jacobian product
with the history folded into the logit gradient, and the second-moment parameter update.
``paper_2609_36738_amd.bom`` is a thin ctypes binding with the same entry-point names.
"""
from . import bom  # noqa: F401
from .bom import (BomError, bom_ema, bom_head_forward, bom_head_vjp, bom_residual, bom_update,  # noqa: F401
                  make_update_cfg)
