"""MI355X (gfx950) hot path of Non-blocking SGD (He & Dube, arXiv 2211.00889).

The product is the C-ABI library ``libnbsgd.so`` (declared in ``include/nbsgd.h``);
``_lib`` is its ctypes binding with the same names.
"""

from ._lib import (  # noqa: F401
    DELAY_CONST,
    DELAY_EXP,
    DELAY_LOMAX,
    MIX_THEN_STEP,
    STEP_THEN_MIX,
    Matcha,
    NbsgdError,
    accumulate,
    iteration_accounting,
    load,
    minibatch_indices,
    mix,
    mlp_grad,
    mlp_grad_noalloc,
    mlp_grad_strided,
    mlp_loss,
    mlp_param_count,
    mlp_workspace_bytes,
    row_stride,
    sample_mask,
    step,
    step_server,
    step_strided,
    update,
    w_allreduce,
    w_ring,
)
