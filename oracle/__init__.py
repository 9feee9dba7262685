"""CPU oracle of MoNe test-time learning: test infrastructure only (see mone_oracle)."""
from .mone_oracle import (  # noqa: F401
    ACTIVATIONS, LOSSES, memory_forward, memory_kv, segment_grad, segment_loss, sigmoid, silu,
    silu_grad, targets, ttl_run, ttl_run_layers, ttl_step,
)
from .paper_optimizer import (  # noqa: F401
    momentum_decay, paper_run, paper_step, renormalise, row_norms, softplus, token_rates,
    weighted_grad,
)
from .memory_attention import memory_attention  # noqa: F401
from . import swiglu_memory  # noqa: F401  (paper-form memory; names overlap the config form's)
