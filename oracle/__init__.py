"""fp64 CPU oracle for the policy-gradient hot path — TEST INFRASTRUCTURE ONLY.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
or call anything in this package.  The product path (the HIP library and its
Python binding) never does, and shares no code with it.
"""
from .rl_oracle import (  # noqa: F401
    AGG_SEQ,
    AGG_TOKEN,
    compact,
    group_index,
    group_advantage,
    token_logprob,
    token_weights,
    surrogate,
    tis_weight,
    kl_sampled,
    pg_loss_fwd_bwd,
    sampled_rows,
    loss_from_token_values,
    token_grad_weights,
    dw_rows,
    gae,
    value_loss,
    value_head,
    value_head_grads,
    tree_pack,
)
