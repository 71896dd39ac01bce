"""Seeded synthetic inputs shaped like agentic-RL policy-gradient batches.

This package is the only code shared by the GPU path's tests/benchmark and the
fp64 oracle.  It holds no part of the method's arithmetic: it draws lengths,
loss masks, target ids, rewards, group ids, hidden states, LM-head weights and
the Gaussian noise that perturbs old log-probs, and nothing else.

Integer structure and per-token noise come from NumPy's PCG64 so they are
reproducible bit-for-bit on any host; the large float tensors (hidden states
and LM-head weights) come from torch's generator on the requested device.
"""
from .configs import CONFIGS, Config, get_config, scaled_config
from .gen import (Structure, make_structure, make_tensors, old_logp_from_anchor, perturbed_logps,
                  sample_policy_rows, token_values)

__all__ = [
    "CONFIGS",
    "Config",
    "get_config",
    "scaled_config",
    "Structure",
    "make_structure",
    "make_tensors",
    "old_logp_from_anchor",
    "perturbed_logps",
    "sample_policy_rows",
    "token_values",
]
