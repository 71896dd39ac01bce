"""The five workload configurations and their scaled-down parity instances.

Each configuration is an agentic-RL update batch: G rollouts for each of Q task
(or task-harness) groups, packed back to back, with a loss mask that alternates
harness/tool observation segments (mask 0) and policy-generated segments
(mask 1).  Shapes follow the RL batch sizes of the paper's experiments section
(GRPO: tasks x rollouts per update; 64K-token context) and Qwen-shaped LM heads.

Conventions fixed here (they are input recipes, not arithmetic):
  * a std written as "N(0, x)" in a configuration is the standard deviation x;
  * every rollout starts with a masked (prompt/tool) segment, then policy and tool
    segments alternate with geometric lengths on {1, 2, ...}; the policy-segment
    mean is tool_mean * (1 - f) / f for a masked fraction f;
  * group ids are opaque int32 keys (random distinct values), and for the larger
    batches the rollouts of different groups are interleaved in the packed
    order, since task-harness pairs are randomly mixed within a batch.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    number: int                 # 1..5; the structure seed is 20260000 + number
    groups: int                 # Q
    rollouts_per_group: int     # G
    len_min: int                # rollout length range (inclusive); equal => fixed T
    len_max: int
    d: int
    V: int
    dtype: str                  # "f32" or "bf16": hidden, W and dhidden
    h_std: float
    w_std: float
    masked_frac: float          # expected fraction of tokens with mask 0
    tool_mean: float            # mean masked-segment length
    reward: str                 # "bernoulli" | "uniform" | "uniform_ties"
    reward_p: float = 0.5
    eps_low: float = 0.2
    eps_high: float = 0.2
    entropy_coef: float = 0.0
    sigma_old: float = 0.1
    anchor: str = "gaussian"    # how old log-probs are placed: "oracle" | "gaussian"
    interleave_groups: bool = False
    forced_equal_groups: tuple = ()   # reward values of groups forced all-equal
    n_excluded: int = 0         # rollouts marked excluded (group id < 0)
    seed_offset: int = 0

    @property
    def R(self) -> int:
        return self.groups * self.rollouts_per_group

    @property
    def seed(self) -> int:
        return 20260000 + self.number + self.seed_offset

    @property
    def policy_mean(self) -> float:
        f = self.masked_frac
        return self.tool_mean * (1.0 - f) / f

    def with_(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


CONFIGS = {
    # 2 groups x 4 rollouts, T = 256; d = 256, V = 4096, fp32; W std 1/sqrt(256);
    # policy/tool segments of mean 32; Bernoulli(0.5) rewards; eps 0.2; old = oracle + N(0, 0.05).
    "tiny_fp32": Config(
        name="tiny_fp32", number=1, groups=2, rollouts_per_group=4, len_min=256, len_max=256,
        d=256, V=4096, dtype="f32", h_std=1.0, w_std=1.0 / 16.0, masked_frac=0.5, tool_mean=32.0,
        reward="bernoulli", reward_p=0.5, eps_low=0.2, eps_high=0.2, sigma_old=0.05, anchor="oracle"),
    # 8 x 8 rollouts, T = 2048; d = 2048, V = 32768, bf16; W std 1/sqrt(d); 40% masked in
    # tool segments of mean 64; rewards U[0, 1); eps 0.2; old perturbed by N(0, 0.1).
    "small_bf16": Config(
        name="small_bf16", number=2, groups=8, rollouts_per_group=8, len_min=2048, len_max=2048,
        d=2048, V=32768, dtype="bf16", h_std=1.0, w_std=1.0 / math.sqrt(2048.0), masked_frac=0.4,
        tool_mean=64.0, reward="uniform", eps_low=0.2, eps_high=0.2, sigma_old=0.1),
    # Qwen-8B-shaped LM head: 16 x 8 rollouts, T = 4096; d = 4096, V = 151936; W std 0.02;
    # 60% masked tool tokens; Bernoulli(0.3) rewards; eps_low 0.2, eps_high 0.28.
    "qwen8b_bf16": Config(
        name="qwen8b_bf16", number=3, groups=16, rollouts_per_group=8, len_min=4096, len_max=4096,
        d=4096, V=151936, dtype="bf16", h_std=1.0, w_std=0.02, masked_frac=0.6, tool_mean=64.0,
        reward="bernoulli", reward_p=0.3, eps_low=0.2, eps_high=0.28, sigma_old=0.1,
        interleave_groups=True),
    # Long-horizon: 4 x 8 rollouts of U{8192..32768} tokens, varlen packed; d = 5120;
    # 70% masked harness/tool tokens in segments of mean 256; Bernoulli(0.2) rewards.
    "long_bf16": Config(
        name="long_bf16", number=4, groups=4, rollouts_per_group=8, len_min=8192, len_max=32768,
        d=5120, V=151936, dtype="bf16", h_std=1.0, w_std=0.02, masked_frac=0.7, tool_mean=256.0,
        reward="bernoulli", reward_p=0.2, eps_low=0.2, eps_high=0.2, sigma_old=0.1),
    # Large batch: 64 x 16 rollouts of U{1024..8192} tokens; d = 4096; 50% masked;
    # rewards on a 1/8 grid (ties) plus groups forced all-equal; entropy coefficient 1e-3.
    "large_bf16": Config(
        name="large_bf16", number=5, groups=64, rollouts_per_group=16, len_min=1024, len_max=8192,
        d=4096, V=151936, dtype="bf16", h_std=1.0, w_std=0.02, masked_frac=0.5, tool_mean=64.0,
        reward="uniform_ties", eps_low=0.2, eps_high=0.2, entropy_coef=1e-3, sigma_old=0.1,
        interleave_groups=True, forced_equal_groups=(0.0, 1.0, 0.3, 0.625)),
}

ORDER = ["tiny_fp32", "small_bf16", "qwen8b_bf16", "long_bf16", "large_bf16"]


def get_config(name: str) -> Config:
    return CONFIGS[name]


# Scaled instances keep d, V, dtype, value laws, mask statistics, reward law, eps and the
# entropy coefficient of their configuration, and shrink the number of rollouts and their
# lengths so the fp64 oracle finishes in seconds while the batch still spans several token
# tiles, several vocabulary tiles and a ragged tail.
_SCALED = {
    "tiny_fp32": dict(),
    "small_bf16": dict(groups=2, rollouts_per_group=4, len_min=640, len_max=640),
    "qwen8b_bf16": dict(groups=2, rollouts_per_group=4, len_min=240, len_max=240),
    "long_bf16": dict(groups=2, rollouts_per_group=3, len_min=300, len_max=520, tool_mean=48.0),
    "large_bf16": dict(groups=3, rollouts_per_group=4, len_min=100, len_max=240,
                       forced_equal_groups=(0.625,)),
}


def scaled_config(name: str, **overrides) -> Config:
    kw = dict(_SCALED[name])
    kw.update(overrides)
    base = CONFIGS[name]
    return base.with_(name=base.name + "_scaled", seed_offset=base.seed_offset + 100, **kw)


def describe(cfg: Config, n_tokens: Optional[int] = None) -> dict:
    out = {"workload": cfg.name, "rollouts": cfg.R, "groups": cfg.groups, "d": cfg.d,
           "V": cfg.V, "dtype": cfg.dtype}
    if cfg.len_min == cfg.len_max:
        out["T"] = cfg.len_min
    else:
        out["T_range"] = [cfg.len_min, cfg.len_max]
    if n_tokens is not None:
        out["N"] = int(n_tokens)
    return out
