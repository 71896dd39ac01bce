"""Seeded generators for packed agentic-RL batches (no method arithmetic here)."""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

from .configs import Config


@dataclasses.dataclass
class Structure:
    """Integer structure and per-token noise of one packed batch (host arrays)."""
    cfg: Config
    lengths: np.ndarray      # int64 [R]
    cu_seqlens: np.ndarray   # int32 [R+1], cu[0] = 0, cu[R] = N
    mask: np.ndarray         # uint8 [N], 1 = policy-generated token, 0 = harness/tool token
    targets: np.ndarray      # int32 [N], sampled token id aligned with hidden row t
    rewards: np.ndarray      # float32 [R]
    group_ids: np.ndarray    # int32 [R], opaque keys; < 0 marks an excluded rollout
    noise: np.ndarray        # float32 [N], standard normal draws for the old log-prob perturbation

    @property
    def N(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def R(self) -> int:
        return int(self.lengths.shape[0])


def _geometric(rng: np.random.Generator, mean: float, size: int) -> np.ndarray:
    # Geometric on {1, 2, ...} with the given mean (success probability 1 / mean).
    p = min(1.0, 1.0 / max(mean, 1.0))
    return rng.geometric(p, size=size).astype(np.int64)


def _rollout_mask(rng: np.random.Generator, T: int, tool_mean: float, policy_mean: float) -> np.ndarray:
    m = np.zeros(T, dtype=np.uint8)
    pos = 0
    is_policy = False  # every rollout opens with a prompt/tool segment
    batch = max(8, int(2 * T / max(1.0, min(tool_mean, policy_mean))) + 8)
    tool_len = _geometric(rng, tool_mean, batch)
    pol_len = _geometric(rng, policy_mean, batch)
    i = 0
    while pos < T:
        if i >= batch:
            tool_len = np.concatenate([tool_len, _geometric(rng, tool_mean, batch)])
            pol_len = np.concatenate([pol_len, _geometric(rng, policy_mean, batch)])
            batch *= 2
        L = int(pol_len[i] if is_policy else tool_len[i])
        end = min(T, pos + L)
        if is_policy:
            m[pos:end] = 1
            i += 1
        pos = end
        is_policy = not is_policy
    return m


def make_structure(cfg: Config, seed: Optional[int] = None) -> Structure:
    rng = np.random.Generator(np.random.PCG64(cfg.seed if seed is None else seed))
    R, Q, G = cfg.R, cfg.groups, cfg.rollouts_per_group
    if cfg.len_min == cfg.len_max:
        lengths = np.full(R, cfg.len_min, dtype=np.int64)
    else:
        lengths = rng.integers(cfg.len_min, cfg.len_max + 1, size=R).astype(np.int64)
    cu = np.zeros(R + 1, dtype=np.int64)
    np.cumsum(lengths, out=cu[1:])
    N = int(cu[-1])
    if N >= 2**31:
        raise ValueError("packed batch too large for int32 offsets")
    mask = np.concatenate([_rollout_mask(rng, int(T), cfg.tool_mean, cfg.policy_mean) for T in lengths])
    targets = rng.integers(0, cfg.V, size=N, dtype=np.int64).astype(np.int32)

    # Rewards, drawn per group (rows of G rollouts).
    if cfg.reward == "bernoulli":
        rew = (rng.random((Q, G)) < cfg.reward_p).astype(np.float32)
    elif cfg.reward == "uniform":
        rew = rng.random((Q, G)).astype(np.float32)
    elif cfg.reward == "uniform_ties":
        rew = (np.round(8.0 * rng.random((Q, G))) / 8.0).astype(np.float32)
    else:
        raise ValueError(cfg.reward)
    for gi, val in enumerate(cfg.forced_equal_groups):
        if gi < Q:
            rew[gi, :] = np.float32(val)

    # Opaque distinct group keys.
    keys = np.zeros(0, dtype=np.int64)
    while keys.shape[0] < Q:
        draw = rng.integers(1, 2**31 - 1, size=Q - keys.shape[0], dtype=np.int64)
        keys = np.concatenate([keys, draw[~np.isin(draw, keys)]])
        keys = keys[np.sort(np.unique(keys, return_index=True)[1])]
    keys = keys.astype(np.int32)
    gid = np.repeat(keys, G)
    rew = rew.reshape(-1)
    if cfg.interleave_groups:
        perm = rng.permutation(R)
        gid = gid[perm]
        rew = rew[perm]
    gid = gid.astype(np.int32)
    if cfg.n_excluded:
        ex = rng.choice(R, size=cfg.n_excluded, replace=False)
        gid[ex] = -1
    noise = rng.standard_normal(N).astype(np.float32)
    return Structure(cfg=cfg, lengths=lengths, cu_seqlens=cu.astype(np.int32), mask=mask,
                     targets=targets, rewards=rew.astype(np.float32), group_ids=gid, noise=noise)


def make_tensors(cfg: Config, N: int, device="cpu", seed: Optional[int] = None, chunk_rows: int = 65536):
    """Hidden states h [N, d] and LM-head weight W [V, d] in the configuration dtype.

    Drawn as float32 standard normals from a torch generator seeded with the
    configuration seed, scaled by the configured std, then cast (bf16 rounds to
    nearest-even).  Generation is chunked so the float32 temporary stays small.
    """
    import torch

    dt = {"f32": torch.float32, "bf16": torch.bfloat16}[cfg.dtype]
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(int(cfg.seed if seed is None else seed))

    def draw(rows: int, std: float):
        out = torch.empty((rows, cfg.d), dtype=dt, device=dev)
        for r0 in range(0, rows, chunk_rows):
            r1 = min(rows, r0 + chunk_rows)
            tmp = torch.randn((r1 - r0, cfg.d), generator=gen, dtype=torch.float32, device=dev)
            tmp.mul_(std)
            out[r0:r1].copy_(tmp)
            del tmp
        return out

    W = draw(cfg.V, cfg.w_std)
    h = draw(N, cfg.h_std)
    return h, W


def old_logp_from_anchor(anchor: np.ndarray, st: Structure) -> np.ndarray:
    """Old log-probs = anchor + sigma_old * noise on policy rows, 0 on masked rows (float32)."""
    a = np.asarray(anchor, dtype=np.float64)
    out = a + float(st.cfg.sigma_old) * st.noise.astype(np.float64)
    out = np.where(st.mask.astype(bool), out, 0.0)
    return out.astype(np.float32)


def perturbed_logps(old: np.ndarray, st: Structure, sigma: float, seed: int) -> np.ndarray:
    """Log-probs of another policy for the same sampled tokens (the inference engine's
    rollout log-probs, or a reference policy's): old + sigma * N(0,1) on policy rows, 0 on masked
    rows (float32, seeded)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    noise = rng.standard_normal(np.asarray(old).shape[0])
    out = np.asarray(old, dtype=np.float64) + float(sigma) * noise
    return np.where(st.mask.astype(bool), out, 0.0).astype(np.float32)


def token_values(st: Structure, seed: int, scale: float = 1.0) -> np.ndarray:
    """Value-model outputs V(s_t) for every packed row: scale * N(0,1) (float32, seeded)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return (float(scale) * rng.standard_normal(st.N)).astype(np.float32)


def sample_policy_rows(candidates: np.ndarray, k: int, seed: int) -> np.ndarray:
    """k distinct rows drawn (seeded) from the given candidate positions, sorted."""
    rng = np.random.Generator(np.random.PCG64(seed))
    k = min(int(k), int(candidates.shape[0]))
    pick = rng.choice(candidates.shape[0], size=k, replace=False)
    return np.sort(candidates[pick])
