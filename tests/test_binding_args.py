"""Argument checks of the Python binding: wrong dtypes, shapes, layouts or devices raise before any
pointer crosses the C ABI (the library is not even loaded)."""
import pytest
import torch

import paper_2608_16798_amd as rlk


@pytest.fixture(autouse=True)
def no_library(monkeypatch):
    def refuse(*a, **k):
        raise AssertionError("the C ABI was reached")

    monkeypatch.setattr(rlk, "load_library", refuse)


N, d, V, R = 12, 16, 40, 3


def batch(**over):
    b = dict(hidden=torch.zeros(N, d, dtype=torch.bfloat16), W=torch.zeros(V, d, dtype=torch.bfloat16),
             targets=torch.zeros(N, dtype=torch.int32), mask=torch.ones(N, dtype=torch.uint8),
             cu_seqlens=torch.tensor([0, 4, 8, 12], dtype=torch.int32), old_logp=torch.zeros(N),
             rewards=torch.zeros(R), group_ids=torch.zeros(R, dtype=torch.int32))
    b.update(over)
    return b


def pg(b, **kw):
    return rlk.pg_loss_fwd_bwd(b["hidden"], b["W"], b["targets"], b["mask"], b["cu_seqlens"], b["old_logp"],
                               b["rewards"], b["group_ids"], rlk.make_params(), **kw)


def lp(b, **kw):
    return rlk.logprob_fwd(b["hidden"], b["W"], b["targets"], b["mask"], b["cu_seqlens"], **kw)


BAD = [
    ("W narrower than hidden", dict(W=torch.zeros(V, d - 8, dtype=torch.bfloat16)), {}, ValueError, "W has shape"),
    ("W dtype differs from hidden", dict(W=torch.zeros(V, d)), {}, TypeError, "W has dtype"),
    ("transposed W", dict(W=torch.zeros(d, V, dtype=torch.bfloat16).t()), {}, ValueError, "contiguous"),
    ("int64 targets", dict(targets=torch.zeros(N, dtype=torch.int64)), {}, TypeError, "targets has dtype"),
    ("short targets", dict(targets=torch.zeros(N - 1, dtype=torch.int32)), {}, ValueError, "targets has shape"),
    ("float mask", dict(mask=torch.ones(N)), {}, TypeError, "mask has dtype"),
    ("fp16 hidden", dict(hidden=torch.zeros(N, d, dtype=torch.float16), W=torch.zeros(V, d, dtype=torch.float16)),
     {}, TypeError, "hidden has dtype"),
    ("int64 cu_seqlens", dict(cu_seqlens=torch.tensor([0, 4, 8, 12])), {}, TypeError, "cu_seqlens has dtype"),
    ("fp64 old_logp", dict(old_logp=torch.zeros(N, dtype=torch.float64)), {}, TypeError, "old_logp has dtype"),
    ("old_logp of the wrong length", dict(old_logp=torch.zeros(N + 1)), {}, ValueError, "old_logp has shape"),
    ("rewards per token", dict(rewards=torch.zeros(N)), {}, ValueError, "rewards has shape"),
    ("int64 group ids", dict(group_ids=torch.zeros(R, dtype=torch.int64)), {}, TypeError, "group_ids has dtype"),
    ("bf16 dW", {}, dict(dW=torch.zeros(V, d, dtype=torch.bfloat16)), TypeError, "dW has dtype"),
    ("dW of the wrong shape", {}, dict(dW=torch.zeros(V - 1, d)), ValueError, "dW has shape"),
    ("fp32 dhidden for bf16 hidden", {}, dict(dhidden=torch.zeros(N, d)), TypeError, "dhidden has dtype"),
    ("dhidden of the wrong shape", {}, dict(dhidden=torch.zeros(N, d + 8, dtype=torch.bfloat16)), ValueError,
     "dhidden has shape"),
    ("short stats buffer", {}, dict(stats=torch.zeros(8, dtype=torch.uint8)), ValueError, "stats holds"),
    ("fp32 workspace", {}, dict(ws=torch.zeros(64)), TypeError, "ws has dtype"),
    ("rollout_logp of the wrong length", {}, dict(rollout_logp=torch.zeros(N - 2)), ValueError,
     "rollout_logp has shape"),
    ("int token_adv", {}, dict(token_adv=torch.zeros(N, dtype=torch.int32)), TypeError, "token_adv has dtype"),
    ("list hidden", dict(hidden=[[0.0]]), {},
     TypeError, "hidden must be a torch.Tensor"),
]


@pytest.mark.parametrize("what,over,kw,exc,msg", BAD, ids=[b[0] for b in BAD])
def test_pg_loss_rejects(what, over, kw, exc, msg):
    with pytest.raises(exc, match=msg):
        pg(batch(**over), **kw)


def test_pg_loss_rejects_host_tensors_after_the_shape_checks():
    with pytest.raises(ValueError, match="must be a GPU tensor"):
        pg(batch())


@pytest.mark.parametrize("over,kw,exc,msg", [
    (dict(W=torch.zeros(V, 8, dtype=torch.bfloat16)), {}, ValueError, "W has shape"),
    (dict(targets=torch.zeros(N, dtype=torch.int64)), {}, TypeError, "targets has dtype"),
    ({}, dict(logp=torch.zeros(N, dtype=torch.float64)), TypeError, "logp has dtype"),
    ({}, dict(entropy=torch.zeros(N - 1)), ValueError, "entropy has shape"),
    ({}, {}, ValueError, "must be a GPU tensor"),
])
def test_logprob_rejects(over, kw, exc, msg):
    with pytest.raises(exc, match=msg):
        lp(batch(**over), **kw)


def test_advantage_ppo_and_value_head_reject():
    with pytest.raises(TypeError, match="rewards has dtype"):
        rlk.group_advantage(torch.zeros(R, dtype=torch.float64), torch.zeros(R, dtype=torch.int32))
    with pytest.raises(ValueError, match="group_ids has shape"):
        rlk.group_advantage(torch.zeros(R), torch.zeros(R + 1, dtype=torch.int32))
    cu = torch.tensor([0, 4, 8, 12], dtype=torch.int32)
    m = torch.ones(N, dtype=torch.uint8)
    with pytest.raises(ValueError, match="cu_seqlens has shape"):
        rlk.gae(torch.zeros(N), torch.zeros(R), m, torch.tensor([0, 12], dtype=torch.int32))
    with pytest.raises(TypeError, match="values has dtype"):
        rlk.value_loss(torch.zeros(N, dtype=torch.float64), torch.zeros(N), m, cu)
    h = torch.zeros(N, d, dtype=torch.bfloat16)
    with pytest.raises(TypeError, match="w_v has dtype"):
        rlk.value_head_fwd(h, torch.zeros(d), 0.0, m, cu)
    with pytest.raises(ValueError, match="dvalues has shape"):
        rlk.value_head_bwd(h, torch.zeros(d, dtype=torch.bfloat16), m, cu, None, torch.zeros(N + 3))
    with pytest.raises(ValueError, match="must be a GPU tensor"):
        rlk.value_head_fwd(h, torch.zeros(d, dtype=torch.bfloat16), 0.0, m, cu)


# The chunk-planning hint counts the trained tokens in groups of unequal rewards; the oracle's group
# advantage (Sec. 2.3.1) is exactly 0 for the rollouts of the other groups and, with continuous rewards,
# nonzero for every rollout of a mixed group, so the two counts agree.
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_grad_token_hint_counts_the_oracle_nonzero_advantage_tokens(seed):
    import numpy as np

    import oracle as O

    rng = np.random.default_rng(seed)
    R = 24
    lens = rng.integers(1, 40, R)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    mask = (rng.random(cu[-1]) < 0.7).astype(np.uint8)
    gid = rng.integers(-1, 6, R).astype(np.int32)          # -1: excluded rollouts
    rewards = rng.standard_normal(R)
    for g in (1, 3):
        rewards[gid == g] = 0.5 * g                        # two all-equal groups
    adv = O.group_advantage(rewards, gid)["adv"]
    tok_adv = np.repeat(adv, lens)
    tok_live = np.repeat(gid >= 0, lens)
    expect = int(((mask == 1) & tok_live & (tok_adv != 0.0)).sum())
    assert rlk.grad_token_hint(mask, cu, rewards, gid) == expect
    assert rlk.grad_token_hint(mask, cu, np.zeros(R), gid) == 0
