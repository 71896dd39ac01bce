"""The seeded generators: determinism and realised statistics of each workload."""
import numpy as np
import pytest

import workloads as WL
from workloads.configs import ORDER


@pytest.mark.parametrize("name", ORDER)
def test_structure_deterministic_and_shaped(name):
    cfg = WL.get_config(name)
    a = WL.make_structure(cfg)
    b = WL.make_structure(cfg)
    for f in ("cu_seqlens", "mask", "targets", "rewards", "group_ids", "noise"):
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
    assert a.R == cfg.R
    assert a.cu_seqlens[0] == 0 and np.all(np.diff(a.cu_seqlens) >= cfg.len_min)
    assert np.all(np.diff(a.cu_seqlens) <= cfg.len_max)
    assert a.targets.min() >= 0 and a.targets.max() < cfg.V
    frac = 1.0 - a.mask.mean()
    assert abs(frac - cfg.masked_frac) < 0.06, frac
    # every rollout opens with a masked segment
    assert np.all(a.mask[a.cu_seqlens[:-1]] == 0)
    # opaque distinct keys, G rollouts each
    keys, counts = np.unique(a.group_ids, return_counts=True)
    assert len(keys) == cfg.groups and np.all(counts == cfg.rollouts_per_group)


def test_large_batch_has_all_equal_groups_and_ties():
    cfg = WL.get_config("large_bf16")
    st = WL.make_structure(cfg)
    eq = 0
    for k in np.unique(st.group_ids):
        r = st.rewards[st.group_ids == k]
        eq += int(r.max() == r.min())
        assert len(np.unique(r)) < len(r)          # ties inside every group
    assert eq >= 4


def test_scaled_instances_keep_shape_laws():
    for name in ORDER:
        base = WL.get_config(name)
        s = WL.scaled_config(name)
        assert (s.d, s.V, s.dtype, s.eps_low, s.eps_high, s.entropy_coef) == \
            (base.d, base.V, base.dtype, base.eps_low, base.eps_high, base.entropy_coef)
        st = WL.make_structure(s)
        assert st.N <= 8192


def test_tensors_seeded():
    torch = pytest.importorskip("torch")
    cfg = WL.get_config("tiny_fp32")
    h1, W1 = WL.make_tensors(cfg, 300, device="cpu", chunk_rows=128)
    h2, W2 = WL.make_tensors(cfg, 300, device="cpu", chunk_rows=300)
    assert torch.equal(h1, h2) and torch.equal(W1, W2)
    assert h1.shape == (300, cfg.d) and W1.shape == (cfg.V, cfg.d)
    assert abs(float(W1.float().std()) - cfg.w_std) < 0.01 * cfg.w_std * 10


def test_old_logp_placement():
    cfg = WL.get_config("tiny_fp32")
    st = WL.make_structure(cfg)
    anchor = np.linspace(-9, -7, st.N)
    old = WL.old_logp_from_anchor(anchor, st)
    pol = st.mask.astype(bool)
    assert np.all(old[~pol] == 0)
    resid = (old[pol] - anchor[pol]) / cfg.sigma_old
    assert abs(resid.std() - 1.0) < 0.1
