"""rlk_group_advantage_noalloc (the library's fixed device scratch instead of a workspace) against
rlk_group_advantage: two calls in a row, the second with fewer rollouts, each bitwise equal to the
workspace entry point and within tolerance of the fp64 oracle."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _groups(R, seed):
    """R rollouts in groups of 1-16 under opaque int32 keys, interleaved; rewards on a 1/8 grid (ties,
    all-equal groups); about 3 % of the rollouts excluded (key -1)."""
    rng = np.random.default_rng(seed)
    sizes = []
    while sum(sizes) < R:
        sizes.append(int(rng.integers(1, 17)))
    sizes[-1] -= sum(sizes) - R
    keys = rng.choice(np.arange(0, 2**31 - 1, 7919, dtype=np.int64), size=len(sizes), replace=False)
    gid = rng.permutation(np.repeat(keys, sizes)).astype(np.int32)
    gid[rng.random(R) < 0.03] = -1
    rewards = (np.round(8 * rng.random(R)) / 8).astype(np.float32)
    return rewards, gid


def test_noalloc_advantage_matches_the_workspace_entry_point():
    import torch

    from gpu_common import O, ensure_library, log, rlk

    ensure_library()
    for R, seed in ((16384, 5), (1000, 6)):
        rewards, gid = _groups(R, seed)
        log(f"noalloc advantage R={R} seed={seed}")
        r_d = torch.as_tensor(rewards, device="cuda")
        g_d = torch.as_tensor(gid, device="cuda")
        a_ws = torch.full((R,), 7.0, dtype=torch.float32, device="cuda")
        gi_ws = torch.full((R,), 9, dtype=torch.int32, device="cuda")
        q_ws = torch.zeros(1, dtype=torch.int32, device="cuda")
        rlk.group_advantage(r_d, g_d, 1e-6, adv=a_ws, group_index=gi_ws, n_groups=q_ws)
        a_na = torch.full((R,), -7.0, dtype=torch.float32, device="cuda")
        gi_na = torch.full((R,), -9, dtype=torch.int32, device="cuda")
        q_na = torch.zeros(1, dtype=torch.int32, device="cuda")
        rlk.group_advantage_noalloc(r_d, g_d, 1e-6, adv=a_na, group_index=gi_na, n_groups=q_na)
        torch.cuda.synchronize()
        assert torch.equal(a_na, a_ws) and torch.equal(gi_na, gi_ws) and int(q_na.item()) == int(q_ws.item())
        ref = O.group_advantage(rewards, gid, 1e-6)
        np.testing.assert_array_equal(gi_na.cpu().numpy(), ref["group_index"])
        assert int(q_na.item()) == ref["n_groups"]
        a = a_na.cpu().numpy().astype(np.float64)
        scale = np.maximum(1.0, np.abs(ref["adv"]))
        assert float(np.max(np.abs(a - ref["adv"]) / scale)) <= 1e-6
        assert np.all(a[ref["adv"] == 0] == 0)     # excluded rollouts and all-equal groups are exactly 0
        log(f"  Q={ref['n_groups']} bitwise equal to rlk_group_advantage")


def test_noalloc_advantage_rejects_too_many_rollouts():
    import torch

    from gpu_common import ensure_library, rlk

    ensure_library()
    R = 16385
    with pytest.raises(rlk.RlkError) as e:
        rlk.group_advantage_noalloc(torch.zeros(R, device="cuda"), torch.zeros(R, dtype=torch.int32, device="cuda"))
    assert e.value.code == rlk.RLK_ESHAPE
