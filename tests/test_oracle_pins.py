"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

None of these re-derive the oracle's own formulas: each checks a closed form,
an invariant, a special case that reduces to a library routine, or finite
differences of the loss, chosen so that a dropped term, a wrong sign, a wrong
index or a transposed operand in the oracle fails at least one of them.
"""
import math

import numpy as np
import pytest

import oracle as O

EPS = 1e-6


def tiny_batch(seed=0, d=8, V=16, groups=3, per_group=(2, 3, 2), lens=None, masked=0.4,
               excluded=(), w_std=0.5, old_sigma=0.3):
    rng = np.random.default_rng(seed)
    R = sum(per_group)
    if lens is None:
        lens = rng.integers(3, 9, size=R)
    cu = np.zeros(R + 1, dtype=np.int64)
    cu[1:] = np.cumsum(lens)
    N = int(cu[-1])
    h = rng.standard_normal((N, d))
    W = rng.standard_normal((V, d)) * w_std
    targets = rng.integers(0, V, size=N)
    mask = (rng.random(N) > masked).astype(np.uint8)
    keys = rng.choice(1000, size=groups, replace=False) + 7
    gid = np.concatenate([np.full(c, keys[i]) for i, c in enumerate(per_group)])
    gid = rng.permutation(gid).astype(np.int64)
    for r in excluded:
        gid[r] = -1
    rewards = rng.random(R).astype(np.float32)
    old = rng.standard_normal(N) * old_sigma - 2.5
    return dict(h=h, W=W, targets=targets, mask=mask, cu_seqlens=cu, old_logp=old,
                rewards=rewards, group_ids=gid)


# ---------------------------------------------------------------- compaction
def test_compact_brute_force():
    rng = np.random.default_rng(1)
    lens = [5, 0, 7, 3, 9]
    cu = np.concatenate([[0], np.cumsum(lens)])
    N = cu[-1]
    mask = (rng.random(N) > 0.5).astype(np.uint8)
    gid = np.array([0, 9, -1, 0, 2])   # 0 is a valid key; rollout 1 is empty
    idx, tr, npol = O.compact(mask, cu, gid)
    exp_idx, exp_tr = [], []
    exp_n = [0] * len(lens)
    for r in range(len(lens)):
        for t in range(cu[r], cu[r + 1]):
            if mask[t] and gid[r] >= 0:
                exp_idx.append(t)
                exp_tr.append(r)
                exp_n[r] += 1
    assert idx.tolist() == exp_idx
    assert tr.tolist() == exp_tr
    assert npol.tolist() == exp_n
    # without group ids nothing is excluded; mask None keeps every token
    idx2, _, _ = O.compact(mask, cu)
    assert idx2.tolist() == np.flatnonzero(mask).tolist()
    idx3, tr3, n3 = O.compact(None, cu)
    assert idx3.tolist() == list(range(N)) and n3.tolist() == lens


def test_group_index_opaque_keys():
    gid = np.array([50, -3, 7, 50, 1000, 7, -1])
    gi, Q = O.group_index(gid)
    assert Q == 3
    assert gi.tolist() == [1, -1, 0, 1, 2, 0, -1]


# ---------------------------------------------------------------- log-softmax
def test_logprob_sums_to_one_and_bounds():
    rng = np.random.default_rng(2)
    V, d = 16, 8
    W = rng.standard_normal((V, d))
    h = rng.standard_normal((3, d))
    tot = np.zeros(3)
    Hs = None
    for y in range(V):
        lse, lp, H = O.token_logprob(h, W, np.full(3, y))
        tot += np.exp(lp)
        Hs = H
    np.testing.assert_allclose(tot, 1.0, rtol=0, atol=1e-13)
    assert np.all(Hs >= 0) and np.all(Hs <= math.log(V) + 1e-12)


def test_logprob_matches_torch_log_softmax():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(3)
    V, d, n = 37, 5, 11
    W = rng.standard_normal((V, d)) * 2
    h = rng.standard_normal((n, d))
    y = rng.integers(0, V, size=n)
    lse, lp, H = O.token_logprob(h, W, y)
    z = torch.from_numpy(h) @ torch.from_numpy(W).T
    ls = torch.log_softmax(z, dim=1)
    np.testing.assert_allclose(lp, ls[torch.arange(n), torch.from_numpy(y)].numpy(), atol=1e-12)
    np.testing.assert_allclose(lse, torch.logsumexp(z, dim=1).numpy(), atol=1e-12)
    ent = torch.distributions.Categorical(logits=z).entropy().numpy()
    np.testing.assert_allclose(H, ent, atol=1e-12)


def test_logprob_special_cases():
    d, V = 4, 9
    h = np.random.default_rng(4).standard_normal((2, d))
    lse, lp, H = O.token_logprob(h, np.zeros((V, d)), np.array([0, 5]))
    np.testing.assert_allclose(lse, math.log(V), atol=1e-14)
    np.testing.assert_allclose(H, math.log(V), atol=1e-14)
    np.testing.assert_allclose(lp, -math.log(V), atol=1e-14)
    lse1, lp1, H1 = O.token_logprob(h, np.ones((1, d)), np.array([0, 0]))
    np.testing.assert_allclose(lp1, 0.0, atol=1e-14)
    np.testing.assert_allclose(H1, 0.0, atol=1e-14)
    np.testing.assert_allclose(lse1, h.sum(1), atol=1e-14)


def test_logprob_shift_invariance():
    rng = np.random.default_rng(5)
    V, d = 23, 6
    W = rng.standard_normal((V, d))
    h = rng.standard_normal((4, d))
    y = rng.integers(0, V, size=4)
    u = rng.standard_normal(d)
    lse, lp, H = O.token_logprob(h, W, y)
    lse2, lp2, H2 = O.token_logprob(h, W + u[None, :], y)   # every logit of a row shifts by u.h
    np.testing.assert_allclose(lse2, lse + h @ u, atol=1e-12)
    np.testing.assert_allclose(lp2, lp, atol=1e-12)
    np.testing.assert_allclose(H2, H, atol=1e-12)


# ---------------------------------------------------------------- advantages
def test_advantage_zero_mean_unit_std():
    rng = np.random.default_rng(6)
    gid = np.repeat([11, 3, 8], [5, 8, 3])
    rew = rng.random(16)
    a = O.group_advantage(rew, gid, EPS)
    for key in (11, 3, 8):
        m = gid == key
        A = a["adv"][m]
        sig = np.std(rew[m])             # library population std
        assert abs(A.sum()) < 1e-12
        np.testing.assert_allclose(np.std(A), sig / (sig + EPS), rtol=1e-12)


@pytest.mark.parametrize("n,k", [(2, 1), (8, 3), (8, 1), (5, 4)])
def test_advantage_binary_closed_form(n, k):
    rew = np.array([1.0] * k + [0.0] * (n - k))
    a = O.group_advantage(rew, np.zeros(n, dtype=int), EPS)["adv"]
    p = k / n
    s = math.sqrt(p * (1 - p))
    np.testing.assert_allclose(a[:k], (1 - p) / (s + EPS), rtol=1e-13)
    np.testing.assert_allclose(a[k:], -p / (s + EPS), rtol=1e-13)
    if n == 2:
        np.testing.assert_allclose(a, [0.5 / (0.5 + EPS), -0.5 / (0.5 + EPS)], rtol=1e-13)


def test_advantage_degenerate_and_invariances():
    rng = np.random.default_rng(7)
    gid = np.array([5, 5, 5, 9, 9, 2, 4, 4])
    rew = np.array([0.3, 0.3, 0.3, 0.1, 0.9, 0.7, 1.0, 1.0], dtype=np.float32)
    a = O.group_advantage(rew, gid, EPS)["adv"]
    assert a[0] == 0 and a[1] == 0 and a[2] == 0          # all-equal group
    assert a[5] == 0                                       # group of one
    assert a[6] == 0 and a[7] == 0
    # shift invariance
    a2 = O.group_advantage(rew.astype(np.float64) + 3.25, gid, EPS)["adv"]
    np.testing.assert_allclose(a2, a, atol=1e-9)
    # permutation equivariance and opaque relabeling
    perm = rng.permutation(8)
    a3 = O.group_advantage(rew[perm], gid[perm] * 17 + 1, EPS)["adv"]
    np.testing.assert_allclose(a3, a[perm], atol=1e-15)


def test_advantage_exclusion_removes_rollout():
    gid = np.array([1, 1, 1, 1])
    rew = np.array([1.0, 0.0, 0.0, 5.0])
    ex = gid.copy()
    ex[3] = -1
    a = O.group_advantage(rew, ex, EPS)["adv"]
    ref = O.group_advantage(rew[:3], gid[:3], EPS)["adv"]
    np.testing.assert_allclose(a[:3], ref, rtol=1e-15)
    assert a[3] == 0


# ---------------------------------------------------------------- surrogate
def test_surrogate_quadrants():
    A = np.array([2.0, 2.0, -2.0, -2.0, 2.0, -2.0])
    rho = np.array([1.3, 0.5, 0.5, 1.5, 1.28, 0.8])
    s, r, c = O.surrogate(np.log(rho), np.zeros(6), A, 0.2, 0.28)
    np.testing.assert_allclose(r, rho, rtol=1e-15)
    np.testing.assert_allclose(s, [1.28 * 2, 0.5 * 2, 0.8 * -2, 1.5 * -2, 1.28 * 2, 0.8 * -2], rtol=1e-13)
    # clipped: A>0 & rho>1.28 ; A<0 & rho<0.8 ; exactly on the bound the gradient passes
    assert c.tolist() == [True, False, True, False, False, False]


def test_surrogate_large_eps_is_importance_weighted_pg():
    rng = np.random.default_rng(8)
    lp = rng.standard_normal(50)
    old = lp + rng.standard_normal(50)
    A = rng.standard_normal(50)
    s, r, c = O.surrogate(lp, old, A, 1e9, 1e9)
    np.testing.assert_allclose(s, np.exp(lp - old) * A, rtol=1e-14)
    assert not c.any()


# ---------------------------------------------------------------- loss identities
def _loss(b, **kw):
    return O.pg_loss_fwd_bwd(b["h"], b["W"], b["targets"], b["mask"], b["cu_seqlens"], b["old_logp"],
                             b["rewards"], b["group_ids"], **kw)


def test_ratio_one_token_mode_is_minus_masked_mean_advantage():
    b = tiny_batch(9)
    lse, lp, H = O.token_logprob(b["h"], b["W"], b["targets"])
    b["old_logp"] = lp.copy()       # rho == 1 exactly
    c = 0.01
    out = _loss(b, agg=O.AGG_TOKEN, entropy_coef=c, eps_low=0.2, eps_high=0.28)
    idx, tr, _ = O.compact(b["mask"], b["cu_seqlens"], b["group_ids"])
    adv = O.group_advantage(b["rewards"], b["group_ids"], EPS)["adv"]
    exp = -adv[tr].mean() - c * H[idx].mean()
    np.testing.assert_allclose(out["loss"], exp, rtol=1e-12)
    np.testing.assert_allclose(out["stats"]["ratio_mean"], 1.0, rtol=1e-14)
    # seq mode with every rollout non-empty and no entropy: the group sums of A vanish
    b2 = tiny_batch(10, masked=0.0)
    lse2, lp2, H2 = O.token_logprob(b2["h"], b2["W"], b2["targets"])
    b2["old_logp"] = lp2
    assert abs(_loss(b2)["loss"]) < 1e-12


def test_seq_equals_token_when_balanced():
    b = tiny_batch(11, per_group=(2, 2, 2), lens=np.full(6, 5), masked=0.0)
    s = _loss(b, agg=O.AGG_SEQ, eps_low=0.2, eps_high=0.2)
    t = _loss(b, agg=O.AGG_TOKEN, eps_low=0.2, eps_high=0.2)
    np.testing.assert_allclose(s["loss"], t["loss"], rtol=1e-12)
    np.testing.assert_allclose(s["dW"], t["dW"], rtol=1e-10, atol=1e-14)


def test_single_rollout_seq_is_masked_token_mean():
    b = tiny_batch(12, groups=1, per_group=(1,), lens=np.array([17]))
    out = _loss(b, eps_low=0.2, eps_high=0.2)
    # a group of one has advantage 0, so the surrogate is 0 for every token
    assert out["loss"] == 0.0
    assert np.all(out["dW"] == 0) and np.all(out["dh"] == 0)


def test_duplicated_group_leaves_seq_loss_unchanged():
    b = tiny_batch(13)
    R = len(b["rewards"])
    out = _loss(b, eps_low=0.2, eps_high=0.28)
    lens = np.diff(b["cu_seqlens"])
    N = b["h"].shape[0]
    dup = dict(
        h=np.concatenate([b["h"], b["h"]]), W=b["W"],
        targets=np.concatenate([b["targets"], b["targets"]]),
        mask=np.concatenate([b["mask"], b["mask"]]),
        cu_seqlens=np.concatenate([[0], np.cumsum(np.concatenate([lens, lens]))]),
        old_logp=np.concatenate([b["old_logp"], b["old_logp"]]),
        rewards=np.concatenate([b["rewards"], b["rewards"]]),
        group_ids=np.concatenate([b["group_ids"], np.where(b["group_ids"] >= 0, b["group_ids"] + 100000, -1)]))
    out2 = _loss(dup, eps_low=0.2, eps_high=0.28)
    np.testing.assert_allclose(out2["loss"], out["loss"], rtol=1e-12)
    np.testing.assert_allclose(out2["dW"], out["dW"], rtol=1e-10, atol=1e-15)
    np.testing.assert_allclose(out2["dh"][:N], out["dh"] / 2, rtol=1e-10, atol=1e-15)
    assert R == out["stats"]["n_valid_rollouts"]


def test_microbatch_norm_override_adds_up():
    b = tiny_batch(14, groups=3, per_group=(3, 2, 3))
    full = _loss(b, eps_low=0.2, eps_high=0.28, entropy_coef=0.02)
    Q = full["n_groups"]
    gid = b["group_ids"]
    cu = b["cu_seqlens"]
    tot_loss, tot_dW = 0.0, np.zeros_like(full["dW"])
    for key in np.unique(gid[gid >= 0]):
        rs = np.flatnonzero(gid == key)
        rows = np.concatenate([np.arange(cu[r], cu[r + 1]) for r in rs])
        lens = np.array([cu[r + 1] - cu[r] for r in rs])
        part = dict(h=b["h"][rows], W=b["W"], targets=b["targets"][rows], mask=b["mask"][rows],
                    cu_seqlens=np.concatenate([[0], np.cumsum(lens)]), old_logp=b["old_logp"][rows],
                    rewards=b["rewards"][rs], group_ids=gid[rs])
        o = _loss(part, eps_low=0.2, eps_high=0.28, entropy_coef=0.02, norm_override=Q)
        tot_loss += o["loss"]
        tot_dW += o["dW"]
    np.testing.assert_allclose(tot_loss, full["loss"], rtol=1e-12)
    np.testing.assert_allclose(tot_dW, full["dW"], rtol=1e-10, atol=1e-15)


def test_excluded_rollout_contributes_nothing():
    b = tiny_batch(15, excluded=(1,))
    out = _loss(b, eps_low=0.2, eps_high=0.2)
    cu = b["cu_seqlens"]
    assert np.all(out["dh"][cu[1]:cu[2]] == 0)
    assert out["stats"]["n_valid_rollouts"] == len(b["rewards"]) - 1
    # perturbing the excluded rollout's inputs changes nothing
    b2 = dict(b)
    b2["h"] = b["h"].copy()
    b2["h"][cu[1]:cu[2]] += 10.0
    b2["rewards"] = b["rewards"].copy()
    b2["rewards"][1] = 123.0
    out2 = _loss(b2, eps_low=0.2, eps_high=0.2)
    assert out2["loss"] == out["loss"]
    np.testing.assert_array_equal(out2["dW"], out["dW"])


def test_empty_batch():
    b = tiny_batch(16)
    b["mask"] = np.zeros_like(b["mask"])
    out = _loss(b)
    assert out["loss"] == 0.0 and np.all(out["dh"] == 0) and np.all(out["dW"] == 0)
    b = tiny_batch(16)
    b["group_ids"] = np.full_like(b["group_ids"], -1)
    out = _loss(b)
    assert out["loss"] == 0.0 and out["n_groups"] == 0 and np.all(out["dW"] == 0)


# ---------------------------------------------------------------- gradients
def _kink_safe(b, eps_low, eps_high, margin=1e-3, temperature=1.0):
    lse, lp, H = O.token_logprob(b["h"], b["W"], b["targets"], temperature=temperature)
    rho = np.exp(lp - b["old_logp"])
    for bound in (1 - eps_low, 1 + eps_high):
        near = np.abs(rho - bound) < margin
        b["old_logp"][near] -= 5 * margin
    return b


@pytest.mark.parametrize("agg,c_ent", [(O.AGG_SEQ, 0.0), (O.AGG_SEQ, 0.05), (O.AGG_TOKEN, 0.03)])
def test_gradients_match_finite_differences(agg, c_ent):
    b = tiny_batch(17, excluded=(4,), old_sigma=0.4)
    lse, lp, H = O.token_logprob(b["h"], b["W"], b["targets"])
    b["old_logp"] = lp + np.random.default_rng(18).standard_normal(lp.shape) * 0.25
    b = _kink_safe(b, 0.2, 0.28)
    kw = dict(eps_low=0.2, eps_high=0.28, agg=agg, entropy_coef=c_ent)
    out = _loss(b, **kw)
    assert 0 < out["stats"]["clip_frac"] < 1      # both branches exercised
    step = 1e-6
    rng = np.random.default_rng(19)
    for name, grad in (("h", out["dh"]), ("W", out["dW"])):
        X = b[name]
        picks = [tuple(rng.integers(0, s) for s in X.shape) for _ in range(25)]
        for ij in picks:
            bp = dict(b)
            bp[name] = X.copy()
            bp[name][ij] += step
            lp_ = _loss(bp, grads=False, **kw)["loss"]
            bp[name][ij] -= 2 * step
            lm_ = _loss(bp, grads=False, **kw)["loss"]
            fd = (lp_ - lm_) / (2 * step)
            assert abs(fd - grad[ij]) <= 1e-6 * max(1.0, abs(grad).max()), (name, ij, fd, grad[ij])


def test_gradients_match_torch_autograd():
    torch = pytest.importorskip("torch")
    b = tiny_batch(20, excluded=(2,))
    lse, lp, H = O.token_logprob(b["h"], b["W"], b["targets"])
    b["old_logp"] = lp + np.random.default_rng(21).standard_normal(lp.shape) * 0.3
    kw = dict(eps_low=0.2, eps_high=0.28, entropy_coef=0.04)
    out = _loss(b, **kw)
    idx, tr, npol = O.compact(b["mask"], b["cu_seqlens"], b["group_ids"])
    ga = O.group_advantage(b["rewards"], b["group_ids"], EPS)
    gi, Q, G = ga["group_index"], ga["n_groups"], ga["G"]
    h = torch.tensor(b["h"], requires_grad=True)
    W = torch.tensor(b["W"], requires_grad=True)
    z = h[torch.from_numpy(idx)] @ W.T
    ls = torch.log_softmax(z, dim=1)
    lpy = ls[torch.arange(len(idx)), torch.from_numpy(b["targets"][idx])]
    ent = -(ls.exp() * ls).sum(1)
    rho = torch.exp(lpy - torch.from_numpy(b["old_logp"][idx]))
    A = torch.from_numpy(ga["adv"][tr])
    s = torch.minimum(rho * A, torch.clamp(rho, 0.8, 1.28) * A)
    val = s + 0.04 * ent
    # seq aggregation built from torch segment sums (not the oracle's weights)
    per_r = torch.zeros(len(b["rewards"]), dtype=torch.float64).index_add(0, torch.from_numpy(tr), val)
    ell = per_r / torch.from_numpy(np.maximum(npol, 1)).double()
    J = sum(ell[torch.from_numpy(np.flatnonzero(gi == q))].sum() / G[q] for q in range(Q)) / Q
    (-J).backward()
    np.testing.assert_allclose(float(-J), out["loss"], rtol=1e-12)
    np.testing.assert_allclose(h.grad.numpy(), out["dh"], rtol=1e-9, atol=1e-13)
    np.testing.assert_allclose(W.grad.numpy(), out["dW"], rtol=1e-9, atol=1e-13)


def test_gradient_invariants():
    b = tiny_batch(22, excluded=(0,))
    lse, lp, H = O.token_logprob(b["h"], b["W"], b["targets"])
    b["old_logp"] = lp + np.random.default_rng(23).standard_normal(lp.shape) * 0.2
    kw = dict(eps_low=0.2, eps_high=0.28, entropy_coef=0.02)
    out = _loss(b, **kw)
    # every dz row sums to 0, so the columns of dW sum to 0
    np.testing.assert_allclose(out["dW"].sum(axis=0), 0.0, atol=1e-14)
    # masked rows of dhidden are exactly 0
    idx = out["idx"]
    keep = np.zeros(b["h"].shape[0], dtype=bool)
    keep[idx] = True
    assert np.all(out["dh"][~keep] == 0)
    # W + 1 c^T shifts each logit row by c.h: loss and gradients unchanged
    c = np.random.default_rng(24).standard_normal(b["W"].shape[1])
    b2 = dict(b)
    b2["W"] = b["W"] + c[None, :]
    out2 = _loss(b2, **kw)
    np.testing.assert_allclose(out2["loss"], out["loss"], rtol=1e-11)
    np.testing.assert_allclose(out2["dW"], out["dW"], atol=1e-12)
    # masked tokens' inputs do not matter
    b3 = dict(b)
    b3["h"] = b["h"].copy()
    b3["h"][~keep] *= -3.0
    b3["targets"] = b["targets"].copy()
    b3["targets"][~keep] = 0
    b3["old_logp"] = b["old_logp"].copy()
    b3["old_logp"][~keep] = 99.0
    out3 = _loss(b3, **kw)
    assert out3["loss"] == out["loss"]
    np.testing.assert_array_equal(out3["dW"], out["dW"])


# ------------------------------------------- truncated IS (Sec. 3.2.4) and the KL term (Sec. 2.3.2)
def _with_old_from_current(seed, sigma=0.25, **kw):
    b = tiny_batch(seed, **kw)
    lse, lp, H = O.token_logprob(b["h"], b["W"], b["targets"])
    b["old_logp"] = lp + np.random.default_rng(seed + 1).standard_normal(lp.shape) * sigma
    return b


def test_tis_identity_when_rollout_equals_old():
    b = _with_old_from_current(30, excluded=(1,))
    kw = dict(eps_low=0.2, eps_high=0.28, entropy_coef=0.05)
    plain = _loss(b, **kw)
    tis = _loss(b, rollout_logp=b["old_logp"].copy(), tis_cap=2.0, **kw)
    assert tis["loss"] == plain["loss"]
    np.testing.assert_array_equal(tis["dh"], plain["dh"])
    np.testing.assert_array_equal(tis["dW"], plain["dW"])
    assert tis["stats"]["tis_mean"] == 1.0


@pytest.mark.parametrize("shift,cap,expect", [(0.4, 5.0, math.exp(0.4)), (3.0, 2.5, 2.5), (-0.7, 4.0, math.exp(-0.7))])
def test_tis_constant_weight_scales_the_whole_token_loss(shift, cap, expect):
    # rollout = old - shift on every token: w_t = min(e^shift, cap) is one constant, so the loss
    # (surrogate, entropy and KL terms alike) and both gradients scale by exactly that constant
    b = _with_old_from_current(31, excluded=(3,))
    ref = b["old_logp"] - 0.3
    kw = dict(eps_low=0.2, eps_high=0.28, entropy_coef=0.07, ref_logp=ref, kl_coef=0.05)
    plain = _loss(b, **kw)
    tis = _loss(b, rollout_logp=b["old_logp"] - shift, tis_cap=cap, **kw)
    np.testing.assert_allclose(tis["loss"], expect * plain["loss"], rtol=1e-12)
    np.testing.assert_allclose(tis["pg_loss"], expect * plain["pg_loss"], rtol=1e-12)
    np.testing.assert_allclose(tis["dh"], expect * plain["dh"], rtol=1e-10, atol=1e-15)
    np.testing.assert_allclose(tis["dW"], expect * plain["dW"], rtol=1e-10, atol=1e-15)


def test_kl_sampled_estimator_is_unbiased_by_enumeration():
    # E_{a ~ p}[q_a/p_a - log(q_a/p_a) - 1] = KL(p || q) exactly, summing over the whole vocabulary
    rng = np.random.default_rng(32)
    for _ in range(5):
        zp, zq = rng.standard_normal(24) * 2.0, rng.standard_normal(24) * 2.0
        lp = zp - np.log(np.exp(zp).sum())
        lq = zq - np.log(np.exp(zq).sum())
        est, _ = O.kl_sampled(lp, lq)
        assert np.all(est >= 0)
        kl_exact = float((np.exp(lp) * (lp - lq)).sum())
        np.testing.assert_allclose(float((np.exp(lp) * est).sum()), kl_exact, rtol=1e-12)
    est, d = O.kl_sampled(np.array([-1.3]), np.array([-1.3]))
    assert est[0] == 0.0 and d[0] == 0.0


def test_kl_term_enters_the_loss_with_minus_beta():
    # at rho = 1 with zero advantages (all rewards equal) the loss is beta times the mean sampled KL
    b = _with_old_from_current(33, sigma=0.0)
    b["rewards"][:] = 0.5
    lse, lp, H = O.token_logprob(b["h"], b["W"], b["targets"])
    ref = lp + np.random.default_rng(34).standard_normal(lp.shape) * 0.5
    out = _loss(b, agg=O.AGG_TOKEN, ref_logp=ref, kl_coef=0.1)
    idx = out["idx"]
    r = ref[idx] - lp[idx]
    np.testing.assert_allclose(out["loss"], 0.1 * np.mean(np.exp(r) - r - 1.0), rtol=1e-12)
    np.testing.assert_allclose(out["stats"]["kl_mean"], np.mean(np.exp(r) - r - 1.0), rtol=1e-12)


@pytest.mark.parametrize("agg", [O.AGG_SEQ, O.AGG_TOKEN])
def test_tis_and_kl_gradients_match_finite_differences(agg):
    b = _with_old_from_current(35, excluded=(4,), sigma=0.4)
    b = _kink_safe(b, 0.2, 0.28)
    rng = np.random.default_rng(36)
    rollout = b["old_logp"] + rng.standard_normal(b["old_logp"].shape) * 0.6
    ref = b["old_logp"] + rng.standard_normal(b["old_logp"].shape) * 0.5
    kw = dict(eps_low=0.2, eps_high=0.28, agg=agg, entropy_coef=0.03, rollout_logp=rollout, tis_cap=1.5,
              ref_logp=ref, kl_coef=0.2)
    out = _loss(b, **kw)
    assert 0 < out["stats"]["clip_frac"] < 1
    assert np.any(out["tis"] == 1.5) and np.any(out["tis"] < 1.5)   # both sides of the cap
    step = 1e-6
    for name, grad in (("h", out["dh"]), ("W", out["dW"])):
        X = b[name]
        for ij in [tuple(rng.integers(0, s) for s in X.shape) for _ in range(20)]:
            bp = dict(b)
            bp[name] = X.copy()
            bp[name][ij] += step
            lp_ = _loss(bp, grads=False, **kw)["loss"]
            bp[name][ij] -= 2 * step
            lm_ = _loss(bp, grads=False, **kw)["loss"]
            fd = (lp_ - lm_) / (2 * step)
            assert abs(fd - grad[ij]) <= 1e-6 * max(1.0, abs(grad).max()), (name, ij, fd, grad[ij])


# ------------------------------------------------ PPO path: GAE, value loss, token advantages
def _gae_case(seed=40, R=4):
    rng = np.random.default_rng(seed)
    lens = rng.integers(5, 14, size=R)
    cu = np.concatenate([[0], np.cumsum(lens)])
    N = int(cu[-1])
    mask = (rng.random(N) > 0.35).astype(np.uint8)
    values = rng.standard_normal(N)
    rewards = rng.random(R)
    return dict(values=values, rewards=rewards, mask=mask, cu=cu)


def test_gae_gamma_lambda_one_is_reward_minus_value():
    # Sec. 3.2.3: with gamma = lambda = 1 the recursion degenerates to A_t = R_i - V(s_t)
    c = _gae_case()
    adv, ret = O.gae(c["values"], c["rewards"], c["mask"], c["cu"], None, 1.0, 1.0)
    for r in range(len(c["rewards"])):
        for t in range(c["cu"][r], c["cu"][r + 1]):
            if c["mask"][t]:
                np.testing.assert_allclose(adv[t], c["rewards"][r] - c["values"][t], rtol=0, atol=1e-12)
                np.testing.assert_allclose(ret[t], c["rewards"][r], rtol=0, atol=1e-12)
            else:
                assert adv[t] == 0 and ret[t] == 0


def _policy_seq(c, r):
    return [t for t in range(c["cu"][r], c["cu"][r + 1]) if c["mask"][t]]


@pytest.mark.parametrize("gamma,lam", [(0.9, 0.0), (0.97, 0.8), (1.0, 0.5), (0.5, 1.0)])
def test_gae_is_the_discounted_sum_of_td_residuals(gamma, lam):
    # brute force on the definition: A_t = sum_l (gamma lam)^l delta_{t+l}, delta from next policy token
    c = _gae_case(41)
    adv, ret = O.gae(c["values"], c["rewards"], c["mask"], c["cu"], None, gamma, lam)
    V = c["values"]
    for r in range(len(c["rewards"])):
        pos = _policy_seq(c, r)
        deltas = []
        for j, t in enumerate(pos):
            nxt = gamma * V[pos[j + 1]] if j + 1 < len(pos) else c["rewards"][r]
            deltas.append(nxt - V[t])
        for j, t in enumerate(pos):
            want = sum((gamma * lam) ** l * deltas[j + l] for l in range(len(pos) - j))
            np.testing.assert_allclose(adv[t], want, rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(ret[t], want + V[t], rtol=1e-12, atol=1e-12)
        if lam == 0.0:   # one-step residuals
            np.testing.assert_allclose(adv[pos], deltas, rtol=1e-12, atol=1e-12)


def test_gae_steps_over_tool_tokens_and_skips_excluded_rollouts():
    c = _gae_case(42)
    adv, _ = O.gae(c["values"], c["rewards"], c["mask"], c["cu"], None, 0.95, 0.9)
    # drop every tool token: the policy tokens' advantages are unchanged
    keep = c["mask"].astype(bool)
    cu2 = np.concatenate([[0], np.cumsum([keep[c["cu"][r]:c["cu"][r + 1]].sum() for r in range(len(c["rewards"]))])])
    adv2, _ = O.gae(c["values"][keep], c["rewards"], np.ones(keep.sum(), np.uint8), cu2, None, 0.95, 0.9)
    np.testing.assert_allclose(adv[keep], adv2, rtol=1e-12, atol=1e-14)
    gid = np.array([3, -1, 3, 5])
    adv3, ret3 = O.gae(c["values"], c["rewards"], c["mask"], c["cu"], gid, 0.95, 0.9)
    ex = slice(c["cu"][1], c["cu"][2])
    assert np.all(adv3[ex] == 0) and np.all(ret3[ex] == 0)
    np.testing.assert_array_equal(adv3[:c["cu"][1]], adv[:c["cu"][1]])


def test_value_loss_closed_form_and_finite_differences():
    c = _gae_case(43)
    G = np.random.default_rng(44).standard_normal(c["values"].shape)
    loss, dV = O.value_loss(c["values"], G, c["mask"], c["cu"])
    m = c["mask"].astype(bool)
    np.testing.assert_allclose(loss, np.mean((c["values"][m] - G[m]) ** 2), rtol=1e-12)
    assert np.all(dV[~m] == 0)
    for t in np.flatnonzero(m)[:10]:
        vp = c["values"].copy()
        vp[t] += 1e-6
        lp_, _ = O.value_loss(vp, G, c["mask"], c["cu"])
        vp[t] -= 2e-6
        lm_, _ = O.value_loss(vp, G, c["mask"], c["cu"])
        np.testing.assert_allclose((lp_ - lm_) / 2e-6, dV[t], rtol=1e-6, atol=1e-10)


def test_token_advantages_reduce_to_the_group_advantages():
    b = _with_old_from_current(45, excluded=(2,))
    kw = dict(eps_low=0.2, eps_high=0.28, entropy_coef=0.02)
    grpo = _loss(b, **kw)
    tok = np.zeros(b["h"].shape[0])
    tok[grpo["idx"]] = grpo["adv"][grpo["tok_rollout"]]
    ppo = _loss(b, token_adv=tok, **kw)
    assert ppo["loss"] == grpo["loss"]
    np.testing.assert_array_equal(ppo["dh"], grpo["dh"])
    np.testing.assert_array_equal(ppo["dW"], grpo["dW"])


def test_token_advantage_gradients_match_finite_differences():
    b = _with_old_from_current(47, excluded=(1,), sigma=0.6)
    b = _kink_safe(b, 0.2, 0.2)
    tok = np.random.default_rng(47).standard_normal(b["h"].shape[0])
    kw = dict(eps_low=0.2, eps_high=0.2, agg=O.AGG_TOKEN, token_adv=tok)
    out = _loss(b, **kw)
    assert 0 < out["stats"]["clip_frac"] < 1
    rng = np.random.default_rng(48)
    for name, grad in (("h", out["dh"]), ("W", out["dW"])):
        X = b[name]
        for ij in [tuple(rng.integers(0, s) for s in X.shape) for _ in range(15)]:
            bp = dict(b)
            bp[name] = X.copy()
            bp[name][ij] += 1e-6
            lp_ = _loss(bp, grads=False, **kw)["loss"]
            bp[name][ij] -= 2e-6
            lm_ = _loss(bp, grads=False, **kw)["loss"]
            assert abs((lp_ - lm_) / 2e-6 - grad[ij]) <= 1e-6 * max(1.0, abs(grad).max())


# ------------------------------------- row-restricted helpers used by the full-size GPU checks
@pytest.mark.parametrize("agg", [O.AGG_SEQ, O.AGG_TOKEN])
def test_loss_from_token_values_matches_the_full_pass(agg):
    b = _with_old_from_current(61, excluded=(2,))
    kw = dict(eps_low=0.2, eps_high=0.28, entropy_coef=0.03, agg=agg)
    out = _loss(b, **kw)
    idx, tr, npol = out["idx"], out["tok_rollout"], out["n_pol"]
    ga = O.group_advantage(b["rewards"], b["group_ids"], EPS)
    got = O.loss_from_token_values(out["logp"], out["H"], b["old_logp"][idx], ga["adv"][tr], tr, npol,
                                   ga["group_index"], ga["G"], ga["n_groups"], eps_low=0.2, eps_high=0.28,
                                   entropy_coef=0.03, agg=agg)
    np.testing.assert_allclose(got, out["loss"], rtol=1e-12, atol=1e-15)
    omega = O.token_weights(tr, npol, ga["group_index"], ga["G"], ga["n_groups"], agg)
    g, e = O.token_grad_weights(out["logp"], b["old_logp"][idx], ga["adv"][tr], omega, eps_low=0.2,
                                eps_high=0.28, entropy_coef=0.03)
    np.testing.assert_allclose(g, out["g"], rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(e, out["e"], rtol=1e-13, atol=1e-16)


def test_dw_rows_match_the_full_gradient():
    b = _with_old_from_current(62, V=24, excluded=(1,))
    kw = dict(eps_low=0.2, eps_high=0.28, entropy_coef=0.05)
    out = _loss(b, **kw)
    idx = out["idx"]
    y = b["targets"][idx]
    # every row, so the selection includes each target id and the zero column sum applies
    v_all = np.arange(b["W"].shape[0])
    rows = O.dw_rows(b["h"][idx], b["W"], v_all, y, out["logp"], out["H"], out["g"], out["e"], block=7)
    np.testing.assert_allclose(rows, out["dW"], rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(rows.sum(axis=0), 0.0, atol=1e-13)
    sel = np.array([y[0], 3, 17, y[-1]])
    part = O.dw_rows(b["h"][idx], b["W"], sel, y, out["logp"], out["H"], out["g"], out["e"])
    np.testing.assert_allclose(part, out["dW"][sel], rtol=1e-11, atol=1e-14)


# ------------------------------------------------------------- linear value head (PPO critic)
def test_value_head_closed_form_and_exclusion():
    c = _gae_case(45)
    N = c["mask"].shape[0]
    d = 6
    h = np.zeros((N, d))
    h[np.arange(N), np.arange(N) % d] = 1.0          # row t is the unit vector e_{t mod d}
    w = np.arange(1.0, d + 1.0)
    V = O.value_head(h, w, 0.5, c["mask"], c["cu"])
    m = c["mask"].astype(bool)
    np.testing.assert_array_equal(V[m], w[np.arange(N) % d][m] + 0.5)
    assert np.all(V[~m] == 0)
    gid = np.zeros(c["cu"].shape[0] - 1, dtype=np.int64)
    gid[0] = -1                                       # excluded rollout: no values
    V2 = O.value_head(h, w, 0.5, c["mask"], c["cu"], gid)
    assert np.all(V2[c["cu"][0]:c["cu"][1]] == 0)


def test_value_head_gradients_match_finite_differences():
    c = _gae_case(46)
    rng = np.random.default_rng(47)
    N = c["mask"].shape[0]
    d = 5
    h = rng.standard_normal((N, d))
    w = rng.standard_normal(d)
    b = 0.3
    G = rng.standard_normal(N)
    gid = np.zeros(c["cu"].shape[0] - 1, dtype=np.int64)
    gid[-1] = -1

    def loss(hh, ww, bb):
        return O.value_loss(O.value_head(hh, ww, bb, c["mask"], c["cu"], gid), G, c["mask"], c["cu"], gid)[0]

    _, dV = O.value_loss(O.value_head(h, w, b, c["mask"], c["cu"], gid), G, c["mask"], c["cu"], gid)
    dh, dw, db = O.value_head_grads(h, w, dV, c["mask"], c["cu"], gid)
    eps = 1e-6
    for t in range(N):
        for j in (0, d - 1):
            hp, hm = h.copy(), h.copy()
            hp[t, j] += eps
            hm[t, j] -= eps
            np.testing.assert_allclose((loss(hp, w, b) - loss(hm, w, b)) / (2 * eps), dh[t, j], atol=1e-8)
    for j in range(d):
        wp, wm = w.copy(), w.copy()
        wp[j] += eps
        wm[j] -= eps
        np.testing.assert_allclose((loss(h, wp, b) - loss(h, wm, b)) / (2 * eps), dw[j], rtol=1e-6, atol=1e-9)
    np.testing.assert_allclose((loss(h, w, b + eps) - loss(h, w, b - eps)) / (2 * eps), db, rtol=1e-6, atol=1e-9)


# ------------------------------------------------- sampling temperature (logits z = W h / tau)
def test_temperature_is_a_rescaled_lm_head():
    # z = W h / tau is the tau = 1 computation with W / tau: the same loss, log-probs and dhidden,
    # and dW scaled by 1 / tau (chain rule through W -> W / tau)
    b = _with_old_from_current(81, excluded=(1,))
    tau = 0.7
    kw = dict(eps_low=0.2, eps_high=0.28, entropy_coef=0.03)
    out = _loss(b, temperature=tau, **kw)
    b1 = dict(b)
    b1["W"] = b["W"] / tau
    ref = _loss(b1, **kw)
    np.testing.assert_allclose(out["loss"], ref["loss"], rtol=1e-12)
    np.testing.assert_allclose(out["logp"], ref["logp"], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(out["dh"], ref["dh"], rtol=1e-11, atol=1e-15)
    np.testing.assert_allclose(out["dW"], ref["dW"] / tau, rtol=1e-11, atol=1e-15)
    lse, lp, H = O.token_logprob(b["h"][out["idx"]], b["W"], b["targets"][out["idx"]], temperature=tau)
    np.testing.assert_allclose(lp, out["logp"], rtol=1e-12, atol=1e-14)


def test_temperature_gradients_match_finite_differences():
    b = _with_old_from_current(82, excluded=(2,))
    tau = 1.6
    b = _kink_safe(b, 0.2, 0.28, temperature=tau)
    kw = dict(eps_low=0.2, eps_high=0.28, entropy_coef=0.05, temperature=tau)
    out = _loss(b, **kw)
    rng = np.random.default_rng(83)
    step = 1e-6
    for name, grad in (("h", out["dh"]), ("W", out["dW"])):
        X = b[name]
        for _ in range(15):
            ij = tuple(rng.integers(0, s) for s in X.shape)
            bp = dict(b)
            bp[name] = X.copy()
            bp[name][ij] += step
            lp_ = _loss(bp, grads=False, **kw)["loss"]
            bp[name][ij] -= 2 * step
            lm_ = _loss(bp, grads=False, **kw)["loss"]
            assert abs((lp_ - lm_) / (2 * step) - grad[ij]) <= 1e-6 * max(1.0, abs(grad).max()), (name, ij)
    # the row-restricted helpers follow the same temperature
    idx = out["idx"]
    rows = O.dw_rows(b["h"][idx], b["W"], np.arange(b["W"].shape[0]), b["targets"][idx], out["logp"], out["H"],
                     out["g"], out["e"], temperature=tau)
    np.testing.assert_allclose(rows, out["dW"], rtol=1e-10, atol=1e-14)


# ---------------------- sampled_rows: the per-row checker of the full-size GPU parity tests
def _sampled_rows_case(seed, agg, temperature):
    b = _with_old_from_current(seed, sigma=0.5, excluded=(3,), per_group=(3, 4, 3))
    b = _kink_safe(b, 0.2, 0.28, temperature=temperature)
    rng = np.random.default_rng(seed + 7)
    N = b["h"].shape[0]
    b["rollout_logp"] = b["old_logp"] + rng.standard_normal(N) * 0.4   # TIS cap binds on part of the rows
    b["ref_logp"] = b["old_logp"] + rng.standard_normal(N) * 0.3
    kw = dict(eps_low=0.2, eps_high=0.28, entropy_coef=0.04, agg=agg, rollout_logp=b["rollout_logp"],
              tis_cap=1.1, ref_logp=b["ref_logp"], kl_coef=0.07, temperature=temperature)
    return b, kw


@pytest.mark.parametrize("agg,temperature", [(O.AGG_SEQ, 1.0), (O.AGG_SEQ, 1.3), (O.AGG_TOKEN, 0.8)])
def test_sampled_rows_reproduce_the_full_pass(agg, temperature):
    # Sec. 2.3.1-2.3.2: a row's log-prob, entropy, chain-rule weights and dhidden depend only on the
    # row and on its per-rollout scalars, so the row-restricted pass equals the full pass (itself
    # pinned by finite differences and torch autograd) row by row, with every option switched on
    b, kw = _sampled_rows_case(91, agg, temperature)
    out = _loss(b, **kw)
    assert 0 < out["clipped"].mean() < 1 and (out["tis"] < 1.1).any() and (out["tis"] == 1.1).any()
    idx = out["idx"]
    perm = np.random.default_rng(5).permutation(idx.shape[0])   # rows in any order and any block size
    sel = idx[perm]
    got = O.sampled_rows(b["h"][sel], b["W"], b["targets"][sel], b["old_logp"][sel], out["adv_tok"][perm],
                         out["omega"][perm], eps_low=0.2, eps_high=0.28, entropy_coef=0.04,
                         tis_rows=out["tis"][perm], ref_rows=b["ref_logp"][sel], kl_coef=0.07,
                         temperature=temperature, block=5)
    for k in ("lse", "logp", "H", "rho", "g", "e"):
        np.testing.assert_allclose(got[k], out[k][perm], rtol=1e-12, atol=1e-15, err_msg=k)
    np.testing.assert_array_equal(got["clipped"], out["clipped"][perm])
    np.testing.assert_allclose(got["dh"], out["dh"][sel], rtol=1e-11, atol=1e-15)


def test_sampled_rows_dhidden_matches_finite_differences_of_the_row_loss():
    # independent of pg_loss_fwd_bwd: the row's loss term omega_t w_t (s_t + c H_t - beta KL_t) built
    # from the log-softmax (pinned against torch.log_softmax) and differentiated numerically in h_t
    tau = 1.3
    b, kw = _sampled_rows_case(92, O.AGG_SEQ, tau)
    out = _loss(b, grads=False, **kw)
    idx = out["idx"]
    pick = np.arange(0, idx.shape[0], max(1, idx.shape[0] // 6))
    sel = idx[pick]
    A, om, w = out["adv_tok"][pick], out["omega"][pick], out["tis"][pick]
    got = O.sampled_rows(b["h"][sel], b["W"], b["targets"][sel], b["old_logp"][sel], A, om, eps_low=0.2,
                         eps_high=0.28, entropy_coef=0.04, tis_rows=w, ref_rows=b["ref_logp"][sel], kl_coef=0.07,
                         temperature=tau)

    def row_loss(i, hrow):
        _, lp, H = O.token_logprob(hrow[None, :], b["W"], b["targets"][sel[i]:sel[i] + 1], temperature=tau)
        rho = math.exp(lp[0] - b["old_logp"][sel[i]])
        s = min(rho * A[i], min(max(rho, 0.8), 1.28) * A[i])
        r = b["ref_logp"][sel[i]] - lp[0]
        kl = math.expm1(r) - r
        return om[i] * w[i] * (s + 0.04 * H[0] - 0.07 * kl)

    step = 1e-6
    for i in range(sel.shape[0]):
        h0 = b["h"][sel[i]].astype(np.float64)
        for j in range(h0.shape[0]):
            hp, hm = h0.copy(), h0.copy()
            hp[j] += step
            hm[j] -= step
            fd = (row_loss(i, hp) - row_loss(i, hm)) / (2 * step)
            assert abs(fd - got["dh"][i, j]) <= 1e-7 * max(1.0, abs(got["dh"][i]).max()), (i, j, fd, got["dh"][i, j])
