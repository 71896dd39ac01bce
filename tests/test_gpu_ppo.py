"""GPU parity of the PPO path through the C ABI: masked GAE (rlk_gae), the masked value loss
(rlk_value_loss) and the clipped loss with per-token advantages, against the fp64 oracle."""
import numpy as np
import pytest

from gpu_common import (O, WL, build_instance, compare_full, ensure_library, log, params_for, rlk, run_gpu,
                        run_oracle)

pytestmark = pytest.mark.gpu


def _structure_tensors(st):
    import torch

    dev = "cuda"
    return dict(mask=torch.as_tensor(st.mask, device=dev), cu=torch.as_tensor(st.cu_seqlens, device=dev),
                rewards=torch.as_tensor(st.rewards, device=dev), gid=torch.as_tensor(st.group_ids, device=dev))


GAE_CASES = [("small_bf16", True), ("long_bf16", False), ("large_bf16", True)]


@pytest.mark.parametrize("name,scaled", GAE_CASES)
def test_gae_parity(name, scaled):
    import torch

    ensure_library()
    cfg = WL.scaled_config(name) if scaled else WL.get_config(name)
    if name == "large_bf16":
        cfg = cfg.with_(n_excluded=3)
    st = WL.make_structure(cfg)
    T = _structure_tensors(st)
    vals = WL.token_values(st, cfg.seed + 501, scale=0.5)
    v_dev = torch.as_tensor(vals, device="cuda")
    for gamma, lam in ((1.0, 1.0), (0.99, 0.95), (1.0, 0.0), (0.5, 0.9)):
        adv, ret = rlk.gae(v_dev, T["rewards"], T["mask"], T["cu"], T["gid"], gamma, lam)
        torch.cuda.synchronize()
        ra, rr = O.gae(vals, st.rewards, st.mask, st.cu_seqlens, st.group_ids, gamma, lam)
        a, r = adv.cpu().numpy().astype(np.float64), ret.cpu().numpy().astype(np.float64)
        scale = max(1.0, float(np.abs(ra).max()))
        ea, er = float(np.abs(a - ra).max()) / scale, float(np.abs(r - rr).max()) / max(1.0, float(np.abs(rr).max()))
        log(f"gae {cfg.name} N={st.N} R={st.R} gamma={gamma} lam={lam}: adv err {ea:.2e}, returns err {er:.2e}")
        assert ea <= 2e-6 and er <= 2e-6
        zero = ra == 0
        assert np.all(a[zero] == 0)   # tool rows and excluded rollouts are exactly 0


def test_gae_edge_cases():
    import torch

    ensure_library()
    # a rollout with no policy token, an empty rollout, a 1-token rollout, a long all-policy one
    lens = [5, 0, 1, 700]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    N = int(cu[-1])
    mask = np.ones(N, np.uint8)
    mask[:5] = 0
    vals = np.random.default_rng(3).standard_normal(N).astype(np.float32)
    rew = np.array([1.0, 0.5, -2.0, 0.25], np.float32)
    d = lambda x: torch.as_tensor(x, device="cuda")
    adv, ret = rlk.gae(d(vals), d(rew), d(mask), d(cu), None, 0.9, 0.7)
    torch.cuda.synchronize()
    ra, rr = O.gae(vals, rew, mask, cu, None, 0.9, 0.7)
    np.testing.assert_allclose(adv.cpu().numpy(), ra, rtol=0, atol=2e-6 * max(1, np.abs(ra).max()))
    np.testing.assert_allclose(ret.cpu().numpy(), rr, rtol=0, atol=2e-6 * max(1, np.abs(rr).max()))
    # N = 0 and R = 0 are no-ops
    e = torch.empty(0, dtype=torch.float32, device="cuda")
    rlk.gae(e, torch.empty(0, device="cuda"), torch.empty(0, dtype=torch.uint8, device="cuda"),
            torch.zeros(1, dtype=torch.int32, device="cuda"))


@pytest.mark.parametrize("name,scaled", [("small_bf16", True), ("large_bf16", False)])
def test_value_loss_parity(name, scaled):
    import torch

    ensure_library()
    cfg = WL.scaled_config(name) if scaled else WL.get_config(name)
    cfg = cfg.with_(n_excluded=2)
    st = WL.make_structure(cfg)
    T = _structure_tensors(st)
    vals = WL.token_values(st, cfg.seed + 502, scale=0.5)
    rets = WL.token_values(st, cfg.seed + 503, scale=1.0)
    loss, dv = rlk.value_loss(torch.as_tensor(vals, device="cuda"), torch.as_tensor(rets, device="cuda"), T["mask"],
                              T["cu"], T["gid"])
    torch.cuda.synchronize()
    rl, rdv = O.value_loss(vals, rets, st.mask, st.cu_seqlens, st.group_ids)
    g = dv.cpu().numpy().astype(np.float64)
    log(f"value loss {cfg.name}: {float(loss.item()):.6f} vs {rl:.6f}")
    assert abs(float(loss.item()) - rl) <= 1e-6 * max(1.0, abs(rl))
    assert float(np.abs(g - rdv).max()) <= 1e-6 * max(1e-30, float(np.abs(rdv).max()))
    assert np.all(g[rdv == 0] == 0)


@pytest.mark.parametrize("name,scaled,agg", [("tiny_fp32", False, rlk.AGG_TOKEN), ("qwen8b_bf16", True, rlk.AGG_TOKEN),
                                             ("small_bf16", True, rlk.AGG_SEQ)])
def test_ppo_loss_parity(name, scaled, agg):
    """The clipped loss with per-token advantages from rlk_gae (gamma = lambda = 1)."""
    import torch

    cfg = WL.scaled_config(name) if scaled else WL.get_config(name)
    inst = build_instance(cfg)
    st = inst["st"]
    vals = WL.token_values(st, cfg.seed + 504, scale=0.3)
    adv_dev, _ = rlk.gae(torch.as_tensor(vals, device="cuda"), inst["rewards"], inst["mask"], inst["cu"], inst["gid"])
    ra, _ = O.gae(vals, st.rewards, st.mask, st.cu_seqlens, st.group_ids)
    p = params_for(cfg, agg=agg, chunk_rows=256 if scaled else 0)
    gpu = run_gpu(inst, p, token_adv=adv_dev)
    ref = run_oracle(inst, p, token_adv=ra)
    compare_full(inst, gpu, ref, p, tag="ppo")


# ------------------------------------------------------------------ linear value head
HEAD_CASES = [("tiny_fp32", False), ("small_bf16", True), ("qwen8b_bf16", True)]


@pytest.mark.parametrize("name,scaled", HEAD_CASES)
def test_value_head_parity(name, scaled):
    """values = w_v . h + b_v on the policy rows of non-excluded rollouts; the backward from the
    value loss (dhidden written and accumulated, dw_v, db_v) against the oracle, bitwise repeatable."""
    import torch

    from gpu_common import rel_fro, to_host

    ensure_library()
    cfg = WL.scaled_config(name) if scaled else WL.get_config(name)
    cfg = cfg.with_(n_excluded=1)
    inst = build_instance(cfg)
    st = inst["st"]
    h = inst["h"]
    rng = np.random.default_rng(cfg.seed + 77)
    w_host = (rng.standard_normal(cfg.d) / np.sqrt(cfg.d)).astype(np.float32)
    w = torch.as_tensor(w_host, device="cuda").to(h.dtype)
    b_v = 0.25
    vals = rlk.value_head_fwd(h, w, b_v, inst["mask"], inst["cu"], inst["gid"])
    torch.cuda.synchronize()
    h_host, w64 = to_host(h), to_host(w)
    ref = O.value_head(h_host, w64, b_v, st.mask, st.cu_seqlens, st.group_ids)
    ev = float(np.abs(vals.cpu().numpy() - ref).max()) / max(1.0, float(np.abs(ref).max()))
    assert np.all(vals.cpu().numpy()[ref == 0] == 0)
    # backward of the value loss against seeded returns
    G = rng.standard_normal(st.N).astype(np.float32)
    _, dV = O.value_loss(ref, G, st.mask, st.cu_seqlens, st.group_ids)
    dV_dev = torch.as_tensor(dV.astype(np.float32), device="cuda")
    r_dh, r_dw, r_db = O.value_head_grads(h_host, w64, dV.astype(np.float32), st.mask, st.cu_seqlens, st.group_ids)
    dh = torch.full_like(h, 7.0)
    dh, dw, db = rlk.value_head_bwd(h, w, inst["mask"], inst["cu"], inst["gid"], dV_dev, dhidden=dh)
    torch.cuda.synchronize()
    e_dh = rel_fro(to_host(dh), r_dh)
    e_dw = rel_fro(dw.cpu().numpy(), r_dw)
    e_db = abs(float(db.item()) - r_db) / max(1e-30, float(np.abs(dV).sum()))
    # accumulate: kept rows get the gradient added, the other rows keep their values
    # a base of the gradient's own magnitude, so bf16 rounding of the sum stays relative
    scale = float(np.abs(r_dh).max())
    base = torch.as_tensor((scale * rng.standard_normal((st.N, cfg.d))).astype(np.float32), device="cuda").to(h.dtype)
    acc = base.clone()
    rlk.value_head_bwd(h, w, inst["mask"], inst["cu"], inst["gid"], dV_dev, dhidden=acc, accumulate=True)
    _, dw2, db2 = rlk.value_head_bwd(h, w, inst["mask"], inst["cu"], inst["gid"], dV_dev)
    torch.cuda.synchronize()
    e_acc = rel_fro(to_host(acc), to_host(base) + r_dh)   # the accumulated result against its exact value
    keep = np.zeros(st.N, dtype=bool)
    keep[O.compact(st.mask, st.cu_seqlens, st.group_ids)[0]] = True
    unchanged = bool(torch.equal(acc[torch.as_tensor(~keep, device="cuda")], base[torch.as_tensor(~keep, device="cuda")]))
    log(f"value head {cfg.name} N={st.N} d={cfg.d}: values {ev:.2e}, dh {e_dh:.2e}, dw {e_dw:.2e}, db {e_db:.2e}, "
        f"accumulated dh {e_acc:.2e}")
    tol_v = 1e-5 if cfg.dtype == "f32" else 1e-4
    tol_h = 1e-6 if cfg.dtype == "f32" else 1e-2
    assert ev <= tol_v and e_dh <= tol_h and e_dw <= 1e-5 and e_db <= 1e-6
    assert e_acc <= (1e-6 if cfg.dtype == "f32" else 1e-2) and unchanged
    assert torch.equal(dw, dw2) and torch.equal(db, db2)
    assert int(torch.count_nonzero(dh[torch.as_tensor(~keep, device="cuda")])) == 0
