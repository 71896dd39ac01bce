"""GPU parity of the HIP hot path against the fp64 oracle, through the C ABI.

Integer outputs (compaction lists, group indices, counts) must be bit-exact; floating
outputs meet the tolerances in gpu_common.  Full parity runs on every configuration at a
scaled size the oracle finishes in seconds (several token and vocabulary tiles, ragged
tails, several backward chunks); the full-size runs are checked on seeded sampled rows
that the oracle computes one by one and on properties that hold at any size.
"""
import numpy as np
import pytest

from gpu_common import (TOL_GRAD, TOL_LOSS, aux_logps, loss_error, TOL_LOGP, O, WL, build_instance, compare_full, ensure_library, log,
                        expected_grad_tokens, params_for, ref_layout, rel_fro, rlk, run_gpu, run_oracle, to_host, with_far_target)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ensure_library()


def _dev(a, dt):
    import torch

    return torch.as_tensor(a, dtype=dt, device="cuda")


# ------------------------------------------------------------------ a1: compaction (bit-exact)
@pytest.mark.parametrize("name,scaled,excl", [("tiny_fp32", False, 0), ("qwen8b_bf16", False, 3),
                                               ("large_bf16", False, 7), ("long_bf16", True, 1)])
def test_compaction_bit_exact(name, scaled, excl):
    import torch

    cfg = WL.scaled_config(name) if scaled else WL.get_config(name)
    cfg = cfg.with_(n_excluded=excl)
    st = WL.make_structure(cfg)
    log(f"compaction {cfg.name} N={st.N} R={st.R} excluded={excl}")
    idx, tokr, npol, neff, ws = rlk.compact(_dev(st.cu_seqlens, torch.int32), _dev(st.mask, torch.uint8),
                                            _dev(st.group_ids, torch.int32), _dev(st.targets, torch.int32),
                                            V=cfg.V)
    torch.cuda.synchronize()
    ri, rt, rn = O.compact(st.mask, st.cu_seqlens, st.group_ids)
    n = int(neff.item())
    assert n == ri.shape[0]
    assert np.array_equal(idx[:n].cpu().numpy(), ri)
    assert np.array_equal(tokr[:n].cpu().numpy(), rt)
    assert np.array_equal(npol.cpu().numpy(), rn)
    assert rlk.check_status(ws) == 0


def test_compaction_edge_cases():
    import torch

    # empty rollouts, a rollout of length 1, all-masked rollout, mask NULL
    lens = np.array([0, 1, 5, 0, 300, 4096, 4097, 2])
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    N = int(cu[-1])
    rng = np.random.default_rng(5)
    mask = (rng.random(N) < 0.5).astype(np.uint8)
    mask[cu[4]:cu[5]] = 0
    gid = np.array([3, 3, 0, 9, 9, -1, 0, 3], dtype=np.int32)
    for m in (mask, None):
        idx, tokr, npol, neff, ws = rlk.compact(_dev(cu, torch.int32), None if m is None else _dev(m, torch.uint8),
                                                _dev(gid, torch.int32), N=N)
        ri, rt, rn = O.compact(m, cu, gid)
        n = int(neff.item())
        assert n == len(ri)
        assert np.array_equal(idx[:n].cpu().numpy(), ri) and np.array_equal(tokr[:n].cpu().numpy(), rt)
        assert np.array_equal(npol.cpu().numpy(), rn)


# ------------------------------------------------------------------ a2: advantages
@pytest.mark.parametrize("name,excl", [("large_bf16", 5), ("qwen8b_bf16", 0), ("tiny_fp32", 1)])
def test_group_advantage(name, excl):
    import torch

    cfg = WL.get_config(name).with_(n_excluded=excl)
    st = WL.make_structure(cfg)
    R = st.R
    gi = torch.empty(R, dtype=torch.int32, device="cuda")
    ng = torch.empty(1, dtype=torch.int32, device="cuda")
    adv = rlk.group_advantage(_dev(st.rewards, torch.float32), _dev(st.group_ids, torch.int32), 1e-6,
                              group_index=gi, n_groups=ng)
    ref = O.group_advantage(st.rewards, st.group_ids, 1e-6)
    a = adv.cpu().numpy()
    assert np.array_equal(gi.cpu().numpy(), ref["group_index"])
    assert int(ng.item()) == ref["n_groups"]
    err = np.abs(a - ref["adv"]).max()
    log(f"advantage {name}: max abs err {err:.3g}")
    assert err <= 1e-6 * max(1.0, np.abs(ref["adv"]).max())
    # all-equal groups and excluded rollouts are exactly zero
    zero = np.flatnonzero(ref["adv"] == 0)
    assert np.all(a[zero] == 0)


def test_group_advantage_small_cases():
    import torch

    rew = np.array([1, 0, 0, 0, 0.5, 0.5, 7, 1, 0], dtype=np.float32)
    gid = np.array([2, 2, 2, 2, 5, 5, 0, -1, 11], dtype=np.int32)
    adv = rlk.group_advantage(_dev(rew, torch.float32), _dev(gid, torch.int32), 1e-6).cpu().numpy()
    p = 0.25
    s = np.sqrt(p * (1 - p))
    np.testing.assert_allclose(adv[:4], [(1 - p) / (s + 1e-6)] + [-p / (s + 1e-6)] * 3, rtol=1e-6)
    assert np.all(adv[4:] == 0)


# ------------------------------------------------------------------ a3: log-prob forward
@pytest.mark.parametrize("name,scaled", [("tiny_fp32", False), ("small_bf16", True), ("qwen8b_bf16", True)])
def test_logprob_fwd(name, scaled):
    import torch

    cfg = WL.scaled_config(name) if scaled else WL.get_config(name)
    st = WL.make_structure(cfg)
    h, W = WL.make_tensors(cfg, st.N, device="cuda")
    N = st.N
    log(f"logprob {cfg.name} N={N} d={cfg.d} V={cfg.V}")
    ent = torch.empty(N, dtype=torch.float32, device="cuda")
    lse = torch.empty(N, dtype=torch.float32, device="cuda")
    logp, _, _, ws = rlk.logprob_fwd(h, W, _dev(st.targets, torch.int32), _dev(st.mask, torch.uint8),
                                     _dev(st.cu_seqlens, torch.int32), entropy=ent, lse=lse)
    torch.cuda.synchronize()
    assert rlk.check_status(ws) == 0
    idx, _, _ = O.compact(st.mask, st.cu_seqlens)
    rl, rp, rH = O.token_logprob(to_host(h)[idx], to_host(W), st.targets[idx])
    g = {k: v.cpu().numpy() for k, v in (("logp", logp), ("ent", ent), ("lse", lse))}
    e = dict(logp=np.abs(g["logp"][idx] - rp).max(), ent=np.abs(g["ent"][idx] - rH).max(),
             lse=np.abs(g["lse"][idx] - rl).max())
    log(f"  max abs err {e}")
    tol = TOL_LOGP[cfg.dtype]
    assert e["logp"] <= tol and e["ent"] <= tol and e["lse"] <= tol * max(1.0, np.abs(rl).max())
    keep = np.zeros(N, dtype=bool)
    keep[idx] = True
    for k in g:
        assert np.all(g[k][~keep] == 0)


# ------------------------------------------------------------------ a1-a7: loss forward + backward
PARITY = [("tiny_fp32", False, 0), ("small_bf16", True, 0), ("qwen8b_bf16", True, 256),
          ("long_bf16", True, 512), ("large_bf16", True, 256)]


@pytest.mark.parametrize("name,scaled,chunk", PARITY)
def test_pg_loss_parity(name, scaled, chunk):
    cfg = WL.scaled_config(name) if scaled else WL.get_config(name)
    if name == "large_bf16":
        cfg = cfg.with_(n_excluded=1)
    inst = build_instance(cfg)
    p = params_for(cfg, chunk_rows=chunk)
    log(f"pg_loss {cfg.name} N={inst['st'].N} chunk_rows={chunk}")
    gpu = run_gpu(inst, p)
    ref = run_oracle(inst, p)
    compare_full(inst, gpu, ref, p, tag="seq")


@pytest.mark.parametrize("name,scaled,agg,ent", [("tiny_fp32", False, rlk.AGG_SEQ, 0.01),
                                                 ("small_bf16", True, rlk.AGG_SEQ, 0.01),
                                                 ("qwen8b_bf16", True, rlk.AGG_TOKEN, 0.01),
                                                 ("qwen8b_bf16", True, rlk.AGG_SEQ, 0.0)])
def test_pg_loss_tis_and_kl_parity(name, scaled, agg, ent):
    """Truncated importance sampling (Sec. 3.2.4) and the KL term (Sec. 2.3.2), both on, the cap
    binding on part of the tokens; without the entropy term through the token-reference layout."""
    cfg = WL.scaled_config(name) if scaled else WL.get_config(name)
    inst = build_instance(cfg)
    aux = aux_logps(inst)
    p = params_for(cfg, agg=agg, tis_cap=1.1, kl_coef=0.05, entropy_coef=ent, chunk_rows=256 if scaled else 0)
    log(f"pg_loss tis+kl {cfg.name} N={inst['st'].N}")
    gpu = run_gpu(inst, p, aux=aux)
    ref = run_oracle(inst, p, aux=aux)
    assert 0 < np.mean(ref["tis"] == np.float64(p.tis_cap)) < 1
    compare_full(inst, gpu, ref, p, tag="tis+kl")


def test_pg_loss_token_mean_and_override():
    cfg = WL.scaled_config("qwen8b_bf16")
    inst = build_instance(cfg)
    for kw in (dict(agg=rlk.AGG_TOKEN), dict(agg=rlk.AGG_SEQ, norm_override=5.0),
               dict(agg=rlk.AGG_TOKEN, norm_override=1234.0, entropy_coef=0.01)):
        p = params_for(cfg, chunk_rows=512, **kw)
        compare_full(inst, run_gpu(inst, p), run_oracle(inst, p), p, tag=str(kw))


def test_microbatch_accumulation_matches_one_call():
    """Per-group calls with accumulate_dW and norm_override = Q add up to the one-call gradient."""
    import torch

    cfg = WL.scaled_config("small_bf16")
    inst = build_instance(cfg)
    st = inst["st"]
    p = params_for(cfg)
    full = run_gpu(inst, p)
    Q = full["stats"]["n_groups"]
    dW = torch.zeros_like(full["dW"])
    tot = 0.0
    for key in np.unique(st.group_ids):
        rs = np.flatnonzero(st.group_ids == key)
        rows = np.concatenate([np.arange(st.cu_seqlens[r], st.cu_seqlens[r + 1]) for r in rs])
        lens = st.cu_seqlens[rs + 1] - st.cu_seqlens[rs]
        rows_t = torch.as_tensor(rows, device="cuda")
        sub = dict(inst)
        sub.update(h=inst["h"][rows_t].contiguous(), targets=inst["targets"][rows_t].contiguous(),
                   mask=inst["mask"][rows_t].contiguous(), old=inst["old"][rows_t].contiguous(),
                   cu=_dev(np.concatenate([[0], np.cumsum(lens)]), torch.int32),
                   rewards=_dev(st.rewards[rs], torch.float32), gid=_dev(st.group_ids[rs], torch.int32))
        out = run_gpu(sub, params_for(cfg, accumulate_dW=True, norm_override=float(Q)), dW=dW)
        tot += out["loss"]
    err = rel_fro(to_host(dW), to_host(full["dW"]))
    log(f"microbatch dW rel err {err:.3g}; loss {tot:.6g} vs {full['loss']:.6g}")
    assert err <= 1e-3
    assert abs(tot - full["loss"]) <= 1e-4 * max(1e-3, abs(full["loss"]))


def test_determinism_and_masked_invariance():
    import torch

    cfg = WL.scaled_config("large_bf16")
    inst = build_instance(cfg)
    p = params_for(cfg, chunk_rows=256)
    a = run_gpu(inst, p)
    b = run_gpu(inst, p)
    assert a["loss"] == b["loss"]
    assert torch.equal(a["dh"], b["dh"]) and torch.equal(a["dW"], b["dW"])
    # change every input on masked rows: outputs on trained rows are bitwise unchanged
    st = inst["st"]
    masked = torch.as_tensor(st.mask == 0, device="cuda")
    pert = dict(inst)
    h2 = inst["h"].clone()
    h2[masked] = -3.0 * h2[masked]
    t2 = inst["targets"].clone()
    t2[masked] = 0
    o2 = inst["old"].clone()
    o2[masked] = 5.0
    pert.update(h=h2, targets=t2, old=o2)
    c = run_gpu(pert, p)
    assert c["loss"] == a["loss"]
    assert torch.equal(c["dW"], a["dW"]) and torch.equal(c["dh"], a["dh"])


def test_empty_and_fully_excluded_batches():
    import torch

    cfg = WL.scaled_config("small_bf16")
    inst = build_instance(cfg)
    p = params_for(cfg)
    dW0 = torch.full(inst["W"].shape, 7.0, dtype=torch.float32, device="cuda")
    out = run_gpu(inst, p, mask=torch.zeros_like(inst["mask"]), dW=dW0)
    assert out["loss"] == 0.0 and out["flags"] == 0
    assert int(torch.count_nonzero(out["dh"])) == 0 and int(torch.count_nonzero(out["dW"])) == 0
    assert out["stats"]["n_policy_tokens"] == 0
    gid = torch.full_like(inst["gid"], -1)
    out = run_gpu(inst, p, gid=gid)
    assert out["loss"] == 0.0 and out["stats"]["n_groups"] == 0
    assert int(torch.count_nonzero(out["dh"])) == 0 and int(torch.count_nonzero(out["dW"])) == 0


def test_device_data_errors_are_flagged():
    import torch

    cfg = WL.scaled_config("small_bf16")
    inst = build_instance(cfg)
    p = params_for(cfg)
    st = inst["st"]
    t2 = inst["targets"].clone()
    pol = int(np.flatnonzero(st.mask)[3])
    t2[pol] = cfg.V + 5
    bad = dict(inst)
    bad["targets"] = t2
    assert run_gpu(bad, p)["flags"] & rlk.DERR_TARGET
    cu2 = inst["cu"].clone()
    cu2[-1] = cu2[-1] - 3
    bad = dict(inst)
    bad["cu"] = cu2
    assert run_gpu(bad, p)["flags"] & rlk.DERR_CU_SEQLENS
    assert run_gpu(inst, p)["flags"] == 0


@pytest.mark.parametrize("name,chunk", [("qwen8b_bf16", 512), ("large_bf16", 256), ("tiny_fp32", 0)])
def test_policy_token_bound(name, chunk):
    """A host-known bound on the trained tokens sizes the chunk loop: exact and loose bounds give the
    oracle's results, per-token outputs and dhidden bitwise equal to the unbounded call (rows do not
    depend on the chunking); a bound below the batch's count is flagged."""
    import torch

    cfg = WL.scaled_config(name) if name != "tiny_fp32" else WL.get_config(name)
    inst = build_instance(cfg)
    p = params_for(cfg, chunk_rows=chunk)
    free = run_gpu(inst, p)
    n_eff = int(free["stats"]["n_policy_tokens"])
    ref = run_oracle(inst, p)
    for bound in (n_eff, n_eff + 777):
        log(f"bound {cfg.name}: n_eff={n_eff} max_policy_tokens={bound} chunk_rows={chunk}")
        got = run_gpu(inst, p, max_policy_tokens=bound)
        compare_full(inst, got, ref, p, tag=f"bound {bound}")
        assert got["loss"] == free["loss"]
        assert torch.equal(got["logp"], free["logp"]) and torch.equal(got["dh"], free["dh"])
        assert rel_fro(to_host(got["dW"]), to_host(free["dW"])) <= 1e-5
    log(f"bound {cfg.name}: max_policy_tokens={n_eff - 1} (below the count)")
    assert run_gpu(inst, p, max_policy_tokens=n_eff - 1)["flags"] & rlk.DERR_POLICY_BOUND


# ------------------------------------------------------------------ full-size, sampled rows
class _CompactRows:
    """Compacted policy rows of a device tensor, fetched to the host block by block."""

    def __init__(self, h, idx):
        import torch

        self.h = h
        self.idx = torch.as_tensor(idx, device=h.device)
        self.shape = (int(idx.shape[0]), int(h.shape[1]))

    def __getitem__(self, sl):
        return to_host(self.h[self.idx[sl]])


N_SAMPLED_ROWS = 1024
N_DW_ROWS = 64


@pytest.mark.parametrize("name,far", [("small_bf16", False), ("qwen8b_bf16", False), ("long_bf16", False),
                                      ("large_bf16", False), ("qwen8b_bf16", True)])
def test_full_size_sampled_rows(name, far):
    """Full-size batch in the configuration the benchmark times: integer outputs bit-exact;
    per-token log-prob / entropy and dhidden rows exact on 1,024 seeded sampled rows (a row
    depends only on itself and per-rollout scalars); the loss re-aggregated in fp64 from the
    GPU's per-token log-probs and entropies; 64 seeded dW rows from the GPU's per-token values
    (each is a sum over every policy token); the zero column sum of dW.  With far, one policy token
    in the middle of the batch gets a target about 700 nats below its largest logit, so its chunk
    (one of the full-size chunks) forms dz explicitly; that token joins the sampled rows."""
    import time

    import torch

    cfg = WL.get_config(name)
    inst = build_instance(cfg)
    st = inst["st"]
    p = params_for(cfg)
    idx, tr, npol = O.compact(st.mask, st.cu_seqlens, st.group_ids)
    far_pos = None
    if far:
        far_pos = idx.shape[0] // 2 + 12345
        inst, lp_far = with_far_target(inst, int(idx[far_pos]))
        st = inst["st"]
        log(f"  far target at policy token {far_pos} (row {int(idx[far_pos])}), log-prob {lp_far:.1f}")
    # the benchmark passes the host-known count of trained tokens as the bound (without far: chunks sized
    # by it, and dhidden tile rows of a partial last wave split over K; with far: chunks over all N) and
    # the host count of tokens in groups of unequal rewards as the chunk-planning hint
    bound = 0 if far else int(idx.shape[0])
    if bound:
        p = params_for(cfg, grad_tokens=rlk.grad_token_hint(st.mask, st.cu_seqlens, st.rewards, st.group_ids))
    log(f"full-size {name} N={st.N} max_policy_tokens={bound} grad_tokens={p.grad_tokens}")
    gpu = run_gpu(inst, p, max_policy_tokens=bound)
    assert gpu["flags"] == 0
    sg = gpu["stats"]
    log(f"  explicit dz in {sg['n_dz_chunks']} of {sg['n_chunks']} chunks")
    # every chunk of these batches keeps the token-reference layout when it applies (with far: all but one)
    if far:
        assert sg["n_dz_chunks"] == 1
    else:
        assert sg["n_dz_chunks"] == (0 if ref_layout(cfg, p) else sg["n_chunks"])
    ga = O.group_advantage(st.rewards, st.group_ids, p.adv_eps)
    assert gpu["stats"]["n_policy_tokens"] == idx.shape[0] and gpu["stats"]["n_groups"] == ga["n_groups"]
    omega = O.token_weights(tr, npol, ga["group_index"], ga["G"], ga["n_groups"], p.agg)
    adv_tok = ga["adv"][tr]
    # surrogate-only loss: the tokens of zero-advantage rollouts skip the backward
    n_grad = int(np.count_nonzero(adv_tok)) if p.entropy_coef == 0.0 else int(idx.shape[0])
    assert sg["n_grad_tokens"] == n_grad
    old_pol = inst["old_host"][idx]
    W_host = to_host(inst["W"])
    t0 = time.time()

    # sampled rows: forward and dhidden
    pick = np.sort(WL.sample_policy_rows(np.arange(idx.shape[0]), N_SAMPLED_ROWS, seed=cfg.seed + 7))
    if far_pos is not None:
        pick = np.unique(np.append(pick, far_pos))
    rows = idx[pick]
    rows_t = torch.as_tensor(rows, device="cuda")
    ref = O.sampled_rows(to_host(inst["h"][rows_t]), W_host, st.targets[rows], old_pol[pick], adv_tok[pick],
                         omega[pick], eps_low=p.eps_low, eps_high=p.eps_high, entropy_coef=p.entropy_coef)
    lp = gpu["logp"][rows_t].cpu().numpy()
    en = gpu["ent"][rows_t].cpu().numpy()
    dh = to_host(gpu["dh"][rows_t])
    e_lp, e_en = np.abs(lp - ref["logp"]).max(), np.abs(en - ref["H"]).max()
    e_dh = rel_fro(dh, ref["dh"])

    # loss: the oracle's aggregation of the GPU's per-token values (all policy tokens)
    idx_t = torch.as_tensor(idx, device="cuda")
    lp_all = gpu["logp"][idx_t].double().cpu().numpy()
    en_all = gpu["ent"][idx_t].double().cpu().numpy()
    loss_ref = O.loss_from_token_values(lp_all, en_all, old_pol, adv_tok, tr, npol, ga["group_index"], ga["G"],
                                        ga["n_groups"], eps_low=p.eps_low, eps_high=p.eps_high,
                                        entropy_coef=p.entropy_coef, agg=p.agg)
    s_tok, _, _ = O.surrogate(lp_all, old_pol, adv_tok, p.eps_low, p.eps_high)
    scale = float(np.abs(omega * (s_tok + p.entropy_coef * en_all)).sum())
    e_loss_l1 = abs(gpu["loss"] - loss_ref) / max(scale, 1e-30)
    e_loss = loss_error(gpu["loss"], loss_ref, scale)

    # dW rows: seeded vocabulary ids, a quarter of them targets of policy tokens (the one-hot term)
    rng = np.random.default_rng(cfg.seed + 11)
    tgt = st.targets[idx]
    v_sel = np.unique(np.concatenate([rng.choice(cfg.V, N_DW_ROWS * 3 // 4, replace=False),
                                      rng.choice(tgt, N_DW_ROWS // 4, replace=False)]))
    g, e = O.token_grad_weights(lp_all, old_pol, adv_tok, omega, eps_low=p.eps_low, eps_high=p.eps_high,
                                entropy_coef=p.entropy_coef)
    dw_ref = O.dw_rows(_CompactRows(inst["h"], idx), W_host, v_sel, tgt, lp_all, en_all, g, e)
    dw_gpu = gpu["dW"][torch.as_tensor(v_sel, device="cuda")].double().cpu().numpy()
    e_dw = rel_fro(dw_gpu, dw_ref)

    colsum = to_host(gpu["dW"].sum(dim=0))
    rel_cs = float(np.abs(colsum).max() / max(1e-30, float(gpu["dW"].abs().sum(dim=0).max())))
    log(f"  {N_SAMPLED_ROWS} sampled rows: logp {e_lp:.3g} ent {e_en:.3g} dh {e_dh:.3g}; loss {e_loss:.3g} "
        f"(gpu {gpu['loss']:.6g} ref {loss_ref:.6g}); {v_sel.shape[0]} dW rows {e_dw:.3g}; loss/L1 {e_loss_l1:.3g}; dW colsum rel "
        f"{rel_cs:.3g}; oracle {time.time() - t0:.1f} s")
    tol = TOL_LOGP[cfg.dtype]
    assert e_lp <= tol and e_en <= tol and e_dh <= TOL_GRAD
    assert e_loss <= TOL_LOSS
    assert e_dw <= TOL_GRAD
    assert rel_cs <= 1e-2


# Ragged shapes: hidden sizes that are not a multiple of the 64-element K slice (the forward GEMM's
# K tail, the dhidden/dW GEMMs' ragged N), vocabularies that are not a multiple of the 256-row
# tile (and smaller than one tile), token counts that leave partial token tiles.
# The bf16 shapes run with and without the entropy term (without it, the token-reference layout).
RAGGED = [("tiny_fp32", dict(d=264, V=1000), 0.02), ("tiny_fp32", dict(d=40, V=100), 0.02),
          ("small_bf16", dict(d=136, V=777), 0.02), ("small_bf16", dict(d=520, V=4099), 0.02),
          ("small_bf16", dict(d=136, V=777), 0.0), ("small_bf16", dict(d=520, V=4099), 0.0)]


@pytest.mark.parametrize("name,kw,ent", RAGGED)
def test_pg_loss_parity_ragged_shapes(name, kw, ent):
    base = WL.get_config(name) if name == "tiny_fp32" else WL.scaled_config(name)
    cfg = base.with_(name=f"{base.name}_d{kw['d']}_V{kw['V']}", w_std=1.0 / np.sqrt(kw["d"]), **kw)
    inst = build_instance(cfg)
    p = params_for(cfg, entropy_coef=ent, chunk_rows=256)
    log(f"pg_loss ragged {cfg.name} N={inst['st'].N}")
    compare_full(inst, run_gpu(inst, p), run_oracle(inst, p), p, tag="ragged")
    # the log-prob forward alone on the same shapes
    import torch

    ws = rlk.alloc_workspace(rlk.workspace_size(rlk.make_batch(inst["h"], inst["W"], inst["cu"])), "cuda")
    logp = torch.empty(inst["st"].N, dtype=torch.float32, device="cuda")
    rlk.logprob_fwd(inst["h"], inst["W"], inst["targets"], inst["mask"], inst["cu"], logp=logp, ws=ws)
    torch.cuda.synchronize()
    ref = run_oracle(inst, p, grads=False)
    err = float(np.abs(logp.cpu().numpy()[ref["idx"]] - ref["logp"]).max())
    assert err <= TOL_LOGP[cfg.dtype], err


# Split K: with d = 256 and V = 4096 the dhidden and dW GEMMs have fewer than 128 output tiles, so
# both split K and reduce fp32 partials.  Several chunks exercise the dW accumulation across
# chunks.  accumulate_dW adds the gradient to a preset dW (expected: preset + oracle gradient).
def test_split_k_accumulates_into_preset_dw():
    import torch

    cfg = WL.get_config("tiny_fp32")
    inst = build_instance(cfg)
    p = params_for(cfg, chunk_rows=256)
    ref = run_oracle(inst, p)
    compare_full(inst, run_gpu(inst, p), ref, p, tag="split-k")
    g = torch.Generator(device="cuda").manual_seed(11)
    dW0 = torch.randn(inst["W"].shape, generator=g, device="cuda", dtype=torch.float32)
    pa = params_for(cfg, chunk_rows=256, accumulate_dW=True)
    out = run_gpu(inst, pa, dW=dW0.clone())
    expect = to_host(dW0).astype(np.float64) + ref["dW"]
    err = float(np.abs(to_host(out["dW"]) - expect).max())
    scale = float(np.abs(ref["dW"]).max())
    log(f"split-K accumulate: max |dW - (dW0 + ref)| = {err:.3g} (ref max {scale:.3g})")
    assert err <= 2e-2 * scale + 1e-6


# Degenerate vocabulary: with V = 1 every policy token has log-prob 0, entropy 0 and a zero
# logit gradient, so dhidden and dW are 0 (one valid row in a 256-row tile); the GPU reaches
# them up to the fp32 rounding of exp2 / log at z = max.
@pytest.mark.parametrize("name,d,ent", [("tiny_fp32", 64, 0.02), ("small_bf16", 128, 0.02), ("small_bf16", 128, 0.0)])
def test_pg_loss_single_entry_vocabulary(name, d, ent):
    base = WL.get_config(name) if name == "tiny_fp32" else WL.scaled_config(name)
    cfg = base.with_(name=f"{base.name}_V1", d=d, V=1, w_std=1.0 / np.sqrt(d))
    inst = build_instance(cfg)
    p = params_for(cfg, entropy_coef=ent)
    gpu = run_gpu(inst, p)
    compare_full(inst, gpu, run_oracle(inst, p), p, tag="V=1")
    assert float(gpu["logp"].abs().max()) <= 1e-6 and float(gpu["ent"].abs().max()) <= 1e-6
    assert float(gpu["dh"].float().abs().max()) <= 1e-6 and float(gpu["dW"].abs().max()) <= 1e-6


# The largest batch the library accepts in rollouts: 16,384 rollouts (2,048 groups of 8) of 8
# tokens each, many of them with no policy token at all.
def test_pg_loss_maximum_rollout_count():
    base = WL.get_config("tiny_fp32")
    cfg = base.with_(name="tiny_fp32_R16384", groups=2048, rollouts_per_group=8, len_min=8, len_max=8, d=64,
                     V=512, w_std=1.0 / 8.0, tool_mean=2.0)
    inst = build_instance(cfg)
    assert inst["st"].group_ids.shape[0] == 16384   # the documented maximum R
    p = params_for(cfg, entropy_coef=0.01)
    log(f"pg_loss max rollouts R={cfg.R} N={inst['st'].N}")
    compare_full(inst, run_gpu(inst, p), run_oracle(inst, p), p, tag="max R")


# Sampling temperature: logits z = W h / tau in the forward and the gradients.
@pytest.mark.parametrize("name,scaled,tau,ent", [("tiny_fp32", False, 0.7, 0.02), ("small_bf16", True, 1.3, 0.02),
                                                  ("small_bf16", True, 0.6, 0.0)])
def test_pg_loss_temperature_parity(name, scaled, tau, ent):
    import torch

    cfg = WL.scaled_config(name) if scaled else WL.get_config(name)
    inst = build_instance(cfg)
    p = params_for(cfg, entropy_coef=ent, chunk_rows=256 if scaled else 0)
    log(f"pg_loss temperature {tau} {cfg.name} N={inst['st'].N}")
    compare_full(inst, run_gpu(inst, p, temperature=tau), run_oracle(inst, p, temperature=tau), p, tag=f"tau={tau}")
    logp, ent, lse, ws = rlk.logprob_fwd(inst["h"], inst["W"], inst["targets"], inst["mask"], inst["cu"],
                                         entropy=torch.empty(inst["st"].N, device="cuda"),
                                         lse=torch.empty(inst["st"].N, device="cuda"), temperature=tau)
    torch.cuda.synchronize()
    idx = O.compact(inst["st"].mask, inst["st"].cu_seqlens)[0]
    rl, rp, rH = O.token_logprob(to_host(inst["h"])[idx], to_host(inst["W"]), inst["st"].targets[idx], temperature=tau)
    tol = TOL_LOGP[cfg.dtype]
    assert np.abs(logp.cpu().numpy()[idx] - rp).max() <= tol and np.abs(ent.cpu().numpy()[idx] - rH).max() <= tol


# Token-reference layout (bf16 without an entropy term): the stored probabilities are taken against
# each token's target logit, dz = diag(s) q is applied inside the GEMMs and no chunk needs the
# explicit dz pass.  One token whose hidden row is scaled by 64 (exact in bf16) and whose target is
# its smallest logit (log-prob near -700, far beyond the 40-nat span) sends exactly its own chunk to
# the explicit pass; its old log-prob is set next to the new one so that its gradient is not zero.
def test_token_reference_layout_and_its_fallback():
    cfg = WL.scaled_config("qwen8b_bf16")
    inst = build_instance(cfg)
    p = params_for(cfg, chunk_rows=256)
    gpu = run_gpu(inst, p)
    compare_full(inst, gpu, run_oracle(inst, p), p, tag="ref layout")
    assert gpu["stats"]["n_chunks"] >= 3 and gpu["stats"]["n_dz_chunks"] == 0

    st = inst["st"]
    idx = O.compact(st.mask, st.cu_seqlens, st.group_ids)[0]
    t = int(idx[len(idx) // 2])
    inst2, lp = with_far_target(inst, t)
    assert lp < -100.0, lp
    log(f"fallback token {t} (chunk {int(np.searchsorted(idx, t)) // 256}): log-prob {lp:.1f}")
    gpu2 = run_gpu(inst2, p)
    compare_full(inst2, gpu2, run_oracle(inst2, p), p, tag="ref fallback")
    assert gpu2["stats"]["n_dz_chunks"] == 1

    # the scale bound: a normaliser of 1e24 puts g_t near 1e-26 and the row scales s_t = -g_t p_y
    # below 1e-30 (fp32 denormals once multiplied), so those chunks form dz explicitly as well
    p3 = params_for(cfg, chunk_rows=256, norm_override=1e24)
    gpu3 = run_gpu(inst, p3)
    compare_full(inst, gpu3, run_oracle(inst, p3), p3, tag="ref tiny scales")
    assert gpu3["stats"]["n_dz_chunks"] >= 1


# The dhidden GEMM's partial last wave of 256 tiles, split over K in a second launch (chunk rows known
# from the bound): d = 1024 (4 tile columns), V = 4096 and 20,610 trained tokens in one chunk give 81
# tile rows, 324 tiles and a 68-tile tail (17 tile rows), split 7 ways.  Parity with and without the
# bound (without it the chunk is one launch).
def test_dhidden_tail_split_over_k():
    base = WL.scaled_config("small_bf16")
    cfg = base.with_(name="small_bf16_d1024_V4096", groups=4, rollouts_per_group=8, len_min=1024, len_max=1024,
                     d=1024, V=4096, w_std=1.0 / 32.0)
    inst = build_instance(cfg)
    st = inst["st"]
    n_eff = int(O.compact(st.mask, st.cu_seqlens, st.group_ids)[0].shape[0])
    assert 256 * 64 < n_eff <= 65536 and (n_eff + 255) // 256 * 4 % 256 > 0
    p = params_for(cfg)
    ref = run_oracle(inst, p)
    for bound in (n_eff, 0):
        log(f"dhidden tail split: N_eff={n_eff} bound={bound}")
        gpu = run_gpu(inst, p, max_policy_tokens=bound)
        compare_full(inst, gpu, ref, p, tag=f"dh tail bound={bound}")


# Zero-advantage rollouts (Sec. 2.3.2: every rollout of an all-equal group has advantage 0): with the
# surrogate as the only term their tokens get the forward but skip the backward GEMMs; log-probs and
# entropies are still written for them, their dhidden rows are exactly 0, and a batch where no token
# carries a gradient overwrites dW with zeros (or leaves an accumulated dW as it was).
def test_zero_advantage_rollouts_skip_the_backward():
    import torch

    cfg = WL.scaled_config("qwen8b_bf16")
    inst = build_instance(cfg)
    st = inst["st"]
    gid = st.group_ids
    g0 = gid[gid >= 0][0]
    rewards = st.rewards.copy()
    rewards[gid == g0] = 1.0                       # one all-equal group
    inst1 = dict(inst, rewards=torch.as_tensor(rewards, device="cuda"),
                 st=__import__("dataclasses").replace(st, rewards=rewards))
    p = params_for(cfg, chunk_rows=256)
    gpu = run_gpu(inst1, p)
    ref = run_oracle(inst1, p)
    compare_full(inst1, gpu, ref, p, tag="zero-advantage group")
    zero_rows = ref["idx"][ref["adv_tok"] == 0]
    assert zero_rows.size > 0 and gpu["stats"]["n_grad_tokens"] == ref["idx"].size - zero_rows.size
    rows_t = torch.as_tensor(zero_rows, device="cuda")
    assert float(gpu["dh"][rows_t].float().abs().max()) == 0.0
    assert float(gpu["logp"][rows_t].abs().min()) > 0.0
    # the same batch with an entropy term: no skipping
    pe = params_for(cfg, chunk_rows=256, entropy_coef=0.01)
    ge = run_gpu(inst1, pe)
    assert ge["stats"]["n_grad_tokens"] == ref["idx"].size

    # every group all-equal: nothing carries a gradient
    rewards_all = np.full_like(st.rewards, 0.25)
    inst2 = dict(inst, rewards=torch.as_tensor(rewards_all, device="cuda"),
                 st=__import__("dataclasses").replace(st, rewards=rewards_all))
    g2 = run_gpu(inst2, p)
    ref2 = run_oracle(inst2, p)
    compare_full(inst2, g2, ref2, p, tag="all groups equal")
    assert g2["stats"]["n_grad_tokens"] == 0 and g2["loss"] == 0.0
    assert float(g2["dW"].abs().max()) == 0.0 and float(g2["dh"].float().abs().max()) == 0.0
    dW0 = torch.randn(inst["W"].shape, device="cuda", dtype=torch.float32)
    g3 = run_gpu(inst2, params_for(cfg, chunk_rows=256, accumulate_dW=True), dW=dW0.clone())
    assert torch.equal(g3["dW"], dW0)


# The host hint of gradient-carrying tokens (groups of unequal rewards) only plans the chunk loop:
# chunks over the first grad_tokens compacted rows, then over the rest.  Exact, too small, too large
# and out-of-range hints, and a hint the loss cannot use (an entropy term), all give the oracle's
# results; the exact hint puts the boundary at N_grad.
def test_grad_token_hint_only_plans_the_chunks():
    import torch

    base = WL.scaled_config("small_bf16")
    cfg = base.with_(name="small_bf16_d1024_V4096", groups=4, rollouts_per_group=8, len_min=512, len_max=1024,
                     d=1024, V=4096, w_std=1.0 / 32.0)
    inst = build_instance(cfg)
    st = inst["st"]
    gid = st.group_ids
    rewards = st.rewards.copy()
    live = np.unique(gid[gid >= 0])
    for g in live[1::2]:
        rewards[gid == g] = 1.0                    # every other group all-equal
    st1 = __import__("dataclasses").replace(st, rewards=rewards)
    inst1 = dict(inst, rewards=torch.as_tensor(rewards, device="cuda"), st=st1)
    n_eff = int(O.compact(st.mask, st.cu_seqlens, st.group_ids)[0].shape[0])
    G = rlk.grad_token_hint(st.mask, st.cu_seqlens, rewards, gid)
    assert 0 < G < n_eff
    p0 = params_for(cfg, chunk_rows=4096)
    ref = run_oracle(inst1, p0)
    assert G == expected_grad_tokens(ref, p0, False)
    for hint in (G, G // 3, min(G + 3000, n_eff - 1), 1, n_eff - 1, n_eff, 10 * n_eff):
        p = params_for(cfg, chunk_rows=4096, grad_tokens=hint)
        log(f"grad-token hint {hint} (N_grad={G}, N_eff={n_eff})")
        gpu = run_gpu(inst1, p, max_policy_tokens=n_eff)
        compare_full(inst1, gpu, ref, p, tag=f"grad hint {hint}")
    # without the policy-token bound the hint is not used
    p = params_for(cfg, chunk_rows=4096, grad_tokens=G)
    compare_full(inst1, run_gpu(inst1, p), ref, p, tag="grad hint without a bound")
    pe = params_for(cfg, chunk_rows=4096, entropy_coef=0.01, grad_tokens=G)
    gpu = run_gpu(inst1, pe, max_policy_tokens=n_eff)
    compare_full(inst1, gpu, run_oracle(inst1, pe), pe, tag="grad hint with an entropy term")


# Truncated importance sampling scales the surrogate by a constant weight, so a zero-advantage rollout
# still has an exactly zero gradient and skips the backward; in both aggregation modes the loss
# normalisers still count its tokens.
@pytest.mark.parametrize("agg", [rlk.AGG_SEQ, rlk.AGG_TOKEN])
def test_tis_alone_keeps_the_zero_advantage_skip(agg):
    import torch

    cfg = WL.scaled_config("qwen8b_bf16")
    inst = build_instance(cfg)
    st = inst["st"]
    gid = st.group_ids
    rewards = st.rewards.copy()
    rewards[gid == gid[gid >= 0][-1]] = 0.0        # one all-equal group
    inst1 = dict(inst, rewards=torch.as_tensor(rewards, device="cuda"),
                 st=__import__("dataclasses").replace(st, rewards=rewards))
    aux = aux_logps(inst1)
    p = params_for(cfg, agg=agg, tis_cap=1.1, chunk_rows=256)
    gpu = run_gpu(inst1, p, aux=aux)
    ref = run_oracle(inst1, p, aux=aux)
    assert 0 < np.mean(ref["tis"] == np.float64(p.tis_cap)) < 1
    assert np.count_nonzero(ref["adv_tok"] == 0) > 0
    compare_full(inst1, gpu, ref, p, tag=f"tis, zero-advantage group, agg {agg}")
