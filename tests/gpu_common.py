"""Shared helpers of the GPU parity tests: seeded instances on the device, the call into the
HIP library through the C ABI, and the comparison metrics.  Expected values always come
from the fp64 oracle run on host copies of exactly the bytes the GPU consumed."""
from __future__ import annotations

import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle as O  # noqa: E402
import paper_2608_16798_amd as rlk  # noqa: E402
import workloads as WL  # noqa: E402
from workloads.anchor import gaussian_anchor  # noqa: E402

# Tolerances (per-token log-prob: abs; loss: relative to the L1 size of its terms; gradients:
# relative Frobenius).  fp32 configurations use the tighter log-prob bound.
TOL_LOGP = {"f32": 1e-4, "bf16": 3e-2}
TOL_LOSS = 1e-3
# A loss below this fraction of the L1 size of its terms is a cancellation of signed advantages;
# there the relative bound is taken against that fraction of the L1 size instead of |loss|.
LOSS_CANCEL_FRAC = 1e-2
TOL_GRAD = 2e-2


def log(*a):
    print(*a, flush=True)


def ensure_library():
    if not os.path.exists(rlk.LIB_PATH):
        from paper_2608_16798_amd.build import build

        build(verbose=False)
    return rlk.load_library()


def to_host(t):
    import torch

    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy()
    return t.cpu().numpy()


def build_instance(cfg, device="cuda", structure=None):
    """Seeded instance of a configuration on the device, plus host copies for the oracle."""
    import torch

    st = structure if structure is not None else WL.make_structure(cfg)
    h, W = WL.make_tensors(cfg, st.N, device=device)
    if cfg.anchor == "oracle":
        _, anchor, _ = O.token_logprob(to_host(h), to_host(W), st.targets)
    else:
        anchor = gaussian_anchor(h, W, st.targets, cfg.w_std)
    old = WL.old_logp_from_anchor(anchor, st)
    dev = lambda a, dt: torch.as_tensor(a, dtype=dt, device=device)
    inst = dict(
        cfg=cfg, st=st, h=h, W=W,
        cu=dev(st.cu_seqlens, torch.int32), mask=dev(st.mask, torch.uint8),
        targets=dev(st.targets, torch.int32), rewards=dev(st.rewards, torch.float32),
        gid=dev(st.group_ids, torch.int32), old=dev(old, torch.float32), old_host=old)
    return inst


def params_for(cfg, **kw):
    base = dict(eps_low=cfg.eps_low, eps_high=cfg.eps_high, entropy_coef=cfg.entropy_coef)
    base.update(kw)
    return rlk.make_params(**base)


def aux_logps(inst, *, rollout_sigma=0.15, ref_sigma=0.3):
    """Seeded rollout / reference log-probs of the instance's sampled tokens (host and device)."""
    import torch

    st = inst["st"]
    seed = inst["cfg"].seed
    ro = WL.perturbed_logps(inst["old_host"], st, rollout_sigma, seed + 7001)
    rf = WL.perturbed_logps(inst["old_host"], st, ref_sigma, seed + 7002)
    dev = inst["h"].device
    return dict(rollout_host=ro, ref_host=rf, rollout=torch.as_tensor(ro, device=dev),
                ref=torch.as_tensor(rf, device=dev))


def run_gpu(inst, params, *, gid=None, mask="default", dW=None, ws=None, aux=None, token_adv=None, temperature=1.0,
            max_policy_tokens=0):
    import torch

    h, W = inst["h"], inst["W"]
    N = h.shape[0]
    logp = torch.empty(N, dtype=torch.float32, device=h.device)
    ent = torch.empty(N, dtype=torch.float32, device=h.device)
    stats = rlk.stats_buffer(h.device)
    loss, dh, dWo, ws = rlk.pg_loss_fwd_bwd(
        h, W, inst["targets"], inst["mask"] if mask == "default" else mask, inst["cu"], inst["old"],
        inst["rewards"], inst["gid"] if gid is None else gid, params, dW=dW, logp_out=logp, entropy_out=ent,
        stats=stats, ws=ws, rollout_logp=aux["rollout"] if aux else None, ref_logp=aux["ref"] if aux else None,
        token_adv=token_adv, temperature=temperature, max_policy_tokens=max_policy_tokens)
    torch.cuda.synchronize()
    flags = rlk.check_status(ws)
    return dict(loss=float(loss.item()), dh=dh, dW=dWo, logp=logp, ent=ent, stats=rlk.stats_from_tensor(stats),
                flags=flags, ws=ws, token_adv=token_adv is not None)


def run_oracle(inst, params, *, grads=True, aux=None, token_adv=None, temperature=1.0):
    st = inst["st"]
    extra = {} if token_adv is None else dict(token_adv=token_adv)
    if aux is not None and params.tis_cap > 0:
        extra.update(rollout_logp=aux["rollout_host"], tis_cap=params.tis_cap)
    if aux is not None and params.kl_coef > 0:
        extra.update(ref_logp=aux["ref_host"], kl_coef=params.kl_coef)
    return O.pg_loss_fwd_bwd(
        to_host(inst["h"]), to_host(inst["W"]), st.targets, st.mask, st.cu_seqlens, inst["old_host"],
        st.rewards, st.group_ids, eps_low=params.eps_low, eps_high=params.eps_high, adv_eps=params.adv_eps,
        entropy_coef=params.entropy_coef, agg=params.agg,
        norm_override=params.norm_override if params.norm_override > 0 else None, temperature=temperature,
        grads=grads, **extra)


def rel_fro(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (nb if nb > 0 else 1.0))


def loss_scale(ref, params):
    """L1 size of the loss terms: sum_t |omega_t w_t (s_t + c H_t - beta KL_t)|."""
    A = ref["adv_tok"]
    rho = ref["rho"]
    c = np.clip(rho, 1 - params.eps_low, 1 + params.eps_high)
    sv = np.minimum(rho * A, c * A) + params.entropy_coef * ref["H"] - params.kl_coef * ref["kl"]
    return float(np.abs(ref["omega"] * ref["tis"] * sv).sum())


def loss_error(loss_gpu, loss_ref, scale):
    """Error of the loss against the oracle, relative to |loss_ref| (the stated 1e-3 relative
    tolerance); in the cancellation case |loss_ref| < LOSS_CANCEL_FRAC * scale (scale = L1 size of
    the loss terms) the denominator is LOSS_CANCEL_FRAC * scale, so the bound stays continuous and
    never looser than 1e-3 * 1e-2 of the L1 size."""
    denom = max(abs(loss_ref), LOSS_CANCEL_FRAC * scale)
    if denom == 0.0:
        return abs(loss_gpu)
    return abs(loss_gpu - loss_ref) / denom


def compare_full(inst, gpu, ref, params, tag=""):
    """Element-wise parity of every output against the oracle; returns the metrics."""
    cfg = inst["cfg"]
    idx = ref["idx"]
    N = inst["h"].shape[0]
    keep = np.zeros(N, dtype=bool)
    keep[idx] = True
    logp = gpu["logp"].cpu().numpy()
    ent = gpu["ent"].cpu().numpy()
    m = {}
    m["logp_abs"] = float(np.abs(logp[idx] - ref["logp"]).max()) if idx.size else 0.0
    m["ent_abs"] = float(np.abs(ent[idx] - ref["H"]).max()) if idx.size else 0.0
    m["masked_nonzero"] = int((logp[~keep] != 0).sum() + (ent[~keep] != 0).sum())
    scale = loss_scale(ref, params)
    m["loss_gpu"], m["loss_ref"] = gpu["loss"], ref["loss"]
    m["loss_rel_l1"] = abs(gpu["loss"] - ref["loss"]) / max(scale, 1e-30) if scale > 0 else abs(gpu["loss"])
    m["loss_rel"] = abs(gpu["loss"] - ref["loss"]) / max(abs(ref["loss"]), 1e-30)
    m["loss_err"] = loss_error(gpu["loss"], ref["loss"], scale)
    dh = to_host(gpu["dh"])
    m["dh_rel"] = rel_fro(dh[idx], ref["dh"][idx])
    m["dh_masked_nonzero"] = int(np.count_nonzero(dh[~keep]))
    m["dW_rel"] = rel_fro(to_host(gpu["dW"]), ref["dW"])
    st = gpu["stats"]
    m["stats_ok"] = (st["n_policy_tokens"] == ref["stats"]["n_policy_tokens"]
                     and st["n_groups"] == ref["stats"]["n_groups"]
                     and st["n_valid_rollouts"] == ref["stats"]["n_valid_rollouts"])
    m["kl_mean_err"] = abs(st["kl_mean"] - ref["stats"]["kl_mean"]) / max(1.0, abs(ref["stats"]["kl_mean"]))
    m["tis_mean_err"] = abs(st["tis_mean"] - ref["stats"]["tis_mean"])
    m["flags"] = gpu["flags"]
    m["dz_chunks"] = f"{st['n_dz_chunks']}/{st['n_chunks']}"
    log(f"[{tag}] {cfg.name}: " + ", ".join(f"{k}={v:.3g}" if isinstance(v, float) else f"{k}={v}"
                                            for k, v in m.items()))
    tl = TOL_LOGP[cfg.dtype]
    assert m["flags"] == 0
    assert m["logp_abs"] <= tl and m["ent_abs"] <= tl
    assert m["masked_nonzero"] == 0 and m["dh_masked_nonzero"] == 0
    assert m["loss_err"] <= TOL_LOSS
    assert m["dh_rel"] <= TOL_GRAD and m["dW_rel"] <= TOL_GRAD
    assert m["stats_ok"]
    assert m["kl_mean_err"] <= 1e-3 and m["tis_mean_err"] <= 1e-4
    # the explicit dz pass runs for every chunk unless the token-reference layout applies (bf16
    # without an entropy term), where it runs only for the chunks flagged on the device
    assert st["n_chunks"] >= 1 and 0 <= st["n_dz_chunks"] <= st["n_chunks"]
    if not ref_layout(cfg, params):
        assert st["n_dz_chunks"] == st["n_chunks"]
    # the backward covers the tokens with a surrogate gradient: without an entropy term, a KL term or
    # per-token advantages, those of rollouts with a non-zero advantage
    assert st["n_grad_tokens"] == expected_grad_tokens(ref, params, gpu.get("token_adv", False))
    return m


def expected_grad_tokens(ref, params, token_adv):
    if params.entropy_coef == 0.0 and params.kl_coef == 0.0 and not token_adv:
        return int(np.count_nonzero(ref["adv_tok"]))
    return int(ref["idx"].shape[0])


def ref_layout(cfg, params):
    """Whether a fwd+bwd call of this configuration stores q against the target logits."""
    return cfg.dtype == "bf16" and params.entropy_coef == 0.0


def with_far_target(inst, t):
    """The instance with token t's hidden row scaled by 64 (exact in bf16) and its target set to its
    smallest logit, so that its log-prob is far below -40 (about -700 at the qwen8b shape), and its
    old log-prob set next to the new one so that its gradient is not zero.  Returns (instance, logp)."""
    import dataclasses

    import torch

    st = inst["st"]
    h = inst["h"].clone()
    h[t] *= 64
    W64 = to_host(inst["W"]).astype(np.float64)
    y = int(np.argmin(W64 @ to_host(h[t]).astype(np.float64)))
    targets = st.targets.copy()
    targets[t] = y
    lp = float(O.token_logprob(to_host(h[t:t + 1]), to_host(inst["W"]), np.array([y]))[1][0])
    old = inst["old_host"].copy()
    old[t] = lp + 0.05
    dev = h.device
    out = dict(inst, st=dataclasses.replace(st, targets=targets), h=h,
               targets=torch.as_tensor(targets, dtype=torch.int32, device=dev),
               old=torch.as_tensor(old, dtype=torch.float32, device=dev), old_host=old)
    return out, lp
