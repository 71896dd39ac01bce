"""Plain fp64 reference of the per-token policy-gradient computation.

TEST INFRASTRUCTURE ONLY: imported by tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py, never by the product path.  It shares no code
with the HIP library.

Every quantity is evaluated from its definition in float64 with complete
vocabulary rows of logits (no online/streaming softmax).  Rows of tokens are
processed in blocks purely to bound memory; rows are independent.

Passages followed (ClawGym II):
  * Sec. 2.3.1, masked clipped PPO objective: token ratio
    rho_t = pi_theta(a_t|s_t) / pi_old(a_t|s_t), binary mask M_t (1 for valid
    policy-generated tokens), min(rho A, clip(rho, 1-eps, 1+eps) A).
  * Sec. 2.3.2, GRPO: A_i = (R_i - mu_q) / (sigma_q + eps) with the population
    (1/G) standard deviation; objective = 1/G sum over trajectories of the
    masked token mean of the clipped surrogate.
  * Sec. 3.2.3, tree GRPO: the group is the n rollouts of a task; the rollout's
    advantage goes to each of its trainable tokens, shared-prefix tokens once.
  * Sec. 3.2.4: pi_old is a separate forward pass of the trainer (the log-prob
    forward computed here).
  * Sec. 3.3: under mix-harness training a group is a task-harness pair.
  * Sec. 3.4: rollouts with sandbox failures leave both advantage estimation
    and policy optimization.

Readings where the paper is silent (each one is stated where it is applied):
  * loss = - objective (the equations are objectives to maximise);
  * default aggregation "seq": per-rollout masked token mean, 1/G_q within a
    group, then the mean over the Q groups of the batch; alternative "token":
    one masked token mean over the batch (the hat-E_t form of the PPO equation);
  * advantage eps defaults to 1e-6; a group whose rewards are all bitwise equal
    gets advantage exactly 0 (so does a group of one);
  * asymmetric clip range [1 - eps_low, 1 + eps_high]; at rho exactly on a clip
    bound the gradient passes (clipped only on strict inequality);
  * optional entropy bonus: objective += c_ent * H_t under the same mask and
    aggregation, H_t the full-vocabulary Shannon entropy in nats;
  * the KL term of the GRPO objective (Sec. 2.3.2) is optional (beta = 0 by
    default); when on, D_KL(pi_theta || pi_ref) at a sampled token is the
    estimator r/p - log(r/p) - 1 of the GRPO work the paper builds on, from the
    reference policy's log-prob of the sampled token (no second LM head);
  * PPO (Sec. 2.3.1, simplified per Sec. 3.2.3): GAE runs over a rollout's policy
    tokens in order (tool tokens stepped over), the terminal reward arriving at the
    last policy token; a packed rollout is one trajectory; the value loss is the
    token mean of (V - G)^2 over policy tokens, G = A + V; when the critic shares the
    policy's trunk, V_t = w_v . h_t + b_v is a linear head on its final hidden state;
  * prefix trees (Sec. 3.2.1): a call attaches to the node whose history is the
    longest prefix of its context; a node identical to a sibling is that sibling;
    packing is depth-first, one training row per non-root position;
  * token-level truncated importance sampling (Sec. 3.2.4) is optional (off by
    default); when on, w_t = min(exp(old_t - rollout_t), c_bar) scales the whole
    loss of token t (surrogate, entropy and KL terms) and is held constant in
    the gradient;
  * a rollout with no policy tokens contributes 0 to its group's sum but still
    counts in G_q and in mu/sigma;
  * group_id < 0 marks an excluded rollout: removed from mu, sigma, G_q, Q and
    the loss; group ids are opaque keys, dense index = rank among the sorted
    distinct non-negative ids;
  * logits z = W h / tau (no bias; tau = 1 unless a sampling temperature is given);
  * norm_override replaces Q (seq) or the policy-token count (token), so
    gradients of separately processed micro-batches add up to the one-call
    gradient;
  * with nothing to train (no policy tokens or every rollout excluded) the
    loss is 0, dhidden is 0 and the overwritten dW is 0.
"""
from __future__ import annotations

import numpy as np

AGG_SEQ = 0
AGG_TOKEN = 1


def _f64(a):
    return np.asarray(a, dtype=np.float64)


# --------------------------------------------------------------------------
# Token compaction and rollout segmentation (Sec. 2.3.1 mask, Sec. 3.2.3
# per-rollout token count, Sec. 3.4 exclusion).
# --------------------------------------------------------------------------
def compact(mask, cu_seqlens, group_ids=None):
    """Ascending positions t with M_t = 1 inside non-excluded rollouts.

    Returns (idx int64 [N_eff], tok_rollout int64 [N_eff], n_pol int64 [R]).
    mask None means every token is a policy token.
    """
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    R = cu.shape[0] - 1
    N = int(cu[-1])
    t = np.arange(N, dtype=np.int64)
    rollout_of = np.searchsorted(cu[1:], t, side="right")
    keep = np.ones(N, dtype=bool) if mask is None else (np.asarray(mask)[:N] != 0)
    if group_ids is not None:
        gid = np.asarray(group_ids, dtype=np.int64)
        keep &= gid[rollout_of] >= 0
    idx = np.flatnonzero(keep).astype(np.int64)
    tok_rollout = rollout_of[idx]
    n_pol = np.bincount(tok_rollout, minlength=R).astype(np.int64)
    return idx, tok_rollout, n_pol


def group_index(group_ids):
    """Dense group index per rollout (-1 if excluded) and the number of groups Q."""
    gid = np.asarray(group_ids, dtype=np.int64)
    valid = gid >= 0
    gi = np.full(gid.shape[0], -1, dtype=np.int64)
    uniq, inv = np.unique(gid[valid], return_inverse=True)
    gi[valid] = inv
    return gi, int(uniq.shape[0])


def group_advantage(rewards, group_ids, adv_eps=1e-6):
    """GRPO advantage per rollout (Sec. 2.3.2 / Sec. 3.2.3), fp64.

    Returns dict(adv [R], group_index [R], n_groups, G [Q], mu [Q], sigma [Q]).
    """
    r = _f64(rewards)
    gi, Q = group_index(group_ids)
    adv = np.zeros(r.shape[0], dtype=np.float64)
    G = np.zeros(Q, dtype=np.int64)
    mu = np.zeros(Q)
    sigma = np.zeros(Q)
    for q in range(Q):
        members = np.flatnonzero(gi == q)
        Rq = r[members]
        n = members.shape[0]
        G[q] = n
        mu[q] = Rq.sum() / n
        sigma[q] = np.sqrt(((Rq - mu[q]) ** 2).sum() / n)
        if Rq.max() == Rq.min():
            adv[members] = 0.0          # all-equal group: exactly 0
        else:
            adv[members] = (Rq - mu[q]) / (sigma[q] + adv_eps)
    return dict(adv=adv, group_index=gi, n_groups=Q, G=G, mu=mu, sigma=sigma)


# --------------------------------------------------------------------------
# Log-prob forward (Sec. 3.2.4) with full-row logits.
# --------------------------------------------------------------------------
def token_logprob(h_rows, W, y, block: int = 256, temperature: float = 1.0):
    """log pi(y_t | s_t), entropy and log-partition per row, from complete logit rows.

    z = W h_t / tau; lse = max z + log sum exp(z - max z); logp = z_y - lse;
    H = -sum_j p_j log p_j with log p_j = z_j - lse.
    """
    W64 = _f64(W)
    y = np.asarray(y, dtype=np.int64)
    n = y.shape[0]
    lse = np.empty(n)
    logp = np.empty(n)
    H = np.empty(n)
    for b0 in range(0, n, block):
        b1 = min(n, b0 + block)
        z = (_f64(h_rows[b0:b1]) @ W64.T) / temperature
        m = z.max(axis=1)
        l = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
        lp = z - l[:, None]
        p = np.exp(lp)
        lse[b0:b1] = l
        logp[b0:b1] = lp[np.arange(b1 - b0), y[b0:b1]]
        H[b0:b1] = -(p * lp).sum(axis=1)
    return lse, logp, H


# --------------------------------------------------------------------------
# Clipped surrogate (Sec. 2.3.1 / 2.3.2) and aggregation weights.
# --------------------------------------------------------------------------
def surrogate(logp, old_logp, adv_tok, eps_low, eps_high):
    """s_t = min(rho A, clip(rho, 1-eps_low, 1+eps_high) A) and the gradient gate.

    Returns (s, rho, clipped) where clipped marks tokens whose surrogate does
    not depend on rho (strict inequality beyond the bound on the side that the
    min selects).
    """
    rho = np.exp(_f64(logp) - _f64(old_logp))
    A = _f64(adv_tok)
    c = np.clip(rho, 1.0 - eps_low, 1.0 + eps_high)
    s = np.minimum(rho * A, c * A)
    clipped = ((A > 0) & (rho > 1.0 + eps_high)) | ((A < 0) & (rho < 1.0 - eps_low))
    return s, rho, clipped


def tis_weight(old_logp, rollout_logp, cap):
    """Sec. 3.2.4, token-level truncated importance-sampling weight:
    w_t = min(exp(log pi_old - log pi_rollout), c_bar)."""
    return np.minimum(np.exp(_f64(old_logp) - _f64(rollout_logp)), float(cap))


def kl_sampled(logp, ref_logp):
    """KL(pi_theta || pi_ref) at a sampled token, the estimator pi_ref/pi - log(pi_ref/pi) - 1
    (GRPO objective, Sec. 2.3.2).  Returns the estimate and its derivative w.r.t. log pi_theta."""
    r = _f64(ref_logp) - _f64(logp)
    return np.expm1(r) - r, -np.expm1(r)


def token_weights(tok_rollout, n_pol, gi, G, n_groups, agg=AGG_SEQ, norm_override=None):
    """d loss / d (s_t + c H_t) per compacted token (negative: loss = -objective).

    seq:   -1 / (Q * G_q * n_r)   (per-rollout token mean, 1/G_q, mean over groups)
    token: -1 / sum_t M_t
    """
    tok_rollout = np.asarray(tok_rollout, dtype=np.int64)
    n = tok_rollout.shape[0]
    if n == 0:
        return np.zeros(0)
    if agg == AGG_SEQ:
        Qn = float(n_groups) if not norm_override else float(norm_override)
        q = gi[tok_rollout]
        return -1.0 / (Qn * G[q].astype(np.float64) * n_pol[tok_rollout].astype(np.float64))
    Mn = float(n) if not norm_override else float(norm_override)
    return np.full(n, -1.0 / Mn)


def _aggregate(val, tok_rollout, n_pol, gi, G, n_groups, R, agg, norm_override):
    """Objective J from per-token values val_t = s_t + c H_t (definitions above)."""
    n = val.shape[0]
    if n == 0 or n_groups == 0:
        return 0.0
    if agg == AGG_SEQ:
        ell = np.zeros(R)
        for r in range(R):
            if gi[r] >= 0 and n_pol[r] > 0:
                ell[r] = val[tok_rollout == r].sum() / n_pol[r]
        J = 0.0
        for q in range(n_groups):
            J += ell[gi == q].sum() / G[q]
        Qn = float(n_groups) if not norm_override else float(norm_override)
        return J / Qn
    Mn = float(n) if not norm_override else float(norm_override)
    return val.sum() / Mn


# --------------------------------------------------------------------------
# Full forward + backward.
# --------------------------------------------------------------------------
def pg_loss_fwd_bwd(h, W, targets, mask, cu_seqlens, old_logp, rewards, group_ids, *,
                    eps_low=0.2, eps_high=0.2, adv_eps=1e-6, entropy_coef=0.0, agg=AGG_SEQ,
                    norm_override=None, rollout_logp=None, tis_cap=None, ref_logp=None, kl_coef=0.0,
                    token_adv=None, temperature=1.0, grads=True, block: int = 128):
    """Loss, per-token outputs and gradients w.r.t. hidden states and the LM-head weight.

    h [N, d], W [V, d] (any float dtype, evaluated in fp64), targets [N], mask [N]
    (None = all policy), cu_seqlens [R+1], old_logp [N], rewards [R], group_ids [R];
    rollout_logp [N] with tis_cap switches on truncated importance sampling, ref_logp [N]
    with kl_coef > 0 the KL term; token_adv [N] (PPO, Sec. 2.3.1) replaces the group advantage
    of each token by a per-token advantage; temperature tau divides the logits (z = W h / tau),
    so the raw-logit gradient is dL/dz / tau.
    """
    h = np.asarray(h)
    W64 = _f64(W)
    N, d = h.shape
    V = W64.shape[0]
    targets = np.asarray(targets, dtype=np.int64)
    old = _f64(old_logp)
    R = np.asarray(cu_seqlens).shape[0] - 1

    idx, tok_r, n_pol = compact(mask, cu_seqlens, group_ids)
    ga = group_advantage(rewards, group_ids, adv_eps)
    adv, gi, Q, G = ga["adv"], ga["group_index"], ga["n_groups"], ga["G"]
    n = idx.shape[0]
    omega = token_weights(tok_r, n_pol, gi, G, Q, agg, norm_override)
    tis = tis_weight(old[idx], _f64(rollout_logp)[idx], tis_cap) if rollout_logp is not None else np.ones(n)
    adv_tok = _f64(token_adv)[idx] if token_adv is not None else adv[tok_r]
    ref = _f64(ref_logp)[idx] if (ref_logp is not None and kl_coef) else None

    lse = np.zeros(n)
    logp = np.zeros(n)
    H = np.zeros(n)
    s = np.zeros(n)
    rho = np.zeros(n)
    clipped = np.zeros(n, dtype=bool)
    kl = np.zeros(n)
    g = np.zeros(n)
    e = np.zeros(n)
    dh = np.zeros((N, d)) if grads else None
    dW = np.zeros((V, d)) if grads else None
    for b0 in range(0, n, block):
        b1 = min(n, b0 + block)
        rows = idx[b0:b1]
        hb = _f64(h[rows])
        z = (hb @ W64.T) / temperature
        m = z.max(axis=1)
        l = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
        lp = z - l[:, None]
        p = np.exp(lp)
        yb = targets[rows]
        ar = np.arange(b1 - b0)
        lse[b0:b1] = l
        logp[b0:b1] = lp[ar, yb]
        H[b0:b1] = -(p * lp).sum(axis=1)
        sb, rb, cb = surrogate(logp[b0:b1], old[rows], adv_tok[b0:b1], eps_low, eps_high)
        s[b0:b1], rho[b0:b1], clipped[b0:b1] = sb, rb, cb
        # chain rule (w = tis weight, constant): dL/dlogp_t = omega_t w_t (A rho_t [not clipped]
        # - beta dKL_t/dlogp_t); dL/dH_t = omega_t w_t c_ent
        dkl = np.zeros(b1 - b0)
        if ref is not None:
            kl[b0:b1], dkl = kl_sampled(logp[b0:b1], ref[b0:b1])
        wb = omega[b0:b1] * tis[b0:b1]
        gb = wb * (adv_tok[b0:b1] * rb * (~cb) - kl_coef * dkl)
        eb = wb * entropy_coef
        g[b0:b1], e[b0:b1] = gb, eb
        if grads:
            onehot = np.zeros_like(z)
            onehot[ar, yb] = 1.0
            # d logp_y / dz_j = [j = y] - p_j ;  d H / dz_j = -p_j (log p_j + H)
            dz = gb[:, None] * (onehot - p) - eb[:, None] * p * (lp + H[b0:b1, None])
            dz /= temperature   # d z / d (W h) = 1 / tau
            dh[rows] = dz @ W64
            dW += dz.T @ hb

    val = tis * (s + entropy_coef * H - kl_coef * kl)
    J = _aggregate(val, tok_r, n_pol, gi, G, Q, R, agg, norm_override)
    Jpg = _aggregate(tis * s, tok_r, n_pol, gi, G, Q, R, agg, norm_override)
    stats = dict(
        loss=-J, pg_loss=-Jpg,
        entropy_mean=float(H.mean()) if n else 0.0,
        clip_frac=float(clipped.mean()) if n else 0.0,
        ratio_mean=float(rho.mean()) if n else 0.0,
        kl_mean=float(kl.mean()) if n else 0.0,
        tis_mean=float(tis.mean()) if n else 0.0,
        n_policy_tokens=int(n), n_groups=int(Q), n_valid_rollouts=int((gi >= 0).sum()))
    logp_full = np.zeros(N)
    H_full = np.zeros(N)
    lse_full = np.zeros(N)
    logp_full[idx] = logp
    H_full[idx] = H
    lse_full[idx] = lse
    return dict(loss=-J, pg_loss=-Jpg, stats=stats, idx=idx, tok_rollout=tok_r, n_pol=n_pol,
                adv=adv, group_index=gi, n_groups=Q, omega=omega, lse=lse, logp=logp, H=H,
                rho=rho, clipped=clipped, kl=kl, tis=tis, adv_tok=adv_tok, g=g, e=e, logp_full=logp_full, entropy_full=H_full,
                lse_full=lse_full, dh=dh, dW=dW)


def sampled_rows(h_rows, W, y_rows, old_rows, adv_rows, omega_rows, *, eps_low, eps_high,
                 entropy_coef=0.0, tis_rows=None, ref_rows=None, kl_coef=0.0, temperature=1.0, block: int = 64):
    """Per-row forward and dhidden for selected policy rows of a large batch.

    A row's log-prob, entropy and dhidden depend only on that row and on
    per-rollout scalars (advantage, aggregation weight), so each can be checked
    exactly without the rest of the batch.
    """
    W64 = _f64(W)
    y = np.asarray(y_rows, dtype=np.int64)
    n = y.shape[0]
    out = {k: np.zeros(n) for k in ("lse", "logp", "H", "rho", "g", "e")}
    out["clipped"] = np.zeros(n, dtype=bool)
    out["dh"] = np.zeros((n, W64.shape[1]))
    for b0 in range(0, n, block):
        b1 = min(n, b0 + block)
        hb = _f64(h_rows[b0:b1])
        z = (hb @ W64.T) / temperature
        m = z.max(axis=1)
        l = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
        lp = z - l[:, None]
        p = np.exp(lp)
        ar = np.arange(b1 - b0)
        lpy = lp[ar, y[b0:b1]]
        Hb = -(p * lp).sum(axis=1)
        A = _f64(adv_rows[b0:b1])
        _, rb, cb = surrogate(lpy, old_rows[b0:b1], A, eps_low, eps_high)
        om = _f64(omega_rows[b0:b1])
        if tis_rows is not None:
            om = om * _f64(tis_rows[b0:b1])
        dkl = kl_sampled(lpy, ref_rows[b0:b1])[1] if (ref_rows is not None and kl_coef) else 0.0
        gb = om * (A * rb * (~cb) - kl_coef * dkl)
        eb = om * entropy_coef
        onehot = np.zeros_like(z)
        onehot[ar, y[b0:b1]] = 1.0
        dz = gb[:, None] * (onehot - p) - eb[:, None] * p * (lp + Hb[:, None])
        out["lse"][b0:b1] = l
        out["logp"][b0:b1] = lpy
        out["H"][b0:b1] = Hb
        out["rho"][b0:b1] = rb
        out["clipped"][b0:b1] = cb
        out["g"][b0:b1] = gb
        out["e"][b0:b1] = eb
        out["dh"][b0:b1] = (dz / temperature) @ W64
    return out


def loss_from_token_values(logp, H, old_logp, adv_tok, tok_rollout, n_pol, gi, G, n_groups, *, eps_low, eps_high,
                           entropy_coef=0.0, agg=AGG_SEQ, norm_override=None):
    """Loss -J (Sec. 2.3.1 / 2.3.2 objectives, readings above) of the compacted policy tokens
    from their log-probs and entropies, for batches too large for a full-logit pass: the
    aggregation of pg_loss_fwd_bwd applied to given per-token values."""
    s, _, _ = surrogate(logp, old_logp, adv_tok, eps_low, eps_high)
    val = s + entropy_coef * _f64(H)
    R = np.asarray(n_pol).shape[0]
    return -_aggregate(val, np.asarray(tok_rollout, dtype=np.int64), np.asarray(n_pol), np.asarray(gi),
                       np.asarray(G), n_groups, R, agg, norm_override)


def token_grad_weights(logp, old_logp, adv_tok, omega, *, eps_low, eps_high, entropy_coef=0.0):
    """Chain-rule weights of the clipped surrogate with the entropy bonus (no importance weight,
    no KL term): g_t = dL/dlogp_t = omega_t A_t rho_t [not clipped], e_t = dL/dH_t = omega_t c_ent,
    omega_t from token_weights."""
    _, rho, clipped = surrogate(logp, old_logp, adv_tok, eps_low, eps_high)
    om = _f64(omega)
    return om * _f64(adv_tok) * rho * (~clipped), om * entropy_coef


def dw_rows(h, W, v_sel, y, logp, H, g, e, block: int = 8192, temperature: float = 1.0):
    """Rows v_sel of dW = sum_t dz_t h_t^T over the compacted policy tokens t, from per-token
    scalars: the log-prob logp_t, entropy H_t and the chain-rule weights g_t = dL/dlogp_t,
    e_t = dL/dH_t.  With z_tv = W_v . h_t / tau, lse_t = z_{t,y_t} - logp_t and p_tv = e^{z_tv - lse_t},
    dz_tv = g_t ([v = y_t] - p_tv) - e_t p_tv (z_tv - lse_t + H_t) (the derivatives noted in
    pg_loss_fwd_bwd; the raw-logit gradient is dz / tau).  h is [n, d], read in row blocks (anything whose slices convert to arrays),
    W is [V, d]; a row's cost is 2 n d per selected v."""
    v_sel = np.asarray(v_sel, dtype=np.int64)
    y = np.asarray(y, dtype=np.int64)
    logp, H, g, e = _f64(logp), _f64(H), _f64(g), _f64(e)
    Wsel = _f64(np.asarray(W)[v_sel])
    n = y.shape[0]
    out = np.zeros((v_sel.shape[0], Wsel.shape[1]))
    for b0 in range(0, n, block):
        b1 = min(n, b0 + block)
        hb = _f64(h[b0:b1])
        yb = y[b0:b1]
        zy = np.einsum("ij,ij->i", hb, _f64(np.asarray(W)[yb])) / temperature
        lse = zy - logp[b0:b1]
        z = (hb @ Wsel.T) / temperature
        p = np.exp(z - lse[:, None])
        dz = -p * (g[b0:b1, None] + e[b0:b1, None] * (z - lse[:, None] + H[b0:b1, None]))
        dz += g[b0:b1, None] * (yb[:, None] == v_sel[None, :])
        out += (dz / temperature).T @ hb
    return out


# --------------------------------------------------------------------------
# PPO path (Sec. 2.3.1 GAE and value loss; Sec. 3.2.3 simplified variant).
# --------------------------------------------------------------------------
def gae(values, rewards, mask, cu_seqlens, group_ids=None, gamma=1.0, lam=1.0):
    """Masked generalised advantage estimation per rollout, and the returns.

    Sec. 2.3.1: A_t = sum_l (gamma lam)^l delta_{t+l} M_{t+l}, delta_t = r_t + gamma V(s_{t+1})
    M_{t+1} - V(s_t); Sec. 3.2.3: the rollout's terminal reward R_i is received at its final
    token.  Reading: the recursion runs over the rollout's policy tokens (M = 1) in order, the
    state after a policy token being the next policy token of the rollout (tool tokens carry no
    value and are stepped over), and the reward arrives at the last policy token; with
    gamma = lam = 1 this gives A_t = R_i - V(s_t), the form Sec. 3.2.3 states.  Returns
    G_t = A_t + V(s_t).  Masked rows and rows of excluded rollouts (group id < 0) are 0.
    """
    V = _f64(values)
    mask = np.asarray(mask).astype(bool)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    R = cu.shape[0] - 1
    gid = np.zeros(R, dtype=np.int64) if group_ids is None else np.asarray(group_ids, dtype=np.int64)
    adv = np.zeros(V.shape[0])
    ret = np.zeros(V.shape[0])
    for r in range(R):
        if gid[r] < 0:
            continue
        pos = [t for t in range(cu[r], cu[r + 1]) if mask[t]]
        a_next, v_next = 0.0, 0.0
        for j in range(len(pos) - 1, -1, -1):
            t = pos[j]
            last = j == len(pos) - 1
            delta = (float(rewards[r]) if last else 0.0) + (0.0 if last else gamma * v_next) - V[t]
            a = delta + gamma * lam * a_next
            adv[t], ret[t] = a, a + V[t]
            a_next, v_next = a, V[t]
    return adv, ret


def value_loss(values, returns, mask, cu_seqlens, group_ids=None):
    """Sec. 2.3.1 masked mean-squared value loss E_t[M_t (V(s_t) - G_t)^2] (token mean over the
    policy tokens of non-excluded rollouts) and its gradient with respect to V."""
    V = _f64(values)
    G = _f64(returns)
    idx, _, _ = compact(mask, cu_seqlens, group_ids)
    dV = np.zeros(V.shape[0])
    if idx.size == 0:
        return 0.0, dV
    diff = V[idx] - G[idx]
    dV[idx] = 2.0 * diff / idx.size
    return float((diff * diff).mean()), dV


def value_head(h, w_v, b_v, mask, cu_seqlens, group_ids=None):
    """Value estimates V(s_t) of the PPO objective (Sec. 2.3.1) from a linear value head on the
    policy's final hidden states (the critic's form is unstated; reading: V_t = w_v . h_t + b_v),
    on the policy tokens of non-excluded rollouts, 0 elsewhere."""
    idx, _, _ = compact(mask, cu_seqlens, group_ids)
    V = np.zeros(np.asarray(h).shape[0])
    if idx.size:
        V[idx] = _f64(np.asarray(h)[idx]) @ _f64(w_v) + float(b_v)
    return V


def value_head_grads(h, w_v, dvalues, mask, cu_seqlens, group_ids=None):
    """Gradients of a loss through value_head given dL/dV (e.g. from value_loss): dL/dh_t =
    dL/dV_t w_v on the rows value_head computes (0 elsewhere), dL/dw_v = sum_t dL/dV_t h_t and
    dL/db_v = sum_t dL/dV_t over those rows."""
    h = np.asarray(h)
    idx, _, _ = compact(mask, cu_seqlens, group_ids)
    dV = _f64(dvalues)
    dh = np.zeros((h.shape[0], h.shape[1]))
    if idx.size == 0:
        return dh, np.zeros(h.shape[1]), 0.0
    dh[idx] = dV[idx, None] * _f64(w_v)[None, :]
    return dh, dV[idx] @ _f64(h[idx]), float(dV[idx].sum())


# --------------------------------------------------------------------------
# Prefix-tree packing of a rollout's model calls (Sec. 3.2.1, used by Sec. 3.2.3).
# --------------------------------------------------------------------------
def tree_pack(calls_per_rollout):
    """Prefix trees of the rollouts' model calls, packed for the trainer.

    calls_per_rollout: list over rollouts of lists of (x, y) token lists, in capture order
    (x = the call's input context, y = the model's response).

    Sec. 3.2.1: the tree is rooted at the initial task prompt, taken to be the first call's
    context (a harness-content node under an empty root); each call attaches to the existing
    node whose accumulated history is the longest prefix of x; the new node holds the
    intervening harness content x[len(history):] (not trainable) followed by y (trainable), and
    its history is x + y.  A context that extends no node's history (not even the prompt)
    attaches to the empty root and starts a separate tree of the rollout.
    Reading: a new node whose content equals that of an existing child of the same parent is
    that child (identical calls collapse, so a shared history is stored once); children keep
    their first-seen order.

    Packing, per rollout: the nodes in depth-first pre-order, each node's tokens in order.
    Every packed position p has parent[p] = the packed position of the previous token on its
    root path (-1 for the first token of a tree) and depth[p] = its index on that path.
    Training rows: one per position with parent >= 0, predicting token[p] from the hidden state
    at parent[p]: row (src = parent[p], target = token[p], mask = 1 if p holds a model-generated
    token).  Shared prefixes therefore yield each trainable token once per rollout (Sec. 3.2.3),
    and a fork yields one row per continuation.

    Returns dict(token, parent, depth, pos_off [R+1], row_src, row_target, row_mask,
    row_cu [R+1], leaves [R]) with positions/rows numbered over the whole batch.
    """
    tok, par, dep, pos_off = [], [], [], [0]
    rsrc, rtgt, rmask, row_cu, leaves = [], [], [], [0], []
    for calls in calls_per_rollout:
        # node: dict(hist=list, content=list, mask=list, children=[node ids])
        nodes = [dict(hist=[], content=[], mask=[], children=[])]
        if calls and len(calls[0][0]) > 0:
            prompt = list(calls[0][0])
            nodes.append(dict(hist=prompt, content=prompt, mask=[0] * len(prompt), children=[]))
            nodes[0]["children"].append(1)
        for x, y in calls:
            x, y = list(x), list(y)
            best, best_len = 0, -1
            for k, n in enumerate(nodes):
                L = len(n["hist"])
                if L <= len(x) and x[:L] == n["hist"] and L > best_len:
                    best, best_len = k, L
            content = x[best_len:] + y
            mask = [0] * (len(x) - best_len) + [1] * len(y)
            same = [c for c in nodes[best]["children"]
                    if nodes[c]["content"] == content and nodes[c]["mask"] == mask]
            if same or not content:
                continue
            nodes.append(dict(hist=x + y, content=content, mask=mask, children=[]))
            nodes[best]["children"].append(len(nodes) - 1)
        base = len(tok)
        nrows = 0

        def emit(k, last_pos, depth):
            nonlocal nrows
            n = nodes[k]
            prev = last_pos
            for t, m in zip(n["content"], n["mask"]):
                p = len(tok)
                tok.append(t)
                par.append(prev)
                dep.append(depth)
                if prev >= 0:
                    rsrc.append(prev)
                    rtgt.append(t)
                    rmask.append(m)
                    nrows += 1
                prev = p
                depth += 1
            for c in n["children"]:
                emit(c, prev, depth)

        emit(0, -1, 0)
        leaves.append(sum(1 for k, n in enumerate(nodes) if k > 0 and not n["children"]))
        pos_off.append(len(tok))
        row_cu.append(row_cu[-1] + nrows)
        assert pos_off[-1] - base >= 0
    i32 = lambda a: np.asarray(a, dtype=np.int32)
    return dict(token=i32(tok), parent=i32(par), depth=i32(dep), pos_off=np.asarray(pos_off, np.int64),
                row_src=i32(rsrc), row_target=i32(rtgt), row_mask=np.asarray(rmask, np.uint8),
                row_cu=i32(row_cu), leaves=i32(leaves))
