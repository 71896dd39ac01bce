"""A tree-packed batch through the GPU loss: rlk_tree_pack's rows (hidden state gathered at the
predicting position, forks giving one row per continuation) feed rlk_pg_loss_fwd_bwd, checked
against the fp64 oracle on the same rows."""
import numpy as np
import pytest

from gpu_common import TOL_LOSS, O, ensure_library, log, loss_error, loss_scale, rel_fro, rlk

pytestmark = pytest.mark.gpu


def _calls(rng, V, n_calls):
    calls, ctx = [], list(rng.integers(0, V, size=int(rng.integers(8, 40))))
    for _ in range(n_calls):
        u = rng.random()
        if calls and u < 0.15:
            x, y = calls[-1][0], list(rng.integers(0, V, size=int(rng.integers(3, 20))))      # retry
        elif calls and u < 0.3:
            x = ctx[:int(rng.integers(1, len(ctx)))] + list(rng.integers(0, V, size=8))       # compaction
            y = list(rng.integers(0, V, size=int(rng.integers(3, 30))))
        else:
            x = ctx + list(rng.integers(0, V, size=int(rng.integers(0, 30))))               # tool output
            y = list(rng.integers(0, V, size=int(rng.integers(3, 30))))
        calls.append(([int(t) for t in x], [int(t) for t in y]))
        ctx = calls[-1][0] + calls[-1][1]
    return calls


def test_tree_packed_batch_loss_parity():
    import torch

    ensure_library()
    rng = np.random.default_rng(11)
    d, V, R = 256, 4096, 6
    rolls = [_calls(rng, V, int(rng.integers(3, 10))) for _ in range(R)]
    pk = rlk.tree_pack(rolls)
    want = O.tree_pack(rolls)
    for k in want:
        np.testing.assert_array_equal(pk[k], want[k])
    n_pos, n_rows = len(pk["token"]), len(pk["row_src"])
    g = torch.Generator(device="cuda").manual_seed(12)
    h_pos = torch.randn(n_pos, d, generator=g, device="cuda")            # the trunk's hidden states
    W = torch.randn(V, d, generator=g, device="cuda") * 0.25
    src = torch.as_tensor(pk["row_src"].astype(np.int64), device="cuda")
    hidden = h_pos[src].contiguous()                                      # one row per prediction
    targets = torch.as_tensor(pk["row_target"], device="cuda")
    mask = torch.as_tensor(pk["row_mask"], device="cuda")
    cu = torch.as_tensor(pk["row_cu"], device="cuda")
    rewards = torch.as_tensor(rng.random(R).astype(np.float32), device="cuda")
    gid = torch.as_tensor(np.array([5, 5, 5, 9, 9, 9], np.int32), device="cuda")
    lse, lp, H = O.token_logprob(hidden.cpu().numpy(), W.cpu().numpy(), pk["row_target"])
    old_host = (lp + rng.standard_normal(n_rows) * 0.1).astype(np.float32)
    old = torch.as_tensor(old_host, device="cuda")
    p = rlk.make_params(eps_low=0.2, eps_high=0.28)
    loss, dh, dW, ws = rlk.pg_loss_fwd_bwd(hidden, W, targets, mask, cu, old, rewards, gid, p)
    torch.cuda.synchronize()
    ref = O.pg_loss_fwd_bwd(hidden.cpu().numpy(), W.cpu().numpy(), pk["row_target"], pk["row_mask"], pk["row_cu"],
                            old_host, rewards.cpu().numpy(), gid.cpu().numpy(), eps_low=0.2, eps_high=0.28)
    e_loss = loss_error(float(loss.item()), ref["loss"], loss_scale(ref, p))
    # fp32 batch: also within 1e-5 of the L1 size of the loss terms
    e_loss_l1 = abs(float(loss.item()) - ref["loss"]) / max(1e-30, loss_scale(ref, p))
    e_dh, e_dW = rel_fro(dh.cpu().numpy(), ref["dh"]), rel_fro(dW.cpu().numpy(), ref["dW"])
    log(f"tree batch: {R} rollouts, {n_pos} positions, {n_rows} rows ({int(pk['row_mask'].sum())} trainable), "
        f"leaves {pk['leaves'].tolist()}; loss err {e_loss:.2e}, dh {e_dh:.2e}, dW {e_dW:.2e}")
    assert rlk.check_status(ws) == 0
    assert e_loss <= TOL_LOSS and e_loss_l1 <= 1e-5 and e_dh <= 1e-4 and e_dW <= 1e-4
    assert max(pk["leaves"]) >= 2       # the batch does contain forks
