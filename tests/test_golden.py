"""The hand-derived worked example (tests/golden/worked_example_clip.json) against the oracle
(CPU) and against the HIP path (GPU, fp32 batch).  The example covers a masked tool token at
each rollout's edge, a two-rollout group with binary rewards, and the three regimes of the
clipped surrogate: on-policy, clipped above with a positive advantage next to an unclipped ratio
with a negative one, and both tokens clipped (zero gradients)."""
from __future__ import annotations

import numpy as np
import pytest

import golden_example as G
import oracle as O

EX = G.load()
CASES = sorted(EX["cases"])


@pytest.mark.parametrize("case", CASES)
def test_oracle_reproduces_the_worked_example(case):
    c = EX["cases"][case]
    r = O.pg_loss_fwd_bwd(EX["h"], EX["W"], EX["targets"], EX["mask"], EX["cu_seqlens"], c["old_logp"],
                          EX["rewards"], EX["group_ids"], eps_low=EX["eps_low"], eps_high=EX["eps_high"],
                          adv_eps=EX["adv_eps"])
    assert r["loss"] == pytest.approx(c["loss"], abs=1e-14)
    np.testing.assert_allclose(r["logp"], EX["logp"], rtol=0, atol=1e-14)
    np.testing.assert_allclose(r["H"], EX["entropy"], rtol=0, atol=1e-14)
    np.testing.assert_allclose(r["dh"], c["dh"], rtol=0, atol=1e-14)
    np.testing.assert_allclose(r["dW"], c["dW"], rtol=0, atol=1e-14)


@pytest.mark.gpu
@pytest.mark.parametrize("case", CASES)
def test_hip_path_reproduces_the_worked_example(case):
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from gpu_common import ensure_library, log

    import paper_2608_16798_amd as rlk

    ensure_library()
    c = EX["cases"][case]
    log(f"worked example {case}")
    dev = lambda a, dt: torch.as_tensor(np.asarray(a), dtype=dt, device="cuda")
    p = rlk.make_params(eps_low=EX["eps_low"], eps_high=EX["eps_high"], adv_eps=EX["adv_eps"])
    N = EX["h"].shape[0]
    logp = torch.empty(N, dtype=torch.float32, device="cuda")
    ent = torch.empty(N, dtype=torch.float32, device="cuda")
    loss, dh, dW, ws = rlk.pg_loss_fwd_bwd(
        dev(EX["h"], torch.float32), dev(EX["W"], torch.float32), dev(EX["targets"], torch.int32),
        dev(EX["mask"], torch.uint8), dev(EX["cu_seqlens"], torch.int32), dev(c["old_logp"], torch.float32),
        dev(EX["rewards"], torch.float32), dev(EX["group_ids"], torch.int32), p, logp_out=logp, entropy_out=ent)
    torch.cuda.synchronize()
    assert rlk.check_status(ws) == 0
    # fp32 inputs (log 3 rounded to fp32) and fp32 arithmetic: a few fp32 ulps of values of order 1
    tol = 2e-6
    assert float(loss.item()) == pytest.approx(c["loss"], abs=tol)
    pol = EX["mask"] == 1
    np.testing.assert_allclose(logp.cpu().numpy()[pol], EX["logp"], rtol=0, atol=tol)
    np.testing.assert_allclose(ent.cpu().numpy()[pol], EX["entropy"], rtol=0, atol=tol)
    np.testing.assert_allclose(dh.cpu().numpy(), c["dh"], rtol=0, atol=tol)
    np.testing.assert_allclose(dW.cpu().numpy(), c["dW"], rtol=0, atol=tol)
