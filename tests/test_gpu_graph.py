"""HIP graph capture of the whole policy-gradient call.

rlk_pg_loss_fwd_bwd enqueues only kernel launches on the caller's stream: no allocation, no host
synchronisation, no memset, and the number of policy tokens is read by the kernels from device
memory.  A graph captured once therefore replays the complete step.  Every replay here is checked
bit for bit against an eager call on the same inputs.  The outputs are overwritten with garbage
before each replay, and unrelated eager work runs between replays.  After an input is changed in
place, the replay must follow it.
"""
from __future__ import annotations

import pytest

from gpu_common import O, WL, build_instance, ensure_library, log, params_for, with_far_target

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ensure_library()


def _buffers(inst, params):
    import torch

    import paper_2608_16798_amd as rlk

    h, W = inst["h"], inst["W"]
    N = h.shape[0]
    b = rlk.make_batch(h, W, inst["cu"])
    return dict(loss=torch.empty(1, dtype=torch.float32, device="cuda"), dh=torch.empty_like(h),
                dW=torch.empty(W.shape, dtype=torch.float32, device="cuda"),
                logp=torch.empty(N, dtype=torch.float32, device="cuda"),
                stats=rlk.stats_buffer(h.device), ws=rlk.alloc_workspace(rlk.workspace_size(b, params), h.device))


def _call(inst, params, buf):
    import paper_2608_16798_amd as rlk

    rlk.pg_loss_fwd_bwd(inst["h"], inst["W"], inst["targets"], inst["mask"], inst["cu"], inst["old"],
                        inst["rewards"], inst["gid"], params, loss=buf["loss"], dhidden=buf["dh"], dW=buf["dW"],
                        logp_out=buf["logp"], stats=buf["stats"], ws=buf["ws"])


def _snapshot(buf):
    import paper_2608_16798_amd as rlk

    snap = {k: buf[k].clone() for k in ("loss", "dh", "dW", "logp")}
    snap["stats"] = rlk.stats_from_tensor(buf["stats"])  # the struct's fields (not its padding)
    return snap


def _assert_same(got, ref, tag):
    import torch

    for k in ref:
        same = got[k] == ref[k] if k == "stats" else torch.equal(got[k], ref[k])
        assert same, f"{tag}: {k} differs from the eager call"


# small_bf16 (no entropy term): the token-reference layout, no chunk flagged; large_bf16: the dz pass in
# every chunk; qwen8b_bf16 with one far target: the layout with exactly one flagged chunk, whose flag
# each replay must clear and set again.
@pytest.mark.parametrize("name,chunk_rows,far", [("small_bf16", 0, False), ("large_bf16", 256, False),
                                                 ("qwen8b_bf16", 256, True)])
def test_pg_loss_graph_replay(name, chunk_rows, far):
    import torch

    import paper_2608_16798_amd as rlk

    cfg = WL.scaled_config(name)
    inst = build_instance(cfg)
    if far:
        st = inst["st"]
        idx = O.compact(st.mask, st.cu_seqlens, st.group_ids)[0]
        inst, _ = with_far_target(inst, int(idx[len(idx) // 2]))
    p = params_for(cfg, chunk_rows=chunk_rows)
    log(f"graph replay {cfg.name} N={inst['h'].shape[0]} chunk_rows={chunk_rows} far target {far}")

    eager = _buffers(inst, p)
    _call(inst, p, eager)
    torch.cuda.synchronize()
    ref = _snapshot(eager)
    if far:
        assert ref["stats"]["n_dz_chunks"] == 1

    buf = _buffers(inst, p)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _call(inst, p, buf)  # warm-up on the capture side of the stream fence
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _call(inst, p, buf)
    torch.cuda.synchronize()

    x = torch.randn(1024, 1024, device="cuda")
    for rep in range(3):
        for k in ("loss", "dh", "dW", "logp", "stats"):
            buf[k].fill_(7)
        y = x @ x  # unrelated eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _assert_same(_snapshot(buf), ref, f"replay {rep}")
        assert rlk.check_status(buf["ws"]) == 0
        del y

    # the captured call reads live input memory: flip the rewards in place and replay
    inst["rewards"].copy_(1.0 - inst["rewards"])
    _call(inst, p, eager)
    torch.cuda.synchronize()
    ref2 = _snapshot(eager)
    assert not torch.equal(ref2["dh"], ref["dh"])
    g.replay()
    torch.cuda.synchronize()
    _assert_same(_snapshot(buf), ref2, "replay after the rewards changed")
