"""Host-side checks of the C ABI: the library loads, exports every declared entry point,
sizes workspaces and rejects invalid arguments before launching anything (no GPU needed)."""
import ctypes
import os
import re

import pytest

import paper_2608_16798_amd as rlk
from workloads import get_config
from workloads.configs import ORDER

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(rlk.LIB_PATH):
        from paper_2608_16798_amd.build import build

        build(verbose=False)
    return rlk.load_library()


def declared_functions():
    src = open(os.path.join(ROOT, "include", "rlk.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(rlk_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert "rlk_pg_loss_fwd_bwd" in names and "rlk_logprob_fwd" in names and "rlk_group_advantage" in names
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(rlk.EXPORTS)


def test_version_and_strings(lib):
    assert lib.rlk_version() == 7
    assert lib.rlk_status_string(rlk.RLK_EWORKSPACE).decode().startswith("workspace")
    assert lib.rlk_kernel_kind_name(10).decode() == "fwd_lse_gemm"


def _batch(cfg, N=4096, R=8, cu=0x1000):
    return rlk.Batch(N=N, R=R, d=cfg.d, V=cfg.V, dtype=rlk.DTYPE_BF16 if cfg.dtype == "bf16" else rlk.DTYPE_F32,
                     cu_seqlens=cu)


@pytest.mark.parametrize("name", ORDER)
def test_workspace_sizes(lib, name):
    cfg = get_config(name)
    b = _batch(cfg)
    fwd = rlk.workspace_size(b)
    bwd = rlk.workspace_size(b, rlk.make_params())
    assert 0 < fwd < bwd
    esz = 2 if cfg.dtype == "bf16" else 4
    Vp = (cfg.V + 255) // 256 * 256
    Mc = 4096  # chunk capped at the token count rounded to 256
    assert bwd >= 2 * Mc * Vp * esz + cfg.d * Vp * esz
    big = rlk.workspace_size(b, rlk.make_params(chunk_rows=8192))
    assert big > bwd


def test_host_validation(lib):
    cfg = get_config("tiny_fp32")
    n = ctypes.c_size_t()
    b = _batch(cfg)
    assert lib.rlk_workspace_size(None, None, ctypes.byref(n)) == rlk.RLK_EINVAL
    bad = _batch(cfg)
    bad.dtype = 7
    assert lib.rlk_workspace_size(ctypes.byref(bad), None, ctypes.byref(n)) == rlk.RLK_EDTYPE
    bad = _batch(cfg)
    bad.d = 12
    assert lib.rlk_workspace_size(ctypes.byref(bad), None, ctypes.byref(n)) == rlk.RLK_ESHAPE
    assert b"multiple of 8" in lib.rlk_last_error()
    bad = _batch(cfg, N=10, R=0)
    assert lib.rlk_workspace_size(ctypes.byref(bad), None, ctypes.byref(n)) == rlk.RLK_ESHAPE
    p = rlk.make_params(chunk_rows=300)
    assert lib.rlk_workspace_size(ctypes.byref(b), ctypes.byref(p), ctypes.byref(n)) == rlk.RLK_ESHAPE
    # size limits of the 32-bit panel addressing
    p = rlk.make_params(chunk_rows=(1 << 20) + 256)
    assert lib.rlk_workspace_size(ctypes.byref(b), ctypes.byref(p), ctypes.byref(n)) == rlk.RLK_ESHAPE
    for field, val in (("V", (1 << 21) + 1), ("d", (1 << 21) + 8), ("V", 0)):
        bad = _batch(cfg)
        setattr(bad, field, val)
        assert lib.rlk_workspace_size(ctypes.byref(bad), None, ctypes.byref(n)) == rlk.RLK_ESHAPE, (field, val)
    big = _batch(cfg)
    big.V = 1 << 21
    assert lib.rlk_workspace_size(ctypes.byref(big), None, ctypes.byref(n)) == rlk.RLK_OK
    assert lib.rlk_advantage_workspace_size(20000, ctypes.byref(n)) == rlk.RLK_ESHAPE

    fake = 0x10000  # never dereferenced: every call below fails validation first
    need = rlk.workspace_size(b)
    # missing / misaligned / short workspace
    assert lib.rlk_logprob_fwd(ctypes.byref(b), fake, fake, fake, None, fake, None, None, None, need, None) \
        == rlk.RLK_EWORKSPACE
    assert lib.rlk_logprob_fwd(ctypes.byref(b), fake, fake, fake, None, fake, None, None, fake + 8, need, None) \
        == rlk.RLK_EWORKSPACE
    assert lib.rlk_logprob_fwd(ctypes.byref(b), fake, fake, fake, None, fake, None, None, fake, need - 1, None) \
        == rlk.RLK_EWORKSPACE
    assert lib.rlk_logprob_fwd(ctypes.byref(b), None, fake, fake, None, fake, None, None, fake, need, None) \
        == rlk.RLK_EINVAL
    # row tensors must be 16-byte aligned (they are moved in 16-byte vectors)
    assert lib.rlk_logprob_fwd(ctypes.byref(b), fake + 8, fake, fake, None, fake, None, None, fake, 256, None) \
        == rlk.RLK_EINVAL
    assert lib.rlk_logprob_fwd(ctypes.byref(b), fake, fake + 4, fake, None, fake, None, None, fake, 256, None) \
        == rlk.RLK_EINVAL
    # loss parameters
    args = lambda p: (ctypes.byref(b), fake, fake, fake, None, fake, fake, fake, ctypes.byref(p), fake, fake, fake,
                      None, None, None, fake, 1 << 40, None)
    for kw in (dict(eps_low=1.0), dict(eps_low=-0.1), dict(agg=3), dict(adv_eps=-1.0)):
        p = rlk.make_params(**kw)
        assert lib.rlk_pg_loss_fwd_bwd(*args(p)) == rlk.RLK_EINVAL, kw
    # truncated importance sampling and the KL term
    for kw, ro, rf in ((dict(tis_cap=1.5), None, None), (dict(), fake, None), (dict(tis_cap=-1.0), fake, None),
                       (dict(tis_cap=float("inf")), fake, None), (dict(kl_coef=0.1), None, None),
                       (dict(kl_coef=-0.1), None, fake), (dict(kl_coef=float("nan")), None, fake)):
        p = rlk.make_params(**kw)
        p.rollout_logp = ro
        p.ref_logp = rf
        assert lib.rlk_pg_loss_fwd_bwd(*args(p)) == rlk.RLK_EINVAL, (kw, ro, rf)
    assert ctypes.sizeof(rlk.PgParams) == 80 and ctypes.sizeof(rlk.PgStats) == 64
    assert ctypes.sizeof(rlk.Batch) == 40
    for tau in (-1.0, float("inf"), float("nan")):
        bad = _batch(cfg)
        bad.temperature = tau
        assert lib.rlk_workspace_size(ctypes.byref(bad), None, ctypes.byref(n)) == rlk.RLK_EINVAL, tau
    bad = _batch(cfg)
    bad.max_policy_tokens = -1
    assert lib.rlk_workspace_size(ctypes.byref(bad), None, ctypes.byref(n)) == rlk.RLK_EINVAL
    for tau in (0.0, 0.5, 2.0):
        ok = _batch(cfg)
        ok.temperature = tau
        assert lib.rlk_workspace_size(ctypes.byref(ok), None, ctypes.byref(n)) == rlk.RLK_OK
    # GAE / value loss
    assert lib.rlk_gae(10, 2, fake, fake, fake, fake, None, ctypes.c_float(1.5), ctypes.c_float(1.0), fake, None,
                       None) == rlk.RLK_EINVAL
    assert lib.rlk_gae(10, 2, None, fake, fake, fake, None, ctypes.c_float(1.0), ctypes.c_float(1.0), fake, None,
                       None) == rlk.RLK_EINVAL
    assert lib.rlk_gae(-1, 2, fake, fake, fake, fake, None, ctypes.c_float(1.0), ctypes.c_float(1.0), fake, None,
                       None) == rlk.RLK_ESHAPE
    need = rlk.value_workspace_size(4)
    assert need > 0
    assert lib.rlk_value_loss(10, 4, fake, fake, fake, fake, None, fake, None, fake, need - 1, None) \
        == rlk.RLK_EWORKSPACE
    assert lib.rlk_value_loss(10, 4, fake, fake, fake, fake, None, None, None, fake, need, None) == rlk.RLK_EINVAL
    # linear value head
    hb = _batch(cfg)
    assert lib.rlk_value_head_fwd(ctypes.byref(hb), fake, fake, ctypes.c_float(float("nan")), None, None, fake,
                                  None) == rlk.RLK_EINVAL
    assert lib.rlk_value_head_fwd(ctypes.byref(hb), None, fake, ctypes.c_float(0.0), None, None, fake,
                                  None) == rlk.RLK_EINVAL
    need = ctypes.c_size_t()
    assert lib.rlk_value_head_workspace_size(ctypes.byref(hb), ctypes.byref(need)) == rlk.RLK_OK
    assert need.value >= (4096 // 1024) * cfg.d * 4
    args_h = lambda acc, wsb: (ctypes.byref(hb), fake, fake, None, None, fake, None, acc, fake, fake, fake, wsb, None)
    assert lib.rlk_value_head_bwd(*args_h(2, need.value)) == rlk.RLK_EINVAL
    assert lib.rlk_value_head_bwd(*args_h(0, need.value - 1)) == rlk.RLK_EWORKSPACE
    p = rlk.make_params()
    p.accumulate_dW = 2
    assert lib.rlk_pg_loss_fwd_bwd(*args(p)) == rlk.RLK_EINVAL
    p = rlk.make_params()
    for pos in (1, 2, 10):  # hidden, W, dhidden
        a = list(args(p))
        a[pos] = fake + 8
        a[16] = 256  # a short workspace too: nothing can be launched if the check were missing
        assert lib.rlk_pg_loss_fwd_bwd(*a) == rlk.RLK_EINVAL, pos
    assert lib.rlk_value_head_fwd(ctypes.byref(hb), fake + 2, fake, ctypes.c_float(0.0), None, None, fake,
                                  None) == rlk.RLK_EINVAL
    assert lib.rlk_group_advantage(8, fake, fake, ctypes.c_float(-1.0), fake, None, None, fake, 1 << 20, None) \
        == rlk.RLK_EINVAL
    assert lib.rlk_group_advantage(8, None, fake, ctypes.c_float(1e-6), fake, None, None, fake, 1 << 20, None) \
        == rlk.RLK_EINVAL


def test_policy_token_bound_sizes_the_chunks(lib):
    # qwen8b shape: a bound on the trained tokens plans the chunk rows from it, within the same
    # 256-row granularity and never above the unbounded chunk
    cfg = get_config("qwen8b_bf16")
    N = 524288
    p = rlk.make_params()
    free = rlk.workspace_size(_batch(cfg, N=N, R=128), p)
    for bound in (211143, 100000, 40000, 1000):
        b = _batch(cfg, N=N, R=128)
        b.max_policy_tokens = bound
        got = rlk.workspace_size(b, p)
        assert 0 < got <= free, bound
    small = _batch(cfg, N=N, R=128)
    small.max_policy_tokens = 1000
    assert rlk.workspace_size(small, p) < rlk.workspace_size(_batch(cfg, N=1280, R=128), p) * 2
    # a bound above N is the same as N
    b = _batch(cfg, N=N, R=128)
    b.max_policy_tokens = N + 5
    bN = _batch(cfg, N=N, R=128)
    bN.max_policy_tokens = N
    assert rlk.workspace_size(b, p) == rlk.workspace_size(bN, p)


def test_grad_token_hint_sizes_stay_bounded(lib):
    # the hint re-plans the chunks of a bounded call; any value (tiny, near or past the bound, huge)
    # gives a workspace within 1 % of the unbounded one (chunks no wider; the K-split partials of a
    # dhidden tail may grow), and it is ignored without the bound or when the loss has another term
    # (the sizes then equal the hint-free ones)
    cfg = get_config("qwen8b_bf16")
    N, bound = 524288, 211143
    free = rlk.workspace_size(_batch(cfg, N=N, R=128), rlk.make_params())
    b = _batch(cfg, N=N, R=128)
    b.max_policy_tokens = bound
    plain = rlk.workspace_size(b, rlk.make_params())
    for hint in (1, 255, 256, 185134, bound - 1, bound, bound + 1, 1 << 62):
        got = rlk.workspace_size(b, rlk.make_params(grad_tokens=hint))
        assert 0 < got <= 1.01 * free, hint
        if hint >= bound - 1:                     # rounded up to whole tiles it reaches the bound
            assert got == plain, hint
        assert rlk.workspace_size(b, rlk.make_params(grad_tokens=hint, entropy_coef=0.01)) == \
            rlk.workspace_size(b, rlk.make_params(entropy_coef=0.01)), hint
    unbounded = _batch(cfg, N=N, R=128)
    assert rlk.workspace_size(unbounded, rlk.make_params(grad_tokens=185134)) == free
