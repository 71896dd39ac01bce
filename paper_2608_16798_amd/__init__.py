"""Python binding of librlk (the MI355X policy-gradient hot path).

Argument marshalling only: every step of the computation runs in the HIP kernels of
librlk.so, reached through its C ABI (include/rlk.h) with ctypes.  torch provides
device memory and streams.  There is no fallback: if the library is missing or no
GPU is present, the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "librlk.so")

RLK_OK, RLK_EINVAL, RLK_ESHAPE, RLK_EDTYPE, RLK_EWORKSPACE, RLK_EHIP, RLK_EDATA = range(7)
DTYPE_F32, DTYPE_BF16 = 0, 1
AGG_SEQ, AGG_TOKEN = 0, 1
DERR_TARGET, DERR_CU_SEQLENS, DERR_POLICY_BOUND = 1, 2, 4

EXPORTS = [
    "rlk_workspace_size", "rlk_advantage_workspace_size", "rlk_compact", "rlk_logprob_fwd", "rlk_group_advantage",
    "rlk_pg_loss_fwd_bwd", "rlk_check_status", "rlk_status_string", "rlk_last_error", "rlk_version",
    "rlk_profile_begin", "rlk_profile_end", "rlk_kernel_kind_name", "rlk_gae", "rlk_value_workspace_size",
    "rlk_value_loss", "rlk_tree_pack", "rlk_value_head_fwd", "rlk_value_head_workspace_size", "rlk_value_head_bwd",
    "rlk_group_advantage_noalloc",
]


class Batch(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("R", ctypes.c_int32), ("d", ctypes.c_int32), ("V", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("cu_seqlens", ctypes.c_void_p), ("temperature", ctypes.c_float),
                ("max_policy_tokens", ctypes.c_int32)]


class PgParams(ctypes.Structure):
    _fields_ = [("eps_low", ctypes.c_float), ("eps_high", ctypes.c_float), ("adv_eps", ctypes.c_float),
                ("entropy_coef", ctypes.c_float), ("agg", ctypes.c_int32), ("accumulate_dW", ctypes.c_int32),
                ("norm_override", ctypes.c_double), ("chunk_rows", ctypes.c_int64),
                ("rollout_logp", ctypes.c_void_p), ("ref_logp", ctypes.c_void_p), ("tis_cap", ctypes.c_float),
                ("kl_coef", ctypes.c_float), ("token_adv", ctypes.c_void_p), ("grad_tokens", ctypes.c_int64)]


class PgStats(ctypes.Structure):
    _fields_ = [("loss", ctypes.c_float), ("pg_loss", ctypes.c_float), ("entropy_mean", ctypes.c_float),
                ("clip_frac", ctypes.c_float), ("ratio_mean", ctypes.c_float), ("n_groups", ctypes.c_int32),
                ("n_valid_rollouts", ctypes.c_int32), ("n_policy_tokens", ctypes.c_int64),
                ("kl_mean", ctypes.c_float), ("tis_mean", ctypes.c_float), ("n_chunks", ctypes.c_int32),
                ("n_dz_chunks", ctypes.c_int32), ("n_grad_tokens", ctypes.c_int64)]


class Calls(ctypes.Structure):
    _fields_ = [("R", ctypes.c_int32), ("call_off", ctypes.c_void_p), ("x_off", ctypes.c_void_p),
                ("x_tok", ctypes.c_void_p), ("y_off", ctypes.c_void_p), ("y_tok", ctypes.c_void_p)]


class TreeOut(ctypes.Structure):
    _fields_ = [("cap_pos", ctypes.c_int64), ("cap_rows", ctypes.c_int64), ("token", ctypes.c_void_p),
                ("parent", ctypes.c_void_p), ("depth", ctypes.c_void_p), ("pos_off", ctypes.c_void_p),
                ("row_src", ctypes.c_void_p), ("row_target", ctypes.c_void_p), ("row_mask", ctypes.c_void_p),
                ("row_cu", ctypes.c_void_p), ("leaves", ctypes.c_void_p), ("n_pos", ctypes.c_int64),
                ("n_rows", ctypes.c_int64)]


class RlkError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"rlk error {code}: {msg}")
        self.code = code


_lib = None


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Load librlk.so (raises if it has not been built).  RLK_LIBRARY (environment) names another
    build of the same library, e.g. the host-sanitizer build librlk_hostsan.so."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or os.environ.get("RLK_LIBRARY") or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"librlk.so not found at {path}; build it with `python -m paper_2608_16798_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i32, i64, sz, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float
    pb, pp = ctypes.POINTER(Batch), ctypes.POINTER(PgParams)
    lib.rlk_workspace_size.argtypes = [pb, pp, ctypes.POINTER(sz)]
    lib.rlk_advantage_workspace_size.argtypes = [i32, ctypes.POINTER(sz)]
    lib.rlk_compact.argtypes = [pb, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.rlk_logprob_fwd.argtypes = [pb, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.rlk_group_advantage.argtypes = [i32, vp, vp, f32, vp, vp, vp, vp, sz, vp]
    lib.rlk_group_advantage_noalloc.argtypes = [i32, vp, vp, f32, vp, vp, vp, vp]
    lib.rlk_pg_loss_fwd_bwd.argtypes = [pb, vp, vp, vp, vp, vp, vp, vp, pp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.rlk_check_status.argtypes = [vp, vp, ctypes.POINTER(i32)]
    lib.rlk_status_string.argtypes = [i32]
    lib.rlk_status_string.restype = ctypes.c_char_p
    lib.rlk_last_error.argtypes = []
    lib.rlk_last_error.restype = ctypes.c_char_p
    lib.rlk_version.restype = i32
    lib.rlk_profile_begin.argtypes = []
    lib.rlk_profile_end.argtypes = [i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32), ctypes.POINTER(i32)]
    lib.rlk_kernel_kind_name.argtypes = [i32]
    i64 = ctypes.c_int64
    lib.rlk_gae.argtypes = [i64, i32, vp, vp, vp, vp, vp, f32, f32, vp, vp, vp]
    lib.rlk_value_workspace_size.argtypes = [i32, ctypes.POINTER(sz)]
    lib.rlk_value_loss.argtypes = [i64, i32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.rlk_tree_pack.argtypes = [ctypes.POINTER(Calls), ctypes.POINTER(TreeOut)]
    lib.rlk_value_head_fwd.argtypes = [ctypes.POINTER(Batch), vp, vp, f32, vp, vp, vp, vp]
    lib.rlk_value_head_workspace_size.argtypes = [ctypes.POINTER(Batch), ctypes.POINTER(sz)]
    lib.rlk_value_head_bwd.argtypes = [ctypes.POINTER(Batch), vp, vp, vp, vp, vp, vp, i32, vp, vp, vp, sz, vp]
    lib.rlk_kernel_kind_name.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name not in ("rlk_status_string", "rlk_last_error", "rlk_kernel_kind_name", "rlk_version"):
            getattr(lib, name).restype = i32
    _lib = lib
    return lib


def _check(code: int):
    if code != RLK_OK:
        raise RlkError(code, load_library().rlk_last_error().decode())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _tensor(t, name: str, shape=None, dtypes=None, optional: bool = False, min_bytes: int = 0):
    """Checks a tensor argument before its pointer crosses the C ABI: a torch tensor of one of
    `dtypes`, of exactly `shape` (None entries match any size) and contiguous (row-major).
    Raises TypeError / ValueError; nothing is launched.  Devices are checked afterwards, for all
    arguments together, by _on_one_gpu."""
    import torch

    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor, got {type(t).__name__}")
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {' or '.join(str(d) for d in dtypes)}")
    if shape is not None:
        ok = t.dim() == len(shape) and all(w is None or int(a) == int(w) for a, w in zip(t.shape, shape))
        if not ok:
            want = "[" + ", ".join("*" if w is None else str(int(w)) for w in shape) + "]"
            raise ValueError(f"{name} has shape {list(t.shape)}, expected {want}")
    if min_bytes and t.numel() * t.element_size() < min_bytes:
        raise ValueError(f"{name} holds {t.numel() * t.element_size()} bytes, needs at least {min_bytes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous (row-major)")


def _on_one_gpu(**tensors):
    """Every given tensor (None entries skipped) lives on one and the same GPU."""
    dev = None
    for name, t in tensors.items():
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError(f"{name} must be a GPU tensor, got device {t.device}")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError(f"{name} is on {t.device}, other arguments on {dev}")


def _float_types():
    import torch

    return (torch.float32, torch.bfloat16)


def _check_rows(hidden, W, targets, mask, cu_seqlens):
    """The batch tensors shared by the log-prob and loss entry points; returns (N, d, V, R, device)."""
    import torch

    _tensor(hidden, "hidden", shape=(None, None), dtypes=_float_types())
    N, d = hidden.shape
    dev = hidden.device
    _tensor(W, "W", shape=(None, d), dtypes=(hidden.dtype,))
    _tensor(targets, "targets", shape=(N,), dtypes=(torch.int32,))
    _tensor(mask, "mask", shape=(N,), dtypes=(torch.uint8, torch.bool), optional=True)
    _tensor(cu_seqlens, "cu_seqlens", shape=(None,), dtypes=(torch.int32,))
    if cu_seqlens.shape[0] < 1:
        raise ValueError("cu_seqlens needs R + 1 >= 1 entries")
    return N, d, W.shape[0], cu_seqlens.shape[0] - 1, dev


def _stream_handle(stream) -> Optional[int]:
    import torch

    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _dtype_code(t) -> int:
    import torch

    if t.dtype == torch.bfloat16:
        return DTYPE_BF16
    if t.dtype == torch.float32:
        return DTYPE_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def make_batch(hidden, W, cu_seqlens, temperature: float = 1.0, max_policy_tokens: int = 0) -> Batch:
    """Batch descriptor; max_policy_tokens is an optional host-known upper bound on the trained
    tokens (0 = unknown), see rlk_batch_t."""
    N, d = hidden.shape
    V = W.shape[0]
    R = cu_seqlens.shape[0] - 1
    return Batch(N=N, R=R, d=d, V=V, dtype=_dtype_code(W), cu_seqlens=_ptr(cu_seqlens), temperature=temperature,
                 max_policy_tokens=int(max_policy_tokens))


def make_params(eps_low=0.2, eps_high=None, adv_eps=1e-6, entropy_coef=0.0, agg=AGG_SEQ, accumulate_dW=False,
                norm_override=0.0, chunk_rows=0, tis_cap=0.0, kl_coef=0.0, grad_tokens=0) -> PgParams:
    """Loss parameters; the rollout / reference log-prob arrays of truncated importance sampling
    and of the KL term are passed to pg_loss_fwd_bwd.  grad_tokens is the optional chunk-planning
    hint (see grad_token_hint)."""
    p = PgParams()
    p.eps_low = eps_low
    p.eps_high = eps_low if eps_high is None else eps_high
    p.adv_eps = adv_eps
    p.entropy_coef = entropy_coef
    p.agg = agg
    p.accumulate_dW = 1 if accumulate_dW else 0
    p.norm_override = float(norm_override or 0.0)
    p.chunk_rows = int(chunk_rows)
    p.tis_cap = float(tis_cap)
    p.kl_coef = float(kl_coef)
    p.grad_tokens = int(grad_tokens)
    return p


def grad_token_hint(mask, cu_seqlens, rewards, group_ids) -> int:
    """Host count for PgParams.grad_tokens: trained tokens (mask = 1) of the rollouts with a group id
    >= 0 whose group's rewards are not all equal.  A group of equal rewards has the advantage 0 for
    every member (Sec. 2.3.1), so without an entropy term, KL term or per-token advantages its tokens
    carry no gradient and the call leaves them out of the backward.  It is a planning hint only: a
    rollout whose advantage comes out 0 in a mixed group is still counted, which any value tolerates."""
    import numpy as np

    cu = np.asarray(cu_seqlens, dtype=np.int64)
    gid = np.asarray(group_ids, dtype=np.int64)
    rw = np.asarray(rewards, dtype=np.float64)
    lens = np.diff(cu)
    live = gid >= 0
    mixed = np.zeros(len(gid), dtype=bool)
    if live.any():
        groups, inv = np.unique(gid[live], return_inverse=True)
        lo = np.full(len(groups), np.inf)
        hi = np.full(len(groups), -np.inf)
        np.minimum.at(lo, inv, rw[live])
        np.maximum.at(hi, inv, rw[live])
        mixed[live] = (hi > lo)[inv]
    keep = np.repeat(mixed, lens)
    m = np.asarray(mask)[:keep.shape[0]].astype(bool)
    return int((m & keep).sum())


def workspace_size(batch: Batch, params: Optional[PgParams] = None) -> int:
    lib = load_library()
    n = ctypes.c_size_t()
    _check(lib.rlk_workspace_size(ctypes.byref(batch), ctypes.byref(params) if params is not None else None,
                                  ctypes.byref(n)))
    return n.value


def advantage_workspace_size(R: int) -> int:
    lib = load_library()
    n = ctypes.c_size_t()
    _check(lib.rlk_advantage_workspace_size(R, ctypes.byref(n)))
    return n.value


def alloc_workspace(nbytes: int, device="cuda"):
    """A 256-byte aligned uint8 device buffer of at least nbytes (torch allocations are)."""
    import torch

    ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws


def logprob_fwd(hidden, W, targets, mask, cu_seqlens, logp=None, entropy=None, lse=None, ws=None, stream=None,
                temperature: float = 1.0, max_policy_tokens: int = 0):
    """Per-token log-prob / entropy / log-partition of the sampled tokens (rows with mask 0 -> 0).
    max_policy_tokens: optional host-known bound on the policy tokens (rlk_batch_t)."""
    import torch

    N, d, V, R, dev = _check_rows(hidden, W, targets, mask, cu_seqlens)
    f32 = (torch.float32,)
    _tensor(logp, "logp", shape=(N,), dtypes=f32, optional=True)
    _tensor(entropy, "entropy", shape=(N,), dtypes=f32, optional=True)
    _tensor(lse, "lse", shape=(N,), dtypes=f32, optional=True)
    _tensor(ws, "ws", dtypes=(torch.uint8,), optional=True)
    _on_one_gpu(hidden=hidden, W=W, targets=targets, mask=mask, cu_seqlens=cu_seqlens, logp=logp, entropy=entropy,
                lse=lse, ws=ws)
    lib = load_library()
    b = make_batch(hidden, W, cu_seqlens, temperature, max_policy_tokens)
    if logp is None:
        logp = torch.empty(N, dtype=torch.float32, device=dev)
    if ws is None:
        ws = alloc_workspace(workspace_size(b), dev)
    _on_one_gpu(hidden=hidden, W=W, targets=targets, mask=mask, cu_seqlens=cu_seqlens, logp=logp, entropy=entropy,
                lse=lse, ws=ws)
    _check(lib.rlk_logprob_fwd(ctypes.byref(b), _ptr(hidden), _ptr(W), _ptr(targets), _ptr(mask), _ptr(logp),
                               _ptr(entropy), _ptr(lse), _ptr(ws), ws.numel(), _stream_handle(stream)))
    return logp, entropy, lse, ws


def compact(cu_seqlens, mask, group_ids=None, targets=None, N=None, V=1, d=8, ws=None, stream=None):
    """Compacted policy-token positions, their rollouts, per-rollout counts and N_eff (device tensors)."""
    import torch

    _tensor(cu_seqlens, "cu_seqlens", shape=(None,), dtypes=(torch.int32,))
    dev = cu_seqlens.device
    R = cu_seqlens.shape[0] - 1
    if N is None:
        if mask is None:
            raise ValueError("compact needs N when mask is None")
        N = mask.shape[0]
    _tensor(mask, "mask", shape=(N,), dtypes=(torch.uint8, torch.bool), optional=True)
    _tensor(group_ids, "group_ids", shape=(R,), dtypes=(torch.int32,), optional=True)
    _tensor(targets, "targets", shape=(N,), dtypes=(torch.int32,), optional=True)
    _tensor(ws, "ws", dtypes=(torch.uint8,), optional=True)
    _on_one_gpu(cu_seqlens=cu_seqlens, mask=mask, group_ids=group_ids, targets=targets, ws=ws)
    lib = load_library()
    b = Batch(N=N, R=R, d=d, V=V, dtype=DTYPE_BF16, cu_seqlens=_ptr(cu_seqlens))
    idx = torch.empty(max(N, 1), dtype=torch.int32, device=dev)
    tokr = torch.empty(max(N, 1), dtype=torch.int32, device=dev)
    n_pol = torch.empty(max(R, 1), dtype=torch.int32, device=dev)
    n_eff = torch.empty(1, dtype=torch.int32, device=dev)
    if ws is None:
        ws = alloc_workspace(workspace_size(b), dev)
    _on_one_gpu(cu_seqlens=cu_seqlens, mask=mask, group_ids=group_ids, targets=targets, idx=idx, tokr=tokr,
                n_pol=n_pol, n_eff=n_eff, ws=ws)
    _check(lib.rlk_compact(ctypes.byref(b), _ptr(mask), _ptr(group_ids), _ptr(targets), _ptr(idx), _ptr(tokr),
                           _ptr(n_pol), _ptr(n_eff), _ptr(ws), ws.numel(), _stream_handle(stream)))
    return idx, tokr, n_pol[:R], n_eff, ws


def group_advantage(rewards, group_ids, adv_eps=1e-6, adv=None, group_index=None, n_groups=None, ws=None,
                    stream=None):
    import torch

    _tensor(rewards, "rewards", shape=(None,), dtypes=(torch.float32,))
    R = rewards.shape[0]
    dev = rewards.device
    _tensor(group_ids, "group_ids", shape=(R,), dtypes=(torch.int32,))
    _tensor(adv, "adv", shape=(R,), dtypes=(torch.float32,), optional=True)
    _tensor(group_index, "group_index", shape=(R,), dtypes=(torch.int32,), optional=True)
    _tensor(n_groups, "n_groups", shape=(None,), dtypes=(torch.int32,), optional=True, min_bytes=4)
    _tensor(ws, "ws", dtypes=(torch.uint8,), optional=True)
    _on_one_gpu(rewards=rewards, group_ids=group_ids, adv=adv, group_index=group_index, n_groups=n_groups, ws=ws)
    lib = load_library()
    if adv is None:
        adv = torch.empty(R, dtype=torch.float32, device=dev)
    if ws is None:
        ws = alloc_workspace(advantage_workspace_size(R), dev)
    _on_one_gpu(rewards=rewards, group_ids=group_ids, adv=adv, group_index=group_index, n_groups=n_groups, ws=ws)
    _check(lib.rlk_group_advantage(R, _ptr(rewards), _ptr(group_ids), adv_eps, _ptr(adv), _ptr(group_index),
                                   _ptr(n_groups), _ptr(ws), ws.numel(), _stream_handle(stream)))
    return adv


def group_advantage_noalloc(rewards, group_ids, adv_eps=1e-6, adv=None, group_index=None, n_groups=None,
                            stream=None):
    """group_advantage through rlk_group_advantage_noalloc: the library's fixed device scratch instead
    of a workspace (for callers that cannot allocate; calls overlapping on one GPU race)."""
    import torch

    _tensor(rewards, "rewards", shape=(None,), dtypes=(torch.float32,))
    R = rewards.shape[0]
    _tensor(group_ids, "group_ids", shape=(R,), dtypes=(torch.int32,))
    _tensor(adv, "adv", shape=(R,), dtypes=(torch.float32,), optional=True)
    _tensor(group_index, "group_index", shape=(R,), dtypes=(torch.int32,), optional=True)
    _tensor(n_groups, "n_groups", shape=(None,), dtypes=(torch.int32,), optional=True, min_bytes=4)
    _on_one_gpu(rewards=rewards, group_ids=group_ids, adv=adv, group_index=group_index, n_groups=n_groups)
    lib = load_library()
    if adv is None:
        adv = torch.empty(R, dtype=torch.float32, device=rewards.device)
    _on_one_gpu(rewards=rewards, adv=adv)
    _check(lib.rlk_group_advantage_noalloc(R, _ptr(rewards), _ptr(group_ids), adv_eps, _ptr(adv), _ptr(group_index),
                                           _ptr(n_groups), _stream_handle(stream)))
    return adv


def pg_loss_fwd_bwd(hidden, W, targets, mask, cu_seqlens, old_logp, rewards, group_ids, params: PgParams,
                    loss=None, dhidden=None, dW=None, logp_out=None, entropy_out=None, stats=None, ws=None,
                    stream=None, rollout_logp=None, ref_logp=None, token_adv=None, temperature: float = 1.0,
                    max_policy_tokens: int = 0):
    """Loss, dL/dhidden and dL/dW of the masked clipped policy-gradient objective.
    rollout_logp / ref_logp ([N] fp32 device tensors or None) feed truncated importance sampling
    (params.tis_cap) and the KL term (params.kl_coef); token_adv ([N] fp32, e.g. from gae())
    replaces the group advantages (PPO); max_policy_tokens is an optional host-known bound on the
    trained tokens that sizes the chunk loop (rlk_batch_t; the workspace must be sized with it)."""
    import torch

    N, d, V, R, dev = _check_rows(hidden, W, targets, mask, cu_seqlens)
    f32 = (torch.float32,)
    _tensor(old_logp, "old_logp", shape=(N,), dtypes=f32)
    _tensor(rewards, "rewards", shape=(R,), dtypes=f32)
    _tensor(group_ids, "group_ids", shape=(R,), dtypes=(torch.int32,))
    _tensor(loss, "loss", shape=(None,), dtypes=f32, optional=True, min_bytes=4)
    _tensor(dhidden, "dhidden", shape=(N, d), dtypes=(hidden.dtype,), optional=True)
    _tensor(dW, "dW", shape=(V, d), dtypes=f32, optional=True)
    _tensor(logp_out, "logp_out", shape=(N,), dtypes=f32, optional=True)
    _tensor(entropy_out, "entropy_out", shape=(N,), dtypes=f32, optional=True)
    _tensor(stats, "stats", shape=(None,), dtypes=(torch.uint8,), optional=True,
            min_bytes=ctypes.sizeof(PgStats))
    _tensor(ws, "ws", dtypes=(torch.uint8,), optional=True)
    for name, t in (("rollout_logp", rollout_logp), ("ref_logp", ref_logp), ("token_adv", token_adv)):
        _tensor(t, name, shape=(N,), dtypes=f32, optional=True)
    _on_one_gpu(hidden=hidden, W=W, targets=targets, mask=mask, cu_seqlens=cu_seqlens, old_logp=old_logp,
                rewards=rewards, group_ids=group_ids, loss=loss, dhidden=dhidden, dW=dW, logp_out=logp_out,
                entropy_out=entropy_out, stats=stats, ws=ws, rollout_logp=rollout_logp, ref_logp=ref_logp,
                token_adv=token_adv)
    lib = load_library()
    if rollout_logp is not None or ref_logp is not None or token_adv is not None:
        params = PgParams.from_buffer_copy(bytes(params))
        params.rollout_logp = _ptr(rollout_logp)
        params.ref_logp = _ptr(ref_logp)
        params.token_adv = _ptr(token_adv)
    b = make_batch(hidden, W, cu_seqlens, temperature, max_policy_tokens)
    if loss is None:
        loss = torch.empty(1, dtype=torch.float32, device=dev)
    if dhidden is None:
        dhidden = torch.empty_like(hidden)
    if dW is None:
        dW = torch.empty(W.shape, dtype=torch.float32, device=dev)
    if ws is None:
        ws = alloc_workspace(workspace_size(b, params), dev)
    _on_one_gpu(hidden=hidden, loss=loss, dhidden=dhidden, dW=dW, ws=ws)
    _check(lib.rlk_pg_loss_fwd_bwd(ctypes.byref(b), _ptr(hidden), _ptr(W), _ptr(targets), _ptr(mask),
                                   _ptr(old_logp), _ptr(rewards), _ptr(group_ids), ctypes.byref(params), _ptr(loss),
                                   _ptr(dhidden), _ptr(dW), _ptr(logp_out), _ptr(entropy_out), _ptr(stats),
                                   _ptr(ws), ws.numel(), _stream_handle(stream)))
    return loss, dhidden, dW, ws


def gae(values, rewards, mask, cu_seqlens, group_ids=None, gamma=1.0, lam=1.0, adv=None, returns=None, stream=None):
    """Masked GAE per rollout (see rlk_gae); returns (adv, returns) as [N] fp32 device tensors."""
    import torch

    f32 = (torch.float32,)
    _tensor(values, "values", shape=(None,), dtypes=f32)
    dev = values.device
    N = values.shape[0]
    _tensor(rewards, "rewards", shape=(None,), dtypes=f32)
    R = rewards.shape[0]
    _tensor(cu_seqlens, "cu_seqlens", shape=(R + 1,), dtypes=(torch.int32,))
    _tensor(mask, "mask", shape=(N,), dtypes=(torch.uint8, torch.bool))
    _tensor(group_ids, "group_ids", shape=(R,), dtypes=(torch.int32,), optional=True)
    _tensor(adv, "adv", shape=(N,), dtypes=f32, optional=True)
    _tensor(returns, "returns", shape=(N,), dtypes=f32, optional=True)
    _on_one_gpu(values=values, rewards=rewards, cu_seqlens=cu_seqlens, mask=mask, group_ids=group_ids, adv=adv,
                returns=returns)
    lib = load_library()
    if adv is None:
        adv = torch.empty(N, dtype=torch.float32, device=values.device)
    if returns is None:
        returns = torch.empty(N, dtype=torch.float32, device=values.device)
    _on_one_gpu(values=values, adv=adv, returns=returns)
    _check(lib.rlk_gae(N, R, _ptr(cu_seqlens), _ptr(mask), _ptr(values), _ptr(rewards), _ptr(group_ids),
                       gamma, lam, _ptr(adv), _ptr(returns), _stream_handle(stream)))
    return adv, returns


def value_workspace_size(R: int) -> int:
    n = ctypes.c_size_t()
    _check(load_library().rlk_value_workspace_size(R, ctypes.byref(n)))
    return n.value


def value_loss(values, returns, mask, cu_seqlens, group_ids=None, loss=None, dvalues=None, ws=None, stream=None):
    """Masked mean-squared value loss and its gradient (see rlk_value_loss)."""
    import torch

    f32 = (torch.float32,)
    _tensor(values, "values", shape=(None,), dtypes=f32)
    dev = values.device
    N = values.shape[0]
    _tensor(cu_seqlens, "cu_seqlens", shape=(None,), dtypes=(torch.int32,))
    R = cu_seqlens.shape[0] - 1
    _tensor(returns, "returns", shape=(N,), dtypes=f32)
    _tensor(mask, "mask", shape=(N,), dtypes=(torch.uint8, torch.bool))
    _tensor(group_ids, "group_ids", shape=(R,), dtypes=(torch.int32,), optional=True)
    _tensor(loss, "loss", shape=(None,), dtypes=f32, optional=True, min_bytes=4)
    _tensor(dvalues, "dvalues", shape=(N,), dtypes=f32, optional=True)
    _tensor(ws, "ws", dtypes=(torch.uint8,), optional=True)
    _on_one_gpu(values=values, returns=returns, cu_seqlens=cu_seqlens, mask=mask, group_ids=group_ids, loss=loss,
                dvalues=dvalues, ws=ws)
    lib = load_library()
    if loss is None:
        loss = torch.empty(1, dtype=torch.float32, device=dev)
    if dvalues is None:
        dvalues = torch.empty(N, dtype=torch.float32, device=dev)
    if ws is None:
        ws = alloc_workspace(value_workspace_size(R), dev)
    _on_one_gpu(values=values, loss=loss, dvalues=dvalues, ws=ws)
    _check(lib.rlk_value_loss(N, R, _ptr(cu_seqlens), _ptr(mask), _ptr(values), _ptr(returns), _ptr(group_ids),
                              _ptr(loss), _ptr(dvalues), _ptr(ws), ws.numel(), _stream_handle(stream)))
    return loss, dvalues


def _check_head(hidden, w_v, mask, cu_seqlens, group_ids):
    import torch

    _tensor(hidden, "hidden", shape=(None, None), dtypes=_float_types())
    N, d = hidden.shape
    dev = hidden.device
    _tensor(w_v, "w_v", shape=(d,), dtypes=(hidden.dtype,))
    _tensor(mask, "mask", shape=(N,), dtypes=(torch.uint8, torch.bool), optional=True)
    _tensor(cu_seqlens, "cu_seqlens", shape=(None,), dtypes=(torch.int32,))
    _tensor(group_ids, "group_ids", shape=(cu_seqlens.shape[0] - 1,), dtypes=(torch.int32,),
            optional=True)
    return N, d, dev


def _head_batch(hidden, cu_seqlens) -> Batch:
    N, d = hidden.shape
    return Batch(N=N, R=cu_seqlens.shape[0] - 1, d=d, V=1, dtype=_dtype_code(hidden), cu_seqlens=_ptr(cu_seqlens))


def value_head_fwd(hidden, w_v, b_v, mask, cu_seqlens, group_ids=None, values=None, stream=None):
    """Linear value head values[t] = w_v . hidden[t] + b_v on the policy rows (see rlk_value_head_fwd)."""
    import torch

    N, d, dev = _check_head(hidden, w_v, mask, cu_seqlens, group_ids)
    _tensor(values, "values", shape=(N,), dtypes=(torch.float32,), optional=True)
    _on_one_gpu(hidden=hidden, w_v=w_v, mask=mask, cu_seqlens=cu_seqlens, group_ids=group_ids, values=values)
    lib = load_library()
    b = _head_batch(hidden, cu_seqlens)
    if values is None:
        values = torch.empty(hidden.shape[0], dtype=torch.float32, device=hidden.device)
    _on_one_gpu(hidden=hidden, values=values)
    _check(lib.rlk_value_head_fwd(ctypes.byref(b), _ptr(hidden), _ptr(w_v), ctypes.c_float(b_v), _ptr(mask),
                                  _ptr(group_ids), _ptr(values), _stream_handle(stream)))
    return values


def value_head_workspace_size(hidden, cu_seqlens) -> int:
    n = ctypes.c_size_t()
    b = _head_batch(hidden, cu_seqlens)
    _check(load_library().rlk_value_head_workspace_size(ctypes.byref(b), ctypes.byref(n)))
    return n.value


def value_head_bwd(hidden, w_v, mask, cu_seqlens, group_ids, dvalues, dhidden=None, accumulate=False, dw_v=None,
                   db_v=None, ws=None, stream=None):
    """Backward of the linear value head (see rlk_value_head_bwd); returns (dhidden, dw_v, db_v)."""
    import torch

    N, d, dev = _check_head(hidden, w_v, mask, cu_seqlens, group_ids)
    f32 = (torch.float32,)
    _tensor(dvalues, "dvalues", shape=(N,), dtypes=f32)
    _tensor(dhidden, "dhidden", shape=(N, d), dtypes=(hidden.dtype,), optional=True)
    _tensor(dw_v, "dw_v", shape=(d,), dtypes=f32, optional=True)
    _tensor(db_v, "db_v", shape=(None,), dtypes=f32, optional=True, min_bytes=4)
    _tensor(ws, "ws", dtypes=(torch.uint8,), optional=True)
    _on_one_gpu(hidden=hidden, w_v=w_v, mask=mask, cu_seqlens=cu_seqlens, group_ids=group_ids, dvalues=dvalues,
                dhidden=dhidden, dw_v=dw_v, db_v=db_v, ws=ws)
    lib = load_library()
    b = _head_batch(hidden, cu_seqlens)
    if dw_v is None:
        dw_v = torch.empty(hidden.shape[1], dtype=torch.float32, device=dev)
    if db_v is None:
        db_v = torch.empty(1, dtype=torch.float32, device=dev)
    if ws is None:
        ws = alloc_workspace(value_head_workspace_size(hidden, cu_seqlens), dev)
    _on_one_gpu(hidden=hidden, dhidden=dhidden, dw_v=dw_v, db_v=db_v, ws=ws)
    _check(lib.rlk_value_head_bwd(ctypes.byref(b), _ptr(hidden), _ptr(w_v), _ptr(mask), _ptr(group_ids),
                                  _ptr(dvalues), _ptr(dhidden), 1 if accumulate else 0, _ptr(dw_v), _ptr(db_v),
                                  _ptr(ws), ws.numel(), _stream_handle(stream)))
    return dhidden, dw_v, db_v


def _calls_struct(calls_per_rollout):
    """Flat host arrays (kept alive in the returned tuple) and the rlk_calls_t describing them."""
    import numpy as np

    call_off, x_off, y_off, xs, ys = [0], [0], [0], [], []
    for calls in calls_per_rollout:
        for x, y in calls:
            xs.extend(int(t) for t in x)
            ys.extend(int(t) for t in y)
            x_off.append(len(xs))
            y_off.append(len(ys))
        call_off.append(len(x_off) - 1)
    arrs = dict(call_off=np.asarray(call_off, np.int64), x_off=np.asarray(x_off, np.int64),
                y_off=np.asarray(y_off, np.int64), x_tok=np.asarray(xs, np.int32), y_tok=np.asarray(ys, np.int32))
    c = Calls(R=len(calls_per_rollout), **{k: v.ctypes.data for k, v in arrs.items()})
    return c, arrs


def tree_pack_sizes(calls_per_rollout):
    """(packed positions, training rows) that tree_pack will produce."""
    c, keep = _calls_struct(calls_per_rollout)
    o = TreeOut()
    _check(load_library().rlk_tree_pack(ctypes.byref(c), ctypes.byref(o)))
    return o.n_pos, o.n_rows


def tree_pack(calls_per_rollout, cap_pos=None, cap_rows=None) -> dict:
    """Prefix trees of the rollouts' model calls, packed (see rlk_tree_pack).  calls_per_rollout:
    list over rollouts of lists of (context tokens, response tokens).  Host numpy arrays."""
    import numpy as np

    n_pos, n_rows = tree_pack_sizes(calls_per_rollout)
    cap_pos = n_pos if cap_pos is None else cap_pos
    cap_rows = n_rows if cap_rows is None else cap_rows
    R = len(calls_per_rollout)
    out = dict(token=np.zeros(max(cap_pos, 1), np.int32), parent=np.zeros(max(cap_pos, 1), np.int32),
               depth=np.zeros(max(cap_pos, 1), np.int32), pos_off=np.zeros(R + 1, np.int64),
               row_src=np.zeros(max(cap_rows, 1), np.int32), row_target=np.zeros(max(cap_rows, 1), np.int32),
               row_mask=np.zeros(max(cap_rows, 1), np.uint8), row_cu=np.zeros(R + 1, np.int32),
               leaves=np.zeros(max(R, 1), np.int32))
    c, keep = _calls_struct(calls_per_rollout)
    o = TreeOut(cap_pos=cap_pos, cap_rows=cap_rows, **{k: v.ctypes.data for k, v in out.items()})
    _check(load_library().rlk_tree_pack(ctypes.byref(c), ctypes.byref(o)))
    for k in ("token", "parent", "depth"):
        out[k] = out[k][:o.n_pos]
    for k in ("row_src", "row_target", "row_mask"):
        out[k] = out[k][:o.n_rows]
    out["leaves"] = out["leaves"][:R]
    return out


def check_status(ws, stream=None) -> int:
    """Synchronises the stream and returns the device data-error bits left in ws."""
    lib = load_library()
    flags = ctypes.c_int32(0)
    code = lib.rlk_check_status(_ptr(ws), _stream_handle(stream), ctypes.byref(flags))
    if code not in (RLK_OK, RLK_EDATA):
        _check(code)
    return flags.value


def stats_from_tensor(t) -> dict:
    """Decodes a device buffer holding an rlk_pg_stats_t (as returned by stats_buffer())."""
    raw = bytes(t.cpu().numpy().tobytes())
    s = PgStats.from_buffer_copy(raw[:ctypes.sizeof(PgStats)])
    return {f: getattr(s, f) for f, _ in PgStats._fields_}


def stats_buffer(device="cuda"):
    import torch

    return torch.zeros(ctypes.sizeof(PgStats), dtype=torch.uint8, device=device)


def profile_begin():
    _check(load_library().rlk_profile_begin())


def profile_end() -> dict:
    lib = load_library()
    n = 32
    ms = (ctypes.c_double * n)()
    cnt = (ctypes.c_int32 * n)()
    nk = ctypes.c_int32()
    _check(lib.rlk_profile_end(n, ms, cnt, ctypes.byref(nk)))
    out = {}
    for k in range(min(n, nk.value)):
        if cnt[k]:
            out[lib.rlk_kernel_kind_name(k).decode()] = (ms[k], cnt[k])
    return out
