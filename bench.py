"""Benchmark of the policy-gradient hot path on one MI355X.

A step is one pass of the whole path over one synthetic agentic-RL batch already resident
in HBM: rlk_group_advantage + rlk_pg_loss_fwd_bwd (compaction, advantages, LM-head GEMM with
online log-softmax, loss, dz, dhidden and dW GEMMs).  Prints one JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload qwen8b_bf16]

HBM traffic of the GEMMs (the roofline's "traffic"): run one step twice under rocprofv3 counter
collection, once with FETCH_SIZE and once with WRITE_SIZE, each with --calibrate-copy-mib so the
same run holds a plain device copy of known size, then
  python bench.py --traffic-summary FETCH.csv WRITE.csv [--workload ...]
writes profiles/<kernel>_<workload>_traffic.txt (HBM bytes per launch, scaled by the copy's
known/measured ratio, tagged with a digest of the kernel sources).

Shader clock and MFMA pipe occupancy of the GEMMs: one step under rocprofv3 with
GRBM_GUI_ACTIVE SQ_VALU_MFMA_BUSY_CYCLES SQ_WAVE_CYCLES SQ_WAIT_ANY, then
  python bench.py --occupancy-summary COUNTERS.csv TITLE COMMAND
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16 = 2.5e15      # MI355X dense bf16 MFMA, FLOP/s
PEAK_FP32_MFMA = 157.3e12
PEAK_HBM = 8.0e12       # B/s
METRIC = "policy tokens/sec for logprob+PG loss fwd+bwd; % of bf16 MFMA peak"
GEMM_KINDS = ("fwd_lse_gemm", "dh_gemm", "dw_gemm")
PROFILES = os.path.join(ROOT, "profiles")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def build_inputs(cfg, device="cuda"):
    import numpy as np
    import torch

    import workloads as WL
    from workloads.anchor import gaussian_anchor

    st = WL.make_structure(cfg)
    h, W = WL.make_tensors(cfg, st.N, device=device)
    anchor = gaussian_anchor(h, W, st.targets, cfg.w_std)
    old = WL.old_logp_from_anchor(anchor, st)
    dev = lambda a, dt: torch.as_tensor(np.asarray(a), dtype=dt, device=device)
    return dict(st=st, h=h, W=W, cu=dev(st.cu_seqlens, torch.int32), mask=dev(st.mask, torch.uint8),
                targets=dev(st.targets, torch.int32), rewards=dev(st.rewards, torch.float32),
                gid=dev(st.group_ids, torch.int32), old=dev(old, torch.float32), old_host=old)


def kernel_source_digest() -> str:
    """Digest of the code of the GEMM kernels (the roofline kernels), comments and blank lines
    left out: counter summaries taken from other code no longer describe them."""
    import re

    src = open(os.path.join(ROOT, "paper_2608_16798_amd", "csrc", "k_gemm.hip")).read()
    code = [re.sub(r"//.*$", "", l).rstrip() for l in src.splitlines()]
    h = hashlib.sha256("\n".join(l for l in code if l.strip()).encode())
    return h.hexdigest()[:16]


def read_traffic(kernel: str, workload: str, digest: str, launches_per_step=None):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter summary, if it was
    taken from the current kernel sources and (when given) with the same launches per step (else
    None: a per-launch average over another chunk loop does not describe this run's launches)."""
    path = os.path.join(PROFILES, f"{kernel}_{workload}_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_digest") != digest:
        return None
    if launches_per_step is not None and kv.get("launches_per_step") != str(int(launches_per_step)):
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def host_policy_tokens(st, exclusion: bool = True) -> int:
    """Trained tokens of a batch counted on the host from its structure (mask = 1, in rollouts with a
    group id >= 0 when `exclusion`): the bound a data pipeline that builds the masks knows before the
    call.  The log-prob forward has no exclusion (exclusion=False)."""
    import numpy as np

    lens = np.diff(np.asarray(st.cu_seqlens, dtype=np.int64))
    keep = np.repeat(np.asarray(st.group_ids) >= 0 if exclusion else np.ones(len(lens), bool), lens)
    return int((np.asarray(st.mask)[:keep.shape[0]].astype(bool) & keep).sum())


def cpu_baseline(cfg, inp, target_tokens: int, n_eff_full: int):
    """The fp64 oracle, as it stands, on the first rollouts of the same batch (>= target_tokens
    policy tokens): forward, loss terms, dhidden rows and their dW contribution."""
    import numpy as np

    import oracle as O

    st = inp["st"]
    cu = st.cu_seqlens
    keep_rollouts = 0
    n = 0
    while keep_rollouts < st.R and n < target_tokens:
        r = keep_rollouts
        n += int(st.mask[cu[r]:cu[r + 1]].sum())
        keep_rollouts += 1
    Nt = int(cu[keep_rollouts])
    h = inp["h"][:Nt].float().cpu().numpy()
    W = inp["W"].float().cpu().numpy()
    threads = None
    try:
        from threadpoolctl import threadpool_info

        threads = max((i.get("num_threads") or 0) for i in threadpool_info()) or None
    except Exception:
        pass
    t0 = time.perf_counter()
    out = O.pg_loss_fwd_bwd(h, W, st.targets[:Nt], st.mask[:Nt], cu[:keep_rollouts + 1], inp["old_host"][:Nt],
                            st.rewards[:keep_rollouts], st.group_ids[:keep_rollouts], eps_low=cfg.eps_low,
                            eps_high=cfg.eps_high, entropy_coef=cfg.entropy_coef)
    dt = time.perf_counter() - t0
    ntok = out["stats"]["n_policy_tokens"]
    affinity = sorted(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else []
    return {"value": ntok / dt, "unit": "policy tokens/s", "cores": threads or os.cpu_count(), "kind": "oracle",
            "sample": f"first {keep_rollouts} rollouts ({ntok} policy tokens, full V={cfg.V}, d={cfg.d}, "
                      f"fwd+loss+dhidden+dW contribution), fp64 NumPy, {dt:.1f} s",
            "seconds": dt, "blas_threads": threads, "os_cpu_count": os.cpu_count(),
            "affinity_cores": len(affinity), "affinity": _ranges(affinity),
            "full_config_s_extrapolated": n_eff_full * dt / max(1, ntok)}


def _ranges(cpus):
    """Compact text of a CPU list: 0-15,32-47."""
    out, i = [], 0
    while i < len(cpus):
        j = i
        while j + 1 < len(cpus) and cpus[j + 1] == cpus[j] + 1:
            j += 1
        out.append(str(cpus[i]) if i == j else f"{cpus[i]}-{cpus[j]}")
        i = j + 1
    return ",".join(out)


COPY_TAG = "neg"   # the calibration copy is torch.neg on fp32 (reads and writes its size once)
KERNEL_KIND = {"0": "fwd_lse_gemm", "1": "dh_gemm", "2": "dw_gemm"}


def _counter_rows(path):
    import csv
    import re

    per = {}
    for r in csv.DictReader(open(path)):
        name = r["Kernel_Name"]
        m = re.search(r"k_gemm<[^,]+, (\d)", name)
        kind = KERNEL_KIND.get(m.group(1)) if m else ("copy" if COPY_TAG in name else None)
        if kind is None:
            continue
        d = per.setdefault(kind, {})
        d[r["Dispatch_Id"]] = d.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    return per


def traffic_summary(fetch_csv, write_csv, workload, copy_mib, cmd_fetch, cmd_write):
    """Per-launch HBM bytes of the three GEMMs from FETCH_SIZE / WRITE_SIZE (KiB per dispatch),
    each scaled by known / measured for the calibration copy in the same run."""
    fetch, write = _counter_rows(fetch_csv), _counter_rows(write_csv)
    known_kib = copy_mib * 1024.0
    f_copy = max(fetch["copy"].values())
    w_copy = max(write["copy"].values())
    kf, kw = known_kib / f_copy, known_kib / w_copy
    digest = kernel_source_digest()
    paths = []
    for kind in KERNEL_KIND.values():
        if kind not in fetch or kind not in write:
            continue
        n = len(fetch[kind])
        fk = sum(fetch[kind].values()) / n
        wk = sum(write[kind].values()) / len(write[kind])
        hbm = (fk * kf + wk * kw) * 1024.0
        path = os.path.join(PROFILES, f"{kind}_{workload}_traffic.txt")
        with open(path, "w") as f:
            f.write(f"# HBM traffic of {kind} on the {workload} workload, one step, rocprofv3 counters\n")
            f.write(f"# fetch pass: {cmd_fetch}\n# write pass: {cmd_write}\n")
            f.write(f"# summary: python bench.py --traffic-summary <fetch csv> <write csv> --workload {workload} "
                    f"--calibrate-copy-mib {copy_mib}\n")
            f.write(f"launches_per_step: {n}\n")
            f.write(f"fetch_kib_per_launch_raw: {fk:.1f}\nwrite_kib_per_launch_raw: {wk:.1f}\n")
            f.write(f"copy_known_kib: {known_kib:.0f}\ncopy_fetch_kib: {f_copy:.1f}\ncopy_write_kib: {w_copy:.1f}\n")
            f.write(f"fetch_scale: {kf:.4f}\nwrite_scale: {kw:.4f}\n")
            f.write(f"hbm_bytes_per_launch: {hbm:.0f}\n")
            f.write(f"kernel_source_digest: {digest}\n")
        paths.append(path)
    return paths


N_XCD, N_SIMD = 8, 1024   # MI355X: GRBM_GUI_ACTIVE is summed over the XCDs; MFMA busy over the SIMDs


def occupancy_summary(counter_csv, title, cmd):
    """Shader clock and MFMA pipe occupancy of the three GEMMs from one rocprofv3 counter pass
    (GRBM_GUI_ACTIVE, SQ_VALU_MFMA_BUSY_CYCLES, SQ_WAVE_CYCLES, SQ_WAIT_ANY): clock = active cycles
    per XCD / dispatch time, occupancy = MFMA-busy cycles per SIMD / active cycles per XCD.  Launches
    shorter than 1 ms (chunks past the policy tokens) are left out."""
    import csv
    import re

    per = {}
    for r in csv.DictReader(open(counter_csv)):
        m = re.search(r"k_gemm<[^,]+, (\d)", r["Kernel_Name"])
        if not m:
            continue
        d = per.setdefault(KERNEL_KIND[m.group(1)], {}).setdefault(r["Dispatch_Id"], {})
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        d["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    out = [f"# {title}", f"# command: {cmd}",
           "# summary: python bench.py --occupancy-summary <counter_collection.csv> (launches >= 1 ms)",
           f"# clock = GRBM_GUI_ACTIVE / {N_XCD} / time; occupancy = SQ_VALU_MFMA_BUSY_CYCLES / {N_SIMD} / "
           f"(GRBM_GUI_ACTIVE / {N_XCD}); wait = SQ_WAIT_ANY / SQ_WAVE_CYCLES; executed FLOP = "
           f"SQ_INSTS_VALU_MFMA_MOPS_BF16 * 512 (all launches of the step)",
           f"{'kernel':14s} {'launches':>8s} {'avg_ms':>8s} {'clock_GHz':>9s} {'mfma_occ':>8s} {'wait':>6s} "
           f"{'exec_TFLOP':>10s}"]
    total_flop = 0.0
    for kind in GEMM_KINDS:
        allruns = list(per.get(kind, {}).values())
        flop = sum(d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) for d in allruns) * 512.0
        total_flop += flop
        runs = [d for d in allruns if d["ns"] >= 1_000_000 and "GRBM_GUI_ACTIVE" in d]
        if not runs:
            continue
        ns = sum(d["ns"] for d in runs)
        cyc = sum(d["GRBM_GUI_ACTIVE"] for d in runs) / N_XCD
        busy = sum(d["SQ_VALU_MFMA_BUSY_CYCLES"] for d in runs) / N_SIMD
        wait = sum(d["SQ_WAIT_ANY"] for d in runs) / max(1.0, sum(d["SQ_WAVE_CYCLES"] for d in runs))
        out.append(f"{kind:14s} {len(runs):8d} {ns / len(runs) / 1e6:8.2f} {cyc / ns:9.2f} {busy / cyc:8.3f} "
                   f"{wait:6.3f} {flop / 1e12:10.2f}")
    if total_flop > 0:
        out.append(f"executed_mfma_flop_per_step: {total_flop:.6e}")
    out.append(f"kernel_source_digest: {kernel_source_digest()}")
    return "\n".join(out) + "\n"


def read_occupancy(workload: str, digest: str):
    """(executed MFMA FLOP per step, {gemm: MFMA pipe occupancy}) from the committed counter summary of
    this workload, if it was taken from the current GEMM sources (else None)."""
    path = os.path.join(PROFILES, f"gemm_occupancy_{workload}.txt")
    if not os.path.exists(path):
        return None
    flop, occ, dig = None, {}, None
    for line in open(path):
        if line.startswith("executed_mfma_flop_per_step:"):
            flop = float(line.split(":", 1)[1])
        elif line.startswith("kernel_source_digest:"):
            dig = line.split(":", 1)[1].strip()
        else:
            f = line.split()
            if len(f) >= 5 and f[0] in GEMM_KINDS:
                occ[f[0]] = float(f[4])
    if dig != digest or flop is None:
        return None
    return flop, occ


HBM_KERNELS = ("k_dz", "k_dz_flagged", "k_gather", "k_target_logit", "k_hidden_t", "k_transpose_w", "k_zero_fill",
               "k_combine")


def hbm_kernel_summary(fetch_csv, write_csv, workload, copy_mib, cmd_fetch, cmd_write):
    """HBM bytes per step of the bandwidth-bound kernels (FETCH_SIZE / WRITE_SIZE scaled by the
    calibration copy, as for the GEMMs) against their algorithmic bytes per step."""
    import csv
    import re

    import numpy as np

    import workloads as WL

    import paper_2608_16798_amd as rlk

    cfg = WL.get_config(workload)
    st = WL.make_structure(cfg)
    n_eff = host_policy_tokens(st)
    # rows past the backward: those of zero-advantage rollouts when the surrogate is the only term
    n_grad = rlk.grad_token_hint(st.mask, st.cu_seqlens, st.rewards, st.group_ids) if cfg.entropy_coef == 0.0 else n_eff
    esz = 2 if cfg.dtype == "bf16" else 4
    vp = (cfg.V + 255) // 256 * 256
    # token-reference layout (bf16 without an entropy term): no explicit dz pass unless a chunk is
    # flagged, the gather writes h_c only, and the s-scaled h_c^T comes after the combine
    ref = cfg.dtype == "bf16" and cfg.entropy_coef == 0.0
    hrow = n_eff * cfg.d * esz
    alg = {"k_dz": 3 * n_grad * vp * esz, "k_dz_flagged": 0, "k_gather": (2 if ref else 3) * hrow,
           "k_target_logit": 2 * hrow, "k_hidden_t": 2 * n_grad * cfg.d * esz,
           "k_transpose_w": (cfg.V + vp) * cfg.d * esz,
           "k_zero_fill": (st.N - n_eff) * (cfg.d * esz + 8) + (n_eff - n_grad) * cfg.d * esz,
           "k_combine": n_eff * (12 * (vp // 256) + 40)}
    what = {"k_dz": "read q, write dz and dz^T (N_grad rows)",
            "k_dz_flagged": "dz of flagged chunks only; none expected here, every block exits at once",
            "k_gather": "read h rows, write h_c" + ("" if ref else " and h_c^T"),
            "k_target_logit": "read h_c rows and the target rows of W",
            "k_hidden_t": "read h_c, write the row-scaled h_c^T (N_grad rows)",
            "k_transpose_w": "read W, write W^T",
            "k_zero_fill": "zero untrained rows of dh, logp, entropy, and the dh rows past N_grad",
            "k_combine": "read the online-LSE partials, write per-token values"}

    def per_kernel(path):
        tot = {}
        for r in csv.DictReader(open(path)):
            m = re.search(r"rlk::\(anonymous namespace\)::(k_\w+)", r["Kernel_Name"])
            name = m.group(1) if m else ("copy" if COPY_TAG in r["Kernel_Name"] else None)
            if name in HBM_KERNELS or name == "copy":
                d = tot.setdefault(name, {})
                d[r["Dispatch_Id"]] = d.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
        return tot

    fetch, write = per_kernel(fetch_csv), per_kernel(write_csv)
    known_kib = copy_mib * 1024.0
    kf, kw = known_kib / max(fetch["copy"].values()), known_kib / max(write["copy"].values())
    path = os.path.join(PROFILES, f"hbm_kernels_{workload}_traffic.txt")
    with open(path, "w") as f:
        f.write(f"# HBM traffic of the bandwidth-bound kernels on the {workload} workload, one step, rocprofv3 "
                f"counters (N_eff = {n_eff}, N_grad = {n_grad})\n")
        f.write(f"# fetch pass: {cmd_fetch}\n# write pass: {cmd_write}\n")
        f.write(f"# summary: python bench.py --traffic-summary <fetch csv> <write csv> --workload {workload} "
                f"--calibrate-copy-mib {copy_mib}\n")
        f.write(f"# scales from the calibration copy: fetch {kf:.4f}, write {kw:.4f}\n")
        f.write(f"{'kernel':15s} {'launches':>8s} {'hbm_GB':>9s} {'alg_GB':>9s} {'ratio':>6s}  algorithmic bytes\n")
        for k in HBM_KERNELS:
            if k not in fetch or k not in write:
                continue
            hbm = (sum(fetch[k].values()) * kf + sum(write[k].values()) * kw) * 1024.0
            ratio = f"{hbm / alg[k]:6.3f}" if alg[k] else f"{'-':>6s}"
            f.write(f"{k:15s} {len(fetch[k]):8d} {hbm / 1e9:9.3f} {alg[k] / 1e9:9.3f} {ratio}  {what[k]}\n")
    return path


def stats_summary(stats_csv, title, cmd):
    """Text table of the rlk kernels from a rocprofv3 --stats kernel summary CSV."""
    import csv
    import re

    def short(n):
        m = re.search(r"k_gemm<(?:rlk::)?(\w+), (\d), (\w+), (\w+)>", n)
        if m:
            kind = ["fwd_lse", "dh", "dw"][int(m.group(2))]
            return f"k_gemm<{m.group(1)},{kind},store_q={m.group(3)},ktail={m.group(4)}>"
        m = re.search(r"rlk::\(anonymous namespace\)::(k_\w+)(<[^>(]*>)?", n)
        return (m.group(1) + (m.group(2) or "")) if m else None

    out = [f"# {title}", f"# command: {cmd}",
           "# summary: python bench.py --stats-summary <kernel_stats.csv> (rlk kernels only; microseconds)",
           f"{'kernel':58s} {'calls':>6s} {'total_us':>12s} {'avg_us':>10s} {'min_us':>10s} {'max_us':>10s} {'pct':>6s}"]
    for r in csv.DictReader(open(stats_csv)):
        k = short(r["Name"])
        if k:
            out.append(f"{k:58s} {int(r['Calls']):6d} {float(r['TotalDurationNs']) / 1e3:12.1f} "
                       f"{float(r['AverageNs']) / 1e3:10.1f} {float(r['MinNs']) / 1e3:10.1f} "
                       f"{float(r['MaxNs']) / 1e3:10.1f} {float(r['Percentage']):6.2f}")
    return "\n".join(out) + "\n"


def next_rows(cfg, inp, params, steps):
    """Timings of the adjacent paths at the workload's shape: the loss call with truncated
    importance sampling, and with the KL term as well (overheads over the plain call; a KL term
    gives zero-advantage rollouts a gradient, so that call runs the backward on all N_eff tokens);
    the PPO path's
    GAE, value loss and linear value head (time and achieved bandwidth on their algorithmic
    bytes); the host prefix-tree packer on a synthetic call log."""
    import numpy as np
    import torch

    import paper_2608_16798_amd as rlk

    st = inp["st"]
    N, R, d = st.N, st.R, cfg.d
    n_eff = host_policy_tokens(st)
    esz = 2 if cfg.dtype == "bf16" else 4
    dev = "cuda"
    g = torch.Generator(device=dev).manual_seed(cfg.seed + 4242)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    dh = torch.empty_like(inp["h"])
    dW = torch.empty(inp["W"].shape, dtype=torch.float32, device=dev)
    batch = rlk.make_batch(inp["h"], inp["W"], inp["cu"], max_policy_tokens=n_eff)
    pt = rlk.make_params(eps_low=params.eps_low, eps_high=params.eps_high, entropy_coef=params.entropy_coef,
                         tis_cap=2.0, grad_tokens=params.grad_tokens)
    pk = rlk.make_params(eps_low=params.eps_low, eps_high=params.eps_high, entropy_coef=params.entropy_coef,
                         tis_cap=2.0, kl_coef=0.05)
    ws = rlk.alloc_workspace(max(rlk.workspace_size(batch, p) for p in (params, pt, pk)), dev)
    rollout = inp["old"] + 0.1 * torch.randn(N, generator=g, device=dev)
    ref = inp["old"] + 0.2 * torch.randn(N, generator=g, device=dev)

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    def loss_call(p, **kw):
        return lambda: rlk.pg_loss_fwd_bwd(inp["h"], inp["W"], inp["targets"], inp["mask"], inp["cu"], inp["old"],
                                           inp["rewards"], inp["gid"], p, loss=loss, dhidden=dh, dW=dW, ws=ws,
                                           max_policy_tokens=n_eff, **kw)

    out = {"workload": cfg.name, "N": N, "N_eff": n_eff, "grad_tokens": params.grad_tokens}
    base = timed(loss_call(params), steps)
    tt = timed(loss_call(pt, rollout_logp=rollout), steps)
    tk = timed(loss_call(pk, rollout_logp=rollout, ref_logp=ref), steps)
    out["loss_call_ms"] = round(base, 3)
    out["loss_call_tis_ms"] = round(tt, 3)
    out["loss_call_tis_kl_ms"] = round(tk, 3)
    # PPO path
    values = torch.randn(N, generator=g, device=dev)
    adv = torch.empty(N, dtype=torch.float32, device=dev)
    ret = torch.empty(N, dtype=torch.float32, device=dev)
    t_gae = timed(lambda: rlk.gae(values, inp["rewards"], inp["mask"], inp["cu"], inp["gid"], adv=adv, returns=ret), 20)
    vws = rlk.alloc_workspace(rlk.value_workspace_size(R), dev)
    vl = torch.empty(1, dtype=torch.float32, device=dev)
    dv = torch.empty(N, dtype=torch.float32, device=dev)
    t_vl = timed(lambda: rlk.value_loss(values, ret, inp["mask"], inp["cu"], inp["gid"], loss=vl, dvalues=dv,
                                        ws=vws), 20)
    w_v = (0.02 * torch.randn(d, generator=g, device=dev)).to(inp["h"].dtype)
    vals = torch.empty(N, dtype=torch.float32, device=dev)
    t_hf = timed(lambda: rlk.value_head_fwd(inp["h"], w_v, 0.1, inp["mask"], inp["cu"], inp["gid"], values=vals), 20)
    hws = rlk.alloc_workspace(rlk.value_head_workspace_size(inp["h"], inp["cu"]), dev)
    dhv = torch.empty_like(inp["h"])
    dwv = torch.empty(d, dtype=torch.float32, device=dev)
    dbv = torch.empty(1, dtype=torch.float32, device=dev)
    t_hb = timed(lambda: rlk.value_head_bwd(inp["h"], w_v, inp["mask"], inp["cu"], inp["gid"], dv, dhidden=dhv,
                                            dw_v=dwv, db_v=dbv, ws=hws), 20)
    rate = lambda b, ms: round(b / (ms * 1e-3) / 1e12, 2)
    out["gae_ms"] = round(t_gae, 4)
    out["value_loss_ms"] = round(t_vl, 4)
    out["value_head_fwd_ms"] = round(t_hf, 4)
    out["value_head_fwd_TBps"] = rate(n_eff * d * esz, t_hf)          # read the policy rows
    out["value_head_bwd_ms"] = round(t_hb, 4)
    out["value_head_bwd_TBps"] = rate(N * d * esz + n_eff * d * esz, t_hb)  # read policy rows, write all rows
    # group-relative advantages (sort + segmented reduction) at the batch's R and at the largest
    # supported rollout count, 16384 rollouts in groups of 8 under shuffled keys
    adv_r = torch.empty(R, dtype=torch.float32, device=dev)
    aws = rlk.alloc_workspace(rlk.advantage_workspace_size(R), dev)
    out["advantage_ms"] = round(timed(lambda: rlk.group_advantage(inp["rewards"], inp["gid"], 1e-6, adv=adv_r, ws=aws),
                                      20), 4)
    Rm = 16384
    rng_a = np.random.default_rng(cfg.seed + 78)
    gid_m = torch.as_tensor(rng_a.permutation(np.repeat(np.arange(Rm // 8), 8)).astype(np.int32) * 7 + 3, device=dev)
    rew_m = torch.as_tensor(rng_a.random(Rm).astype(np.float32), device=dev)
    adv_m = torch.empty(Rm, dtype=torch.float32, device=dev)
    aws_m = rlk.alloc_workspace(rlk.advantage_workspace_size(Rm), dev)
    out["advantage_16384_rollouts_ms"] = round(timed(lambda: rlk.group_advantage(rew_m, gid_m, 1e-6, adv=adv_m, ws=aws_m),
                                                     20), 4)
    # host prefix-tree packer: 128 rollouts of 8 calls; each call's context is the previous history
    # (prompt, responses, tool observations), and every fourth rollout repeats one call
    rng = np.random.default_rng(cfg.seed + 77)
    calls_per_rollout, n_tok = [], 0
    for r in range(128):
        hist = list(rng.integers(0, cfg.V, 512))
        calls = []
        for c in range(8):
            resp = list(rng.integers(0, cfg.V, 256))
            calls.append((np.asarray(hist, dtype=np.int32), np.asarray(resp, dtype=np.int32)))
            n_tok += len(hist) + len(resp)
            if r % 4 == 0 and c == 3:
                calls.append(calls[-1])
                n_tok += len(hist) + len(resp)
            hist = hist + resp + list(rng.integers(0, cfg.V, 64))
        calls_per_rollout.append(calls)
    t0 = time.perf_counter()
    packed = rlk.tree_pack(calls_per_rollout)
    dt = time.perf_counter() - t0
    out["tree_pack_calls_tokens"] = n_tok
    out["tree_pack_positions"] = int(len(packed["token"]))
    out["tree_pack_rows"] = int(len(packed["row_target"]))
    out["tree_pack_s"] = round(dt, 4)
    out["tree_pack_input_tokens_per_s"] = round(n_tok / dt, 1)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="qwen8b_bf16")
    ap.add_argument("--group-share", type=int, default=1,
                    help="keep 1/K of the workload's groups: one GPU's share of a K-GPU data-parallel step")
    ap.add_argument("--chunk-rows", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--next-rows", action="store_true",
                    help="time the adjacent paths (TIS/KL options, GAE, value loss, value head, tree packing) and exit")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step as a HIP graph and replay it (launch-bound workloads); no per-kernel events")
    ap.add_argument("--cpu-tokens", type=int, default=1024)
    ap.add_argument("--no-policy-bound", action="store_true",
                    help="do not pass the host-known count of policy tokens (max_policy_tokens = 0: the chunk loop "
                         "covers all N rows)")
    ap.add_argument("--no-grad-hint", action="store_true",
                    help="do not pass the host count of tokens in groups of unequal rewards (grad_tokens = 0)")
    ap.add_argument("--logprob-only", action="store_true",
                    help="time rlk_logprob_fwd alone (the pi_old forward pass, 2 N_eff V d FLOP per call)")
    ap.add_argument("--no-kernel-events", action="store_true",
                    help="time the steps without per-kernel HIP events (roofline then null)")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="run a plain device copy of this many MiB first (counter calibration)")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/<kernel>_<workload>_traffic.txt from two counter runs and exit")
    ap.add_argument("--pmc-commands", nargs=2, default=("", ""), help=argparse.SUPPRESS)
    ap.add_argument("--stats-summary", nargs=3, metavar=("STATS_CSV", "TITLE", "COMMAND"),
                    help="print a text table of the rlk kernels from a rocprofv3 --stats CSV and exit")
    ap.add_argument("--occupancy-summary", nargs=3, metavar=("COUNTER_CSV", "TITLE", "COMMAND"),
                    help="print shader clock and MFMA occupancy of the GEMMs from a rocprofv3 counter CSV and exit")
    args = ap.parse_args()

    if args.occupancy_summary:
        sys.stdout.write(occupancy_summary(*args.occupancy_summary))
        return

    if args.stats_summary:
        sys.stdout.write(stats_summary(*args.stats_summary))
        return

    if args.traffic_summary:
        if args.calibrate_copy_mib <= 0:
            raise SystemExit("--traffic-summary needs the --calibrate-copy-mib size the runs used")
        for p in traffic_summary(*args.traffic_summary, args.workload, args.calibrate_copy_mib, *args.pmc_commands):
            print(p)
        print(hbm_kernel_summary(*args.traffic_summary, args.workload, args.calibrate_copy_mib, *args.pmc_commands))
        return

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: this build has no multi-GPU path (--gpus {args.gpus} requested)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2608_16798_amd as rlk
    import workloads as WL

    if not os.path.exists(rlk.LIB_PATH):
        from paper_2608_16798_amd.build import build

        build(verbose=False)
    rlk.load_library()
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    torch.cuda.set_device(0)

    cfg = WL.get_config(args.workload)
    if args.group_share > 1:
        if cfg.groups % args.group_share:
            raise SystemExit(f"{cfg.name} has {cfg.groups} groups, not divisible by {args.group_share}")
        cfg = cfg.with_(name=f"{cfg.name}/{args.group_share}", groups=cfg.groups // args.group_share)
    log(f"[bench] building {cfg.name} inputs")
    inp = build_inputs(cfg)
    st = inp["st"]
    N, R = st.N, st.R
    dev = "cuda"
    params = rlk.make_params(eps_low=cfg.eps_low, eps_high=cfg.eps_high, entropy_coef=cfg.entropy_coef,
                             chunk_rows=args.chunk_rows)
    bound = 0 if args.no_policy_bound else host_policy_tokens(st, exclusion=not args.logprob_only)
    if bound and not args.logprob_only and not args.no_grad_hint:
        params.grad_tokens = rlk.grad_token_hint(st.mask, st.cu_seqlens, st.rewards, st.group_ids)
    batch = rlk.make_batch(inp["h"], inp["W"], inp["cu"], max_policy_tokens=bound)
    ws = rlk.alloc_workspace(rlk.workspace_size(batch, None if args.logprob_only else params), dev)
    ws_adv = rlk.alloc_workspace(rlk.advantage_workspace_size(R), dev)
    adv = torch.empty(R, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    dh = torch.empty_like(inp["h"])
    dW = torch.empty(inp["W"].shape, dtype=torch.float32, device=dev)
    stats = rlk.stats_buffer(dev)
    logp = torch.empty(N, dtype=torch.float32, device=dev)

    def step():
        # both calls go to torch's current stream (the capture stream while a graph is recorded)
        rlk.group_advantage(inp["rewards"], inp["gid"], params.adv_eps, adv=adv, ws=ws_adv)
        rlk.pg_loss_fwd_bwd(inp["h"], inp["W"], inp["targets"], inp["mask"], inp["cu"], inp["old"], inp["rewards"],
                            inp["gid"], params, loss=loss, dhidden=dh, dW=dW, stats=stats, ws=ws,
                            max_policy_tokens=bound)

    def logprob_step():
        rlk.logprob_fwd(inp["h"], inp["W"], inp["targets"], inp["mask"], inp["cu"], logp=logp, ws=ws,
                        max_policy_tokens=bound)

    if args.logprob_only:
        step = logprob_step

    if args.calibrate_copy_mib > 0:
        n = args.calibrate_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)   # reads and writes calibrate_copy_mib MiB once
        torch.cuda.synchronize()
        del src, dst
    log(f"[bench] warmup {args.warmup} step(s), N={N} R={R} ws={ws.numel() / 2**30:.1f} GiB")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if rlk.check_status(ws) != 0:
        raise SystemExit("device data error in the benchmark batch")
    n_eff = host_policy_tokens(st, exclusion=not args.logprob_only)
    if not args.logprob_only and args.warmup > 0:
        s = rlk.stats_from_tensor(stats)
        if int(s["n_policy_tokens"]) != n_eff:
            raise SystemExit(f"policy tokens: device {int(s['n_policy_tokens'])}, host {n_eff}")

    if args.next_rows:
        print(json.dumps(next_rows(cfg, inp, params, args.steps)), flush=True)
        return

    run = step
    if args.graph:
        # one step captured as a HIP graph (the library enqueues kernel launches only), replayed per step
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        run = graph.replay
        log("[bench] step captured as a graph")
    log(f"[bench] timing {args.steps} step(s)")
    use_events = not args.no_kernel_events and not args.graph
    # per-step events on the stream the library launches on (torch's current stream)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    if use_events:
        rlk.profile_begin()   # creates its event pool here, outside the timed region
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(args.steps):
        run()
        ev[i + 1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    kern = rlk.profile_end() if use_events else {}
    step_ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]
    ms_per_step = float(np.median(step_ms))
    value = n_eff / (ms_per_step / 1e3)
    # Algorithmic MFMA work: 2 V d per trained token for the forward, and 2 V d for each gradient GEMM
    # per token that carries a surrogate gradient (the device's count: without an entropy term, a KL
    # term or per-token advantages, the tokens of zero-advantage rollouts skip the backward GEMMs).
    n_grad = n_eff
    if not args.logprob_only:
        n_grad = int(rlk.stats_from_tensor(stats)["n_grad_tokens"])
    alg_flops = 2.0 * (n_eff if args.logprob_only else n_eff + 2 * n_grad) * cfg.V * cfg.d
    peak = PEAK_BF16 if cfg.dtype == "bf16" else PEAK_FP32_MFMA
    mfma_frac = alg_flops / (ms_per_step / 1e3) / peak
    log(f"[bench] {ms_per_step:.2f} ms/step (median; mean {np.mean(step_ms):.2f}, wall {(t1 - t0) * 1e3 / args.steps:.2f}), "
        f"{value:.0f} policy tokens/s, {100 * mfma_frac:.1f}% of MFMA peak")

    roofline = None
    per_kernel = {}
    if kern:
        for k, (ms, cnt) in sorted(kern.items(), key=lambda kv: -kv[1][0]):
            per_kernel[k] = {"ms_per_step": round(ms / args.steps, 4), "launches_per_step": cnt // args.steps}
        dom = max(GEMM_KINDS, key=lambda k: kern.get(k, (0.0, 1))[0])
        ms, cnt = kern[dom]
        avg_ms = ms / cnt
        flops_per_launch = 2.0 * (n_eff if dom == "fwd_lse_gemm" else n_grad) * cfg.V * cfg.d * args.steps / cnt
        achieved = flops_per_launch / (avg_ms / 1e3) / 1e12
        digest = kernel_source_digest()
        traffic = None if args.logprob_only else read_traffic(dom, cfg.name, digest, cnt // args.steps)
        roofline = {"kernel": dom, "bound": "mfma", "achieved": round(achieved, 1), "peak": peak / 1e12,
                    "unit": "TFLOP/s", "frac": round(achieved * 1e12 / peak, 4), "traffic": traffic,
                    "avg_launch_ms": round(avg_ms, 3), "launches": cnt,
                    "flops_per_launch": flops_per_launch, "kernel_source_digest": digest}
        log("[bench] per-kernel ms/step: " + ", ".join(f"{k}={v['ms_per_step']}" for k, v in per_kernel.items()))

    executed = None
    occ = None if (args.logprob_only or args.graph or args.group_share > 1) else read_occupancy(cfg.name, kernel_source_digest())
    if occ is not None:
        flop, pipe = occ
        executed = {"mfma_flop_per_step": flop, "pct_of_peak": round(100 * flop / (ms_per_step / 1e3) / peak, 2),
                    "mfma_pipe_busy": pipe, "source": f"profiles/gemm_occupancy_{cfg.name}.txt"}

    cpu = None
    if not args.no_cpu_baseline:
        log(f"[bench] timing the fp64 oracle on >= {args.cpu_tokens} policy tokens")
        cpu = cpu_baseline(cfg, inp, args.cpu_tokens, n_eff)
        log(f"[bench] oracle {cpu['value']:.1f} policy tokens/s in {cpu['seconds']:.1f} s")

    dz_chunks = None
    if not args.logprob_only:
        s = rlk.stats_from_tensor(stats)
        dz_chunks = {"explicit_dz": int(s["n_dz_chunks"]), "chunks": int(s["n_chunks"])}

    metric = METRIC if not args.logprob_only else "policy tokens/sec for the logprob forward (pi_old pass); % of bf16 MFMA peak"
    out = {
        "metric": metric, "value": round(value, 1), "unit": "policy tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic",
        "config": dict(WL.configs.describe(cfg, N), N_eff=n_eff,
                       **({} if args.logprob_only else {"N_grad": n_grad}), chunk_rows=args.chunk_rows or "auto",
                       max_policy_tokens=bound, **({} if args.logprob_only else {"grad_tokens": params.grad_tokens}),
                       **({"graph": True} if args.graph else {}),
                       **({"call": "rlk_logprob_fwd"} if args.logprob_only else {})),
        "timing": {"ms_per_step_median": round(ms_per_step, 3), "ms_per_step_mean": round(float(np.mean(step_ms)), 3),
                   "ms_per_step_min": round(float(np.min(step_ms)), 3), "ms_per_step_max": round(float(np.max(step_ms)), 3),
                   "ms_wall_per_step": round((t1 - t0) * 1e3 / args.steps, 3),
                   "per_kernel_events": use_events, "dz_chunks": dz_chunks},
        "mfma_pct_of_peak": round(100 * mfma_frac, 2),
        "flop_accounting": {"alg_mfma_flop_per_step": alg_flops, "forward_tokens": n_eff,
                            "backward_tokens": n_grad,
                            "pct_of_peak_at_6_N_eff_V_d": round(100 * (2.0 * (1 if args.logprob_only else 3) * n_eff
                                                                       * cfg.V * cfg.d) / (ms_per_step / 1e3) / peak, 2)},
        "executed_mfma_pct": executed["pct_of_peak"] if executed else None, "executed_mfma": executed,
        "roofline": roofline, "cpu_baseline": cpu, "kernels": per_kernel,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
