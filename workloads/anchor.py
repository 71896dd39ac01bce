"""Placement of old log-probs for batches too large for an exact reference pass.

Old log-probs only decide where the importance ratios fall (near 1, spread by
the configured noise); both implementations consume the same stored bytes.
For an LM head with i.i.d. N(0, s^2) weights, the log-partition of a hidden
state h is close to ln V + s^2 |h|^2 / 2 (the log of the expected sum of V
log-normal terms; relative spread ~ sqrt((e^{s^2|h|^2} - 1) / V)), so

    anchor_t = W[y_t] . h_t - ln V - s^2 |h_t|^2 / 2

lands within a few hundredths of the true log-prob on the Gaussian workloads.
This is an input heuristic, not a log-softmax: neither the oracle nor the GPU
path imports it.
"""
from __future__ import annotations

import math

import numpy as np


def gaussian_anchor(h, W, targets, w_std: float, rows: int = 32768) -> np.ndarray:
    import torch

    N = h.shape[0]
    V = W.shape[0]
    out = torch.empty(N, dtype=torch.float32, device=h.device)
    tg = torch.as_tensor(np.asarray(targets), dtype=torch.int64, device=h.device)
    for r0 in range(0, N, rows):
        r1 = min(N, r0 + rows)
        hb = h[r0:r1].float()
        wy = W.index_select(0, tg[r0:r1]).float()
        zy = (hb * wy).sum(dim=1)
        hn = (hb * hb).sum(dim=1)
        out[r0:r1] = zy - math.log(V) - 0.5 * (w_std ** 2) * hn
    return out.cpu().numpy()
