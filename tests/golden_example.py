"""Reader of the hand-derived worked example in tests/golden/worked_example_clip.json.

Every value in the fixture is an exact closed form (a log, a ratio of small integers); this
module evaluates those expressions with the math module only and lays the instance out as
arrays.  It holds none of the method's arithmetic."""
from __future__ import annotations

import json
import math
import os

import numpy as np

PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "worked_example_clip.json")


def value(expr: str) -> float:
    return float(eval(expr, {"__builtins__": {}}, {"log": math.log}))


def load():
    with open(PATH) as f:
        ex = json.load(f)
    inp = ex["inputs"]
    d = inp["d"]
    N = len(inp["targets"])
    h = np.zeros((N, d))
    for t, row in enumerate(inp["h"]):
        h[t, :len(row)] = [value(x) for x in row]
    W = np.zeros((2, d))
    W[0, 0] = value(inp["W_row0_col0"])
    out = dict(
        h=h, W=W, targets=np.array(inp["targets"], dtype=np.int64), mask=np.array(inp["mask"], dtype=np.uint8),
        cu_seqlens=np.array(inp["cu_seqlens"], dtype=np.int64), rewards=np.array(inp["rewards"]),
        group_ids=np.array(inp["group_ids"], dtype=np.int64), eps_low=inp["eps_low"], eps_high=inp["eps_high"],
        adv_eps=inp["adv_eps"], logp=[value(x) for x in ex["logp"]], entropy=[value(x) for x in ex["entropy"]],
        cases={})
    for name, c in ex["cases"].items():
        dh = np.zeros((N, d))
        dh[:, 0] = [value(x) for x in c["dh_col0"]]
        dW = np.zeros((2, d))
        dW[:, :2] = [[value(x) for x in row] for row in c["dW"]]
        out["cases"][name] = dict(old_logp=np.array([value(x) for x in c["old_logp"]]), loss=value(c["loss"]),
                                  dh=dh, dW=dW)
    return out
