"""Load-balance metrics of executed steps (product side).

Given the per-device workload W_i of every executed step i (Section 2.3,
D virtual devices):
  effective workload of a step   max_d W_i,d                        (Eq. 2)
  utilization                    u = sum_i sum_d W_i,d / (D sum_i max_d W_i,d)  (Eq. 3,
                                 summed over steps instead of layers)
  under-utilization              1 - u  (the paper's reported figure)
  max/mean                       1 / u
"""
from __future__ import annotations

import numpy as np


def utilization(step_loads) -> float:
    W = np.asarray([np.asarray(w, np.int64) for w in step_loads])
    if W.size == 0:
        return 1.0
    eff = int(W.max(axis=1).sum())
    return 1.0 if eff == 0 else float(W.sum()) / (W.shape[1] * eff)


def summary(step_loads) -> dict:
    u = utilization(step_loads)
    return {"steps": len(step_loads), "max_over_mean": 1.0 / u, "idle_fraction": 1.0 - u}


def lockstep_loads(layer_loads: np.ndarray) -> list:
    """Per-layer baseline: step l combines every micro-batch at layer l."""
    return [layer_loads[:, l].sum(axis=0) for l in range(layer_loads.shape[1])]


def separate_loads(layer_loads: np.ndarray) -> list:
    """No combination: every (micro-batch, layer) workload is its own step."""
    N, L, _ = layer_loads.shape
    return [layer_loads[j, l] for l in range(L) for j in range(N)]
