"""Load-balance metrics of a schedule.

* Effective workload of a step (Eq. 2): the maximum over devices of the
  step's combined workload.
* Utilization (Eq. 3) with steps in place of layers (without EasyBalance the
  two coincide): u = sum_i sum_d W_i,d / (D * sum_i max_d W_i,d).
  The paper reports 1 - u ("under-utilization"); max/mean = 1/u.
* Per step, Section 5.3 contrasts sum_j max(w_j) ("maximum workload", what
  running the step's workloads one after another would cost) with
  max(sum_j w_j) ("effective workload", the combined cost).  Worst-case
  safety (Section 4.1): the latter never exceeds the former.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np


def step_workload(loads: np.ndarray, step) -> np.ndarray:
    loads = np.asarray(loads, np.int64)
    W = np.zeros(loads.shape[-1], np.int64)
    for j, l in step:
        W += loads[j, l]
    return W


def utilization(loads: np.ndarray, steps) -> Fraction:
    loads = np.asarray(loads, np.int64)
    D = loads.shape[-1]
    total = sum(int(step_workload(loads, s).sum()) for s in steps)
    eff = sum(int(step_workload(loads, s).max()) for s in steps)
    return Fraction(1) if eff == 0 else Fraction(total, D * eff)


def max_over_mean(loads: np.ndarray, steps) -> Fraction:
    return 1 / utilization(loads, steps)


def per_step_max_vs_effective(loads: np.ndarray, steps) -> list[tuple[int, int]]:
    """[(sum_j max w_j, max sum_j w_j)] per step."""
    loads = np.asarray(loads, np.int64)
    out = []
    for s in steps:
        mx = sum(int(loads[j, l].max()) for j, l in s)
        out.append((mx, int(step_workload(loads, s).max())))
    return out


def summary(loads: np.ndarray, steps) -> dict:
    u = utilization(loads, steps)
    return {"steps": len(steps), "u": float(u), "under_util": float(1 - u),
            "max_over_mean": float(1 / u),
            "effective_total": sum(e for _, e in per_step_max_vs_effective(loads, steps))}
