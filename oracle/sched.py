"""Algorithm 1 (EasyBalance) and its scheduling policies, plain Python.

Algorithm 1 keeps, for every micro-batch j, the layer l_j it is waiting at and
a pool S of unfinished micro-batches.  Each step picks RunSet = Schedule(S, m),
runs the MoE work of every micro-batch in RunSet jointly (each at its own
layer), advances l_j for those micro-batches and drops the ones that reached
the last layer.  Unpicked micro-batches are deferred.

Policies (the workload of micro-batch j in a step is its per-device load
vector w_j at layer l_j, Section 2.3):

* MaxUtil (Section 4.2): the subset of the pool with at least m members that
  maximises the utilization U of its combined workload; if the pool holds
  fewer than m micro-batches all of them run.
* CumUtil (Section 5.2): scan the pool in id order, the first one is always
  taken, each next one joins iff it strictly raises U of the chosen set.
* DiffPeak (Section 5.2): scan in id order, the first one is always taken,
  each next one joins iff its peak device is not a peak device of any member
  already chosen.

U of a combined workload W in Z^D is Eq. (3) restricted to one step:
U = sum_d W_d / (D * max_d W_d).

Readings where the paper is silent:
* U of an all-zero workload is 1.
* MaxUtil ties: higher U, then more members (more progress), then the
  lexicographically smallest ascending id list.  Comparisons are exact
  (integer cross-multiplication), so every implementation picks the same set.
* CumUtil and DiffPeak also respect m: if their pass picks fewer than
  min(m, |S|) members, the remaining ids are added in ascending order.
* DiffPeak's peak device is the lowest device index among the maxima.
"""
from __future__ import annotations

import itertools

import numpy as np

MAXUTIL, CUMUTIL, DIFFPEAK = 0, 1, 2
POLICY_NAMES = {MAXUTIL: "maxutil", CUMUTIL: "cumutil", DIFFPEAK: "diffpeak"}


def util_fraction(W, D: int) -> tuple[int, int]:
    """U as an exact (numerator, denominator) pair of Python ints."""
    W = [int(v) for v in W]
    mx = max(W) if W else 0
    if mx == 0:
        return 1, 1
    return sum(W), D * mx


def util_greater(u1: tuple[int, int], u2: tuple[int, int]) -> bool:
    return u1[0] * u2[1] > u2[0] * u1[1]


def _combined(members, loads) -> list[int]:
    D = len(next(iter(loads.values())))
    W = [0] * D
    for j in members:
        for d, v in enumerate(loads[j]):
            W[d] += int(v)
    return W


def maxutil(pool: list[int], loads: dict, D: int, m: int) -> tuple[int, ...]:
    need = min(m, len(pool))
    best, best_u = None, None
    for size in range(need, len(pool) + 1):
        for R in itertools.combinations(sorted(pool), size):
            u = util_fraction(_combined(R, loads), D)
            if best is None:
                best, best_u = R, u
                continue
            if util_greater(u, best_u):
                best, best_u = R, u
            elif not util_greater(best_u, u):          # equal U
                if len(R) > len(best) or (len(R) == len(best) and R < best):
                    best, best_u = R, u
    return tuple(best) if best is not None else ()


def _pad(chosen: list[int], pool: list[int], need: int) -> tuple[int, ...]:
    for j in sorted(pool):
        if len(chosen) >= need:
            break
        if j not in chosen:
            chosen.append(j)
    return tuple(sorted(chosen))


def cumutil(pool: list[int], loads: dict, D: int, m: int) -> tuple[int, ...]:
    pool = sorted(pool)
    if not pool:
        return ()
    chosen = [pool[0]]
    for j in pool[1:]:
        if util_greater(util_fraction(_combined(chosen + [j], loads), D),
                        util_fraction(_combined(chosen, loads), D)):
            chosen.append(j)
    return _pad(chosen, pool, min(m, len(pool)))


def peak_device(w) -> int:
    w = [int(v) for v in w]
    return w.index(max(w))


def diffpeak(pool: list[int], loads: dict, D: int, m: int) -> tuple[int, ...]:
    pool = sorted(pool)
    if not pool:
        return ()
    chosen = [pool[0]]
    peaks = {peak_device(loads[pool[0]])}
    for j in pool[1:]:
        p = peak_device(loads[j])
        if p not in peaks:
            chosen.append(j)
            peaks.add(p)
    return _pad(chosen, pool, min(m, len(pool)))


POLICIES = {MAXUTIL: maxutil, CUMUTIL: cumutil, DIFFPEAK: diffpeak}


def schedule(pool, loads, D, m, policy=MAXUTIL) -> tuple[int, ...]:
    return POLICIES[policy](list(pool), loads, D, m)


def run_algorithm1(loads: np.ndarray, m: int, policy: int = MAXUTIL) -> list[list[tuple[int, int]]]:
    """Replay Algorithm 1 on a recorded load tensor loads[j][l][d].

    Returns the steps; step i lists (j, l_j) for every micro-batch in RunSet_i,
    in ascending j.
    """
    loads = np.asarray(loads, np.int64)
    N, L, D = loads.shape
    layer = [0] * N
    pool = list(range(N))
    steps = []
    while pool:
        cur = {j: loads[j, layer[j]] for j in pool}
        R = schedule(pool, cur, D, m, policy)
        assert len(R) >= 1
        steps.append([(j, layer[j]) for j in R])
        for j in R:
            layer[j] += 1
        pool = [j for j in pool if layer[j] < L]
    return steps


def lockstep_steps(N: int, L: int) -> list[list[tuple[int, int]]]:
    """Per-layer baseline: step l runs every micro-batch at layer l."""
    return [[(j, l) for j in range(N)] for l in range(L)]


def separate_steps(N: int, L: int) -> list[list[tuple[int, int]]]:
    """No combination at all: every (j, l) workload is its own step."""
    return [[(j, l)] for l in range(L) for j in range(N)]
