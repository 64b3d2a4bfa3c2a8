"""Pins of oracle.sched / oracle.metrics (Algorithm 1, MaxUtil of Section 4.2,
CumUtil / DiffPeak of Section 5.2, Eqs. 2-3): hand-worked examples, an
independent brute force over subsets with exact fractions, and the invariants
the paper states (losslessness, per-micro-batch order, worst-case safety)."""
import functools
import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import metrics, sched

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "schedule_examples.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _golden(), ids=lambda c: c["name"])
def test_hand_worked_schedules(case):
    loads = {j: w for j, w in enumerate(case["loads"])}
    pool = list(range(len(case["loads"])))
    got = sched.schedule(pool, loads, case["D"], case["m"],
                         {"maxutil": sched.MAXUTIL, "cumutil": sched.CUMUTIL,
                          "diffpeak": sched.DIFFPEAK}[case["policy"]])
    assert list(got) == case["runset"]


def _brute_maxutil(pool, loads, D, m):
    """All subsets with >= min(m, |pool|) members, U as a Fraction, best by
    (U, size, lexicographically smallest)."""
    need = min(m, len(pool))
    cands = []
    for size in range(need, len(pool) + 1):
        for R in itertools.combinations(pool, size):
            W = np.sum([loads[j] for j in R], axis=0)
            U = Fraction(1) if W.max() == 0 else Fraction(int(W.sum()), D * int(W.max()))
            cands.append((U, size, tuple(-j for j in R), R))
    return max(cands)[3]


def test_maxutil_matches_brute_force_on_random_pools():
    rng = np.random.default_rng(11)
    for trial in range(4000):
        n = int(rng.integers(1, 7))
        D = int(rng.integers(1, 5))
        m = int(rng.integers(1, n + 2))
        pool = sorted(rng.choice(12, size=n, replace=False).tolist())
        hi = int(rng.choice([2, 4, 50]))       # small ranges force many exact ties
        loads = {j: rng.integers(0, hi, size=D).tolist() for j in pool}
        assert sched.maxutil(pool, loads, D, m) == _brute_maxutil(pool, loads, D, m), (pool, loads, D, m)


def test_cumutil_hand():
    loads = {0: [3, 1], 1: [1, 3], 2: [2, 2], 3: [3, 1]}
    assert sched.cumutil([0, 1, 2, 3], loads, 2, 1) == (0, 1)
    assert sched.cumutil([0, 1, 2, 3], loads, 2, 3) == (0, 1, 2)      # padded in id order
    assert sched.cumutil([2], loads, 2, 3) == (2,)


def test_diffpeak_hand():
    loads = {0: [3, 1, 0], 1: [5, 1, 0], 2: [0, 4, 4], 3: [1, 1, 2], 4: [2, 2, 2]}
    # peaks: 0->0, 1->0 (taken), 2->1 (lowest of the tie), 3->2, 4->0
    assert sched.diffpeak([0, 1, 2, 3, 4], loads, 3, 1) == (0, 2, 3)
    assert sched.diffpeak([0, 1, 2, 3, 4], loads, 3, 4) == (0, 1, 2, 3)
    assert sched.diffpeak([1, 4], loads, 3, 1) == (1,)


def _random_loads(rng, N, L, D, hi=20):
    return rng.integers(0, hi, size=(N, L, D))


@pytest.mark.parametrize("policy", [sched.MAXUTIL, sched.CUMUTIL, sched.DIFFPEAK])
def test_algorithm1_invariants(policy):
    rng = np.random.default_rng(12 + policy)
    for trial in range(300):
        N = int(rng.integers(1, 7))
        L = int(rng.integers(1, 6))
        D = int(rng.integers(1, 6))
        m = int(rng.integers(1, N + 1))
        loads = _random_loads(rng, N, L, D)
        steps = sched.run_algorithm1(loads, m, policy)
        executed = [p for s in steps for p in s]
        # exactly once
        assert sorted(executed) == [(j, l) for j in range(N) for l in range(L)]
        # per-micro-batch order and one layer per step
        for j in range(N):
            seq = [l for s in steps for (jj, l) in s if jj == j]
            assert seq == list(range(L))
        for s in steps:
            js = [j for j, _ in s]
            assert js == sorted(set(js))
        # termination bound and the m rule
        assert len(steps) <= N * L
        # worst-case safety (Section 4.1): sum_i max W_i <= sum_{j,l} max w_jl
        eff = sum(int(metrics.step_workload(loads, s).max()) for s in steps)
        assert eff <= int(loads.max(axis=-1).sum())
        for mx, ef in metrics.per_step_max_vs_effective(loads, steps):
            assert ef <= mx


def test_m_rule_every_step():
    rng = np.random.default_rng(13)
    for trial in range(300):
        N, L, D = int(rng.integers(1, 7)), int(rng.integers(1, 5)), int(rng.integers(1, 5))
        m = int(rng.integers(1, N + 1))
        loads = _random_loads(rng, N, L, D)
        layer = [0] * N
        for s in sched.run_algorithm1(loads, m, sched.MAXUTIL):
            pool = [j for j in range(N) if layer[j] < L]
            assert len(s) >= min(m, len(pool))
            for j, l in s:
                assert l == layer[j]
                layer[j] += 1


def test_special_cases_reduce_to_lockstep():
    rng = np.random.default_rng(14)
    for trial in range(100):
        N, L, D = int(rng.integers(1, 6)), int(rng.integers(1, 5)), int(rng.integers(1, 5))
        loads = _random_loads(rng, N, L, D)
        # m = N: every step must run the whole pool
        assert sched.run_algorithm1(loads, N, sched.MAXUTIL) == sched.lockstep_steps(N, L)
        # D = 1: U = 1 for every set, the tie-break takes the largest set
        assert sched.run_algorithm1(loads[:, :, :1], 1, sched.MAXUTIL) == sched.lockstep_steps(N, L)
        # N = 1: L single steps
        assert sched.run_algorithm1(loads[:1], 1, sched.MAXUTIL) == [[(0, l)] for l in range(L)]


def test_utilization_closed_forms():
    loads = np.array([[[3, 1]], [[1, 3]]])          # N=2, L=1, D=2
    assert metrics.utilization(loads, [[(0, 0), (1, 0)]]) == 1
    assert metrics.utilization(loads, [[(0, 0)], [(1, 0)]]) == Fraction(8, 12)
    assert metrics.max_over_mean(loads, [[(0, 0)], [(1, 0)]]) == Fraction(3, 2)
    bal = np.full((3, 4, 5), 7)
    assert metrics.utilization(bal, sched.lockstep_steps(3, 4)) == 1
    # lock-step equals Eq. 3 summed over layers
    rng = np.random.default_rng(15)
    w = rng.integers(0, 9, size=(4, 3, 6))
    per_layer = w.sum(axis=0)                       # [L][D]
    want = Fraction(int(per_layer.sum()), 6 * int(per_layer.max(axis=1).sum()))
    assert metrics.utilization(w, sched.lockstep_steps(4, 3)) == want


def test_maxutil_never_worse_than_separate():
    rng = np.random.default_rng(16)
    for trial in range(200):
        N, L, D = int(rng.integers(2, 7)), int(rng.integers(1, 5)), int(rng.integers(2, 9))
        loads = _random_loads(rng, N, L, D)
        eb = sched.run_algorithm1(loads, max(1, int(0.75 * N)), sched.MAXUTIL)
        sep = sched.separate_steps(N, L)
        assert metrics.utilization(loads, eb) >= metrics.utilization(loads, sep)


def _offline_optimum(loads: np.ndarray, m: int) -> int:
    """Smallest summed per-step peak load (sum over steps of max_d W_i,d) over
    every schedule Algorithm 1 may run: at each step any set of at least
    min(m, |pool|) micro-batches still in the pool advances one layer.  An
    exhaustive search over the micro-batches' layer positions, written
    independently of oracle.sched."""
    N, L, _ = loads.shape

    @functools.lru_cache(maxsize=None)
    def best(state):
        pool = [j for j in range(N) if state[j] < L]
        if not pool:
            return 0
        cost = None
        for r in range(min(m, len(pool)), len(pool) + 1):
            for R in itertools.combinations(pool, r):
                peak = int(sum(loads[j, state[j]] for j in R).max())
                nxt = tuple(s + (j in R) for j, s in enumerate(state))
                c = peak + best(nxt)
                cost = c if cost is None else min(cost, c)
        return cost

    return best((0,) * N)


def test_offline_optimum_hand_worked():
    # one layer, two devices: complementary loads merge (peak 4 < 3 + 3),
    # identical ones gain nothing (6 either way)
    assert _offline_optimum(np.array([[[3, 1]], [[1, 3]]]), 1) == 4
    assert _offline_optimum(np.array([[[3, 1]], [[3, 1]]]), 1) == 6
    # m = 2 forces both together at every step: the lock-step sum of peaks
    loads = np.array([[[3, 1], [0, 2]], [[1, 3], [2, 2]]])
    assert _offline_optimum(loads, 2) == 4 + 4


def test_greedy_against_offline_optimum():
    """Every policy's schedule is one the search considers, so the optimum is
    never larger; it is also bounded below by the total work over D, and
    above by lock-step (and, for m = 1, by separate steps).  The greedy /
    optimum ratio is reported, not gated."""
    rng = np.random.default_rng(2026_12_02)
    ratios = {p: [] for p in (sched.MAXUTIL, sched.CUMUTIL, sched.DIFFPEAK)}
    for _ in range(400):
        N, L, D = int(rng.integers(1, 4)), int(rng.integers(1, 4)), int(rng.integers(1, 5))
        m = int(rng.integers(1, N + 1))
        loads = rng.integers(0, 6, size=(N, L, D)).astype(np.int64)
        opt = _offline_optimum(loads, m)
        total = int(loads.sum())
        peaks = lambda steps: sum(int(metrics.step_workload(loads, s).max()) for s in steps)
        assert opt * D >= total
        assert opt <= peaks(sched.lockstep_steps(N, L))
        if m == 1:
            assert opt <= peaks(sched.separate_steps(N, L))
        if D == 1:
            assert opt == total
        for p in ratios:
            g = peaks(sched.run_algorithm1(loads, m, p))
            assert g >= opt
            ratios[p].append(Fraction(g, opt) if opt else Fraction(1))
    for p, r in ratios.items():
        print(f"policy {p}: greedy / optimum mean {float(sum(r) / len(r)):.4f}, max {float(max(r)):.3f}, "
              f"optimal in {sum(x == 1 for x in r)}/{len(r)}")
