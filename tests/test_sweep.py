"""Host side of the load-balance sweeps (paper_2608_07964_amd.sweep): loads
from recorded experts against a brute-force count, the replayed passes
against the oracle's Algorithm 1, and the worst-case window statistic on
hand-worked loads."""
import numpy as np
import pytest

from oracle import metrics as ometrics
from oracle import model as omodel
from oracle import sched as osched
from paper_2608_07964_amd import binding as B
from paper_2608_07964_amd import metrics, sweep


def _routes(rng, tokens, L, k, E):
    # k distinct experts per token and layer
    return np.stack([[rng.choice(E, size=k, replace=False) for _ in range(L)] for _ in range(tokens)]
                    ).astype(np.int32)


def test_layer_loads_brute_force():
    rng = np.random.default_rng(1)
    tokens, L, k, E = 24, 3, 2, 8
    r = _routes(rng, tokens, L, k, E)
    for N, D in ((1, 2), (4, 4), (6, 8), (3, 1)):
        got = sweep.layer_loads(r, N, E, D)
        T = tokens // N
        ref = np.zeros((N, L, D), np.int64)
        for t in range(tokens):
            for l in range(L):
                for e in r[t, l]:
                    ref[t // T, l, e // (E // D)] += 1
        assert np.array_equal(got, ref), (N, D)
        assert got.sum() == tokens * L * k
    with pytest.raises(ValueError):
        sweep.layer_loads(r, 5, E, 4)
    with pytest.raises(ValueError):
        sweep.layer_loads(r, 4, E, 3)


@pytest.mark.parametrize("policy", ["maxutil", "cumutil", "diffpeak"])
def test_replayed_pass_matches_oracle(policy):
    pid = {"maxutil": osched.MAXUTIL, "cumutil": osched.CUMUTIL, "diffpeak": osched.DIFFPEAK}[policy]
    rng = np.random.default_rng(7)
    for trial in range(40):
        N, L, D = int(rng.integers(1, 7)), int(rng.integers(1, 5)), int(rng.integers(1, 5))
        w = rng.integers(0, 6, size=(N, L, D))
        for m in sorted({1, max(1, N // 2), N}):
            got = sweep.run_policy(w, policy, m)
            ref = [sum(w[j, l] for j, l in step) for step in osched.run_algorithm1(w, m, pid)]
            assert len(got) == len(ref), (trial, m)
            for a, b in zip(got, ref):
                assert np.array_equal(a, b), (trial, m)


def test_baselines_and_invariants():
    rng = np.random.default_rng(3)
    N, L, D = 4, 5, 4
    w = rng.integers(0, 9, size=(N, L, D))
    lock = sweep.run_policy(w, "lockstep", N)
    assert [list(x) for x in lock] == [list(w[:, l].sum(axis=0)) for l in range(L)]
    sep = sweep.run_policy(w, "separate", N)
    assert len(sep) == N * L
    # m = N forces lock-step (I5); no policy's peak sum exceeds the separate one (I4)
    assert [list(x) for x in sweep.run_policy(w, "maxutil", N)] == [list(x) for x in lock]
    peak = lambda steps: sum(int(np.max(x)) for x in steps)
    for pol in ("maxutil", "cumutil", "diffpeak", "lockstep"):
        assert peak(sweep.run_policy(w, pol, 2)) <= peak(sep), pol
    # every (j, l) workload runs exactly once: total work is conserved
    for pol in ("maxutil", "cumutil", "diffpeak"):
        assert int(np.sum(sweep.run_policy(w, pol, 1))) == int(w.sum())


def test_same_skew_windows_hand_worked():
    # (3,1)+(2,0): peaks on device 0 both, max 5 = 3 + 2 -> worst case
    # (2,0)+(1,3): max 3 < 2 + 3;  (1,3)+(0,2): max 5 = 3 + 2 -> worst case
    w = np.array([[3, 1], [2, 0], [1, 3], [0, 2]])
    assert sweep.same_skew_windows(w, 2) == (2, 3)
    assert sweep.same_skew_windows(w, 3) == (0, 2)
    # a tie counts as a shared peak; a window longer than L has none
    assert sweep.same_skew_windows(np.array([[2, 2], [1, 1]]), 2) == (1, 1)
    assert sweep.same_skew_windows(w, 5) == (0, 0)


def test_sweep_rows_shape():
    rng = np.random.default_rng(5)
    r = _routes(rng, 16, 3, 2, 8)
    rows = sweep.sweep(r, 8, [2, 4], [2, 4])
    # per (N, D): maxutil/cumutil/diffpeak for m = 1..N, lockstep and separate once
    assert len(rows) == sum(3 * n + 2 for n in (2, 4)) * 2
    for row in rows:
        assert 0.0 <= row["under_util"] < 1.0 and row["max_over_mean"] >= 1.0


def test_replicated_placement_hand_worked():
    # history [10, 1, 1, 8] on two devices: largest first onto the least-loaded
    # device with a free slot (two slots each)
    assert sweep.replicated_placement([10, 1, 1, 8], 2, 0) == [[0, 2], [1, 3]]
    assert sweep.replicated_placement([10, 1, 1, 8], 2, 0, first_device=1) == [[1, 3], [0, 2]]
    # two replicas: experts 0 and 3 get a second copy on the other device
    # (expected loads 5, 5, 4, 4, 1, 1; three slots each)
    assert sweep.replicated_placement([10, 1, 1, 8], 2, 2) == [[0, 1, 3], [0, 2, 3]]
    with pytest.raises(ValueError):
        sweep.replicated_placement([1, 2, 3], 2, 0)


def test_replicated_placement_invariants():
    rng = np.random.default_rng(7)
    for E, D, reps in ((8, 8, 0), (8, 8, 8), (60, 4, 4), (64, 8, 8), (16, 4, 0)):
        hist = rng.integers(0, 1000, size=E)
        hist[rng.integers(0, E)] = hist[rng.integers(0, E)]  # a tie
        for first in (0, D - 1):
            slots = sweep.replicated_placement(hist, D, reps, first)
            assert [len(s) for s in slots] == [(E + reps) // D] * D
            held = np.bincount(np.concatenate(slots), minlength=E)
            order = sorted(range(E), key=lambda e: (-hist[e], e))
            assert sorted(np.flatnonzero(held == 2)) == sorted(order[:reps])
            assert set(np.unique(held)) <= {1, 2}
            for s in slots:  # the copies of one expert sit on different devices
                assert len(set(s)) == len(s)


def test_placed_replay_through_the_library_matches_the_oracle():
    """The placement table of the report comes from the library: the step
    loads easybalance_schedule forms under a replicated placement equal the
    oracle's placed loads (Section 5's orthogonality study) replayed by the
    oracle's Algorithm 1, for every policy; the contiguous placement written
    out as one copy per expert gives the layer_loads replay."""
    rng = np.random.default_rng(9)
    r = _routes(rng, 32, 3, 2, 8)
    N, D, E, L = 4, 4, 8, 3
    counts = sweep.expert_counts(r, N, E)
    assert counts.shape == (N, L, E) and counts.sum() == 32 * L * 2
    slots = [sweep.replicated_placement(counts.sum(axis=0)[l], D, D, l) for l in range(L)]
    copies = [sweep.placement_copies(s, E) for s in slots]
    placed = np.stack([omodel.placed_device_loads(counts[:, l], copies[l], D) for l in range(L)], axis=1)
    pl = B.make_placement(copies, D)
    for pol, opol in (("maxutil", osched.MAXUTIL), ("cumutil", osched.CUMUTIL), ("diffpeak", osched.DIFFPEAK)):
        got = sweep.run_policy_counts(counts, D, pol, 3, pl)
        want = [ometrics.step_workload(placed, rs) for rs in osched.run_algorithm1(placed, 3, opol)]
        assert [g.tolist() for g in got] == [w.tolist() for w in want], pol
    assert [g.tolist() for g in sweep.run_policy_counts(counts, D, "lockstep", 3, pl)] == \
        [w.tolist() for w in metrics.lockstep_loads(placed)]
    assert [g.tolist() for g in sweep.run_policy_counts(counts, D, "separate", 3, pl)] == \
        [w.tolist() for w in metrics.separate_loads(placed)]
    contiguous = B.make_placement([[[e // 2] for e in range(E)]] * L, D)
    w = sweep.layer_loads(r, N, E, D)
    for pol in ("maxutil", "lockstep"):
        assert [g.tolist() for g in sweep.run_policy_counts(counts, D, pol, 3, contiguous)] == \
            [g.tolist() for g in sweep.run_policy(w, pol, 3)]
        assert [g.tolist() for g in sweep.run_policy_counts(counts, D, pol, 3, None)] == \
            [g.tolist() for g in sweep.run_policy(w, pol, 3)]


def test_report_sections_on_synthetic_routes():
    # the markdown report of a small stack: every section present, the
    # placement rows for E and E + D physical experts with both tie orders
    from synth import mini, BY_NAME
    cfg = mini(BY_NAME["qwen_moe_bf16"], T=32, L=3)
    rng = np.random.default_rng(11)
    r = _routes(rng, cfg.N * cfg.T, cfg.L, cfg.k, cfg.E)
    rep = sweep.report(r, cfg)
    for head in ("Policies (N =", "MaxUtil over N and m", "Virtual devices D", "Static placement + EasyBalance",
                 "Host time per scheduling decision", "Windows of n consecutive layers"):
        assert head in rep, head
    for phys in (cfg.E, cfg.E + cfg.D):
        for ties in ("ties at device 0", "ties rotated by layer"):
            assert f"placed from history, {phys} physical experts, {ties}" in rep
