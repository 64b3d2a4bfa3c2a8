"""C-ABI checks that need no GPU: the library loads, exports every function
include/easybalance.h declares, and its host scheduler matches the oracle bit
for bit (Algorithm 1's Schedule; MaxUtil of Section 4.2, CumUtil / DiffPeak of
Section 5.2)."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import model as omodel
from oracle import sched as osched
from paper_2608_07964_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    with open(os.path.join(ROOT, "include", "easybalance.h")) as f:
        src = f.read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(easybalance_\w+)\s*\(", src, flags=re.M)))


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    names = _declared_functions()
    assert len(names) >= 9
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B.EXPORTS)
    assert B.easybalance_version().startswith("easybalance-mi355x")


POL = {osched.MAXUTIL: B.EB_POLICY_MAXUTIL, osched.CUMUTIL: B.EB_POLICY_CUMUTIL,
       osched.DIFFPEAK: B.EB_POLICY_DIFFPEAK}


@pytest.mark.parametrize("policy", [osched.MAXUTIL, osched.CUMUTIL, osched.DIFFPEAK])
def test_schedule_matches_oracle_bit_exact(policy):
    rng = np.random.default_rng(30 + policy)
    for trial in range(1500):
        n = int(rng.integers(1, 11 if policy == osched.MAXUTIL else 17))
        D = int(rng.choice([1, 2, 3, 4, 8, 16, 32]))
        per = int(rng.integers(1, 4))
        E = D * per
        m = int(rng.integers(1, n + 2))
        ids = sorted(rng.choice(64, size=n, replace=False).tolist())
        hi = int(rng.choice([2, 5, 1000]))
        counts = rng.integers(0, hi, size=(n, E)).astype(np.int32)
        mask, load = B.easybalance_schedule(ids, counts, E, D, m, POL[policy])
        loads = {j: omodel.device_loads(counts[i], D) for i, j in enumerate(ids)}
        want = osched.schedule(ids, loads, D, m, policy)
        got = tuple(j for j in ids if (mask >> j) & 1)
        assert got == want, (ids, counts.tolist(), D, m)
        assert np.array_equal(load, sum(loads[j] for j in want))


def test_maxutil_large_pools_match_oracle():
    """Pools of 13-16 micro-batches with m from n - 4 to n (the candidate sets
    are the complements of at most 4 excluded ones), small count ranges (many
    ties) and counts near 2^31 (the exact 128-bit comparison decides)."""
    rng = np.random.default_rng(34)
    for trial in range(8):
        n = int(rng.integers(13, 17))
        D, per = int(rng.choice([4, 8])), 2
        E = D * per
        m = int(rng.integers(n - 4, n + 1))
        ids = sorted(rng.choice(64, size=n, replace=False).tolist())
        hi = [3, 1000, 2 ** 31 - 1][trial % 3]
        counts = rng.integers(0, hi, size=(n, E)).astype(np.int32)
        mask, load = B.easybalance_schedule(ids, counts, E, D, m, B.EB_POLICY_MAXUTIL)
        loads = {j: omodel.device_loads(counts[i], D) for i, j in enumerate(ids)}
        want = osched.schedule(ids, loads, D, m, osched.MAXUTIL)
        assert tuple(j for j in ids if (mask >> j) & 1) == want, (n, m, hi)
        assert np.array_equal(load, sum(loads[j] for j in want))


def test_schedule_large_pool_and_overflow_safety():
    # 16 micro-batches (the decode-like stack) and counts near 2^31
    rng = np.random.default_rng(33)
    ids = list(range(16))
    counts = rng.integers(0, 2 ** 31 - 1, size=(16, 8)).astype(np.int32)
    mask, load = B.easybalance_schedule(ids, counts, 8, 8, 12, B.EB_POLICY_MAXUTIL)
    assert bin(mask).count("1") >= 12
    assert load.dtype == np.int64 and np.all(load >= 0)


def test_schedule_empty_pool_and_errors():
    mask, load = B.easybalance_schedule([], np.zeros((0, 4), np.int32), 4, 2, 1)
    assert mask == 0 and np.all(load == 0)
    bad = [
        dict(ids=[1, 0], counts=np.ones((2, 4)), E=4, D=2, m=1, pol=0),       # not ascending
        dict(ids=[0, 64], counts=np.ones((2, 4)), E=4, D=2, m=1, pol=0),      # id out of range
        dict(ids=[0], counts=np.ones((1, 4)), E=4, D=3, m=1, pol=0),          # E % D
        dict(ids=[0], counts=np.ones((1, 4)), E=4, D=2, m=0, pol=0),          # m < 1
        dict(ids=[0], counts=np.ones((1, 4)), E=4, D=2, m=1, pol=7),          # policy
        dict(ids=[0], counts=-np.ones((1, 4)), E=4, D=2, m=1, pol=0),         # negative count
    ]
    for b in bad:
        with pytest.raises(B.EasyBalanceError) as ei:
            B.easybalance_schedule(b["ids"], b["counts"], b["E"], b["D"], b["m"], b["pol"])
        assert ei.value.code == B.EB_ERR_INVALID_ARG
        assert B.easybalance_last_error()
    with pytest.raises(B.EasyBalanceError) as ei:
        B.easybalance_schedule(list(range(21)), np.ones((21, 2)), 2, 2, 1, B.EB_POLICY_MAXUTIL)
    assert ei.value.code == B.EB_ERR_UNSUPPORTED
    # the heuristics take any pool up to 64
    mask, _ = B.easybalance_schedule(list(range(64)), np.ones((64, 2)), 2, 2, 1, B.EB_POLICY_CUMUTIL)
    assert mask & 1


def test_workspace_size_and_desc_checks():
    d = B.make_desc(8, 4096, 14336, 8, 2, 0, 8, "bf16")
    ws = B.easybalance_moe_step_workspace_size(d, [512] * 4)
    P = 4 * 512 * 2
    assert ws >= P * 4096 * 2 + P * 14336 * 2
    assert ws % 256 == 0
    for bad, code in [(B.make_desc(8, 4000, 14336, 8, 2, 0, 8, "bf16"), B.EB_ERR_UNSUPPORTED),
                      (B.make_desc(8, 4096, 14300, 8, 2, 0, 8, "bf16"), B.EB_ERR_UNSUPPORTED),
                      (B.make_desc(8, 4096, 14336, 8, 9, 0, 8, "bf16"), B.EB_ERR_INVALID_ARG),
                      (B.make_desc(8, 4096, 14336, 8, 2, 0, 3, "bf16"), B.EB_ERR_INVALID_ARG),
                      (B.make_desc(8, 4096, 14336, 8, 2, 0, 8, 5), B.EB_ERR_INVALID_ARG),
                      (B.make_desc(8, 4096, 14336, 64, 8, 9, 8, "bf16"), B.EB_ERR_UNSUPPORTED)]:
        with pytest.raises(B.EasyBalanceError) as ei:
            B.easybalance_moe_step_workspace_size(bad, [16])
        assert ei.value.code == code


def test_device_calls_reject_bad_arguments_before_touching_the_gpu():
    d = B.make_desc(2, 256, 512, 8, 2, 0, 4, "f32")
    with pytest.raises(B.EasyBalanceError) as ei:
        B.easybalance_route(d, 2, 4, 1, 1, 1, 1, 1, 1, 1, 1, 1)        # layer out of range
    assert ei.value.code == B.EB_ERR_INVALID_ARG
    with pytest.raises(B.EasyBalanceError):
        B.easybalance_route(d, 0, 4, None, 1, 1, 1, 1, 1, 1, 1, 1)     # NULL x
    run = B.work_array([(0, 5, 4, 1, 1, 1)])                            # layer 5 >= L
    with pytest.raises(B.EasyBalanceError):
        B.easybalance_moe_step(d, run, 1, [1, 1], [1, 1], 256, 1 << 20, 1, 1)
    run = B.work_array([(0, 0, 4, 1, 1, 1)])
    with pytest.raises(B.EasyBalanceError) as ei:
        B.easybalance_moe_step(d, run, 1, [1, 1], [1, 1], 256, 16, 1, 1)   # workspace too small
    assert ei.value.code == B.EB_ERR_WORKSPACE_TOO_SMALL
    with pytest.raises(B.EasyBalanceError):
        B.easybalance_moe_step(d, run, 1, [1, 1], [1, 1], 255, 1 << 30, 1, 1)  # misaligned
    with pytest.raises(B.EasyBalanceError):
        B.easybalance_combine(d, run, 0, [1], 1, 1)                     # n_run = 0


def test_run_pass_rejects_bad_arguments_before_touching_the_gpu():
    d = B.make_desc(2, 256, 128, 8, 2, 0, 4, "bf16")
    need = B.easybalance_pass_state_size(d, 4, 64)
    assert need > 0
    with pytest.raises(B.EasyBalanceError):
        B.easybalance_pass_state_size(d, 0, 64)
    with pytest.raises(B.EasyBalanceError):
        B.easybalance_pass_state_size(d, 65, 64)
    fake = 1 << 20  # non-NULL, 256-byte aligned; never dereferenced on these paths
    args = (d, 4, 64, fake, fake, [fake, fake], fake, [fake, fake], [fake, fake])
    with pytest.raises(B.EasyBalanceError) as e:   # state too small
        B.easybalance_run_pass(*args, B.EB_POLICY_MAXUTIL, 3, fake, need - 1)
    assert e.value.code == B.EB_ERR_WORKSPACE_TOO_SMALL
    with pytest.raises(B.EasyBalanceError) as e:   # unknown policy
        B.easybalance_run_pass(*args, 7, 3, fake, need)
    assert e.value.code == B.EB_ERR_INVALID_ARG
    with pytest.raises(B.EasyBalanceError) as e:   # misaligned state
        B.easybalance_run_pass(*args, B.EB_POLICY_MAXUTIL, 3, fake + 4, need)
    assert e.value.code == B.EB_ERR_INVALID_ARG
    with pytest.raises(B.EasyBalanceError) as e:   # m < 1
        B.easybalance_run_pass(*args, B.EB_POLICY_MAXUTIL, 0, fake, need)
    assert e.value.code == B.EB_ERR_INVALID_ARG
    with pytest.raises(B.EasyBalanceError) as e:   # a flag bit other than EB_PASS_DEVICE_SCHEDULE
        B.easybalance_run_pass(*args, B.EB_POLICY_MAXUTIL | 0x200, 3, fake, need)
    assert e.value.code == B.EB_ERR_INVALID_ARG
    wide = B.make_desc(2, 256, 128, 128, 2, 0, 128, "bf16")   # D = 128 virtual devices
    need_w = B.easybalance_pass_state_size(wide, 4, 64)
    args_w = (wide, 4, 64, fake, fake, [fake, fake], fake, [fake, fake], [fake, fake])
    with pytest.raises(B.EasyBalanceError) as e:   # the device scheduler handles D <= 64
        B.easybalance_run_pass(*args_w, B.EB_POLICY_MAXUTIL | B.EB_PASS_DEVICE_SCHEDULE, 3, fake, need_w)
    assert e.value.code == B.EB_ERR_UNSUPPORTED
    f32 = B.make_desc(2, 256, 128, 128, 2, 0, 4, "f32")        # fp32 routing with E > 64
    need_f = B.easybalance_pass_state_size(f32, 4, 64)
    args_f = (f32, 4, 64, fake, fake, [fake, fake], fake, [fake, fake], [fake, fake])
    with pytest.raises(B.EasyBalanceError) as e:
        B.easybalance_run_pass(*args_f, B.EB_POLICY_CUMUTIL | B.EB_PASS_DEVICE_SCHEDULE, 3, fake, need_f)
    assert e.value.code == B.EB_ERR_UNSUPPORTED


def test_pack_weights_rejects_bad_arguments_before_touching_the_gpu():
    d = B.make_desc(2, 256, 128, 8, 2, 0, 4, "bf16")
    fake, gu_bytes = 1 << 20, 256 * 256 * 2  # one [2F][H] bf16 matrix
    B.easybalance_pack_weights(d, B.EB_WEIGHTS_GATE_UP, 0, None, None)  # nothing to do
    for args, code in [((7, 1, fake, fake + gu_bytes), B.EB_ERR_INVALID_ARG),        # kind
                       ((B.EB_WEIGHTS_DOWN, -1, fake, fake), B.EB_ERR_INVALID_ARG),   # n < 0
                       ((B.EB_WEIGHTS_DOWN, 1, None, fake), B.EB_ERR_INVALID_ARG),    # NULL
                       ((B.EB_WEIGHTS_GATE_UP, 1, fake, fake + gu_bytes - 2), B.EB_ERR_INVALID_ARG),  # overlap
                       ((B.EB_WEIGHTS_GATE_UP, 1, fake + 8, fake + 2 * gu_bytes), B.EB_ERR_INVALID_ARG)]:  # align
        with pytest.raises(B.EasyBalanceError) as ei:
            B.easybalance_pack_weights(d, *args)
        assert ei.value.code == code, args
    big = B.make_desc(2, 16384, 32768, 8, 2, 0, 4, "bf16")  # a gate/up matrix of 2 GiB
    with pytest.raises(B.EasyBalanceError) as ei:
        B.easybalance_pack_weights(big, B.EB_WEIGHTS_GATE_UP, 1, fake, fake * 4096)
    assert ei.value.code == B.EB_ERR_UNSUPPORTED


def test_empty_step_enqueues_nothing():
    """A step whose entries all have T = 0 returns before any HIP call: no
    pointer is dereferenced or checked, so NULL weights and outputs pass."""
    d = B.make_desc(2, 256, 128, 8, 2, 0, 4, "bf16")
    run = B.work_array([(0, 0, 0, None, None, None), (1, 1, 0, None, None, None)])
    assert B.easybalance_moe_step_workspace_size(d, [0, 0]) >= 0
    B.easybalance_moe_step(d, run, 2, [None, None], [None, None], None, 0, None, None)
    B.easybalance_combine(d, run, 2, [None, None], None, None)
    bad = B.work_array([(0, 2, 0, None, None, None)])   # layer outside [0, L) is still rejected
    with pytest.raises(B.EasyBalanceError) as ei:
        B.easybalance_moe_step(d, bad, 1, [None, None], [None, None], None, 0, None, None)
    assert ei.value.code == B.EB_ERR_INVALID_ARG


def _random_placement(rng, L, E, D):
    R = int(rng.integers(1, D + 1))
    copies = [[sorted(rng.choice(D, size=int(rng.integers(1, R + 1)), replace=False).tolist())
               for _ in range(E)] for _ in range(L)]
    return copies


@pytest.mark.parametrize("policy", [osched.MAXUTIL, osched.CUMUTIL, osched.DIFFPEAK])
def test_schedule_on_a_replicated_placement_matches_oracle(policy):
    """Section 5's orthogonality study: Schedule on the loads of a static
    placement with replicas equals the oracle's choice on the oracle's placed
    loads of each pool member at its own layer."""
    rng = np.random.default_rng(60 + policy)
    for trial in range(400):
        n = int(rng.integers(1, 9))
        D = int(rng.choice([1, 2, 3, 4, 8]))
        E = D * int(rng.integers(1, 4))
        L = int(rng.integers(1, 5))
        m = int(rng.integers(1, n + 2))
        ids = sorted(rng.choice(64, size=n, replace=False).tolist())
        layers = rng.integers(0, L, size=n).tolist()
        copies = _random_placement(rng, L, E, D)
        counts = rng.integers(0, int(rng.choice([3, 50])), size=(n, E)).astype(np.int32)
        pl = B.make_placement(copies, D)
        mask, load = B.easybalance_schedule(ids, counts, E, D, m, POL[policy], layers=layers, placement=pl)
        loads = {j: omodel.placed_device_loads(counts[i], copies[layers[i]], D) for i, j in enumerate(ids)}
        want = osched.schedule(ids, loads, D, m, policy)
        got = tuple(j for j in ids if (mask >> j) & 1)
        assert got == want, (ids, layers, copies, counts.tolist(), D, m)
        assert np.array_equal(load, sum(loads[j] for j in want))


def test_placement_argument_checks():
    E, D, L = 4, 2, 2
    ids, counts = [0, 1], np.ones((2, E), np.int32)
    good = [[[0], [0, 1], [1], [1]]] * L
    B.easybalance_schedule(ids, counts, E, D, 1, layers=[0, 1], placement=B.make_placement(good, D))
    bad = {
        "no copy": np.array([[[0, -1], [-1, -1], [1, -1], [1, -1]]] * L),
        "device out of range": np.array([[[0, -1], [2, -1], [1, -1], [1, -1]]] * L),
        "not ascending": np.array([[[1, 0], [0, -1], [1, -1], [1, -1]]] * L),
        "repeated device": np.array([[[0, 0], [0, -1], [1, -1], [1, -1]]] * L),
        "hole": np.array([[[0, -1], [-1, 1], [1, -1], [1, -1]]] * L),
    }
    for what, arr in bad.items():
        with pytest.raises(B.EasyBalanceError) as ei:
            B.easybalance_schedule(ids, counts, E, D, 1, layers=[0, 1], placement=B.make_placement(arr, D))
        assert ei.value.code == B.EB_ERR_INVALID_ARG, what
    pl = B.make_placement(good, D)
    with pytest.raises(B.EasyBalanceError):          # layers are required with a placement
        B.easybalance_schedule(ids, counts, E, D, 1, placement=pl)
    with pytest.raises(B.EasyBalanceError):          # a layer the placement does not cover
        B.easybalance_schedule(ids, counts, E, D, 1, layers=[0, 2], placement=pl)
    with pytest.raises(B.EasyBalanceError):          # made for another E
        B.easybalance_schedule(ids, np.ones((2, 6), np.int32), 6, D, 1, layers=[0, 1], placement=pl)


@pytest.mark.parametrize("name", ["mixtral_bf16", "qwen_moe_bf16", "dsv2_lite_bf16", "dsv3_share_bf16"])
def test_scheduler_cost_native_against_oracle(name):
    """Context for the paper's Table 3 (scheduling time per step): one
    Schedule decision over a full pool of the stack's N micro-batches at its
    D and m, by the native host scheduler (through the binding) and by the
    oracle's plain-Python one, on the same random counts; the run sets agree
    and the per-decision times are printed (reported, not gated)."""
    import time
    from synth import BY_NAME
    cfg = BY_NAME[name]
    rng = np.random.default_rng(17)
    ids = list(range(cfg.N))
    trials = [rng.integers(0, 200, size=(cfg.N, cfg.E)).astype(np.int32) for _ in range(5)]
    B.easybalance_schedule(ids, trials[0], cfg.E, cfg.D, cfg.m, B.EB_POLICY_DIFFPEAK)  # loads the library
    for policy in (osched.MAXUTIL, osched.CUMUTIL, osched.DIFFPEAK):
        t_nat = t_py = 0.0
        for counts in trials:
            t0 = time.perf_counter()
            mask, _ = B.easybalance_schedule(ids, counts, cfg.E, cfg.D, cfg.m, POL[policy])
            t1 = time.perf_counter()
            loads = {j: omodel.device_loads(counts[j], cfg.D) for j in ids}
            want = osched.schedule(ids, loads, cfg.D, cfg.m, policy)
            t2 = time.perf_counter()
            assert tuple(j for j in ids if (mask >> j) & 1) == want
            t_nat += t1 - t0
            t_py += t2 - t1
        print(f"{name} N={cfg.N} D={cfg.D} m={cfg.m} policy {policy}: native {1e6 * t_nat / len(trials):.0f} us, "
              f"oracle (plain Python) {1e3 * t_py / len(trials):.2f} ms per decision")
