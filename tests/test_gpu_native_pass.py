"""The native Algorithm-1 driver (easybalance_run_pass), host- and
device-scheduled, against the Python driver over the same entry points:
identical schedules, loads, group counts and bit-identical hidden states, for
every policy, on the small stacks and on the full-size Mixtral-shaped stack
that bench.py times."""
import numpy as np
import pytest
import torch

from synth import BY_NAME, CONFIGS, mini
from synth.device import DeviceInputs

from gpu_helpers import log, make_stack

pytestmark = pytest.mark.gpu

# plus a split-K down GEMM (F >= 8192) and many pairs of long rows in the
# grouping (k+S = 9 slots of 4 KB rows: four pieces per token)
SMALL = ([c if c.dtype == "f32" else mini(c) for c in CONFIGS]
         + [mini(BY_NAME["mixtral_bf16"], H=256, F=8192, T=96, L=2),
            mini(BY_NAME["dsv3_share_bf16"], H=2048, T=96, L=2)])
SMALL_IDS = [c.name for c in SMALL[:-2]] + [SMALL[-2].name + "_longk", SMALL[-1].name + "_rowonce"]
# the device scheduler's 16- and 64-device forms (the stacks above use 4, 8
# and 32 virtual devices)
SMALL += [mini(BY_NAME["qwen_moe_bf16"], E=64, D=16, H=256, F=128, T=96, L=3).scaled(name="d16_bf16"),
          mini(BY_NAME["dsv3_share_bf16"], E=128, D=64, H=256, F=128, T=96, L=3).scaled(name="d64_bf16")]
SMALL_IDS += ["d16", "d64"]


def _compare(cfg, device, policies):
    inp = DeviceInputs(cfg, device)
    for policy, m in policies:
        st, _ = make_stack(cfg, device, inputs=inp)
        py_steps = st.run(policy, m=m)
        torch.cuda.synchronize()
        x_py, ll_py = st.x.clone(), st.layer_loads.copy()
        for dev_sched in (False, True):
            st.x.copy_(inp.x0)
            nat_steps = st.run_native(policy, m=m, device_schedule=dev_sched)
            torch.cuda.synchronize()
            what = (policy, m, "device" if dev_sched else "host")
            assert torch.equal(st.x, x_py), what
            assert np.array_equal(st.layer_loads, ll_py), what
            assert [s.runset for s in nat_steps] == [s.runset for s in py_steps], what
            for a, b in zip(nat_steps, py_steps):
                assert np.array_equal(a.load, b.load) and a.groups == b.groups and a.pairs == b.pairs, what
            # without records the call returns once the last step is queued
            st.x.copy_(inp.x0)
            assert st.run_native(policy, m=m, record=False, device_schedule=dev_sched) == []
            torch.cuda.synchronize()
            assert torch.equal(st.x, x_py), what + ("unrecorded",)
        log(f"  {cfg.name} {policy} m={m}: {len(nat_steps)} steps identical (host and device schedule)")


@pytest.mark.parametrize("cfg", SMALL, ids=SMALL_IDS)
def test_native_pass_matches_python_driver(cfg, device):
    _compare(cfg, device, [("maxutil", cfg.m), ("maxutil", 1), ("cumutil", cfg.m),
                           ("diffpeak", cfg.m), ("lockstep", None)])


def test_native_pass_full_size_bench_stack(device):
    cfg = [c for c in CONFIGS if c.name == "mixtral_bf16"][0]
    _compare(cfg, device, [("maxutil", cfg.m), ("lockstep", None)])


@pytest.mark.parametrize("name", ["qwen_moe_bf16", "dsv2_lite_bf16", "dsv3_share_bf16"])
def test_native_pass_full_size_other_stacks(name, device):
    """The pass bench.py times (native, host- and device-scheduled) against
    the Python driver's, whose every step the full-size parity test checks
    against the oracle: bit-identical hidden states, loads and steps."""
    cfg = BY_NAME[name]
    _compare(cfg, device, [("maxutil", cfg.m)])


def test_native_pass_pool_over_32_micro_batches(device):
    """40 micro-batches: the routing after a step spans two batch tables
    (32 entries each), host- and device-scheduled (MaxUtil enumerates pools
    of at most 20, so the heuristics and lock-step run here)."""
    cfg = mini(BY_NAME["qwen_moe_bf16"], N=40, T=24, L=2)
    assert cfg.N == 40
    _compare(cfg, device, [("cumutil", 30), ("diffpeak", 30), ("lockstep", None)])


def _record_counts(st):
    """Per-expert counts c[j][l][e] the GPU routing produced, from one
    lock-step pass of the Python driver (a token's experts do not depend on
    the schedule: the stacks are MoE-only and the kernels batch invariant)."""
    counts = np.full((st.N, st.L, st.E), -1, dtype=np.int64)

    def hook(stage, runset):
        if stage == "pre":
            c = st.counts.cpu().numpy()
            for j, layer in runset:
                counts[j, layer] = c[j]

    st.run("lockstep", record=False, hook=hook)
    torch.cuda.synchronize()
    assert (counts >= 0).all()
    return counts


@pytest.mark.parametrize("name", ["mixtral_bf16", "qwen_moe_bf16", "dsv2_lite_bf16"])
def test_native_pass_on_replicated_placement(name, device):
    """EasyBalance on a static placement with replicas (Section 5, orthogonality
    with EPLB) through the library, host- and device-scheduled: the recorded
    per-device loads are the oracle's placed loads of the GPU's counts, every
    executed schedule is the oracle's Algorithm-1 replay on them, each step's
    workload is the oracle's, and the hidden states equal the lock-step pass's
    bit for bit."""
    from oracle import metrics as ometrics
    from oracle import model as omodel
    from oracle import sched as osched
    from paper_2608_07964_amd import binding as B
    from paper_2608_07964_amd import sweep

    cfg = mini(BY_NAME[name])
    log(f"placement {cfg.name}")
    inp = DeviceInputs(cfg, device)
    st, _ = make_stack(cfg, device, inputs=inp)
    counts = _record_counts(st)
    x_ref = st.x.clone()
    # an EPLB-like placement from the batch's own history: D extra copies of
    # the hottest experts, and a random one with up to 3 copies per expert
    rng = np.random.default_rng(77)
    hist = counts.sum(axis=0)
    placements = {
        "history": [sweep.placement_copies(sweep.replicated_placement(hist[l], cfg.D, cfg.D, l % cfg.D), cfg.E)
                    for l in range(cfg.L)],
        "random": [[sorted(rng.choice(cfg.D, size=int(rng.integers(1, min(3, cfg.D) + 1)), replace=False).tolist())
                    for _ in range(cfg.E)] for _ in range(cfg.L)],
    }
    pols = {"maxutil": osched.MAXUTIL, "cumutil": osched.CUMUTIL, "diffpeak": osched.DIFFPEAK}
    for pname, copies in placements.items():
        placed = np.stack([omodel.placed_device_loads(counts[:, l], copies[l], cfg.D) for l in range(cfg.L)],
                          axis=1)
        pl = B.make_placement(copies, cfg.D)
        for policy, m in [("maxutil", cfg.m), ("cumutil", cfg.m), ("diffpeak", cfg.m), ("lockstep", None)]:
            for dev_sched in (False, True):
                st.x.copy_(inp.x0)
                steps = st.run_native(policy, m=m, device_schedule=dev_sched, placement=pl)
                torch.cuda.synchronize()
                what = (pname, policy, m, "device" if dev_sched else "host")
                assert np.array_equal(st.layer_loads, placed), what
                want = (osched.lockstep_steps(cfg.N, cfg.L) if policy == "lockstep"
                        else osched.run_algorithm1(placed, m, pols[policy]))
                assert [s.runset for s in steps] == want, what
                for s in steps:
                    assert np.array_equal(s.load, ometrics.step_workload(placed, s.runset)), what
                assert torch.equal(st.x, x_ref), what
        log(f"  {cfg.name} {pname}: every policy matches the oracle on the placed loads")
