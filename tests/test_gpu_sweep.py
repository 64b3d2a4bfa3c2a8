"""The sweep's recorded experts reproduce what the native Algorithm-1 pass
sees: per-device loads of every (micro-batch, layer) and, replayed through
the scheduler, the native pass's steps."""
import numpy as np
import pytest
import torch

from synth import CONFIGS, mini
from synth.device import DeviceInputs

from gpu_helpers import log, make_stack
from paper_2608_07964_amd import sweep

pytestmark = pytest.mark.gpu

CFGS = [c if c.dtype == "f32" else mini(c) for c in CONFIGS]


@pytest.mark.parametrize("cfg", CFGS, ids=[c.name for c in CFGS])
def test_recorded_routes_reproduce_native_pass(cfg, device):
    inp = DeviceInputs(cfg, device)
    st, _ = make_stack(cfg, device, inputs=inp)
    routes = sweep.record_routes(st)
    torch.cuda.synchronize()
    assert routes.shape == (cfg.N * cfg.T, cfg.L, cfg.k)
    assert ((routes >= 0) & (routes < cfg.E)).all()
    w = sweep.layer_loads(routes, cfg.N, cfg.E, cfg.D)
    for policy, m in (("maxutil", cfg.m), ("cumutil", cfg.m), ("diffpeak", cfg.m), ("lockstep", None)):
        st.x.copy_(inp.x0)
        steps = st.run_native(policy, m=m)
        torch.cuda.synchronize()
        assert np.array_equal(st.layer_loads, w), policy
        replay = sweep.run_policy(w, policy, cfg.N if m is None else m)
        assert len(replay) == len(steps), policy
        for a, s in zip(replay, steps):
            assert np.array_equal(a, s.load), policy
        log(f"  {cfg.name} {policy}: {len(steps)} steps replayed from recorded experts")
