"""Full-size parity of the five stacks, in the launch configuration bench.py
times (one Algorithm-1 pass with MaxUtil and m = 0.75 N, every step one
moe_step + combine), against the CPU oracle:

* every step, all tokens: top-k indices equal the stable top-k of the GPU's
  own logits, counts equal their bincount, the grouping (inv, offsets) equals
  the oracle's stable sort by (layer, expert) -- bit-exact;
* the executed schedule equals the oracle's replay of Algorithm 1 on the
  loads the GPU observed -- bit-exact;
* sampled tokens / pairs of every step (the oracle recomputes them one by
  one, regenerating the expert's weights on the host): a, logits, w, grouped
  rows, h, o and x after the combine -- max-abs error <= 1e-2 * max|ref|
  (bf16 stacks) / 1e-5 * max|ref| (fp32);
* the EB pass and the per-layer lock-step pass end in bit-identical hidden
  states (cross-layer combination is lossless, Section 4.1).
"""
import numpy as np
import pytest
import torch

from oracle import model as omodel
from oracle import permute as operm
from oracle import sched as osched
from oracle.numerics import cast_fn
from synth import CONFIGS
from synth.device import DeviceInputs

from gpu_helpers import assert_close, host_weights, log, make_stack, to_np

pytestmark = pytest.mark.gpu


def _sample(rng, n, k):
    return sorted(rng.choice(n, size=min(k, n), replace=False).tolist()) if n else []


@pytest.mark.parametrize("cfg", CONFIGS, ids=[c.name for c in CONFIGS])
def test_full_size_eb_pass(cfg, device):
    log(f"full-size {cfg.name}: generating inputs")
    inp = DeviceInputs(cfg, device)
    st, _ = make_stack(cfg, device, inputs=inp)
    P_host = host_weights(cfg, cache=False)
    cast = cast_fn(cfg.dtype)
    ES, slots = cfg.E + cfg.S, cfg.k + cfg.S
    P_max = cfg.N * cfg.T * slots
    tdt = st.a.dtype
    views = dict(a_perm=torch.empty(P_max, cfg.H, dtype=tdt, device=device),
                 h=torch.empty(P_max, cfg.F, dtype=tdt, device=device),
                 perm=torch.empty(P_max, dtype=torch.int32, device=device),
                 offsets=torch.empty(cfg.L * ES + 1, dtype=torch.int32, device=device))
    rng = np.random.default_rng(cfg.seed)
    state = {}
    n_steps = [0]

    def hook(stage, runset):
        torch.cuda.synchronize()
        if stage == "pre":
            state["toks"] = {j: _sample(rng, cfg.T, 4) for j, _ in runset}
            state["x_pre"] = {j: to_np(st.x[j][torch.tensor(state["toks"][j], device=device)])
                              for j, _ in runset}
            for j, l in runset:
                z = to_np(st.logits[j])
                idx = st.idx[j].cpu().numpy()
                assert np.array_equal(idx, omodel.topk_indices(z, cfg.k)), (j, l)
                assert np.array_equal(st.counts[j].cpu().numpy(), omodel.expert_counts(idx, cfg.E))
                assert_close(to_np(st.w[j]), omodel.gate_weights(z, idx, cfg.norm_topk), cfg.dtype, "w")
                toks = state["toks"][j]
                a_ref = omodel.rmsnorm_cast(state["x_pre"][j], P_host.gain(l), cfg.eps, cast)
                a_gpu = to_np(st.a[j][torch.tensor(toks, device=device)])
                assert_close(a_gpu, a_ref, cfg.dtype, "a")
                assert_close(z[toks], omodel.router_logits(a_gpu, P_host.router(l), P_host.bias(l)),
                             cfg.dtype, "logits")
            return
        n_steps[0] += 1
        run_np = [(l, st.idx[j].cpu().numpy()) for j, l in runset]
        keys = operm.step_keys(run_np, cfg.E, cfg.S)
        _, inv_ref, off_ref = operm.stable_permutation(keys, cfg.L * ES)
        P = keys.size
        inv = st.inv[:P].cpu().numpy()
        assert np.array_equal(inv, inv_ref)
        assert np.array_equal(views["offsets"].cpu().numpy(), off_ref)
        # one routed and (if any) one shared pair of the step, recomputed by the oracle
        picks = [int(rng.integers(0, P // slots)) * slots + int(rng.integers(0, cfg.k))]
        if cfg.S:
            picks.append(int(rng.integers(0, P // slots)) * slots + cfg.k + int(rng.integers(0, cfg.S)))
        for q in picks:
            rho, rem = divmod(q, cfg.T * slots)
            t, r = divmod(rem, slots)
            j, l = runset[rho]
            e = int(run_np[rho][1][t, r]) if r < cfg.k else cfg.E + (r - cfg.k)
            pos = int(inv[q])
            a_row = to_np(views["a_perm"][pos:pos + 1])
            assert np.array_equal(a_row, to_np(st.a[j][t:t + 1]))
            Wg_, Wu_ = P_host.gate_up(l, e)
            Wd_ = P_host.down(l, e)
            h_ref, _ = omodel.expert_ffn(a_row, Wg_, Wu_, Wd_, cast)
            h_gpu = to_np(views["h"][pos:pos + 1])
            assert_close(h_gpu, h_ref, cfg.dtype, f"h (layer {l}, expert {e})")
            o_ref = cast(h_gpu @ np.asarray(Wd_, np.float64).T)
            assert_close(to_np(st.o[pos:pos + 1]), o_ref, cfg.dtype, f"o (layer {l}, expert {e})")
        # combine on sampled tokens of every entry, from the GPU's o
        for rho, (j, l) in enumerate(runset):
            toks = state["toks"][j]
            q0 = rho * cfg.T * slots
            rows = np.stack([inv[q0 + t * slots:q0 + (t + 1) * slots] for t in toks])
            o_rows = to_np(st.o[torch.from_numpy(rows.reshape(-1)).to(device)]).reshape(len(toks), slots, cfg.H)
            want = omodel.combine(state["x_pre"][j], o_rows[:, :cfg.k], to_np(st.w[j])[toks],
                                  o_rows[:, cfg.k:] if cfg.S else None)
            assert_close(to_np(st.x[j][torch.tensor(toks, device=device)]), want, "f32",
                         "x after combine")
        log(f"  step {n_steps[0]}: {[(j, l) for j, l in runset]} P={P} ok")

    steps = st.run("maxutil", m=cfg.m, views=views, hook=hook)
    torch.cuda.synchronize()
    assert [s.runset for s in steps] == osched.run_algorithm1(st.layer_loads, cfg.m, osched.MAXUTIL)
    x_eb = st.x.clone()
    log(f"full-size {cfg.name}: lock-step pass")
    st.x.copy_(inp.x0)
    st.run("lockstep", record=False)
    torch.cuda.synchronize()
    assert torch.equal(st.x, x_eb), "EB and lock-step hidden states differ"
    log(f"full-size {cfg.name}: {len(steps)} steps verified")
