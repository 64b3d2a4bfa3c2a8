"""Full-size parity of the five stacks, in the launch configuration bench.py
times (one Algorithm-1 pass with MaxUtil and m = 0.75 N, every step one
moe_step + combine), against the CPU oracle:

* every step, all tokens: top-k indices equal the stable top-k of the GPU's
  own logits, counts equal their bincount, the grouping (inv, offsets) equals
  the oracle's stable sort by (layer, expert) -- bit-exact;
* the executed schedule equals the oracle's replay of Algorithm 1 on the
  loads the GPU observed -- bit-exact;
* 64 tokens per micro-batch and step: a, logits, w and x after the combine;
* h and o of every row of the step's largest and smallest (layer, expert)
  groups (at most 8192 of them) and of up to 256 rows (first, last and a spread between) of every
  other group (the DeepSeek-V3 shape: of 48 of its many groups per step),
  each on a random set of output columns, the oracle recomputing them from
  the GPU's grouped rows (h) and SwiGLU activations (o) with the expert's
  weight rows regenerated on the host -- max-abs error <= 1e-2 * max|ref|
  (bf16 stacks) / 1e-5 * max|ref| (fp32);
* the EB pass and the per-layer lock-step pass end in bit-identical hidden
  states (cross-layer combination is lossless, Section 4.1).

test_free_running_drift reports, without gating, how far the bf16 stacks'
free-running GPU pass drifts from the oracle's own free-running run over the
first two layers (routing flips per (micro-batch, layer), max-abs of x): near
ties of the router logits flip some tokens' experts between fp32 on the GPU
and float64 on the host, which is why the gates above are teacher-forced.
"""
import numpy as np
import pytest
import torch

from oracle import model as omodel
from oracle import permute as operm
from oracle import sched as osched
from oracle.numerics import cast_fn
from synth import BY_NAME, CONFIGS, gen
from synth.device import DeviceInputs

from gpu_helpers import assert_close, host_weights, log, make_stack, to_np

pytestmark = pytest.mark.gpu


def _sample(rng, n, k):
    return sorted(rng.choice(n, size=min(k, n), replace=False).tolist()) if n else []


def _weight_rows(cfg, kind, layer, e, rows, row_len, rows_per_expert):
    """Rows of expert slot e's generated weight matrix (stored values, float64),
    regenerated one row at a time on the host."""
    base = e * rows_per_expert * row_len
    return np.stack([gen.tensor_values(cfg, kind, layer, base + int(r) * row_len, row_len)
                     for r in rows]).astype(np.float64)


def _rows_to_check(rng, M, full):
    """All rows of a group (at most 8192: the DeepSeek-V3 shape's hottest
    groups hold tens of thousands), or 256 of them: first, last and the rest
    drawn between."""
    n = min(M, 8192) if full else min(M, 256)
    if n == M:
        return np.arange(M)
    mid = rng.choice(np.arange(1, M - 1), size=n - 2, replace=False)
    return np.sort(np.concatenate([[0, M - 1], mid]))


def _check_groups(cfg, step_no, runset, off, a_perm_dev, h_dev, o_dev, rng, cast):
    """h and o of the step's groups on sampled output columns (see the module
    docstring); returns (groups checked, rows checked)."""
    ES = cfg.E + cfg.S
    sizes = np.diff(off)
    keys = np.nonzero(sizes)[0]
    big, small = keys[np.argmax(sizes[keys])], keys[np.argmin(sizes[keys])]
    ncols = 32 if cfg.H * cfg.F >= 7168 * 2048 else 128
    if len(keys) > 48:
        keys = np.unique(np.concatenate([[big, small], rng.choice(keys, size=46, replace=False)]))
    n_rows = 0
    for key in keys:
        r0, r1 = int(off[key]), int(off[key + 1])
        l, e = divmod(int(key), ES)
        rows = r0 + _rows_to_check(rng, r1 - r0, key in (big, small))
        idx = torch.from_numpy(rows).to(a_perm_dev.device)
        a_rows = to_np(a_perm_dev[idx])
        fs = np.sort(rng.choice(cfg.F, size=min(ncols, cfg.F), replace=False))
        ns = np.sort(rng.choice(cfg.H, size=min(ncols, cfg.H), replace=False))
        Wg_ = _weight_rows(cfg, gen.KIND_GU, l, e, fs, cfg.H, 2 * cfg.F)
        Wu_ = _weight_rows(cfg, gen.KIND_GU, l, e, cfg.F + fs, cfg.H, 2 * cfg.F)
        Wd_ = _weight_rows(cfg, gen.KIND_DN, l, e, ns, cfg.F, cfg.H)
        # h on columns fs: the SwiGLU of the gate / up rows fs (the oracle's
        # expert, its down projection unused here)
        h_ref, _ = omodel.expert_ffn(a_rows, Wg_, Wu_, np.zeros((1, len(fs))), cast)
        h_rows = to_np(h_dev[idx])
        assert_close(h_rows[:, fs], h_ref, cfg.dtype, f"step {step_no} h (layer {l}, expert {e}, {r1 - r0} rows)")
        # o on columns ns, from the GPU's h (all F columns)
        o_ref = cast(h_rows @ Wd_.T)
        assert_close(to_np(o_dev[idx])[:, ns], o_ref, cfg.dtype,
                     f"step {step_no} o (layer {l}, expert {e}, {r1 - r0} rows)")
        n_rows += len(rows)
    return len(keys), n_rows


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
            state["toks"] = {j: _sample(rng, cfg.T, 64) for j, _ in runset}
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
        # grouped rows are exact copies of their tokens' a rows (sampled pairs)
        for q in rng.choice(P, size=min(64, P), replace=False):
            rho, rem = divmod(int(q), cfg.T * slots)
            t = rem // slots
            j, _ = runset[rho]
            pos = int(inv[q])
            assert np.array_equal(to_np(views["a_perm"][pos:pos + 1]), to_np(st.a[j][t:t + 1]))
        ng, nr = _check_groups(cfg, n_steps[0], runset, off_ref, views["a_perm"], views["h"], st.o, rng, cast)
        # combine on the sampled tokens of every entry, from the GPU's o
        for rho, (j, l) in enumerate(runset):
            toks = state["toks"][j]
            q0 = rho * cfg.T * slots
            rows = np.stack([inv[q0 + t * slots:q0 + (t + 1) * slots] for t in toks])
            o_rows = to_np(st.o[torch.from_numpy(rows.reshape(-1)).to(device)]).reshape(len(toks), slots, cfg.H)
            want = omodel.combine(state["x_pre"][j], o_rows[:, :cfg.k], to_np(st.w[j])[toks],
                                  o_rows[:, cfg.k:] if cfg.S else None)
            assert_close(to_np(st.x[j][torch.tensor(toks, device=device)]), want, "f32",
                         "x after combine")
        log(f"  step {n_steps[0]}: {[(j, l) for j, l in runset]} P={P}: h/o of {nr} rows in {ng} groups ok")

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


@pytest.mark.parametrize("name", ["mixtral_bf16", "qwen_moe_bf16", "dsv2_lite_bf16"])
def test_free_running_drift(name, device):
    """Report (not a gate): the GPU's free-running pass against the oracle's
    free-running plain run over the first two layers, per (micro-batch,
    layer): tokens whose expert set differs, and max-abs of x relative to
    max|x_ref|.  Only finiteness and the shapes are asserted."""
    cfg = BY_NAME[name]
    n_layers = 2
    log(f"drift {cfg.name}: GPU pass")
    st, inp = make_stack(cfg, device)
    idx_gpu, x_gpu = {}, {}

    def hook(stage, runset):
        if stage == "pre":
            for j, l in runset:
                if l < n_layers:
                    idx_gpu[(j, l)] = st.idx[j].cpu().numpy()
        else:
            torch.cuda.synchronize()
            for j, l in runset:
                if l < n_layers:
                    x_gpu[(j, l)] = to_np(st.x[j])

    st.run("lockstep", record=False, hook=hook)
    torch.cuda.synchronize()
    P_host = host_weights(cfg, cache=True)
    x = gen.x_all(cfg).astype(np.float64)
    lines = []
    for l in range(n_layers):
        for j in range(cfg.N):
            out = omodel.moe_layer(x[j], l, P_host, E=cfg.E, k=cfg.k, S=cfg.S, eps=cfg.eps, dtype=cfg.dtype,
                                   norm_topk=cfg.norm_topk)
            x[j] = out.x_out
            flips = int(np.sum(np.any(np.sort(out.idx, axis=1) != np.sort(idx_gpu[(j, l)], axis=1), axis=1)))
            err = float(np.abs(x_gpu[(j, l)] - out.x_out).max() / np.abs(out.x_out).max())
            assert np.isfinite(err)
            lines.append(f"  {cfg.name} micro-batch {j} layer {l}: {flips}/{cfg.T} tokens with another "
                         f"expert set, max-abs(x) {err:.2e} of max|x|")
    log("\n".join(lines))
