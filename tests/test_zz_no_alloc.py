"""easybalance_moe_step_noalloc (the entry point for callers that cannot
allocate) against easybalance_moe_step on the same inputs, through the C ABI:
two calls in a row on one device, the second with a smaller step, each giving
the same grouped rows, activations, outputs and permutation bit for bit (the
same kernels run on the library's static scratch instead of a workspace)."""
import numpy as np
import pytest
import torch

from synth import BY_NAME, gen, mini
from synth.device import DeviceInputs, fill_

from gpu_helpers import ensure_packed, log

pytestmark = pytest.mark.gpu

# long K: the down GEMM's split-K partial sums live in the scratch too
LONGK = mini(BY_NAME["mixtral_bf16"], H=256, F=8192, T=96, L=2)
CFGS = [mini(BY_NAME["qwen_moe_bf16"]), LONGK]
IDS = ["qwen_moe_mini", "mixtral_longk"]


def _binding():
    from paper_2608_07964_amd import binding as B
    B.lib()
    return B


def _entries(B, desc, cfg, inp, plan, device):
    ents = []
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    for j, l, T in plan:
        e = dict(j=j, l=l, T=T, x=inp.x0[j, :T].clone(),
                 a=torch.empty(max(T, 1), cfg.H, dtype=tdt, device=device),
                 idx=torch.empty(max(T, 1), cfg.k, dtype=torch.int32, device=device),
                 w=torch.empty(max(T, 1), cfg.k, dtype=torch.float32, device=device),
                 counts=torch.empty(cfg.E, dtype=torch.int32, device=device))
        B.easybalance_route(desc, l, T, e["x"], inp.g[l], inp.Wg[l], inp.bias[l], e["a"], None,
                            e["idx"], e["w"], e["counts"])
        ents.append(e)
    return ents


def _outputs(cfg, P, device):
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    o = torch.full((P, cfg.H), float("nan"), dtype=tdt, device=device)
    inv = torch.full((P,), -1, dtype=torch.int32, device=device)
    views = dict(a_perm=torch.full((P, cfg.H), float("nan"), dtype=tdt, device=device),
                 h=torch.full((P, cfg.F), float("nan"), dtype=tdt, device=device),
                 perm=torch.full((P,), -1, dtype=torch.int32, device=device),
                 offsets=torch.full((cfg.L * (cfg.E + cfg.S) + 1,), -1, dtype=torch.int32, device=device))
    return o, inv, views


def _same(a, b, what):
    if a.dtype == torch.bfloat16:
        a, b = a.view(torch.int16), b.view(torch.int16)
    assert torch.equal(a, b), what


@pytest.mark.parametrize("cfg", CFGS, ids=IDS)
def test_noalloc_matches_workspace_entry_point(cfg, device):
    B = _binding()
    inp = ensure_packed(cfg, DeviceInputs(cfg, device))
    desc = B.make_desc(cfg.L, cfg.H, cfg.F, cfg.E, cfg.k, cfg.S, cfg.D, cfg.dtype, cfg.eps)
    L, N, T = cfg.L, cfg.N, cfg.T
    plans = [[(0, min(1, L - 1), T), (1, L - 1, T - 37), (2 % N, 0, 0), (N - 1, 0, 5)],
             [(1, 0, 11), (N - 1, L - 1, 3)]]           # the second call: a smaller step
    for call, plan in enumerate(plans):
        log(f"no-alloc step {cfg.name} call {call} plan {plan}")
        ents = _entries(B, desc, cfg, inp, plan, device)
        run = B.work_array((e["j"], e["l"], e["T"], e["a"], e["idx"], e["w"]) for e in ents)
        Ts = [e["T"] for e in ents]
        P = sum(Ts) * (cfg.k + cfg.S)
        # existing entry point, caller workspace
        ws_bytes = B.easybalance_moe_step_workspace_size(desc, Ts)
        ws = torch.empty(ws_bytes + 256, dtype=torch.uint8, device=device)
        wsp = ws.data_ptr() + (-ws.data_ptr()) % 256
        o_ref, inv_ref, v_ref = _outputs(cfg, P, device)
        B.easybalance_moe_step(desc, run, len(ents), inp.W_gu, inp.W_dn, wsp, ws_bytes, o_ref, inv_ref, v_ref)
        # no-alloc entry point: perm and offsets in the static scratch on the
        # first call, in the caller's views on the second
        o, inv, v = _outputs(cfg, P, device)
        if call == 0:
            v_pass = dict(a_perm=v["a_perm"], h=v["h"])
        else:
            v_pass = v
        B.easybalance_moe_step_noalloc(desc, run, len(ents), inp.W_gu, inp.W_dn, o, inv, v_pass)
        torch.cuda.synchronize()
        _same(inv, inv_ref, "inv")
        _same(o, o_ref, "o")
        _same(v["a_perm"], v_ref["a_perm"], "a_perm")
        _same(v["h"], v_ref["h"], "h")
        if call == 1:
            _same(v["perm"], v_ref["perm"], "perm")
            _same(v["offsets"], v_ref["offsets"], "offsets")
        assert np.isfinite(o.float().cpu().numpy()).all()


def test_noalloc_argument_errors(device):
    """views with a_perm and h are required; a step whose scratch need exceeds
    the static array is refused before anything is enqueued (every buffer here
    is real and sized for the step, so nothing could go out of bounds)."""
    B = _binding()
    cfg = mini(BY_NAME["mixtral_bf16"], H=256, F=8192, L=1)
    inp = ensure_packed(cfg, DeviceInputs(cfg, device))
    desc = B.make_desc(cfg.L, cfg.H, cfg.F, cfg.E, cfg.k, cfg.S, cfg.D, cfg.dtype, cfg.eps)
    # 41000 tokens, k = 2: split-K partials 2 * 82000 * 256 * 4 B = 160.2 MiB > 160 MiB
    T = 41000
    log(f"no-alloc refusal T={T}")
    a = fill_(torch.empty(T, cfg.H, dtype=torch.bfloat16, device=device), cfg, gen.KIND_X, 0)
    idx = torch.stack([torch.arange(T, device=device) % cfg.E,
                       (torch.arange(T, device=device) + 1) % cfg.E], 1).to(torch.int32).contiguous()
    w = torch.full((T, 2), 0.5, device=device)
    run = B.work_array([(0, 0, T, a, idx, w)])
    P = 2 * T
    o, inv, v = _outputs(cfg, P, device)
    with pytest.raises(B.EasyBalanceError) as ei:
        B.easybalance_moe_step_noalloc(desc, run, 1, inp.W_gu, inp.W_dn, o, inv, dict(a_perm=v["a_perm"]))
    assert ei.value.code == B.EB_ERR_INVALID_ARG
    with pytest.raises(B.EasyBalanceError) as ei:
        B.easybalance_moe_step_noalloc(desc, run, 1, inp.W_gu, inp.W_dn, o, inv, v)
    assert ei.value.code == B.EB_ERR_UNSUPPORTED and "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert (inv == -1).all().item()          # nothing ran
