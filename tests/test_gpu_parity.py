"""GPU parity of every stage of the hot path against the CPU oracle, through
the C ABI, on seeded inputs at sizes the oracle finishes in seconds (several
GEMM tiles, ragged tails, empty entries).

Contract (teacher-forced where floating point decides an integer):
* idx, counts, perm, inv, offsets, a_perm, schedules: bit-exact;
* activations (a, z, w, h, o, x): max-abs error <= 1e-5 * max|ref| (fp32
  stacks) or 1e-2 * max|ref| (bf16 stacks).
"""
import numpy as np
import pytest
import torch

from oracle import metrics as ometrics
from oracle import model as omodel
from oracle import permute as operm
from oracle import sched as osched
from oracle.numerics import cast_fn
from synth import BY_NAME, CONFIGS, Config, gen, mini
from synth.device import DeviceInputs, fill_

from gpu_helpers import assert_close, ensure_packed, host_weights, log, make_stack, to_np

pytestmark = pytest.mark.gpu

MINIS = [c if c.dtype == "f32" else mini(c) for c in CONFIGS]
IDS = [c.name for c in MINIS]
# long K (F >= 8192): the down GEMM runs its two K halves as separate items
LONGK = mini(BY_NAME["mixtral_bf16"], H=256, F=8192, T=96, L=2)
# many pairs of long rows (k+S = 9 slots of 4 KB rows): the grouping copies
# each token's row piece by piece to all its pairs (gather_tokens_kernel)
ROWONCE = mini(BY_NAME["dsv3_share_bf16"], H=2048, T=96, L=2)
STEP_CFGS = MINIS + [LONGK, ROWONCE]
STEP_IDS = IDS + [LONGK.name + "_longk", ROWONCE.name + "_rowonce"]
# the ABI's shape limits and the method's degenerate mixtures:
# * k + S = 16 expert slots per token (12 routed picks of 64, 4 shared), also
#   with rows of several pieces in the grouping;
# * k = E (every token on every expert), bf16 and fp32;
# * L * (E + S) = 15360 keys in one step's grouping, with E = 252 experts
#   (not a multiple of the router's 32-expert blocks);
# * 100 experts (the router's form for 65..128 experts)
MAXSLOTS = Config("maxslots_bf16", L=2, H=256, F=256, E=64, k=12, S=4, D=8, N=4, T=96, dtype="bf16",
                  skew="zipf", skew_param=1.1, seed=20261001)
LIMIT_CFGS = [
    MAXSLOTS,
    MAXSLOTS.scaled(name="maxslots_rowonce_bf16", H=2048, T=64, seed=20261002),
    Config("dense_bf16", L=2, H=256, F=256, E=8, k=8, S=0, D=4, N=4, T=96, dtype="bf16",
           skew="zipf", skew_param=1.0, seed=20261003),
    Config("dense_f32", L=2, H=256, F=128, E=8, k=8, S=1, D=8, N=3, T=70, dtype="f32",
           skew="dirichlet", skew_param=0.3, seed=20261004),
    Config("maxkeys_bf16", L=60, H=256, F=128, E=252, k=2, S=4, D=4, N=4, T=48, dtype="bf16",
           skew="zipf", skew_param=1.2, seed=20261005),
    # 65..128 experts: the router's one-expert-block-per-wavefront form, a
    # 128-token tile plus a ragged one
    Config("experts100_bf16", L=2, H=512, F=256, E=100, k=6, S=2, D=4, N=3, T=150, dtype="bf16",
           skew="dirichlet", skew_param=0.3, seed=20261006),
    # fp32 routing paths: the per-token kernel with rows over 4096 wide and
    # with 9..64 experts, and the separate logits and top-k kernels above 64
    Config("wide_f32", L=2, H=6144, F=128, E=8, k=2, S=0, D=4, N=2, T=40, dtype="f32",
           skew="zipf", skew_param=1.2, seed=20261007),
    Config("experts40_f32", L=2, H=256, F=128, E=40, k=4, S=1, D=8, N=3, T=70, dtype="f32",
           skew="zipf", skew_param=1.1, seed=20261008),
    Config("experts96_f32", L=2, H=256, F=128, E=96, k=3, S=0, D=4, N=3, T=70, dtype="f32",
           skew="dirichlet", skew_param=0.3, seed=20261009),
]
LIMIT_IDS = [c.name for c in LIMIT_CFGS]
# the RMSNorm in front of the separate router kernels, by row length: a
# workgroup per token holding 4 float4 of the row per thread (2048 < H <=
# 4096), 8 (4096 < H <= 8192), and one wavefront per token above that; and
# the matrix-core router with most of its 64 expert rows padding (E = 20)
NORM_CFGS = [
    Config("experts20_bf16", L=1, H=512, F=128, E=20, k=3, S=0, D=4, N=2, T=70, dtype="bf16",
           skew="zipf", skew_param=1.1, seed=20261013),
    Config("norm4_bf16", L=1, H=4096, F=128, E=64, k=4, S=0, D=4, N=2, T=70, dtype="bf16",
           skew="zipf", skew_param=1.1, seed=20261010),
    Config("norm8_f32", L=1, H=5120, F=128, E=96, k=3, S=0, D=4, N=2, T=70, dtype="f32",
           skew="dirichlet", skew_param=0.3, seed=20261011),
    Config("normwave_bf16", L=1, H=8448, F=128, E=100, k=6, S=0, D=4, N=2, T=70, dtype="bf16",
           skew="dirichlet", skew_param=0.3, seed=20261012),
    Config("normwave64_bf16", L=1, H=8448, F=128, E=64, k=6, S=0, D=4, N=2, T=70, dtype="bf16",
           skew="dirichlet", skew_param=0.3, seed=20261014),
]
NORM_IDS = [c.name for c in NORM_CFGS]


def _binding():
    from paper_2608_07964_amd import binding as B
    B.lib()
    return B


def _pack_reference(W: np.ndarray, F: int, gateup: bool) -> np.ndarray:
    """The packed layout as include/easybalance.h states it, for n matrices
    W [n][N][K] of 16-bit patterns: block (s, t) = K columns 64 s .. of
    column tile t, block row r = a weight row (gate/up rows interleaved per
    64), chunk c = the 8 columns of logical chunk c ^ ((r >> 1) & 7)."""
    n, N, K = W.shape
    r = np.arange(256)
    out = np.empty((n, K // 64, N // 256, 256, 8, 8), dtype=W.dtype)
    for t in range(N // 256):
        if gateup:
            q = r % 64
            rows = 128 * t + 32 * (r // 64) + np.where(q < 32, q, q - 32 + F)
        else:
            rows = 256 * t + r
        for s in range(K // 64):
            for c in range(8):
                cols = 64 * s + 8 * (c ^ ((r >> 1) & 7))[:, None] + np.arange(8)[None, :]
                out[:, s, t, :, c, :] = W[:, rows[:, None], cols]
    return out.reshape(n, N * K)


def test_pack_weights_layout(device):
    """easybalance_pack_weights: every element of the packed bf16 gate/up and
    down matrices of three experts sits where the documented layout puts it
    (bit-exact, random bit patterns); fp32 packing is a copy."""
    B = _binding()
    for H, F in ((512, 384), (256, 128)):
        log(f"pack layout H={H} F={F}")
        desc = B.make_desc(1, H, F, 8, 2, 0, 4, "bf16")
        g = torch.Generator(device="cpu").manual_seed(H + F)
        for kind, N, K in ((B.EB_WEIGHTS_GATE_UP, 2 * F, H), (B.EB_WEIGHTS_DOWN, H, F)):
            bits = torch.randint(-32768, 32768, (3, N, K), generator=g, dtype=torch.int32).to(torch.int16)
            src = bits.to(device).view(torch.bfloat16)
            dst = torch.empty_like(src)
            B.easybalance_pack_weights(desc, kind, 3, src, dst)
            torch.cuda.synchronize()
            got = dst.view(torch.int16).cpu().numpy().reshape(3, N * K)
            ref = _pack_reference(bits.numpy(), F, kind == B.EB_WEIGHTS_GATE_UP)
            assert np.array_equal(got, ref), (H, F, kind)
            assert torch.equal(src.view(torch.int16).cpu(), bits)  # src untouched
    d32 = B.make_desc(1, 256, 128, 8, 2, 0, 4, "f32")
    src = torch.randn(2, 256, 128, device=device)
    dst = torch.empty_like(src)
    B.easybalance_pack_weights(d32, B.EB_WEIGHTS_DOWN, 2, src, dst)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)


def test_device_generator_bit_exact(device):
    cfg = MINIS[1]
    for kind, index, dt in [(gen.KIND_X, 0, torch.float32), (gen.KIND_GU, 2, torch.bfloat16),
                            (gen.KIND_WG, 1, torch.float32), (gen.KIND_DN, 0, torch.bfloat16)]:
        t = fill_(torch.empty(100003, dtype=dt, device=device), cfg, kind, index, i0=777)
        ref = gen.normal_f32(gen.stream_key(cfg.seed, kind, index), 777, 100003, gen.sigma_of(kind, cfg.H))
        if dt == torch.bfloat16:
            got = t.view(torch.int16).cpu().numpy().view(np.uint16)
            assert np.array_equal(got, gen.f32_to_bf16_bits(ref))
        else:
            assert np.array_equal(t.cpu().numpy(), ref)


@pytest.mark.parametrize("cfg", MINIS + LIMIT_CFGS + NORM_CFGS, ids=IDS + LIMIT_IDS + NORM_IDS)
def test_route_stage(cfg, device):
    B = _binding()
    log(f"route parity {cfg.name}")
    inp = DeviceInputs(cfg, device, weights=False)
    P = host_weights(cfg)
    desc = B.make_desc(cfg.L, cfg.H, cfg.F, cfg.E, cfg.k, cfg.S, cfg.D, cfg.dtype, cfg.eps)
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    for T, l, j in [(cfg.T, cfg.L - 1, 1), (1, 0, 0), (cfg.T - 3, 0, cfg.N - 1)]:
        x = inp.x0[j, :T].clone()
        a = torch.empty(T, cfg.H, dtype=tdt, device=device)
        z = torch.empty(T, cfg.E, dtype=torch.float32, device=device)
        idx = torch.empty(T, cfg.k, dtype=torch.int32, device=device)
        w = torch.empty(T, cfg.k, dtype=torch.float32, device=device)
        counts = torch.full((cfg.E,), 12345, dtype=torch.int32, device=device)
        B.easybalance_route(desc, l, T, x, inp.g[l], inp.Wg[l], inp.bias[l], a, z, idx, w, counts)
        torch.cuda.synchronize()
        xh = to_np(x)
        a_ref = omodel.rmsnorm_cast(xh, P.gain(l), cfg.eps, cast_fn(cfg.dtype))
        assert_close(to_np(a), a_ref, cfg.dtype, "a")
        zg = to_np(z)
        assert_close(zg, omodel.router_logits(to_np(a), P.router(l), P.bias(l)), cfg.dtype, "logits")
        idx_ref = omodel.topk_indices(zg, cfg.k)                      # teacher-forced on GPU logits
        assert np.array_equal(idx.cpu().numpy(), idx_ref)
        assert_close(to_np(w), omodel.gate_weights(zg, idx_ref, cfg.norm_topk), cfg.dtype, "w")
        assert np.array_equal(counts.cpu().numpy(), omodel.expert_counts(idx_ref, cfg.E))


def _route_entry(B, desc, cfg, inp, j, l, T, device):
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    x = inp.x0[j, :T].clone()
    bufs = dict(x=x, a=torch.zeros(max(T, 1), cfg.H, dtype=tdt, device=device),
                z=torch.empty(max(T, 1), cfg.E, dtype=torch.float32, device=device),
                idx=torch.empty(max(T, 1), cfg.k, dtype=torch.int32, device=device),
                w=torch.empty(max(T, 1), cfg.k, dtype=torch.float32, device=device),
                counts=torch.empty(cfg.E, dtype=torch.int32, device=device), T=T, l=l, j=j)
    B.easybalance_route(desc, l, T, x, inp.g[l], inp.Wg[l], inp.bias[l], bufs["a"], bufs["z"],
                        bufs["idx"], bufs["w"], bufs["counts"])
    return bufs


@pytest.mark.parametrize("cfg", STEP_CFGS + LIMIT_CFGS, ids=STEP_IDS + LIMIT_IDS)
def test_moe_step_and_combine_stage(cfg, device):
    """One cross-layer step with entries at different layers, ragged and empty
    token counts; every stage checked against the oracle on the GPU's inputs."""
    B = _binding()
    log(f"step parity {cfg.name}")
    inp = ensure_packed(cfg, DeviceInputs(cfg, device))
    P = host_weights(cfg)
    cast = cast_fn(cfg.dtype)
    desc = B.make_desc(cfg.L, cfg.H, cfg.F, cfg.E, cfg.k, cfg.S, cfg.D, cfg.dtype, cfg.eps)
    L = cfg.L
    plan = [(0, min(1, L - 1), cfg.T), (1, L - 1, cfg.T - 37), (2 % cfg.N, 0, 0),
            (cfg.N - 1, 0, 5 if cfg.T > 5 else 1)]
    ents = [_route_entry(B, desc, cfg, inp, j, l, T, device) for j, l, T in plan]
    run = B.work_array((e["j"], e["l"], e["T"], e["a"], e["idx"], e["w"]) for e in ents)
    Ts = [e["T"] for e in ents]
    slots = cfg.k + cfg.S
    Ptot = sum(Ts) * slots
    ws_bytes = B.easybalance_moe_step_workspace_size(desc, Ts)
    ws = torch.empty(ws_bytes + 256, dtype=torch.uint8, device=device)
    wsp = ws.data_ptr() + (-ws.data_ptr()) % 256
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    o = torch.empty(Ptot, cfg.H, dtype=tdt, device=device)
    inv = torch.empty(Ptot, dtype=torch.int32, device=device)
    views = dict(a_perm=torch.empty(Ptot, cfg.H, dtype=tdt, device=device),
                 h=torch.empty(Ptot, cfg.F, dtype=tdt, device=device),
                 perm=torch.empty(Ptot, dtype=torch.int32, device=device),
                 offsets=torch.empty(L * (cfg.E + cfg.S) + 1, dtype=torch.int32, device=device))
    B.easybalance_moe_step(desc, run, len(ents), inp.W_gu, inp.W_dn, wsp, ws_bytes, o, inv, views)
    x_before = [to_np(e["x"]) for e in ents]
    B.easybalance_combine(desc, run, len(ents), [e["x"] for e in ents], o, inv)
    torch.cuda.synchronize()

    # permutation: bit-exact against the stable sort of the GPU's own routing
    run_np = [(e["l"], e["idx"].cpu().numpy()[:e["T"]]) for e in ents]
    keys = operm.step_keys(run_np, cfg.E, cfg.S)
    perm_ref, inv_ref, off_ref = operm.stable_permutation(keys, L * (cfg.E + cfg.S))
    assert np.array_equal(inv.cpu().numpy(), inv_ref)
    assert np.array_equal(views["perm"].cpu().numpy(), perm_ref)
    assert np.array_equal(views["offsets"].cpu().numpy(), off_ref)
    # grouped activation rows are exact copies
    src = operm.source_rows(run_np, cfg.S)
    a_all = [to_np(e["a"]) for e in ents]
    a_perm = to_np(views["a_perm"])
    assert np.array_equal(a_perm[inv_ref], np.stack([a_all[r][t] for r, t in src]) if len(src) else a_perm[:0])
    # expert FFN per group, teacher-forced on the GPU's a_perm (h) and h (o)
    h_gpu, o_gpu = to_np(views["h"]), to_np(o)
    h_ref = np.zeros_like(h_gpu)
    o_ref = np.zeros_like(o_gpu)
    for key in range(L * (cfg.E + cfg.S)):
        r0, r1 = off_ref[key], off_ref[key + 1]
        if r0 == r1:
            continue
        l, e = divmod(key, cfg.E + cfg.S)
        Wg_, Wu_ = P.gate_up(l, e)
        Wd_ = P.down(l, e)
        h_ref[r0:r1], _ = omodel.expert_ffn(a_perm[r0:r1], Wg_, Wu_, Wd_, cast)
        o_ref[r0:r1] = cast(h_gpu[r0:r1] @ np.asarray(Wd_, np.float64).T)
    assert_close(h_gpu, h_ref, cfg.dtype, "h")
    assert_close(o_gpu, o_ref, cfg.dtype, "o")
    # combine: x + sum_r w_r o_r + sum_s o_s, on the GPU's o
    q = 0
    for e, xb in zip(ents, x_before):
        T = e["T"]
        if T == 0:
            continue
        rows = inv_ref[q:q + T * slots].reshape(T, slots)
        q += T * slots
        want = omodel.combine(xb, o_gpu[rows[:, :cfg.k]], to_np(e["w"])[:T],
                              o_gpu[rows[:, cfg.k:]] if cfg.S else None)
        assert_close(to_np(e["x"]), want, "f32", "x after combine")


def test_tiny_fp32_end_to_end_free_running(device):
    """The fp32 stack through the whole EB pass against the oracle's plain
    layer-by-layer run: routing, schedule and hidden states."""
    cfg = BY_NAME["tiny_f32"]
    log("end-to-end tiny fp32")
    st, inp = make_stack(cfg, device)
    steps = st.run("maxutil", m=cfg.m)
    torch.cuda.synchronize()
    P = host_weights(cfg)
    ref = omodel.run_plain(gen.x_all(cfg), P, L=cfg.L, E=cfg.E, k=cfg.k, S=cfg.S, D=cfg.D,
                           eps=cfg.eps, dtype=cfg.dtype)
    # the seed gives no near-ties: the k-th and (k+1)-th logits are well apart
    for j in range(cfg.N):
        for l in range(cfg.L):
            a = omodel.rmsnorm_cast(ref.x[l, j], P.gain(l), cfg.eps, cast_fn(cfg.dtype))
            z = np.sort(omodel.router_logits(a, P.router(l), P.bias(l)), axis=1)[:, ::-1]
            assert np.min(z[:, cfg.k - 1] - z[:, cfg.k]) > 1e-4
    assert np.array_equal(st.layer_loads, ref.loads)
    assert [s.runset for s in steps] == osched.run_algorithm1(ref.loads, cfg.m, osched.MAXUTIL)
    assert_close(to_np(st.x), ref.x[cfg.L], cfg.dtype, "x final")


@pytest.mark.parametrize("cfg", STEP_CFGS, ids=STEP_IDS)
def test_schedule_invariance_and_replay(cfg, device):
    """Cross-layer joint execution is lossless (Section 4.1): the EB schedule
    and the per-layer lock-step schedule give bit-identical hidden states, and
    every executed schedule is the oracle's replay of Algorithm 1 on the loads
    the GPU observed."""
    log(f"invariance {cfg.name}")
    inp = DeviceInputs(cfg, device)
    results = {}
    for policy, m in [("lockstep", None), ("maxutil", cfg.m), ("maxutil", 1), ("cumutil", cfg.m),
                      ("diffpeak", cfg.m)]:
        st, _ = make_stack(cfg, device, inputs=inp)
        steps = st.run(policy, m=m)
        torch.cuda.synchronize()
        results[(policy, m)] = (st.x.clone(), steps, st.layer_loads.copy())
        if policy != "lockstep":
            pol = {"maxutil": osched.MAXUTIL, "cumutil": osched.CUMUTIL, "diffpeak": osched.DIFFPEAK}[policy]
            assert [s.runset for s in steps] == osched.run_algorithm1(st.layer_loads, m, pol)
            for s in steps:
                assert np.array_equal(s.load, ometrics.step_workload(st.layer_loads, s.runset))
    x_ls, steps_ls, loads_ls = results[("lockstep", None)]
    assert [s.runset for s in steps_ls] == osched.lockstep_steps(cfg.N, cfg.L)
    for key, (x, steps, loads) in results.items():
        assert np.array_equal(loads, loads_ls), key
        assert torch.equal(x, x_ls), f"{key}: hidden states differ from lock-step"
    # worst-case safety on the observed loads
    eb = results[("maxutil", cfg.m)][1]
    assert (ometrics.utilization(loads_ls, [s.runset for s in eb])
            >= ometrics.utilization(loads_ls, osched.separate_steps(cfg.N, cfg.L)))


# group sizes on both sides of every tile-shape boundary (64 / 128 / 256-row
# m-tiles, 32-row MFMA blocks, rows split evenly over two wavefront rows),
# and groups of more m-tiles than one block of the GEMM's item order (5 and 6
# m-tiles: a block of four and a ragged one)
EDGE_SIZES = [[150, 129, 193, 65, 33, 1, 287, 64], [160, 161, 192, 128, 127, 63, 31, 256],
              [255, 257, 96, 32, 0, 97, 200, 3], [1100, 1500, 300, 0, 500, 7, 64, 1]]


def test_moe_step_group_sizes_span_tile_shapes(device):
    """Crafted routing (not the router's): one entry per row of EDGE_SIZES, at different layers,
    whose (layer, expert) groups take every row count around the tile-shape
    boundaries; every row of h and o checked against the oracle."""
    B = _binding()
    cfg = mini(BY_NAME["mixtral_bf16"], H=256, F=256, L=len(EDGE_SIZES))
    assert cfg.k == 2 and cfg.E == 8 and cfg.S == 0
    log(f"group-size parity {cfg.name}")
    inp = ensure_packed(cfg, DeviceInputs(cfg, device))
    P = host_weights(cfg)
    cast = cast_fn(cfg.dtype)
    desc = B.make_desc(cfg.L, cfg.H, cfg.F, cfg.E, cfg.k, cfg.S, cfg.D, cfg.dtype, cfg.eps)
    ents = []
    for l, sizes in enumerate(EDGE_SIZES):
        T = sum(sizes) // 2
        assert sum(sizes) == 2 * T and max(sizes) <= T
        # slot 0 takes the first T ids of the sorted list, slot 1 the rest: a
        # token's two experts differ because no expert has more than T pairs
        ids = np.repeat(np.arange(cfg.E), sizes).astype(np.int32)
        idx = np.stack([ids[:T], ids[T:]], axis=1)
        assert (idx[:, 0] != idx[:, 1]).all()
        a = fill_(torch.empty(T, cfg.H, dtype=torch.bfloat16, device=device), cfg, gen.KIND_X, l)
        ents.append(dict(j=l, l=l, T=T, a=a, idx=torch.from_numpy(idx).to(device),
                         w=torch.full((T, 2), 0.5, device=device), idx_np=idx))
    run = B.work_array((e["j"], e["l"], e["T"], e["a"], e["idx"], e["w"]) for e in ents)
    Ts = [e["T"] for e in ents]
    Ptot = 2 * sum(Ts)
    ws_bytes = B.easybalance_moe_step_workspace_size(desc, Ts)
    ws = torch.empty(ws_bytes + 256, dtype=torch.uint8, device=device)
    wsp = ws.data_ptr() + (-ws.data_ptr()) % 256
    o = torch.empty(Ptot, cfg.H, dtype=torch.bfloat16, device=device)
    inv = torch.empty(Ptot, dtype=torch.int32, device=device)
    views = dict(a_perm=torch.empty(Ptot, cfg.H, dtype=torch.bfloat16, device=device),
                 h=torch.empty(Ptot, cfg.F, dtype=torch.bfloat16, device=device),
                 perm=torch.empty(Ptot, dtype=torch.int32, device=device),
                 offsets=torch.empty(cfg.L * cfg.E + 1, dtype=torch.int32, device=device))
    B.easybalance_moe_step(desc, run, len(ents), inp.W_gu, inp.W_dn, wsp, ws_bytes, o, inv, views)
    torch.cuda.synchronize()
    off = views["offsets"].cpu().numpy()
    got_sizes = np.diff(off).reshape(cfg.L, cfg.E)
    assert np.array_equal(got_sizes, np.asarray(EDGE_SIZES))
    a_perm, h_gpu, o_gpu = to_np(views["a_perm"]), to_np(views["h"]), to_np(o)
    for key in range(cfg.L * cfg.E):
        r0, r1 = off[key], off[key + 1]
        if r0 == r1:
            continue
        l, e = divmod(key, cfg.E)
        Wg_, Wu_ = P.gate_up(l, e)
        h_ref, _ = omodel.expert_ffn(a_perm[r0:r1], Wg_, Wu_, P.down(l, e), cast)
        assert_close(h_gpu[r0:r1], h_ref, cfg.dtype, f"h rows={r1 - r0}")
        o_ref = cast(h_gpu[r0:r1] @ np.asarray(P.down(l, e), np.float64).T)
        assert_close(o_gpu[r0:r1], o_ref, cfg.dtype, f"o rows={r1 - r0}")


@pytest.mark.parametrize("name", ["mixtral_bf16", "qwen_moe_bf16", "dsv3_share_bf16", "tiny_f32"])
def test_route_nan_logits_pick_distinct_experts(name, device):
    """NaN logits rank after every number: with NaN in the router bias of all
    but a few experts, and with whole NaN rows of x, every token's picks are
    the oracle's stable top-k of the GPU's own logits (NaN last, ids
    ascending) -- k distinct experts -- and the counts follow them.  Covers
    the one-workgroup-per-token router (E <= 8), the matrix-core router with
    8 lanes per token (E = 60, 256) and the fp32 path; logits_out is also
    left NULL once, which changes none of the other outputs."""
    B = _binding()
    cfg = BY_NAME[name] if name == "tiny_f32" else mini(BY_NAME[name])
    log(f"route NaN {cfg.name}")
    inp = DeviceInputs(cfg, device, weights=False)
    desc = B.make_desc(cfg.L, cfg.H, cfg.F, cfg.E, cfg.k, cfg.S, cfg.D, cfg.dtype, cfg.eps)
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    T = min(cfg.T, 96)
    x = inp.x0[0, :T].clone()
    x[5] = float("nan")
    x[T - 1, 3] = float("nan")                  # one NaN element poisons the row
    bias = inp.bias[0].clone()
    keep = [cfg.E - 1, cfg.E // 3] if cfg.k > 1 else [cfg.E // 3]
    nan_mask = torch.ones(cfg.E, dtype=torch.bool, device=device)
    nan_mask[keep] = False
    bias[nan_mask] = float("nan")
    outs = []
    for with_z in (True, False):
        a = torch.empty(T, cfg.H, dtype=tdt, device=device)
        z = torch.empty(T, cfg.E, dtype=torch.float32, device=device)
        idx = torch.empty(T, cfg.k, dtype=torch.int32, device=device)
        w = torch.empty(T, cfg.k, dtype=torch.float32, device=device)
        counts = torch.empty(cfg.E, dtype=torch.int32, device=device)
        B.easybalance_route(desc, 0, T, x, inp.g[0], inp.Wg[0], bias, a, z if with_z else None, idx, w, counts)
        torch.cuda.synchronize()
        outs.append((z.cpu().numpy(), idx.cpu().numpy(), w.cpu().numpy(), counts.cpu().numpy()))
    (z, idx, w, counts), (_, idx2, w2, counts2) = outs
    assert np.isnan(z[5]).all() and np.isnan(z[T - 1]).all()
    assert np.isnan(z[:, nan_mask.cpu().numpy()]).all()
    want = omodel.topk_indices(z.astype(np.float64), cfg.k)
    assert np.array_equal(idx, want)
    assert all(len(set(r)) == cfg.k for r in idx.tolist())
    assert np.array_equal(counts, omodel.expert_counts(idx, cfg.E))
    assert np.array_equal(idx2, idx) and np.array_equal(counts2, counts)
    assert np.array_equal(np.isnan(w), np.isnan(w2)) and np.array_equal(w[~np.isnan(w)], w2[~np.isnan(w2)])
    assert np.isnan(w[5]).all()


@pytest.mark.parametrize("name", ["mixtral_bf16", "qwen_moe_bf16", "dsv3_share_bf16", "tiny_f32"])
def test_route_exact_ties_and_special_values(name, device):
    """Zero router rows make every logit its bias, so crafted biases put exact
    ties (equal values, +0 against -0), infinities, NaN and subnormal values
    among the logits: every token's picks are the oracle's stable top-k of
    the GPU's own logits (larger first, ties to the lower id, NaN last) and
    the counts follow them.  Covers the one-workgroup-per-token router
    (E = 8), the matrix-core routers with 8 lanes per token (E = 60, 256) and
    the fp32 path."""
    B = _binding()
    cfg = BY_NAME[name] if name == "tiny_f32" else mini(BY_NAME[name])
    log(f"route ties {cfg.name}")
    inp = DeviceInputs(cfg, device, weights=False)
    desc = B.make_desc(cfg.L, cfg.H, cfg.F, cfg.E, cfg.k, cfg.S, cfg.D, cfg.dtype, cfg.eps)
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    T = min(cfg.T, 96)
    specials = np.array([1.0, 1.0, 0.0, -0.0, 2.0 ** -130, -1.0, np.inf, -np.inf, np.nan, 1.0, -0.0, 0.5],
                        np.float32)
    rng = np.random.default_rng(cfg.seed)
    for trial in range(3):
        pick = rng.integers(0, len(specials), size=cfg.E) if trial else np.arange(cfg.E) % len(specials)
        bias = torch.from_numpy(specials[pick]).to(device)
        Wg = torch.zeros_like(inp.Wg[0])
        x = inp.x0[0, :T].clone()
        a = torch.empty(T, cfg.H, dtype=tdt, device=device)
        z = torch.empty(T, cfg.E, dtype=torch.float32, device=device)
        idx = torch.empty(T, cfg.k, dtype=torch.int32, device=device)
        w = torch.empty(T, cfg.k, dtype=torch.float32, device=device)
        counts = torch.empty(cfg.E, dtype=torch.int32, device=device)
        B.easybalance_route(desc, 0, T, x, inp.g[0], Wg, bias, a, z, idx, w, counts)
        torch.cuda.synchronize()
        zg = z.cpu().numpy()
        got = idx.cpu().numpy()
        assert np.array_equal(got, omodel.topk_indices(zg.astype(np.float64), cfg.k)), trial
        assert all(len(set(r)) == cfg.k for r in got.tolist())
        assert np.array_equal(counts.cpu().numpy(), omodel.expert_counts(got, cfg.E))


def test_route_stage_one_workgroup_per_token_bf16(device):
    """bf16 stacks with E <= 8 and H > 4096 route one token per workgroup
    (the LDS-staged wavefront router holds H <= 4096): the same parity as
    test_route_stage on that path, ragged token counts included."""
    B = _binding()
    cfg = mini(BY_NAME["mixtral_bf16"], H=8192, F=256, T=70, L=1)
    log(f"route parity {cfg.name} H={cfg.H}")
    inp = DeviceInputs(cfg, device, weights=False)
    P = host_weights(cfg)
    desc = B.make_desc(cfg.L, cfg.H, cfg.F, cfg.E, cfg.k, cfg.S, cfg.D, cfg.dtype, cfg.eps)
    for T in (cfg.T, 1, 33):
        x = inp.x0[0, :T].clone()
        a = torch.empty(T, cfg.H, dtype=torch.bfloat16, device=device)
        z = torch.empty(T, cfg.E, dtype=torch.float32, device=device)
        idx = torch.empty(T, cfg.k, dtype=torch.int32, device=device)
        w = torch.empty(T, cfg.k, dtype=torch.float32, device=device)
        counts = torch.empty(cfg.E, dtype=torch.int32, device=device)
        B.easybalance_route(desc, 0, T, x, inp.g[0], inp.Wg[0], inp.bias[0], a, z, idx, w, counts)
        torch.cuda.synchronize()
        a_ref = omodel.rmsnorm_cast(to_np(x), P.gain(0), cfg.eps, cast_fn(cfg.dtype))
        assert_close(to_np(a), a_ref, cfg.dtype, "a")
        zg = to_np(z)
        assert_close(zg, omodel.router_logits(to_np(a), P.router(0), P.bias(0)), cfg.dtype, "logits")
        idx_np = idx.cpu().numpy()
        assert np.array_equal(idx_np, omodel.topk_indices(zg, cfg.k))
        assert np.array_equal(counts.cpu().numpy(), omodel.expert_counts(idx_np, cfg.E))
        assert_close(to_np(w), omodel.gate_weights(zg, idx_np), cfg.dtype, "w")
