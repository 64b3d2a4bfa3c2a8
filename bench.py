#!/usr/bin/env python3
"""Benchmark of the EasyBalance hot path on one MI355X.

One step = one full pass of Algorithm 1 over one batch: every micro-batch of
the stack through every MoE layer (routing, MaxUtil scheduling, grouped
expert FFN of each step's RunSet, weighted combine), starting from the same
synthetic residual stream each time.  Inputs and weights are generated in HBM
before timing.  Prints ONE JSON line:

  value      expert-FFN TFLOP/s of the whole pass: 6*H*F FLOP per routed or
             shared (token, expert) pair, over the wall time of the pass
  load       max/mean virtual-device load (and idle fraction) of the executed
             schedule vs the per-layer lock-step baseline and vs no combination
  roofline   the grouped gate/up GEMM (the dominant kernel), timed with HIP
             events on its own stream over the timed region
  cpu_baseline  the CPU oracle timed on a bounded sample of the same workload

Only one GPU: --gpus N with N > 1 exits with an error.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_FP32_VALU_TFLOPS = 157.3  # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def gemm_source_hash() -> str:
    with open(os.path.join(ROOT, "paper_2608_07964_amd", "csrc", "gemm.hip"), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(config: str):
    """HBM bytes per gate/up launch from the committed rocprofv3 counter summary,
    if it was taken on the current kernel source (else None)."""
    path = os.path.join(ROOT, "profiles", f"gateup_traffic_{config}.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("gemm_source_sha256_16") != gemm_source_hash():
        return None
    return t.get("hbm_bytes_per_launch")


def gateup_roofline(cfg, pairs: int, groups: int, t_s: float, launches: int, traffic) -> dict:
    """Roofline entry of the grouped gate/up GEMM over launches that together
    hold `pairs` (token, expert) pairs in `groups` distinct (layer, expert)
    groups and took t_s seconds: algorithmic FLOP (4 H F per pair: gate and
    up) and bytes (each group's gate/up weights once, each pair's A row read
    and h row written), the bound whichever takes longer at the peak, and
    both fractions."""
    eb = 2 if cfg.dtype == "bf16" else 4
    flop = 4 * cfg.H * cfg.F * pairs
    nbytes = groups * 2 * cfg.F * cfg.H * eb + pairs * (cfg.H + cfg.F) * eb
    peak_flops = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_FP32_VALU_TFLOPS
    compute_s = flop / (peak_flops * 1e12)
    memory_s = nbytes / (PEAK_HBM_GBS * 1e9)
    if compute_s >= memory_s:
        ach = flop / t_s / 1e12
        roof = {"bound": "mfma" if cfg.dtype == "bf16" else "alu", "achieved": ach,
                "peak": peak_flops, "unit": "TFLOP/s", "frac": ach / peak_flops, "traffic": traffic}
    else:
        ach = nbytes / t_s / 1e9
        roof = {"bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": ach / PEAK_HBM_GBS, "traffic": traffic}
    # both fractions, whichever bound applies: the MFMA share is the figure the
    # 60%-of-bf16-peak target is stated in
    roof["mfma_frac"] = flop / t_s / 1e12 / peak_flops
    roof["hbm_frac"] = nbytes / t_s / 1e9 / PEAK_HBM_GBS
    n = max(launches, 1)
    roof.update({"kernel": "grouped_gemm_bf16<gate/up+SwiGLU>" if cfg.dtype == "bf16" else "grouped_gemm_f32<gate/up>",
                 "launches": launches, "avg_launch_ms": t_s * 1e3 / n,
                 "algorithmic_flop_per_launch": flop / n,
                 "algorithmic_bytes_per_launch": nbytes / n,
                 "time_at_mfma_peak_ms": compute_s * 1e3 / n,
                 "time_at_hbm_peak_ms": memory_s * 1e3 / n})
    return roof


def kernel_algorithmic_bytes(cfg, tokens: int, pairs: int, groups: int, route_launches: int) -> dict:
    """Algorithmic HBM bytes of the memory-bound kernel classes (and the down
    GEMM) for a span of work that routes `tokens` (micro-batch, layer) tokens,
    groups `pairs` (token, expert) pairs in `groups` distinct (layer, expert)
    groups, with `route_launches` routing launches."""
    eb = 2 if cfg.dtype == "bf16" else 4
    return {
        # x read (fp32), a written, logits / picks / weights written, each
        # launch's router rows read once
        "route_logits": tokens * (4 * cfg.H + eb * cfg.H + 4 * cfg.E + 8 * cfg.k)
                        + route_launches * cfg.E * cfg.H * eb,
        # grouped rows: a token's row read once, written per pair
        "perm_gather": (tokens + pairs) * cfg.H * eb,
        # o rows read per pair (and its routing weight and position), x read
        # and written per token
        "combine": pairs * (cfg.H * eb + 8) + tokens * 8 * cfg.H,
        # weights of the distinct groups, h read, o written
        "down": groups * cfg.F * cfg.H * eb + pairs * (cfg.F + cfg.H) * eb,
    }


def cpu_baseline(cfg, budget_s: float) -> dict:
    """The oracle (float64 NumPy) on whole MoE layers of the same stack, layer
    by layer over all micro-batches (each carrying its hidden state forward),
    as many as fit in ~budget_s; each layer's weights are generated before its
    layers are timed."""
    import numpy as np
    import threadpoolctl

    from oracle import model as omodel
    from synth import gen

    bias = gen.router_bias(cfg)
    info = threadpoolctl.threadpool_info()
    cores = max([i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"] or [1])
    xs = [gen.x_rows(cfg, j, 0, cfg.T).astype(np.float64) for j in range(cfg.N)]
    done, t_total, t_gen, layers = 0, 0.0, 0.0, 0
    for layer in range(cfg.L):
        t0 = time.perf_counter()
        gu = {e: gen.expert_gate_up(cfg, layer, e) for e in range(cfg.E + cfg.S)}
        dn = {e: gen.expert_down(cfg, layer, e) for e in range(cfg.E + cfg.S)}
        Wr = gen.router_weight(cfg, layer)
        t_gen += time.perf_counter() - t0
        P = omodel.Weights(gain=lambda l: gen.rms_gain(cfg), router=lambda l: Wr,
                           bias=lambda l: bias[l], gate_up=lambda l, e: gu[e], down=lambda l, e: dn[e])
        layers += 1
        for j in range(cfg.N):
            t0 = time.perf_counter()
            out = omodel.moe_layer(xs[j], layer, P, E=cfg.E, k=cfg.k, S=cfg.S, eps=cfg.eps,
                                   dtype=cfg.dtype)
            t_total += time.perf_counter() - t0
            xs[j] = out.x_out
            done += 1
            if t_total >= budget_s:
                break
        del gu, dn, P
        if t_total >= budget_s:
            break
    log(f"cpu baseline: {done} (micro-batch, layer) MoE layers in {t_total:.1f}s "
        f"(weights generated in {t_gen:.1f}s, not timed)")
    flops = done * cfg.T * (cfg.k + cfg.S) * cfg.ffn_flop_per_pair
    return {"value": flops / t_total / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"oracle MoE layers 0..{layers - 1}, {done} (micro-batch, layer) workloads of "
                       f"{cfg.T} tokens ({cfg.name}), float64 NumPy/OpenBLAS, {t_total:.1f}s; "
                       f"expert-FFN FLOP counted as on the GPU")}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="mixtral_bf16")
    ap.add_argument("--policy", default="maxutil", choices=["maxutil", "cumutil", "diffpeak", "lockstep"])
    ap.add_argument("--m", type=int, default=None, help="minimum combination size (default 0.75 N)")
    ap.add_argument("--schedule", default="device", choices=["host", "device"],
                    help="where Algorithm 1's Schedule runs: on the host after a copy of the pool's "
                         "expert counts each step, or in a kernel on the GPU with the host queueing "
                         "steps ahead")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-lockstep", action="store_true", help="skip the lock-step comparison pass")
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="after timing, copy a buffer of this many MiB once (a plain copy kernel "
                         "of known size for calibrating rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); an expert-parallel "
              "run over several GPUs is not implemented", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2608_07964_amd import binding as B
    from paper_2608_07964_amd import metrics
    from paper_2608_07964_amd.driver import Stack, pack_expert_weights
    from synth import BY_NAME
    from synth.device import DeviceInputs

    cfg = BY_NAME[args.config]
    m = args.m if args.m is not None else cfg.m
    B.lib()
    dev = "cuda:0"
    t0 = time.perf_counter()
    inp = DeviceInputs(cfg, dev)
    torch.cuda.synchronize()
    log(f"{cfg.name}: inputs generated in HBM in {time.perf_counter() - t0:.2f}s "
        f"({inp.weight_bytes() / 1e9:.1f} GB of expert weights)")
    t0 = time.perf_counter()
    pack_expert_weights(B.make_desc(cfg.L, cfg.H, cfg.F, cfg.E, cfg.k, cfg.S, cfg.D, cfg.dtype, cfg.eps,
                                    cfg.norm_topk), inp.W_gu, inp.W_dn)
    torch.cuda.synchronize()
    log(f"{cfg.name}: expert weights packed for the grouped GEMMs in {time.perf_counter() - t0:.2f}s")
    st = Stack(L=cfg.L, H=cfg.H, F=cfg.F, E=cfg.E, k=cfg.k, S=cfg.S, D=cfg.D, N=cfg.N, T=cfg.T,
               dtype=cfg.dtype, x=inp.x0.clone(), gain=inp.g, Wg=inp.Wg, bias=inp.bias,
               W_gu=inp.W_gu, W_dn=inp.W_dn, eps=cfg.eps, norm_topk=cfg.norm_topk, device=dev)
    stream = torch.cuda.current_stream()

    def one_pass(policy, record=False):
        # one Algorithm-1 pass through the library's native driver
        st.x.copy_(inp.x0)
        return st.run_native(policy, m=m, record=record, stream=stream,
                             device_schedule=args.schedule == "device")

    flop_pass = cfg.total_ffn_flop
    pairs_pass = cfg.N * cfg.T * (cfg.k + cfg.S) * cfg.L

    def timed(policy, K, W, profile):
        """K timed passes after W warm-up passes; profile: kernel classes whose
        launches are bracketed by HIP events during the timed passes."""
        for _ in range(W):
            one_pass(policy)
        torch.cuda.synchronize()
        if profile:
            B.easybalance_profile_begin(profile)
        t = time.perf_counter()
        for _ in range(K):
            one_pass(policy)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t
        prof = B.easybalance_profile_end() if profile else None
        return dt, prof

    # the timed passes bracket only the roofline kernel (gate/up) with events
    dt, prof = timed(args.policy, args.steps, args.warmup, ["gateup"])
    ms_step = dt / args.steps * 1e3
    value = flop_pass * args.steps / dt / 1e12
    log(f"{args.policy}: {ms_step:.3f} ms/pass, {value:.1f} TFLOP/s")
    # per-kernel breakdown from separate, fully instrumented passes
    n_bd = min(args.steps, 3)
    _, prof_all = timed(args.policy, n_bd, 0, list(B.KERNEL_NAMES))

    steps = one_pass(args.policy, record=True)
    torch.cuda.synchronize()
    layer_loads = st.layer_loads.copy()
    load = {
        "schedule": metrics.summary([s.load for s in steps]),
        "per_layer_baseline": metrics.summary(metrics.lockstep_loads(layer_loads)),
        "no_combination": metrics.summary(metrics.separate_loads(layer_loads)),
    }
    extra = {}
    if not args.no_lockstep and args.policy != "lockstep":
        dt_ls, _ = timed("lockstep", args.steps, 1, False)
        extra["lockstep_tflops"] = flop_pass * args.steps / dt_ls / 1e12
        extra["lockstep_ms_per_pass"] = dt_ls / args.steps * 1e3

    # roofline of the grouped gate/up GEMM over the timed region
    gu_ms, gu_n = prof["gateup"]
    groups = sum(s.groups for s in steps) * args.steps
    roof = gateup_roofline(cfg, pairs_pass * args.steps, groups, gu_ms / 1e3, gu_n, measured_traffic(cfg.name))
    peak_flops = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_FP32_VALU_TFLOPS
    kernels = {name: {"ms_per_pass": ms / n_bd, "launches_per_pass": n / n_bd}
               for name, (ms, n) in prof_all.items()}
    # algorithmic HBM bytes per pass of the memory-bound kernels (and the down
    # GEMM) against the 8 TB/s peak, from the per-kernel event times above
    tokens_pass = cfg.N * cfg.T * cfg.L            # every (micro-batch, layer) routed once
    alg_bytes = kernel_algorithmic_bytes(cfg, tokens_pass, pairs_pass, groups // args.steps,
                                         round(prof_all["route_logits"][1] / n_bd))
    for name, b in alg_bytes.items():
        ms = kernels[name]["ms_per_pass"]
        kernels[name]["algorithmic_bytes_per_pass"] = b
        kernels[name]["hbm_gbs"] = b / (ms / 1e3) / 1e9 if ms > 0 else None
        kernels[name]["hbm_frac"] = b / (ms / 1e3) / 1e9 / PEAK_HBM_GBS if ms > 0 else None
    down_flop = 2 * cfg.H * cfg.F * pairs_pass
    if kernels["down"]["ms_per_pass"] > 0:
        kernels["down"]["mfma_frac"] = down_flop / (kernels["down"]["ms_per_pass"] / 1e3) / 1e12 / peak_flops
    # gate/up + down GEMM time; in the device-scheduled pass the split-K sum of
    # the long-K down GEMM is done inside the combine, not counted here
    ffn_tflops = 6 * cfg.H * cfg.F * pairs_pass / ((prof_all["gateup"][0] + prof_all["down"][0]) / n_bd / 1e3) / 1e12

    out = {
        "metric": "expert-FFN TFLOP/s (1 GPU) + max/mean virtual-device load vs per-layer base",
        "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": cfg.name, "L": cfg.L, "H": cfg.H, "F": cfg.F, "E": cfg.E, "k": cfg.k,
                   "S": cfg.S, "D": cfg.D, "N": cfg.N, "T": cfg.T, "m": m, "policy": args.policy,
                   "schedule": args.schedule,
                   "step": "one Algorithm-1 pass: every micro-batch through every layer",
                   "tokens_per_pass": cfg.N * cfg.T, "ffn_flop_per_pass": flop_pass},
        "load": load,
        "steps_per_pass": len(steps),
        "ffn_kernels_tflops": ffn_tflops,
        "kernels": kernels,
        "roofline": roof,
        **extra,
    }
    if args.calib_copy_mb:
        src = torch.empty(args.calib_copy_mb << 18, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["calib_copy_bytes"] = src.numel() * 4
        del src, dst
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_budget)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
