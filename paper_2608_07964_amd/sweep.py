"""Load-balance sweeps over recorded routing: scheduling policies, number of
micro-batches N, minimum combination size m and number of virtual devices
D (the studies of Section 5: scheduling strategies, micro-batch count and
m, EP size, and the worst-case statistic of Section 4.1), EasyBalance on top
of a static replicated expert placement (the orthogonality study of Section 5
and the appendix on redundant experts; the library forms the placed loads and
the decisions itself), and the scheduler's cost per step
(the context of Table 3), on the synthetic stacks.

The stacks are MoE-only (x <- x + MoE_l(RMSNorm(x))), so a token's hidden
state at layer l, and with it its experts there, depends on that token
alone: the experts every token picks at every layer are fixed by the inputs,
whatever the schedule or the split into micro-batches (the kernels are
batch invariant, so the GPU routing is the same in every schedule too).
One lock-step pass on the GPU records them; every (policy, N, m, D) is
then a host computation: per-device loads of each (micro-batch, layer)
from the recorded experts, Algorithm 1 replayed with the library's
scheduler (easybalance_schedule), and the under-utilization 1 - u of
Eq. 3 over the executed steps.

    python -m paper_2608_07964_amd.sweep --config mixtral_bf16

prints the tables (markdown); --save-routes / --routes keep or reuse the
recorded experts (.npy).
"""
from __future__ import annotations

import argparse
import sys
import time

import numpy as np

from . import binding as B
from . import metrics

POLICIES = ("maxutil", "cumutil", "diffpeak", "lockstep", "separate")
_NATIVE = {"maxutil": B.EB_POLICY_MAXUTIL, "cumutil": B.EB_POLICY_CUMUTIL,
           "diffpeak": B.EB_POLICY_DIFFPEAK}


def record_routes(stack) -> np.ndarray:
    """Routed experts of every token at every layer, [N*T][L][k] int32,
    from one lock-step pass of `stack` (a driver.Stack; x is updated)."""
    N, T, L, k = stack.N, stack.T, stack.L, stack.k
    routes = np.full((N * T, L, k), -1, dtype=np.int32)

    def hook(stage, runset):
        if stage == "pre":
            for j, layer in runset:
                routes[j * T:(j + 1) * T, layer] = stack.idx[j].cpu().numpy()

    stack.run("lockstep", record=False, hook=hook)
    assert (routes >= 0).all(), "a (micro-batch, layer) was never routed"
    return routes


def layer_loads(routes: np.ndarray, N: int, E: int, D: int) -> np.ndarray:
    """Per-device load w[j][l][d] (routed pairs, Section 2.3) when the tokens
    are split into N contiguous micro-batches and expert e lives on device
    e // (E / D)."""
    routes = np.asarray(routes)
    tokens, L, k = routes.shape
    if tokens % N or E % D:
        raise ValueError(f"{tokens} tokens into {N} micro-batches / {E} experts onto {D} devices")
    dev = routes // (E // D)                                    # [tokens][L][k]
    T = tokens // N
    out = np.zeros((N, L, D), dtype=np.int64)
    for j in range(N):
        d = dev[j * T:(j + 1) * T]
        for layer in range(L):
            out[j, layer] = np.bincount(d[:, layer].ravel(), minlength=D)
    return out


def expert_counts(routes: np.ndarray, N: int, E: int) -> np.ndarray:
    """Routed pairs per expert, c[j][l][e], of N contiguous micro-batches."""
    routes = np.asarray(routes)
    tokens, L, k = routes.shape
    if tokens % N:
        raise ValueError(f"{tokens} tokens into {N} micro-batches")
    T = tokens // N
    out = np.zeros((N, L, E), dtype=np.int64)
    for j in range(N):
        for layer in range(L):
            out[j, layer] = np.bincount(routes[j * T:(j + 1) * T, layer].ravel(), minlength=E)
    return out


def replicated_placement(hist, D: int, replicas: int, first_device: int = 0) -> list[list[int]]:
    """Static placement of one layer's experts on D devices from a history of
    per-expert loads hist[E], in the manner of EPLB-style replication (the
    placement of the orthogonality study; the heuristic is this module's own):

      * the `replicas` hottest experts (history load descending, ties ->
        lower id) get one extra copy each, and a copy carries hist[e] /
        copies(e) of expected load;
      * copies are placed largest expected load first (ties -> lower expert
        id) on the device with the least expected load so far that has a free
        slot, preferring devices that hold no copy of the same expert (ties
        -> the first device in the order first_device, first_device + 1, ...
        mod D); every device has (E + replicas) / D slots.

    Returns slots[d], the logical experts device d holds (ascending)."""
    hist = np.asarray(hist, dtype=np.int64)
    E = hist.shape[0]
    if D < 1 or not 0 <= replicas <= E or (E + replicas) % D:
        raise ValueError(f"E={E} + replicas={replicas} not a multiple of D={D}")
    per = (E + replicas) // D
    order = sorted(range(E), key=lambda e: (-hist[e], e))
    copies = np.ones(E, dtype=np.int64)
    copies[order[:replicas]] = 2
    items = [(e, c) for e in range(E) for c in range(int(copies[e]))]
    # expected load hist/copies, compared exactly as hist[a]*copies[b] vs hist[b]*copies[a]
    items.sort(key=lambda ec: (-(hist[ec[0]] * 2 // copies[ec[0]]), ec[0], ec[1]))
    load2 = np.zeros(D, dtype=np.int64)   # twice the expected load (integer)
    slots = [[] for _ in range(D)]
    for e, _ in items:
        free = [d for d in range(D) if len(slots[d]) < per]
        fresh = [d for d in free if e not in slots[d]]
        d = min(fresh or free, key=lambda x: (load2[x], (x - first_device) % D))
        slots[d].append(e)
        load2[d] += hist[e] * 2 // copies[e]
    return [sorted(s) for s in slots]


def run_policy_counts(counts: np.ndarray, D: int, policy: str, m: int, placement=None) -> list[np.ndarray]:
    """Per-device workload of every executed step of one pass of Algorithm 1
    replayed with the library's scheduler on per-expert counts c[j][l][e]:
    the loads come from easybalance_schedule itself, under `placement` (a
    binding.make_placement struct: static placement with replicas) or, when
    it is None, the contiguous E/D mapping.  lockstep: step l runs every
    micro-batch at layer l (the scheduler asked for the whole pool);
    separate: every (j, l) alone."""
    counts = np.asarray(counts, np.int64)
    N, L, E = counts.shape
    if counts.max(initial=0) > np.iinfo(np.int32).max:
        raise ValueError("counts exceed int32")
    if policy == "separate":
        steps = []
        for layer in range(L):
            for j in range(N):
                _, load = B.easybalance_schedule([j], counts[[j], layer], E, D, 1, B.EB_POLICY_MAXUTIL,
                                                 layers=[layer], placement=placement)
                steps.append(load.copy())
        return steps
    layer = np.zeros(N, dtype=np.int64)
    pool = list(range(N))
    steps = []
    while pool:
        cur = counts[pool, layer[pool]]
        if policy == "lockstep":
            pol, mm = B.EB_POLICY_MAXUTIL, len(pool)     # the only candidate: the whole pool
        else:
            pol, mm = _NATIVE[policy], m
        mask, load = B.easybalance_schedule(pool, cur, E, D, mm, pol, layers=layer[pool], placement=placement)
        R = [j for j in pool if (mask >> j) & 1]
        if not R:
            raise RuntimeError("scheduler returned an empty run set")
        steps.append(load.copy())
        layer[R] += 1
        pool = [j for j in pool if layer[j] < L]
    return steps


def placement_copies(slots, E: int) -> list[list[int]]:
    """Per expert, the devices holding a copy (ascending), from a layer's
    slots[d] (the experts device d holds)."""
    holders = [[] for _ in range(E)]
    for d, held in enumerate(slots):
        for e in held:
            holders[e].append(d)
    if any(not h for h in holders):
        raise ValueError("an expert has no device")
    return holders


def run_policy(loads: np.ndarray, policy: str, m: int) -> list[np.ndarray]:
    """Per-device workload of every executed step of one pass of Algorithm 1
    over loads[j][l][d] under `policy` (lockstep: step l runs every
    micro-batch at layer l; separate: every (j, l) alone)."""
    loads = np.asarray(loads, np.int64)
    N, L, D = loads.shape
    if policy == "lockstep":
        return metrics.lockstep_loads(loads)
    if policy == "separate":
        return metrics.separate_loads(loads)
    if loads.max(initial=0) > np.iinfo(np.int32).max:
        raise ValueError("loads exceed int32")
    pol = _NATIVE[policy]
    layer = np.zeros(N, dtype=np.int64)
    pool = list(range(N))
    steps = []
    while pool:
        # device loads passed as counts of D one-expert devices
        cur = loads[pool, layer[pool]]
        mask, load = B.easybalance_schedule(pool, cur, D, D, m, pol)
        R = [j for j in pool if (mask >> j) & 1]
        if not R:
            raise RuntimeError("scheduler returned an empty run set")
        steps.append(load.copy())
        layer[R] += 1
        pool = [j for j in pool if layer[j] < L]
    return steps


def same_skew_windows(layer_load: np.ndarray, n: int) -> tuple[int, int]:
    """Windows of n consecutive layers whose loads combine in the worst case
    of Section 4.1, max(sum of w) == sum of max(w) (some device is a peak of
    every layer in the window), over the per-layer load layer_load[l][d] of
    the whole batch.  Returns (worst-case windows, windows)."""
    w = np.asarray(layer_load, np.int64)
    L = w.shape[0]
    hits = 0
    for l0 in range(L - n + 1):
        win = w[l0:l0 + n]
        hits += int(win.sum(axis=0).max() == win.max(axis=1).sum())
    return hits, max(0, L - n + 1)


def _divisors(x: int) -> list[int]:
    return [d for d in range(1, x + 1) if x % d == 0]


def sweep(routes: np.ndarray, E: int, Ns, Ds, ms_for=None, policies=POLICIES) -> list[dict]:
    """One row per (N, D, policy, m): steps, max/mean and under-utilization.
    ms_for(N) gives the m values (default 1..N); lockstep and separate do
    not depend on m and get one row each (m = None)."""
    rows = []
    for N in Ns:
        ms = list(ms_for(N)) if ms_for else list(range(1, N + 1))
        for D in Ds:
            w = layer_loads(routes, N, E, D)
            for pol in policies:
                for m in (ms if pol in _NATIVE else [None]):
                    s = metrics.summary(run_policy(w, pol, m if m is not None else N))
                    rows.append({"N": N, "D": D, "policy": pol, "m": m, "steps": s["steps"],
                                 "max_over_mean": s["max_over_mean"], "under_util": s["idle_fraction"]})
    return rows


def _table(rows, header, fmt) -> str:
    out = ["| " + " | ".join(header) + " |", "|" + "---|" * len(header)]
    out += ["| " + " | ".join(fmt(r)) + " |" for r in rows]
    return "\n".join(out)


def report(routes: np.ndarray, cfg) -> str:
    """The markdown tables for one stack."""
    tokens = routes.shape[0]
    Ns = [n for n in (2, 4, 8, 16) if tokens % n == 0 and n <= tokens]
    Ds = sorted({d for d in _divisors(cfg.E) if 2 <= d <= 64 and (d & (d - 1)) == 0} | {cfg.D})
    m_def = lambda n: max(1, (3 * n) // 4)
    parts = [f"## {cfg.name}: {tokens} tokens, L = {cfg.L}, E = {cfg.E}, k = {cfg.k}\n"]

    # policies at the stack's own N, D and the default m
    rows = sweep(routes, cfg.E, [cfg.N], [cfg.D], ms_for=lambda n: [m_def(n)])
    parts.append(f"Policies (N = {cfg.N}, D = {cfg.D}, m = {m_def(cfg.N)}):\n")
    parts.append(_table(rows, ["policy", "steps", "max/mean", "under-utilization"],
                        lambda r: [r["policy"], str(r["steps"]), f"{r['max_over_mean']:.3f}",
                                   f"{r['under_util']:.3f}"]))
    # N and m (MaxUtil) at the stack's D
    ms_for = lambda n: sorted({1, max(1, n // 4), max(1, n // 2), m_def(n), n})
    rows = sweep(routes, cfg.E, Ns, [cfg.D], ms_for=ms_for, policies=("maxutil", "lockstep"))
    parts.append(f"\nMaxUtil over N and m (D = {cfg.D}; lockstep = per-layer baseline):\n")
    parts.append(_table(rows, ["N", "policy", "m", "steps", "under-utilization"],
                        lambda r: [str(r["N"]), r["policy"], "-" if r["m"] is None else str(r["m"]),
                                   str(r["steps"]), f"{r['under_util']:.3f}"]))
    # D at the stack's N (same tokens spread over more devices)
    rows = sweep(routes, cfg.E, [cfg.N], Ds, ms_for=lambda n: [m_def(n)],
                 policies=("maxutil", "cumutil", "diffpeak", "lockstep"))
    parts.append(f"\nVirtual devices D (N = {cfg.N}, m = {m_def(cfg.N)}):\n")
    parts.append(_table(rows, ["D", "policy", "under-utilization"],
                        lambda r: [str(r["D"]), r["policy"], f"{r['under_util']:.3f}"]))
    # EasyBalance on a static replicated placement; history = the batch's own
    # per-layer expert counts (the most favourable history a placement can have)
    counts = expert_counts(routes, cfg.N, cfg.E)
    hist = counts.sum(axis=0)
    # Ties at device 0 in every layer put every layer's hottest expert on one
    # device (its peaks coincide: the worst case of Section 4.1); rotating the
    # tie order by layer does not.
    mappings = [("contiguous, E/D experts per device", None)]
    for reps in (0, cfg.D):
        for rot in (False, True):
            pl = [replicated_placement(hist[layer], cfg.D, reps, layer % cfg.D if rot else 0)
                  for layer in range(cfg.L)]
            ties = "ties rotated by layer" if rot else "ties at device 0"
            mappings.append((f"placed from history, {cfg.E + reps} physical experts, {ties}",
                             B.make_placement([placement_copies(s, cfg.E) for s in pl], cfg.D)))
    rows = []
    for name, placement in mappings:
        r = {"mapping": name}
        for pol in ("lockstep", "maxutil", "cumutil", "diffpeak"):
            r[pol] = metrics.summary(run_policy_counts(counts, cfg.D, pol, m_def(cfg.N),
                                                       placement))["idle_fraction"]
        rows.append(r)
    parts.append(f"\nStatic placement + EasyBalance (N = {cfg.N}, D = {cfg.D}, m = {m_def(cfg.N)}; "
                 "under-utilization):\n")
    parts.append(_table(rows, ["mapping", "lock-step", "MaxUtil", "CumUtil", "DiffPeak"],
                        lambda r: [r["mapping"]] + [f"{r[p]:.3f}" for p in
                                                    ("lockstep", "maxutil", "cumutil", "diffpeak")]))
    # scheduler cost per decision at the stack's own N, D, m
    w = layer_loads(routes, cfg.N, cfg.E, cfg.D)
    cost = []
    for pol in ("maxutil", "cumutil", "diffpeak"):
        t0 = time.perf_counter()
        n_steps = len(run_policy(w, pol, m_def(cfg.N)))
        cost.append(f"{pol} {(time.perf_counter() - t0) / n_steps * 1e6:.0f} µs")
    parts.append("\nHost time per scheduling decision (one replayed pass, including the Python "
                 "replay loop and the binding call): " + ", ".join(cost) + "\n")
    # worst-case windows over the whole batch's per-layer loads
    whole = layer_loads(routes, 1, cfg.E, cfg.D)[0]
    stats = []
    for n in (2, 3):
        h, t = same_skew_windows(whole, n)
        stats.append(f"n = {n}: {h}/{t}" + (f" = {h / t:.3f}" if t else ""))
    parts.append(f"\nWindows of n consecutive layers combining in the worst case (whole batch, "
                 f"D = {cfg.D}): " + "; ".join(stats) + "\n")
    return "\n".join(parts)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--config", default="mixtral_bf16")
    ap.add_argument("--routes", help="recorded experts (.npy) to use instead of a GPU pass")
    ap.add_argument("--save-routes", help="write the recorded experts here (.npy)")
    args = ap.parse_args(argv)

    from synth import BY_NAME
    cfg = BY_NAME[args.config]
    if args.routes:
        routes = np.load(args.routes)
    else:
        import torch
        from synth.device import DeviceInputs
        from .driver import Stack, pack_expert_weights
        B.lib()
        dev = "cuda:0"
        inp = DeviceInputs(cfg, dev)
        pack_expert_weights(B.make_desc(cfg.L, cfg.H, cfg.F, cfg.E, cfg.k, cfg.S, cfg.D, cfg.dtype,
                                        cfg.eps, cfg.norm_topk), inp.W_gu, inp.W_dn)
        st = Stack(L=cfg.L, H=cfg.H, F=cfg.F, E=cfg.E, k=cfg.k, S=cfg.S, D=cfg.D, N=cfg.N, T=cfg.T,
                   dtype=cfg.dtype, x=inp.x0.clone(), gain=inp.g, Wg=inp.Wg, bias=inp.bias,
                   W_gu=inp.W_gu, W_dn=inp.W_dn, eps=cfg.eps, norm_topk=cfg.norm_topk, device=dev)
        routes = record_routes(st)
        torch.cuda.synchronize()
        if args.save_routes:
            np.save(args.save_routes, routes)
    print(report(routes, cfg))
    return 0


if __name__ == "__main__":
    sys.exit(main())
