"""Algorithm 1 (EasyBalance) on one GPU, driving the C ABI.

    l_j <- 0 for every micro-batch; pool S <- all micro-batches
    route every micro-batch at layer 0                      (Attn_Route_Dispatch)
    while S is not empty:
        RunSet <- Schedule(S, m)                            (easybalance_schedule)
        expert FFNs of RunSet, each at its own layer,
        jointly, then the weighted combine                  (easybalance_moe_step/combine)
        l_j += 1 for j in RunSet; route those not finished  (easybalance_route)
        S <- {j in S : l_j < L}

The only host<->device synchronisation per step is the copy of the pool's
expert counts (N x E int32) into pinned memory for the scheduler.  Torch
provides device memory and the stream; every step of the path runs in the
library's kernels (or its host scheduler).
"""
from __future__ import annotations

import dataclasses
import weakref

import numpy as np
import torch

from . import binding as B

POLICIES = {"maxutil": B.EB_POLICY_MAXUTIL, "cumutil": B.EB_POLICY_CUMUTIL,
            "diffpeak": B.EB_POLICY_DIFFPEAK, "lockstep": None}


# tensors whose contents are packed expert weights (id -> tensor)
_packed: "weakref.WeakValueDictionary[int, torch.Tensor]" = weakref.WeakValueDictionary()


def is_packed(t: torch.Tensor) -> bool:
    return _packed.get(id(t)) is t


def pack_expert_weights(desc, W_gu, W_dn) -> None:
    """Relays every layer's expert weights, in place, into the layout the
    grouped GEMMs read (easybalance_pack_weights), through a one-layer
    temporary copy.  W_gu [L] -> [E+S][2F][H], W_dn [L] -> [E+S][H][F],
    row-major on entry.  Each tensor is packed once."""
    for layers, kind in ((W_gu, B.EB_WEIGHTS_GATE_UP), (W_dn, B.EB_WEIGHTS_DOWN)):
        for t in layers:
            if is_packed(t):
                raise ValueError("these expert weights are already packed")
            if not (t.is_cuda and t.is_contiguous()):
                raise ValueError("expert weights must be contiguous device tensors")
            stream = torch.cuda.current_stream(t.device)
            src = t.clone()
            B.easybalance_pack_weights(desc, kind, t.shape[0], src, t, stream.cuda_stream)
            del src  # freed in stream order, after the pack
            _packed[id(t)] = t


@dataclasses.dataclass
class StepRecord:
    runset: list            # [(j, l_j)] in ascending j
    load: np.ndarray        # combined per-device workload W of the step [D]
    pairs: int              # grouped rows P of the step
    groups: int             # distinct (layer, expert) keys with rows


class Stack:
    """Device state of one MoE stack: N micro-batches of T tokens, L layers.

    x [N][T][H] fp32 is updated in place.  Inputs: gain [L][H] fp32,
    Wg [L] -> [E][H], bias [L][E] fp32, W_gu [L] -> [E+S][2F][H],
    W_dn [L] -> [E+S][H][F] (dtype of the stack), the expert weights packed
    by pack_expert_weights.
    """

    def __init__(self, *, L, H, F, E, k, S, D, N, T, dtype, x, gain, Wg, bias, W_gu, W_dn,
                 eps=1e-6, norm_topk=0, device="cuda:0"):
        self.L, self.H, self.F, self.E, self.k, self.S, self.D, self.N, self.T = \
            L, H, F, E, k, S, D, N, T
        self.dtype = dtype
        self.desc = B.make_desc(L, H, F, E, k, S, D, dtype, eps, norm_topk)
        self.dev = torch.device(device)
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.x, self.gain, self.Wg, self.bias, self.W_gu, self.W_dn = x, gain, Wg, bias, W_gu, W_dn
        assert x.shape == (N, T, H) and x.dtype == torch.float32 and x.is_contiguous()
        if not all(is_packed(t) for t in list(W_gu) + list(W_dn)):
            raise ValueError("expert weights must be packed with pack_expert_weights first")
        self.a = torch.empty(N, T, H, dtype=tdt, device=self.dev)
        self.logits = torch.empty(N, T, E, dtype=torch.float32, device=self.dev)
        self.idx = torch.empty(N, T, k, dtype=torch.int32, device=self.dev)
        self.w = torch.empty(N, T, k, dtype=torch.float32, device=self.dev)
        self.counts = torch.zeros(N, E, dtype=torch.int32, device=self.dev)
        self.counts_host = torch.zeros(N, E, dtype=torch.int32, pin_memory=True)
        P_max = N * T * (k + S)
        self.o = torch.empty(P_max, H, dtype=tdt, device=self.dev)
        self.inv = torch.empty(P_max, dtype=torch.int32, device=self.dev)
        self.ws_bytes = B.easybalance_moe_step_workspace_size(self.desc, [T] * N)
        self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=self.dev)
        off = (-self.ws.data_ptr()) % 256
        self.ws_ptr = self.ws.data_ptr() + off

    # ---- the three operations of Algorithm 1 -------------------------------
    def route(self, j: int, layer: int, stream) -> None:
        B.easybalance_route(self.desc, layer, self.T, self.x[j], self.gain[layer], self.Wg[layer],
                            self.bias[layer], self.a[j], self.logits[j], self.idx[j], self.w[j],
                            self.counts[j], stream)

    def work(self, runset) -> tuple:
        return B.work_array((j, l, self.T, self.a[j], self.idx[j], self.w[j]) for j, l in runset)

    def moe_compute_combine(self, runset, stream, views=None) -> None:
        run = self.work(runset)
        B.easybalance_moe_step(self.desc, run, len(runset), self.W_gu, self.W_dn, self.ws_ptr,
                               self.ws_bytes, self.o, self.inv, views, stream)
        B.easybalance_combine(self.desc, run, len(runset), [self.x[j] for j, _ in runset],
                              self.o, self.inv, stream)

    # ---- Algorithm 1, natively ----------------------------------------------
    def run_native(self, policy: str = "maxutil", m: int | None = None, record: bool = True,
                   stream=None, device_schedule: bool = False, placement=None) -> list[StepRecord]:
        """The same pass as run(), driven by easybalance_run_pass (the host
        loop in the library; device_schedule: Schedule on the GPU, the host
        queueing steps ahead).  Fills layer_loads and returns the steps when
        record (records cover the first N*L steps, i.e. all of them).
        placement: a binding.make_placement struct (static expert placement
        with replicas) from which the loads and decisions are formed."""
        if stream is None:
            stream = torch.cuda.current_stream(self.dev)
        pol = B.EB_POLICY_LOCKSTEP if policy == "lockstep" else POLICIES[policy]
        if device_schedule:
            pol |= B.EB_PASS_DEVICE_SCHEDULE
        m = self.N if m is None else m
        if not hasattr(self, "_state"):
            self._state_bytes = B.easybalance_pass_state_size(self.desc, self.N, self.T)
            self._state = torch.empty(self._state_bytes + 256, dtype=torch.uint8, device=self.dev)
        sp = self._state.data_ptr() + (-self._state.data_ptr()) % 256
        n, rs, ly, sl, gr, ll = B.easybalance_run_pass(
            self.desc, self.N, self.T, self.x, self.gain, self.Wg, self.bias, self.W_gu, self.W_dn,
            pol, m, sp, self._state_bytes, max_steps=self.N * self.L, record=record,
            stream=stream.cuda_stream, placement=placement)
        if not record:
            return []
        self.layer_loads = ll.astype(np.int64)
        steps = []
        for i in range(n):
            runset = [(j, int(ly[i, j])) for j in range(self.N) if (int(rs[i]) >> j) & 1]
            steps.append(StepRecord(runset=runset, load=sl[i].copy(),
                                    pairs=len(runset) * self.T * (self.k + self.S),
                                    groups=int(gr[i])))
        return steps

    # ---- Algorithm 1 --------------------------------------------------------
    def run(self, policy: str = "maxutil", m: int | None = None, record: bool = True,
            stream=None, views=None, hook=None) -> list[StepRecord]:
        """One pass of every micro-batch through every layer.  Returns the steps.

        views: optional eb_step_views buffers (dict) the steps write into;
        hook(stage, runset): called with stage "pre" after scheduling and
        "post" after the combine of every step (tests use it to sample).
        """
        if stream is None:
            stream = torch.cuda.current_stream(self.dev)
        sp = stream.cuda_stream
        self.layer_loads = np.full((self.N, self.L, self.D), -1, dtype=np.int64)
        pol = POLICIES[policy]
        m = self.N if m is None else m
        layer = [0] * self.N
        pool = list(range(self.N))
        for j in pool:
            self.route(j, 0, sp)
        steps = []
        per = self.E // self.D
        while pool:
            with torch.cuda.stream(stream):
                self.counts_host.copy_(self.counts, non_blocking=True)
            stream.synchronize()
            cnt = self.counts_host.numpy()
            for j in pool:
                self.layer_loads[j, layer[j]] = cnt[j].reshape(self.D, per).sum(axis=1)
            if pol is None:
                R = list(pool)
                load = cnt[R].reshape(len(R), self.D, per).sum(axis=(0, 2)).astype(np.int64)
            else:
                mask, load = B.easybalance_schedule(pool, cnt[pool], self.E, self.D, m, pol)
                R = [j for j in pool if (mask >> j) & 1]
            runset = [(j, layer[j]) for j in R]
            if hook:
                hook("pre", runset)
            self.moe_compute_combine(runset, sp, views)
            if hook:
                hook("post", runset)
            if record:
                routed = {(layer[j], int(e)) for j in R for e in np.nonzero(cnt[j])[0]}
                n_layers = len({layer[j] for j in R})
                steps.append(StepRecord(runset=runset, load=np.asarray(load),
                                        pairs=len(R) * self.T * (self.k + self.S),
                                        groups=len(routed) + self.S * n_layers))
            for j in R:
                layer[j] += 1
                if layer[j] < self.L:
                    self.route(j, layer[j], sp)
            pool = [j for j in pool if layer[j] < self.L]
        return steps
