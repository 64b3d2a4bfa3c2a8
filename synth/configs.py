"""Workload definitions: the five synthetic MoE stacks and their routing skew.

These are inputs, not method: shapes, seeds, distributions and the minimum
combination size m.  Both the CPU oracle and the GPU path read them.

The paper measures on LongBench prompts run through Qwen3-30B-A3B,
Moonlight-16B-A3B and Qwen3-235B-A22B (Section 5, "Models"/"Benchmark");
none of those are available here, so seeded synthetic stacks with skewed
routers stand in for them.  Every stack is MoE-only:
    x <- x + MoE_l(RMSNorm(x))          for l = 0 .. L-1
which is the MLP half of the residual block in Section 2.1 (attention is
outside the method, Appendix B).
"""
from __future__ import annotations

import dataclasses
import math


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    L: int          # MoE layers
    H: int          # hidden size
    F: int          # expert FFN size
    E: int          # routed experts
    k: int          # top-k
    S: int          # always-on shared experts (weight 1, not in the load vectors)
    D: int          # virtual expert-parallel devices (E/D experts each)
    N: int          # micro-batches
    T: int          # tokens per micro-batch
    dtype: str      # "f32" or "bf16" (storage of activations/weights; fp32 accumulate)
    skew: str       # "zipf" | "zipf_drift" | "dirichlet"
    skew_param: float
    seed: int
    eps: float = 1e-6
    norm_topk: int = 0

    @property
    def m(self) -> int:
        """Minimum combination size: 0.75 of the micro-batch count, at least 1.

        Section 4.2 suggests m between 0.5 and 0.75 of the number of
        micro-batches, and Section 5 uses m=3 at 4 micro-batches.
        """
        return max(1, math.floor(0.75 * self.N))

    @property
    def experts_per_device(self) -> int:
        return self.E // self.D

    @property
    def slots(self) -> int:
        """Expert slots per token: k routed plus S shared."""
        return self.k + self.S

    @property
    def ffn_flop_per_pair(self) -> int:
        """Gate+up GEMM (4HF) plus down GEMM (2HF) for one (token, expert) pair."""
        return 6 * self.H * self.F

    @property
    def total_ffn_flop(self) -> int:
        return self.ffn_flop_per_pair * self.N * self.T * self.slots * self.L

    def scaled(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


CONFIGS = [
    # 0: tiny fp32 stack that the oracle finishes in well under a second.
    Config("tiny_f32", L=2, H=256, F=512, E=8, k=2, S=0, D=4, N=2, T=64,
           dtype="f32", skew="zipf", skew_param=1.2, seed=20260000),
    # 1: Mixtral-8x7B-shaped layers.
    Config("mixtral_bf16", L=8, H=4096, F=14336, E=8, k=2, S=0, D=8, N=4, T=512,
           dtype="bf16", skew="zipf", skew_param=1.0, seed=20260001),
    # 2: Qwen1.5-MoE-shaped layers.
    Config("qwen_moe_bf16", L=12, H=2048, F=1408, E=60, k=4, S=4, D=4, N=8, T=1024,
           dtype="bf16", skew="zipf", skew_param=1.1, seed=20260002),
    # 3: DeepSeek-V2-Lite-shaped layers, decode-like small micro-batches.
    Config("dsv2_lite_bf16", L=26, H=2048, F=1408, E=64, k=6, S=2, D=8, N=16, T=256,
           dtype="bf16", skew="dirichlet", skew_param=0.3, seed=20260003),
    # 4: DeepSeek-V3-shaped layers, one GPU's share of an EP group.
    Config("dsv3_share_bf16", L=8, H=7168, F=2048, E=256, k=8, S=1, D=32, N=8, T=4096,
           dtype="bf16", skew="zipf_drift", skew_param=1.3, seed=20260004),
]

BY_NAME = {c.name: c for c in CONFIGS}


def mini(cfg: Config, **kw) -> Config:
    """A reduced copy of a stack for parity tests: same E/k/S/D/N structure and
    skew model, smaller H/F/T/L so the oracle runs in seconds while the GPU
    kernels still span several tiles and ragged tails."""
    base = dict(H=512, F=384, T=200, L=min(cfg.L, 3))
    base.update(kw)
    return cfg.scaled(name=cfg.name + "_mini", **base)
