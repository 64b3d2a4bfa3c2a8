"""Shared helpers of the GPU parity tests (not collected by pytest)."""
from __future__ import annotations

import functools
import sys

import numpy as np
import torch

from oracle import model as omodel
from synth import gen
from synth.device import DeviceInputs


def tol_factor(dtype: str) -> float:
    """Activation tolerance: max-abs error <= factor * max|ref|."""
    return 1e-5 if dtype == "f32" else 1e-2


def assert_close(got, ref, dtype: str, what: str) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    scale = max(float(np.abs(ref).max()) if ref.size else 0.0, 1e-30)
    err = float(np.abs(got - ref).max()) if ref.size else 0.0
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    assert err <= tol_factor(dtype) * scale, f"{what}: max-abs err {err:.3e} > {tol_factor(dtype)} * {scale:.3e}"
    return err / scale


def to_np(t: torch.Tensor) -> np.ndarray:
    t = t.detach()
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy().astype(np.float64) if t.is_floating_point() else t.cpu().numpy()


def host_weights(cfg, cache: bool = True) -> omodel.Weights:
    """Oracle parameter provider regenerating the same synthetic weights on the host."""
    bias = gen.router_bias(cfg)
    gu = functools.lru_cache(maxsize=64 if cache else 2)(lambda l, e: gen.expert_gate_up(cfg, l, e))
    dn = functools.lru_cache(maxsize=64 if cache else 2)(lambda l, e: gen.expert_down(cfg, l, e))
    rw = functools.lru_cache(maxsize=None)(lambda l: gen.router_weight(cfg, l))
    return omodel.Weights(gain=lambda l: gen.rms_gain(cfg), router=rw, bias=lambda l: bias[l],
                          gate_up=gu, down=dn)


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def ensure_packed(cfg, inp: DeviceInputs) -> DeviceInputs:
    """Packs the inputs' expert weights, once, into the layout the library's
    grouped GEMMs read (the host oracle regenerates its own row-major copies)."""
    from paper_2608_07964_amd import binding as B
    from paper_2608_07964_amd.driver import is_packed, pack_expert_weights
    if inp.W_gu and not is_packed(inp.W_gu[0]):
        desc = B.make_desc(cfg.L, cfg.H, cfg.F, cfg.E, cfg.k, cfg.S, cfg.D, cfg.dtype, cfg.eps,
                           cfg.norm_topk)
        pack_expert_weights(desc, inp.W_gu, inp.W_dn)
    return inp


def make_stack(cfg, device="cuda:0", inputs: DeviceInputs | None = None):
    from paper_2608_07964_amd.driver import Stack
    inp = ensure_packed(cfg, inputs or DeviceInputs(cfg, device))
    x = inp.x0.clone()
    st = Stack(L=cfg.L, H=cfg.H, F=cfg.F, E=cfg.E, k=cfg.k, S=cfg.S, D=cfg.D, N=cfg.N, T=cfg.T,
               dtype=cfg.dtype, x=x, gain=inp.g, Wg=inp.Wg, bias=inp.bias, W_gu=inp.W_gu,
               W_dn=inp.W_dn, eps=cfg.eps, norm_topk=cfg.norm_topk, device=device)
    return st, inp
