"""Device-resident synthetic inputs (fills torch tensors through libebsynth.so).

The values are bit-identical to ``synth.gen`` (host).  Used by the GPU tests,
``smoke()`` and ``bench.py`` so that every input is generated directly in HBM.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

from . import gen
from .configs import Config

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libebsynth.so")
_lib = None
_tables: dict = {}


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        l = ctypes.CDLL(LIB_PATH)
        l.synth_fill_normal.restype = ctypes.c_int
        l.synth_fill_normal.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                        ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p,
                                        ctypes.c_float, ctypes.c_void_p]
        _lib = l
    return _lib


def _table(device: torch.device) -> torch.Tensor:
    key = str(device)
    if key not in _tables:
        _tables[key] = torch.from_numpy(gen.normal_table().copy()).to(device)
    return _tables[key]


def torch_dtype(cfg: Config) -> torch.dtype:
    return torch.bfloat16 if cfg.dtype == "bf16" else torch.float32


def fill_(t: torch.Tensor, cfg: Config, kind: int, index: int, i0: int = 0) -> torch.Tensor:
    """Fill a contiguous device tensor with elements i0.. of the (kind, index) stream."""
    assert t.is_cuda and t.is_contiguous()
    if t.dtype == torch.bfloat16:
        dt = 1
    elif t.dtype == torch.float32:
        dt = 0
    else:
        raise TypeError(t.dtype)
    key = gen.stream_key(cfg.seed, kind, index)
    sigma = float(gen.sigma_of(kind, cfg.H))
    stream = torch.cuda.current_stream(t.device).cuda_stream
    rc = lib().synth_fill_normal(ctypes.c_void_p(t.data_ptr()), t.numel(), dt, key, i0,
                                 ctypes.c_void_p(_table(t.device).data_ptr()), sigma,
                                 ctypes.c_void_p(stream))
    if rc != 0:
        raise RuntimeError(f"synth_fill_normal failed: hip error {rc}")
    return t


class DeviceInputs:
    """All inputs of one stack, resident on the device.

    x      [N][T][H] fp32          (residual stream, overwritten by combine)
    g      [L][H] fp32             (RMSNorm gain, ones)
    Wg     [L] -> [E][H] dtype      (router weights)
    bias   [L][E] fp32             (router logit bias that skews the load)
    W_gu   [L] -> [E+S][2F][H] dtype (rows 0..F-1 gate, F..2F-1 up)
    W_dn   [L] -> [E+S][H][F] dtype
    """

    def __init__(self, cfg: Config, device="cuda:0", weights: bool = True):
        self.cfg = cfg
        dev = torch.device(device)
        dt = torch_dtype(cfg)
        L, H, F, E, S = cfg.L, cfg.H, cfg.F, cfg.E, cfg.S
        self.x0 = fill_(torch.empty(cfg.N, cfg.T, H, dtype=torch.float32, device=dev),
                        cfg, gen.KIND_X, 0)
        self.g = torch.ones(L, H, dtype=torch.float32, device=dev)
        self.Wg = [fill_(torch.empty(E, H, dtype=dt, device=dev), cfg, gen.KIND_WG, l)
                   for l in range(L)]
        self.bias = torch.from_numpy(gen.router_bias(cfg)).to(dev)
        self.W_gu, self.W_dn = [], []
        if weights:
            for l in range(L):
                self.W_gu.append(fill_(torch.empty(E + S, 2 * F, H, dtype=dt, device=dev),
                                       cfg, gen.KIND_GU, l))
                self.W_dn.append(fill_(torch.empty(E + S, H, F, dtype=dt, device=dev),
                                       cfg, gen.KIND_DN, l))

    def weight_bytes(self) -> int:
        return sum(t.numel() * t.element_size() for t in self.W_gu + self.W_dn)


def host_bias(cfg: Config) -> np.ndarray:
    return gen.router_bias(cfg)
