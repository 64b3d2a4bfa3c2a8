"""Seeded, counter-based input generator (host side, NumPy).

Every large synthetic tensor (residual stream x, router weights, expert
weights) is a pure function of (seed, tensor kind, tensor index, element
index), so any slice can be regenerated on its own -- the oracle rebuilds one
expert's weights at a time -- and the device fill kernel in ``fill.hip``
produces the same bits.  The definition is:

    key      = mix64((seed << 24) | (kind << 16) | index)
    u_i      = mix64(key + (i + 1) * GAMMA)            (mod 2^64)
    normal_i = float32(TABLE[u_i >> 48]) * float32(sigma)   (one IEEE fp32 multiply)
    bf16_i   = round-to-nearest-even of normal_i to bfloat16 (integer bit arithmetic)

mix64 is the SplitMix64 output function (Steele, Lea & Flood, "Fast
splittable pseudorandom number generators", OOPSLA 2014) and u_i is the i-th
output of a SplitMix64 stream whose state starts at ``key``.  TABLE holds the
standard normal quantiles at the midpoints (j + 0.5) / 65536, j = 0..65535,
computed in float64 with ``statistics.NormalDist().inv_cdf`` and rounded to
fp32.  Only integer operations, one table load and one fp32 multiply are
involved, so host and device agree bit for bit.

Small per-layer vectors (the router bias that skews the load) come from
NumPy's PCG64 generator; they are handed to both sides as inputs.

This module holds no arithmetic of the method itself.
"""
from __future__ import annotations

import ctypes
import functools
import os
import statistics

import numpy as np

from .configs import Config

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB

# tensor kinds
KIND_X = 1      # residual stream x [N][T][H] fp32, sigma 1
KIND_WG = 2     # router weights of layer l [E][H], sigma 1/sqrt(H)
KIND_GU = 3     # gate|up weights of layer l [E+S][2F][H], sigma 0.02
KIND_DN = 4     # down weights of layer l [E+S][H][F], sigma 0.02

EXPERT_SIGMA = 0.02


def mix64_int(z: int) -> int:
    z &= MASK64
    z ^= z >> 30
    z = (z * MIX1) & MASK64
    z ^= z >> 27
    z = (z * MIX2) & MASK64
    z ^= z >> 31
    return z


def stream_key(seed: int, kind: int, index: int) -> int:
    assert 0 <= kind < 256 and 0 <= index < 65536 and 0 <= seed < (1 << 40)
    return mix64_int((seed << 24) | (kind << 16) | index)


@functools.lru_cache(maxsize=1)
def normal_table() -> np.ndarray:
    nd = statistics.NormalDist()
    return np.array([nd.inv_cdf((j + 0.5) / 65536.0) for j in range(65536)],
                    dtype=np.float64).astype(np.float32)


def sigma_of(kind: int, H: int) -> np.float32:
    if kind == KIND_X:
        return np.float32(1.0)
    if kind == KIND_WG:
        return np.float32(1.0 / np.sqrt(np.float64(H)))
    return np.float32(EXPERT_SIGMA)


def _mix64_np(z: np.ndarray) -> np.ndarray:
    z = z ^ (z >> np.uint64(30))
    z = z * np.uint64(MIX1)
    z = z ^ (z >> np.uint64(27))
    z = z * np.uint64(MIX2)
    z = z ^ (z >> np.uint64(31))
    return z


_HOST_LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsynthhost.so")
_host = None


def _host_lib():
    """The C/OpenMP implementation of the same stream (gen_host.c), if built."""
    global _host
    if _host is None and os.path.exists(_HOST_LIB):
        l = ctypes.CDLL(_HOST_LIB)
        l.synth_host_normal.restype = None
        l.synth_host_normal.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64,
                                        ctypes.c_void_p, ctypes.c_float, ctypes.c_int,
                                        ctypes.c_void_p]
        _host = l
    return _host


def normal_values(key: int, i0: int, n: int, sigma: np.float32, as_bf16: bool) -> np.ndarray:
    """Elements i0 .. i0+n-1 of stream ``key`` as fp32 (rounded to bf16 values
    if ``as_bf16``); uses the compiled generator when it is built."""
    l = _host_lib()
    if l is None:
        v = normal_f32(key, i0, n, sigma)
        return bf16_bits_to_f32(f32_to_bf16_bits(v)) if as_bf16 else v
    out = np.empty(n, dtype=np.float32)
    tab = normal_table()
    l.synth_host_normal(key, i0, n, tab.ctypes.data, float(sigma), int(as_bf16), out.ctypes.data)
    return out


def normal_f32(key: int, i0: int, n: int, sigma: np.float32,
               chunk: int = 1 << 23) -> np.ndarray:
    """fp32 values of elements i0 .. i0+n-1 of the stream ``key`` (NumPy
    reference implementation of the definition above)."""
    tab = normal_table()
    out = np.empty(n, dtype=np.float32)
    k = np.uint64(key)
    g = np.uint64(GAMMA)
    with np.errstate(over="ignore"):
        for s in range(0, n, chunk):
            e = min(n, s + chunk)
            i = np.arange(i0 + s + 1, i0 + e + 1, dtype=np.uint64)
            u = _mix64_np(k + i * g)
            out[s:e] = tab[(u >> np.uint64(48)).astype(np.int64)] * np.float32(sigma)
    return out


def f32_to_bf16_bits(v: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 on the bit pattern (finite inputs)."""
    b = v.astype(np.float32).view(np.uint32).astype(np.uint64)
    r = (b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return (r & np.uint64(0xFFFF)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def tensor_values(cfg: Config, kind: int, index: int, i0: int, n: int) -> np.ndarray:
    """Elements [i0, i0+n) of a generated tensor as the stored values, in fp32
    (for bf16 storage: the fp32 value of the stored bf16).  x is always fp32."""
    return normal_values(stream_key(cfg.seed, kind, index), i0, n, sigma_of(kind, cfg.H),
                         cfg.dtype == "bf16" and kind != KIND_X)


# ---- whole tensors / slices used by tests and the oracle -------------------

def x_all(cfg: Config) -> np.ndarray:
    return tensor_values(cfg, KIND_X, 0, 0, cfg.N * cfg.T * cfg.H).reshape(cfg.N, cfg.T, cfg.H)


def x_rows(cfg: Config, j: int, t0: int, nt: int) -> np.ndarray:
    i0 = (j * cfg.T + t0) * cfg.H
    return tensor_values(cfg, KIND_X, 0, i0, nt * cfg.H).reshape(nt, cfg.H)


def router_weight(cfg: Config, layer: int) -> np.ndarray:
    return tensor_values(cfg, KIND_WG, layer, 0, cfg.E * cfg.H).reshape(cfg.E, cfg.H)


def expert_gate_up(cfg: Config, layer: int, e: int) -> tuple[np.ndarray, np.ndarray]:
    """(W_gate [F][H], W_up [F][H]) of expert slot e (e >= E: shared expert e-E)."""
    F, H = cfg.F, cfg.H
    v = tensor_values(cfg, KIND_GU, layer, e * 2 * F * H, 2 * F * H).reshape(2 * F, H)
    return v[:F], v[F:]


def expert_down(cfg: Config, layer: int, e: int) -> np.ndarray:
    """W_down [H][F] of expert slot e."""
    F, H = cfg.F, cfg.H
    return tensor_values(cfg, KIND_DN, layer, e * H * F, H * F).reshape(H, F)


def rms_gain(cfg: Config) -> np.ndarray:
    return np.ones(cfg.H, dtype=np.float32)


def router_bias(cfg: Config) -> np.ndarray:
    """Per-layer logit bias ln(p_l[e]) [L][E] fp32 that skews the routing.

    zipf:       p[pi_l(r)] ~ r^-s for rank r = 1..E, fresh uniform permutation per layer
    zipf_drift: as zipf, but pi_{l+1} is pi_l after E/8 random rank transpositions
    dirichlet:  p ~ Dirichlet(alpha * 1_E), resampled per layer
    """
    rng = np.random.Generator(np.random.PCG64(cfg.seed))
    E, L, s = cfg.E, cfg.L, cfg.skew_param
    out = np.empty((L, E), dtype=np.float32)
    ranks = np.arange(1, E + 1, dtype=np.float64)
    zipf = ranks ** (-s)
    zipf /= zipf.sum()
    perm = rng.permutation(E)
    for l in range(L):
        if cfg.skew == "zipf":
            perm = rng.permutation(E)
            p = np.empty(E)
            p[perm] = zipf
        elif cfg.skew == "zipf_drift":
            if l > 0:
                for _ in range(max(1, E // 8)):
                    a, b = rng.integers(0, E, size=2)
                    perm[a], perm[b] = perm[b], perm[a]
            p = np.empty(E)
            p[perm] = zipf
        elif cfg.skew == "dirichlet":
            p = rng.dirichlet(np.full(E, s))
        else:
            raise ValueError(cfg.skew)
        out[l] = np.log(np.maximum(p, 1e-30)).astype(np.float32)
    return out
