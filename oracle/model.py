"""The MoE computation that EasyBalance schedules, written from its definition.

One layer of a micro-batch (Section 2.1 of EasyBalance, arXiv 2608.07964):

    a   = cast(RMSNorm(x))                          normalised input h'_l
    W,I = topk(G(a))                                Section 2.1, routing
    MLP = sum_{i in I} W_i * expert_i(a)            Eq. (1)
    x  <- x + MLP + sum_s shared_s(a)               residual of Section 2.1

with SwiGLU experts expert(a) = cast( cast(SiLU(a Wg^T) * (a Wu^T)) Wd^T ).

Readings where the paper is silent:
* G is a linear router with a per-layer logit bias, z = a Wg^T + b, and the
  gating probabilities are the softmax of z over all E experts; the top-k
  weights are NOT renormalised (Eq. 1 taken literally).  ``norm_topk=1``
  renormalises them over the selected k, as an option.
* Top-k selects on the logits z; equal logits go to the lower expert id.
* Shared (always-on) experts have weight 1 and no gate; they are replicated on
  every device, so they are left out of the per-device load vectors.
* RMSNorm: r = 1/sqrt(mean(x^2) + eps), eps = 1e-6, gain g.
* Precision: float64 arithmetic, rounding to bf16 at a, h and o when the stack
  stores bf16 (``cast``); the residual stream x stays at full precision.
* Expert placement: E/D contiguous experts per device, device(e) = e // (E/D)
  (the paper's evenly distributed mapping, Section 5 "Models").
* Workload unit: number of routed (token, expert) pairs per device.
"""
from __future__ import annotations

import dataclasses
from typing import Callable

import numpy as np

from .numerics import cast_fn, silu, softmax_rows


# --------------------------------------------------------------------------
# routing (Section 2.1: W, I = topk(G(h')))
# --------------------------------------------------------------------------

def rmsnorm_cast(x: np.ndarray, g: np.ndarray, eps: float, cast) -> np.ndarray:
    """a = cast(x * r * g), r = 1/sqrt(mean(x^2) + eps), per row."""
    x = np.asarray(x, dtype=np.float64)
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return cast(x * r * np.asarray(g, dtype=np.float64))


def router_logits(a: np.ndarray, Wg: np.ndarray, bias: np.ndarray) -> np.ndarray:
    """z = a Wg^T + b, [T][E]."""
    return np.asarray(a, np.float64) @ np.asarray(Wg, np.float64).T + np.asarray(bias, np.float64)


def topk_indices(z: np.ndarray, k: int) -> np.ndarray:
    """Ids of the k largest logits per row, largest first; ties -> lower id."""
    return np.argsort(-np.asarray(z, np.float64), axis=-1, kind="stable")[:, :k].astype(np.int32)


def gate_weights(z: np.ndarray, idx: np.ndarray, norm_topk: int = 0) -> np.ndarray:
    """W_r = softmax(z)[idx_r]; optionally renormalised over the k picks."""
    p = softmax_rows(z)
    w = np.take_along_axis(p, idx.astype(np.int64), axis=-1)
    if norm_topk:
        w = w / w.sum(axis=-1, keepdims=True)
    return w


def expert_counts(idx: np.ndarray, E: int) -> np.ndarray:
    """Routed (token, expert) pairs per expert."""
    return np.bincount(np.asarray(idx).reshape(-1), minlength=E)[:E].astype(np.int64)


def device_loads(counts: np.ndarray, D: int) -> np.ndarray:
    """Workload vector w in Z^D (Section 2.3): pairs per device, E/D contiguous
    experts per device.  Works on the last axis of ``counts``."""
    counts = np.asarray(counts, dtype=np.int64)
    E = counts.shape[-1]
    assert E % D == 0
    return counts.reshape(counts.shape[:-1] + (D, E // D)).sum(axis=-1)


def placed_device_loads(counts: np.ndarray, copies, D: int) -> np.ndarray:
    """Workload vector under a static placement with replicas (the redundant
    experts of Section 5's orthogonality study with EPLB): copies[e] lists the
    devices holding expert e in ascending order; an expert's c routed pairs
    are split as evenly as possible over its r copies, the i-th copy taking
    c // r pairs plus one if i < c % r.  Works on the last axis of counts."""
    counts = np.asarray(counts, dtype=np.int64)
    E = counts.shape[-1]
    assert len(copies) == E
    out = np.zeros(counts.shape[:-1] + (D,), dtype=np.int64)
    for e in range(E):
        devs = list(copies[e])
        r = len(devs)
        assert r >= 1 and devs == sorted(set(devs)) and all(0 <= d < D for d in devs)
        c = counts[..., e]
        for i, d in enumerate(devs):
            out[..., d] += c // r + (c % r > i)
    return out


# --------------------------------------------------------------------------
# experts and combine (Eq. 1 plus the residual add)
# --------------------------------------------------------------------------

def expert_ffn(a_rows: np.ndarray, W_gate: np.ndarray, W_up: np.ndarray,
               W_down: np.ndarray, cast) -> tuple[np.ndarray, np.ndarray]:
    """SwiGLU expert on a block of rows: returns (h, o).

    h = cast(SiLU(a W_gate^T) * (a W_up^T))   [M][F]
    o = cast(h W_down^T)                      [M][H]
    """
    a = np.asarray(a_rows, np.float64)
    gate = a @ np.asarray(W_gate, np.float64).T
    up = a @ np.asarray(W_up, np.float64).T
    h = cast(silu(gate) * up)
    o = cast(h @ np.asarray(W_down, np.float64).T)
    return h, o


def combine(x: np.ndarray, o_routed: np.ndarray, w: np.ndarray,
            o_shared: np.ndarray | None) -> np.ndarray:
    """x + sum_r w_r o_r + sum_s o_s  (Eq. 1 and the residual of Section 2.1).

    x [T][H], o_routed [T][k][H], w [T][k], o_shared [T][S][H] or None.
    """
    out = np.asarray(x, np.float64) + np.einsum("tk,tkh->th", np.asarray(w, np.float64),
                                                np.asarray(o_routed, np.float64))
    if o_shared is not None and o_shared.shape[1] > 0:
        out = out + np.asarray(o_shared, np.float64).sum(axis=1)
    return out


# --------------------------------------------------------------------------
# weights provider and a plain layer-by-layer run
# --------------------------------------------------------------------------

@dataclasses.dataclass
class Weights:
    """Callables that return one layer's / one expert's parameters as arrays.

    gain(l) -> [H]; router(l) -> Wg [E][H]; bias(l) -> [E];
    gate_up(l, e) -> (W_gate [F][H], W_up [F][H]); down(l, e) -> W_down [H][F];
    expert slot e in [0, E) is routed, e in [E, E+S) is shared expert e-E.
    """
    gain: Callable[[int], np.ndarray]
    router: Callable[[int], np.ndarray]
    bias: Callable[[int], np.ndarray]
    gate_up: Callable[[int, int], tuple[np.ndarray, np.ndarray]]
    down: Callable[[int, int], np.ndarray]


@dataclasses.dataclass
class LayerOut:
    a: np.ndarray        # [T][H]
    z: np.ndarray        # [T][E]
    idx: np.ndarray      # [T][k]
    w: np.ndarray        # [T][k]
    counts: np.ndarray   # [E]
    x_out: np.ndarray    # [T][H]


def route(x: np.ndarray, l: int, P: Weights, *, k: int, eps: float, dtype: str,
          norm_topk: int = 0):
    """Routing stage of one (micro-batch, layer): (a, z, idx, w, counts)."""
    cast = cast_fn(dtype)
    a = rmsnorm_cast(x, P.gain(l), eps, cast)
    z = router_logits(a, P.router(l), P.bias(l))
    idx = topk_indices(z, k)
    w = gate_weights(z, idx, norm_topk)
    E = z.shape[1]
    return a, z, idx, w, expert_counts(idx, E)


def moe_layer(x: np.ndarray, l: int, P: Weights, *, E: int, k: int, S: int, eps: float,
              dtype: str, norm_topk: int = 0) -> LayerOut:
    """One MoE layer of one micro-batch, all experts, plain definition."""
    cast = cast_fn(dtype)
    a, z, idx, w, counts = route(x, l, P, k=k, eps=eps, dtype=dtype, norm_topk=norm_topk)
    T, H = a.shape
    o_routed = np.zeros((T, k, H))
    for e in np.unique(idx):
        rows, slots = np.nonzero(idx == e)
        Wg_, Wu_ = P.gate_up(l, int(e))
        _, o = expert_ffn(a[rows], Wg_, Wu_, P.down(l, int(e)), cast)
        o_routed[rows, slots] = o
    o_shared = np.zeros((T, S, H))
    for s in range(S):
        Wg_, Wu_ = P.gate_up(l, E + s)
        _, o_shared[:, s] = expert_ffn(a, Wg_, Wu_, P.down(l, E + s), cast)
    return LayerOut(a=a, z=z, idx=idx, w=w, counts=counts,
                    x_out=combine(x, o_routed, w, o_shared))


@dataclasses.dataclass
class PlainRun:
    x: np.ndarray        # [L+1][N][T][H]: x before layer 0 .. after layer L-1
    idx: np.ndarray      # [N][L][T][k]
    w: np.ndarray        # [N][L][T][k]
    counts: np.ndarray   # [N][L][E]
    loads: np.ndarray    # [N][L][D]


def run_plain(x0: np.ndarray, P: Weights, *, L: int, E: int, k: int, S: int, D: int,
              eps: float, dtype: str, norm_topk: int = 0) -> PlainRun:
    """Every micro-batch through every layer in order, no scheduling.

    EasyBalance is lossless (Section 4.1: each micro-batch keeps its own layer
    order), so any schedule must reproduce these hidden states; routing of
    (j, l) depends only on x_j at layer l, so the load tensor recorded here is
    the input of every schedule.
    """
    x0 = np.asarray(x0, np.float64)
    N, T, H = x0.shape
    xs = np.zeros((L + 1, N, T, H))
    xs[0] = x0
    idx = np.zeros((N, L, T, k), np.int32)
    w = np.zeros((N, L, T, k))
    counts = np.zeros((N, L, E), np.int64)
    for l in range(L):
        for j in range(N):
            out = moe_layer(xs[l, j], l, P, E=E, k=k, S=S, eps=eps, dtype=dtype,
                            norm_topk=norm_topk)
            xs[l + 1, j] = out.x_out
            idx[j, l], w[j, l], counts[j, l] = out.idx, out.w, out.counts
    return PlainRun(x=xs, idx=idx, w=w, counts=counts, loads=device_loads(counts, D))
