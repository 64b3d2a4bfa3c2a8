"""Per-step grouping of routed work by (layer, expert).

On a real expert-parallel group an all-to-all sends each (token, expert) pair
to the device that owns the expert and a second all-to-all brings the result
back (Section 2.2).  When the work of several micro-batches at different
layers runs jointly in one step (Section 4.1, cross-layer workload
combination), one GPU groups all pairs of the step by the key
(layer, expert); the permutation below is that grouping.

Definition used here:
* pairs are enumerated micro-batch by micro-batch in run order (ascending
  micro-batch id), then token t ascending, then slot r ascending; slots
  0..k-1 are the routed picks idx[t][r], slots k..k+S-1 are the shared
  experts, given expert slot ids E..E+S-1;
* key(pair) = layer * (E + S) + expert slot;
* perm is the stable sort of the pairs by key (equal keys keep enumeration
  order), inv[q] is the position of pair q in perm, offsets is the exclusive
  prefix sum of the per-key pair counts over all L*(E+S) keys.
"""
from __future__ import annotations

import numpy as np


def step_keys(run: list[tuple[int, np.ndarray]], E: int, S: int) -> np.ndarray:
    """Keys of all pairs of a step.  run = [(layer, idx [T][k]), ...] in run order."""
    keys = []
    for layer, idx in run:
        idx = np.asarray(idx, np.int64)
        T = idx.shape[0]
        slots = np.concatenate([idx, np.broadcast_to(E + np.arange(S, dtype=np.int64), (T, S))],
                               axis=1)
        keys.append(layer * (E + S) + slots.reshape(-1))
    return np.concatenate(keys) if keys else np.zeros(0, np.int64)


def stable_permutation(keys: np.ndarray, n_keys: int):
    """(perm, inv, offsets) of the stable sort of ``keys``."""
    keys = np.asarray(keys, np.int64)
    perm = np.argsort(keys, kind="stable")
    inv = np.empty_like(perm)
    inv[perm] = np.arange(keys.size)
    offsets = np.zeros(n_keys + 1, np.int64)
    offsets[1:] = np.cumsum(np.bincount(keys, minlength=n_keys)[:n_keys])
    return perm.astype(np.int64), inv.astype(np.int64), offsets


def source_rows(run: list[tuple[int, np.ndarray]], S: int) -> np.ndarray:
    """For each pair q of the step: (entry, token) whose activation row it carries."""
    out = []
    for rho, (_, idx) in enumerate(run):
        T, k = np.asarray(idx).shape
        t = np.repeat(np.arange(T), k + S)
        out.append(np.stack([np.full_like(t, rho), t], axis=1))
    return np.concatenate(out) if out else np.zeros((0, 2), np.int64)
