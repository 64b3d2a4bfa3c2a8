"""ctypes binding of libeasybalance.so (include/easybalance.h).

Argument marshalling only: every function here forwards to the C entry
point of the same name and raises ``EasyBalanceError`` on a non-zero status.
Device buffers may be passed as torch tensors (their data pointers are used)
or as integer addresses.  There is no fallback: if the library is missing,
``lib()`` raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libeasybalance.so")

EB_OK = 0
EB_ERR_INVALID_ARG = -1
EB_ERR_UNSUPPORTED = -2
EB_ERR_HIP = -3
EB_ERR_WORKSPACE_TOO_SMALL = -4
EB_DTYPE_F32, EB_DTYPE_BF16 = 0, 1
EB_POLICY_MAXUTIL, EB_POLICY_CUMUTIL, EB_POLICY_DIFFPEAK, EB_POLICY_LOCKSTEP = 0, 1, 2, 3
EB_PASS_DEVICE_SCHEDULE = 0x100  # OR-ed into easybalance_run_pass's policy
EB_WEIGHTS_GATE_UP, EB_WEIGHTS_DOWN = 0, 1
EB_MAX_POOL = 64
EB_MAXUTIL_MAX_POOL = 20
KERNEL_NAMES = ["route_norm", "route_logits", "route_topk", "perm_count", "perm_scan",
                "perm_scatter", "gateup", "down", "combine", "perm_gather"]
EB_NUM_KERNELS = len(KERNEL_NAMES)
EB_PROFILE_ALL = (1 << EB_NUM_KERNELS) - 1

EXPORTS = ["easybalance_version", "easybalance_last_error", "easybalance_route",
           "easybalance_schedule", "easybalance_moe_step_workspace_size", "easybalance_moe_step",
           "easybalance_combine", "easybalance_profile_begin", "easybalance_profile_end",
           "easybalance_pass_state_size", "easybalance_run_pass", "easybalance_pack_weights",
           "easybalance_moe_step_noalloc"]
EB_NOALLOC_SCRATCH_BYTES = 160 * 1024 * 1024


class eb_model_desc(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("H", ctypes.c_int32), ("F", ctypes.c_int32),
                ("E", ctypes.c_int32), ("k", ctypes.c_int32), ("S", ctypes.c_int32),
                ("D", ctypes.c_int32), ("dtype", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("norm_topk", ctypes.c_int32)]


class eb_work(ctypes.Structure):
    _fields_ = [("mb_id", ctypes.c_int32), ("layer", ctypes.c_int32), ("T", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("a", ctypes.c_void_p), ("idx", ctypes.c_void_p),
                ("w", ctypes.c_void_p)]


class eb_step_views(ctypes.Structure):
    _fields_ = [("a_perm", ctypes.c_void_p), ("h", ctypes.c_void_p), ("perm", ctypes.c_void_p),
                ("offsets", ctypes.c_void_p)]


class eb_placement(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("E", ctypes.c_int32), ("D", ctypes.c_int32),
                ("R", ctypes.c_int32), ("copies", ctypes.c_void_p)]


def make_placement(copies, D: int):
    """copies: int32 array [L][E][R] (device of each copy, ascending, -1
    padded), or per layer a list over experts of device lists.  Returns the
    eb_placement struct (it keeps the array alive)."""
    if not isinstance(copies, np.ndarray):
        L, E = len(copies), len(copies[0])
        R = max(len(c) for layer in copies for c in layer)
        arr = np.full((L, E, R), -1, dtype=np.int32)
        for l, layer in enumerate(copies):
            for e, c in enumerate(layer):
                arr[l, e, :len(c)] = c
        copies = arr
    arr = np.ascontiguousarray(copies, dtype=np.int32)
    L, E, R = arr.shape
    p = eb_placement(L, E, D, R, arr.ctypes.data)
    p._keep = arr
    return p


class EasyBalanceError(RuntimeError):
    def __init__(self, fn: str, code: int, msg: str):
        super().__init__(f"{fn} failed with status {code}: {msg}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    l = ctypes.CDLL(LIB_PATH)
    P, I32, U64P, I64P, SZP = (ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_uint64),
                               ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_size_t))
    D = ctypes.POINTER(eb_model_desc)
    W = ctypes.POINTER(eb_work)
    l.easybalance_version.restype = ctypes.c_char_p
    l.easybalance_version.argtypes = []
    l.easybalance_last_error.restype = ctypes.c_char_p
    l.easybalance_last_error.argtypes = []
    l.easybalance_route.restype = ctypes.c_int
    l.easybalance_route.argtypes = [D, I32, I32, P, P, P, P, P, P, P, P, P, P]
    l.easybalance_schedule.restype = ctypes.c_int
    l.easybalance_schedule.argtypes = [I32, P, P, I32, I32, I32, I32, U64P, I64P, P,
                                       ctypes.POINTER(eb_placement)]
    l.easybalance_moe_step_workspace_size.restype = ctypes.c_int
    l.easybalance_moe_step_workspace_size.argtypes = [D, I32, P, SZP]
    l.easybalance_moe_step.restype = ctypes.c_int
    l.easybalance_moe_step.argtypes = [D, I32, W, P, P, P, ctypes.c_size_t, P, P,
                                       ctypes.POINTER(eb_step_views), P]
    l.easybalance_moe_step_noalloc.restype = ctypes.c_int
    l.easybalance_moe_step_noalloc.argtypes = [D, I32, W, P, P, P, P, ctypes.POINTER(eb_step_views), P]
    l.easybalance_combine.restype = ctypes.c_int
    l.easybalance_combine.argtypes = [D, I32, W, P, P, P, P]
    l.easybalance_pass_state_size.restype = ctypes.c_int
    l.easybalance_pass_state_size.argtypes = [D, I32, I32, SZP]
    l.easybalance_run_pass.restype = ctypes.c_int
    l.easybalance_run_pass.argtypes = [D, I32, I32, P, P, P, P, P, P, I32, I32, P, ctypes.c_size_t,
                                       I32, ctypes.POINTER(ctypes.c_int32), U64P,
                                       ctypes.POINTER(ctypes.c_int32), I64P,
                                       ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32),
                                       ctypes.POINTER(eb_placement), P]
    l.easybalance_pack_weights.restype = ctypes.c_int
    l.easybalance_pack_weights.argtypes = [D, I32, I32, P, P, P]
    l.easybalance_profile_begin.restype = ctypes.c_int
    l.easybalance_profile_begin.argtypes = [ctypes.c_uint32]
    l.easybalance_profile_end.restype = ctypes.c_int
    l.easybalance_profile_end.argtypes = [ctypes.POINTER(ctypes.c_double), I64P]
    _lib = l
    return l


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _check(fn: str, rc: int) -> None:
    if rc != EB_OK:
        raise EasyBalanceError(fn, rc, lib().easybalance_last_error().decode())


def make_desc(L, H, F, E, k, S, D, dtype, rms_eps=1e-6, norm_topk=0) -> eb_model_desc:
    dt = dtype if isinstance(dtype, int) else (EB_DTYPE_BF16 if dtype == "bf16" else EB_DTYPE_F32)
    return eb_model_desc(L, H, F, E, k, S, D, dt, rms_eps, norm_topk)


def easybalance_version() -> str:
    return lib().easybalance_version().decode()


def easybalance_last_error() -> str:
    return lib().easybalance_last_error().decode()


def easybalance_route(desc, layer, T, x, gain, Wg, bias, a_out, logits_out, idx_out, w_out,
                      counts_out, stream=None) -> None:
    _check("easybalance_route", lib().easybalance_route(
        ctypes.byref(desc), layer, T, _ptr(x), _ptr(gain), _ptr(Wg), _ptr(bias), _ptr(a_out),
        _ptr(logits_out), _ptr(idx_out), _ptr(w_out), _ptr(counts_out), stream))


def easybalance_schedule(pool_ids, counts, E, D, m, policy=EB_POLICY_MAXUTIL, want_load=True,
                         layers=None, placement=None):
    """pool_ids: ascending ids; counts: [len(pool)][E] host ints; layers: the
    pool members' layers (with a placement from make_placement).
    Returns (runset_mask, step_load or None)."""
    ids = np.ascontiguousarray(pool_ids, dtype=np.int32)
    cnt = np.ascontiguousarray(counts, dtype=np.int32).reshape(len(ids), E) if len(ids) else \
        np.zeros((0, E), np.int32)
    lay = np.ascontiguousarray(layers, dtype=np.int32) if layers is not None else None
    mask = ctypes.c_uint64(0)
    load = np.zeros(D, dtype=np.int64)
    rc = lib().easybalance_schedule(
        len(ids), ids.ctypes.data if len(ids) else None, cnt.ctypes.data if len(ids) else None,
        E, D, m, policy, ctypes.byref(mask),
        load.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)) if want_load else None,
        lay.ctypes.data if lay is not None and len(lay) else None,
        ctypes.byref(placement) if placement is not None else None)
    _check("easybalance_schedule", rc)
    return mask.value, (load if want_load else None)


def easybalance_moe_step_workspace_size(desc, T_list) -> int:
    T = np.ascontiguousarray(T_list, dtype=np.int32)
    out = ctypes.c_size_t(0)
    _check("easybalance_moe_step_workspace_size", lib().easybalance_moe_step_workspace_size(
        ctypes.byref(desc), len(T), T.ctypes.data, ctypes.byref(out)))
    return out.value


def work_array(entries) -> ctypes.Array:
    """entries: iterable of (mb_id, layer, T, a, idx, w) with tensors or addresses."""
    entries = list(entries)
    arr = (eb_work * max(1, len(entries)))()
    for i, (j, l, T, a, idx, w) in enumerate(entries):
        arr[i] = eb_work(j, l, T, 0, _ptr(a), _ptr(idx), _ptr(w))
    return arr


def _ptr_array(items) -> ctypes.Array:
    items = list(items)
    arr = (ctypes.c_void_p * max(1, len(items)))()
    for i, t in enumerate(items):
        arr[i] = _ptr(t)
    return arr


def easybalance_moe_step(desc, run, n_run, W_gu, W_dn, ws, ws_bytes, o_out, inv_out,
                         views=None, stream=None) -> None:
    """run: a ``work_array``; W_gu/W_dn: per-layer lists of device tensors."""
    gu, dn = _ptr_array(W_gu), _ptr_array(W_dn)
    v = None
    if views is not None:
        v = ctypes.byref(eb_step_views(_ptr(views.get("a_perm")), _ptr(views.get("h")),
                                       _ptr(views.get("perm")), _ptr(views.get("offsets"))))
    _check("easybalance_moe_step", lib().easybalance_moe_step(
        ctypes.byref(desc), n_run, run, gu, dn, _ptr(ws), ws_bytes, _ptr(o_out), _ptr(inv_out),
        v, stream))


def easybalance_moe_step_noalloc(desc, run, n_run, W_gu, W_dn, o_out, inv_out, views,
                                 stream=None) -> None:
    """views: dict with at least "a_perm" and "h" (the caller's buffers)."""
    gu, dn = _ptr_array(W_gu), _ptr_array(W_dn)
    v = None
    if views is not None:
        v = ctypes.byref(eb_step_views(_ptr(views.get("a_perm")), _ptr(views.get("h")),
                                       _ptr(views.get("perm")), _ptr(views.get("offsets"))))
    _check("easybalance_moe_step_noalloc", lib().easybalance_moe_step_noalloc(
        ctypes.byref(desc), n_run, run, gu, dn, _ptr(o_out), _ptr(inv_out), v, stream))


def easybalance_pack_weights(desc, kind, n, src, dst, stream=None) -> None:
    _check("easybalance_pack_weights", lib().easybalance_pack_weights(
        ctypes.byref(desc), kind, n, _ptr(src), _ptr(dst), stream))


def easybalance_combine(desc, run, n_run, x_list, o, inv, stream=None) -> None:
    xs = _ptr_array(x_list)
    _check("easybalance_combine", lib().easybalance_combine(
        ctypes.byref(desc), n_run, run, xs, _ptr(o), _ptr(inv), stream))


def easybalance_pass_state_size(desc, N, T) -> int:
    out = ctypes.c_size_t(0)
    _check("easybalance_pass_state_size",
           lib().easybalance_pass_state_size(ctypes.byref(desc), N, T, ctypes.byref(out)))
    return out.value


def easybalance_run_pass(desc, N, T, x, gain, Wg, bias, W_gu, W_dn, policy, m, state, state_bytes,
                         max_steps=0, record=False, stream=None, placement=None):
    """Returns (n_steps, runsets [n], layers [n][N], step_load [n][D], groups [n],
    layer_loads [N][L][D]) when record, else (n_steps, None, None, None, None, None)."""
    n = ctypes.c_int32(0)
    if record:
        rs = np.zeros(max_steps, dtype=np.uint64)
        ly = np.zeros((max_steps, N), dtype=np.int32)
        sl = np.zeros((max_steps, desc.D), dtype=np.int64)
        gr = np.zeros(max_steps, dtype=np.int32)
        ll = np.zeros((N, desc.L, desc.D), dtype=np.int32)
        ptrs = (rs.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)),
                ly.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                sl.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                gr.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                ll.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))
    else:
        ptrs = (None, None, None, None, None)
    wg, gu, dn = _ptr_array(Wg), _ptr_array(W_gu), _ptr_array(W_dn)
    _check("easybalance_run_pass", lib().easybalance_run_pass(
        ctypes.byref(desc), N, T, _ptr(x), _ptr(gain), wg, _ptr(bias), gu, dn, policy, m,
        _ptr(state), state_bytes, max_steps if record else 0, ctypes.byref(n), *ptrs,
        ctypes.byref(placement) if placement is not None else None, stream))
    k = min(n.value, max_steps) if record else 0
    if not record:
        return n.value, None, None, None, None, None
    return n.value, rs[:k], ly[:k], sl[:k], gr[:k], ll


def easybalance_profile_begin(kernels=None) -> None:
    """kernels: iterable of KERNEL_NAMES entries to time (default: all)."""
    mask = EB_PROFILE_ALL if kernels is None else sum(1 << KERNEL_NAMES.index(k) for k in kernels)
    _check("easybalance_profile_begin", lib().easybalance_profile_begin(mask))


def easybalance_profile_end() -> dict:
    ms = (ctypes.c_double * EB_NUM_KERNELS)()
    n = (ctypes.c_int64 * EB_NUM_KERNELS)()
    _check("easybalance_profile_end", lib().easybalance_profile_end(ms, n))
    return {name: (ms[i], n[i]) for i, name in enumerate(KERNEL_NAMES)}
