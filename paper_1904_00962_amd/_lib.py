"""ctypes binding of ``liblamb_mi355x.so`` (include/lamb_mi355x.h).

Argument marshalling only: every step of the optimizer runs in the HIP
kernels behind these calls. The functions keep the C names; failures raise
:class:`LambError` carrying the status code and the library's error detail.
The library is loaded on first use and its absence is an error: there is no
fallback implementation.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np

from . import build as _build

LIBRARY = _build.LIBRARY

LAMB_OK = 0
LAMB_EINVAL = -1
LAMB_ENULL = -2
LAMB_EALIGN = -3
LAMB_EOVERLAP = -4
LAMB_EHIP = -5
LAMB_ENOMEM = -6
LAMB_EPLAN = -7
LAMB_ESYNC = -8

LAMB_GRAD_F32 = 0
LAMB_GRAD_BF16 = 1
LAMB_ALGO_LAMB = 0
LAMB_ALGO_LARS = 1

LAMB_VARIANT_LAMB = 0
LAMB_VARIANT_NLAMB = 1
LAMB_VARIANT_NNLAMB = 2
LAMB_VARIANT_LARS = 3
VARIANTS = {"lamb": LAMB_VARIANT_LAMB, "n-lamb": LAMB_VARIANT_NLAMB,
            "nn-lamb": LAMB_VARIANT_NNLAMB, "lars": LAMB_VARIANT_LARS}

LAMB_NORM_L2 = 0
LAMB_NORM_L1 = 1
LAMB_NORM_LINF = 2
NORMS = {"l2": LAMB_NORM_L2, "l1": LAMB_NORM_L1, "linf": LAMB_NORM_LINF}

LAMB_PATH_AUTO = 0
LAMB_PATH_TWO_PASS = 1
PATHS = {"auto": LAMB_PATH_AUTO, "two-pass": LAMB_PATH_TWO_PASS}

# Every symbol the header declares (checked by the test suite).
EXPORTS = ("lamb_plan_create", "lamb_plan_destroy", "lamb_plan_info",
           "lamb_plan_set_bf16_copies", "lamb_hparams_init",
           "lamb_step_ex", "lamb_step", "nlamb_step", "lars_step", "lamb_lr_at",
           "lamb_sqrt_scaled_lr", "lamb_chunk_table", "lamb_plan_set_timing", "lamb_plan_timing",
           "lamb_plan_set_path", "lamb_plan_tiles", "lamb_plan_check", "lamb_tile_schedule",
           "lamb_step_partials", "lamb_step_finish", "lamb_plan_set_u_check",
           "lamb_plan_u_partials", "lamb_step_static", "lamb_plan_set_trace", "lamb_status_str",
           "lamb_last_error")


class LambError(RuntimeError):
    def __init__(self, status: int, func: str, detail: str):
        self.status = status
        super().__init__("%s failed with status %d (%s): %s"
                         % (func, status, status_str(status), detail))


class lamb_tensor(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("g", ctypes.c_void_p), ("m", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("numel", ctypes.c_int64), ("wd", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class lamb_hparams(ctypes.Structure):
    _fields_ = [("variant", ctypes.c_int32), ("norm", ctypes.c_int32), ("step", ctypes.c_int64),
                ("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("gamma_l", ctypes.c_float), ("gamma_u", ctypes.c_float),
                ("trust_coef", ctypes.c_float), ("grad_scale", ctypes.c_float),
                ("bias_correction", ctypes.c_int32), ("skip_nonfinite", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class lamb_lr_stage(ctypes.Structure):
    _fields_ = [("steps", ctypes.c_int64), ("warmup_steps", ctypes.c_int64),
                ("peak_lr", ctypes.c_double), ("power", ctypes.c_double)]


_lib: Optional[ctypes.CDLL] = None


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Open the HIP library (once). Raises if it has not been built.

    ``LAMB_MI355X_LIBRARY`` may name another build of the same library (for
    comparing compile-time variants); the default is the in-tree build.
    """
    global _lib
    if _lib is not None:
        return _lib
    path = path or os.environ.get("LAMB_MI355X_LIBRARY") or LIBRARY
    if not os.path.exists(path):
        raise RuntimeError("HIP library %s is missing; run `python -m paper_1904_00962_amd.build` "
                           "(there is no CPU fallback)" % path)
    lib = ctypes.CDLL(path)
    i32, i64, f32, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p
    P = ctypes.POINTER
    lib.lamb_plan_create.argtypes = [P(lamb_tensor), i32, i32, i32, i32, P(vp)]
    lib.lamb_plan_destroy.argtypes = [vp]
    lib.lamb_plan_info.argtypes = [vp, P(i32), P(i32), P(i32)]
    lib.lamb_plan_set_bf16_copies.argtypes = [vp, P(vp)]
    lib.lamb_step.argtypes = [vp, f32, f32, f32, f32, f32, f32, f32, i64, i32, vp, vp, vp]
    lib.nlamb_step.argtypes = [vp, f32, f32, f32, f32, f32, f32, f32, i64, i32, vp, vp, vp]
    lib.lamb_hparams_init.argtypes = [P(lamb_hparams), i32]
    lib.lamb_lr_at.argtypes = [P(lamb_lr_stage), i32, i64, P(ctypes.c_double)]
    lib.lamb_sqrt_scaled_lr.argtypes = [ctypes.c_double, i64, i64, P(ctypes.c_double)]
    lib.lamb_step_ex.argtypes = [vp, P(lamb_hparams), vp, vp, vp, vp]
    lib.lars_step.argtypes = [vp, f32, f32, f32, f32, f32, f32, vp, vp, vp]
    lib.lamb_chunk_table.argtypes = [P(i64), i32, i32, i32, P(i32), P(i64), P(i32), P(i32)]
    lib.lamb_plan_set_timing.argtypes = [vp, i32, i32]
    lib.lamb_plan_timing.argtypes = [vp, P(ctypes.c_double), P(i64)]
    lib.lamb_plan_set_path.argtypes = [vp, i32]
    lib.lamb_plan_tiles.argtypes = [vp, P(i32), P(i32), P(i32), P(i64)]
    lib.lamb_plan_check.argtypes = [vp, vp]
    lib.lamb_tile_schedule.argtypes = [P(i64), i32, i32, i32, i32, P(i32), P(i64), P(i32),
                                       P(i32), P(i32), P(i32), P(i32), P(i32)]
    lib.lamb_step_partials.argtypes = [vp, P(lamb_hparams), vp, vp]
    lib.lamb_step_finish.argtypes = [vp, P(lamb_hparams), vp, vp, vp, vp, vp]
    lib.lamb_plan_set_u_check.argtypes = [vp, i32]
    lib.lamb_plan_set_trace.argtypes = [vp, vp]
    lib.lamb_plan_u_partials.argtypes = [vp, vp, i32, vp, vp, P(i32)]
    lib.lamb_step_static.argtypes = [P(lamb_tensor), i32, i32, i32, P(lamb_hparams), vp, vp, vp,
                                     vp]
    lib.lamb_status_str.argtypes = [i32]
    lib.lamb_status_str.restype = ctypes.c_char_p
    lib.lamb_last_error.argtypes = []
    lib.lamb_last_error.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name not in ("lamb_status_str", "lamb_last_error"):
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def status_str(status: int) -> str:
    return load().lamb_status_str(status).decode()


def last_error() -> str:
    return load().lamb_last_error().decode()


def _check(status: int, func: str) -> None:
    if status != LAMB_OK:
        raise LambError(status, func, last_error())


def _vp(p) -> ctypes.c_void_p:
    return ctypes.c_void_p(int(p) if p else 0)


class Plan:
    """Owning handle on a ``lamb_plan``; destroyed with :meth:`close` or on collection."""

    def __init__(self, handle: int):
        self.handle = handle

    def close(self) -> None:
        if self.handle:
            h, self.handle = self.handle, 0
            _check(load().lamb_plan_destroy(_vp(h)), "lamb_plan_destroy")

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def lamb_plan_create(tensors: Sequence[Tuple[int, int, int, int, int, int]], g_dtype: int,
                     algo: int, chunk_elems: int = 0) -> Plan:
    """tensors: (x_ptr, g_ptr, m_ptr, v_ptr, numel, wd) per block, device pointers."""
    lib = load()
    n = len(tensors)
    arr = (lamb_tensor * max(n, 1))()
    for i, (x, g, m, v, numel, wd) in enumerate(tensors):
        arr[i] = lamb_tensor(int(x) or None, int(g) or None, int(m) or None,
                             int(v) if v else None, int(numel), int(wd), 0)
    out = ctypes.c_void_p()
    _check(lib.lamb_plan_create(arr, n, int(g_dtype), int(algo), int(chunk_elems),
                                ctypes.byref(out)), "lamb_plan_create")
    return Plan(out.value)


def lamb_plan_destroy(plan: Plan) -> None:
    plan.close()


def lamb_plan_set_bf16_copies(plan: Plan, copies: Optional[Sequence[int]]) -> None:
    """Attach bf16 copies (device pointers, one per tensor, 0 for none) or
    detach all (None)."""
    if copies is None:
        arr = None
    else:
        arr = (ctypes.c_void_p * max(len(copies), 1))(*[int(c) or None for c in copies])
    _check(load().lamb_plan_set_bf16_copies(_vp(plan.handle), arr), "lamb_plan_set_bf16_copies")


def lamb_plan_info(plan: Plan) -> Tuple[int, int, int]:
    a, b, c = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    _check(load().lamb_plan_info(_vp(plan.handle), ctypes.byref(a), ctypes.byref(b),
                                 ctypes.byref(c)), "lamb_plan_info")
    return a.value, b.value, c.value


def lamb_hparams_init(variant="lamb", **fields) -> lamb_hparams:
    """The paper's defaults for ``variant`` (a name or LAMB_VARIANT_*), then
    ``fields`` set by name (``norm`` may be "l2", "l1" or "linf")."""
    hp = lamb_hparams()
    v = VARIANTS[variant] if isinstance(variant, str) else int(variant)
    _check(load().lamb_hparams_init(ctypes.byref(hp), v), "lamb_hparams_init")
    for k, val in fields.items():
        if k == "norm" and isinstance(val, str):
            val = NORMS[val]
        if not hasattr(hp, k):
            raise AttributeError("lamb_hparams has no field %r" % k)
        setattr(hp, k, val)
    return hp


def lamb_step_ex(plan: Plan, hp: lamb_hparams, stream: int = 0, ratio_out: int = 0,
                 norms_out: int = 0, nonfinite_out: int = 0) -> None:
    _check(load().lamb_step_ex(_vp(plan.handle), ctypes.byref(hp), _vp(stream), _vp(ratio_out),
                               _vp(norms_out), _vp(nonfinite_out)), "lamb_step_ex")


def lamb_step(plan: Plan, lr: float, beta1: float, beta2: float, eps: float,
              weight_decay: float, gamma_l: float, gamma_u: float, step: int,
              bias_correction: bool = True, stream: int = 0, ratio_out: int = 0,
              norms_out: int = 0) -> None:
    _check(load().lamb_step(_vp(plan.handle), lr, beta1, beta2, eps, weight_decay, gamma_l,
                            gamma_u, int(step), int(bool(bias_correction)), _vp(stream),
                            _vp(ratio_out), _vp(norms_out)), "lamb_step")


def nlamb_step(plan: Plan, lr: float, beta1: float, beta2: float, eps: float,
               weight_decay: float, gamma_l: float, gamma_u: float, step: int,
               nesterov_v: bool = False, stream: int = 0, ratio_out: int = 0,
               norms_out: int = 0) -> None:
    _check(load().nlamb_step(_vp(plan.handle), lr, beta1, beta2, eps, weight_decay, gamma_l,
                             gamma_u, int(step), int(bool(nesterov_v)), _vp(stream),
                             _vp(ratio_out), _vp(norms_out)), "nlamb_step")


def lars_step(plan: Plan, lr: float, momentum: float, weight_decay: float, gamma_l: float,
              gamma_u: float, trust_coef: float, stream: int = 0, ratio_out: int = 0,
              norms_out: int = 0) -> None:
    _check(load().lars_step(_vp(plan.handle), lr, momentum, weight_decay, gamma_l, gamma_u,
                            trust_coef, _vp(stream), _vp(ratio_out), _vp(norms_out)),
           "lars_step")


def lamb_chunk_table(numel: Sequence[int], chunk_elems: int = 0):
    """(tensor, start, len) arrays of the chunk table a plan would build."""
    lib = load()
    n = len(numel)
    sizes = np.ascontiguousarray(np.asarray(numel, dtype=np.int64))
    count = ctypes.c_int32()
    p64 = sizes.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)) if n else None
    _check(lib.lamb_chunk_table(p64, n, int(chunk_elems), 0, None, None, None,
                                ctypes.byref(count)), "lamb_chunk_table")
    k = count.value
    ct = np.zeros(k, np.int32)
    cs = np.zeros(k, np.int64)
    cl = np.zeros(k, np.int32)
    _check(lib.lamb_chunk_table(p64, n, int(chunk_elems), k,
                                ct.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                cs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                cl.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                ctypes.byref(count)), "lamb_chunk_table")
    return ct, cs, cl


def lamb_lr_at(stages: Sequence[Tuple[int, int, float, float]], step: int) -> float:
    """Learning rate at step ``step`` (>= 1) of back-to-back stages given as
    (steps, warmup_steps, peak_lr, power)."""
    arr = (lamb_lr_stage * max(len(stages), 1))(*[lamb_lr_stage(int(a), int(b), float(c), float(d))
                                                  for a, b, c, d in stages])
    out = ctypes.c_double()
    _check(load().lamb_lr_at(arr, len(stages), int(step), ctypes.byref(out)), "lamb_lr_at")
    return out.value


def lamb_sqrt_scaled_lr(base_lr: float, base_batch: int, batch: int) -> float:
    out = ctypes.c_double()
    _check(load().lamb_sqrt_scaled_lr(float(base_lr), int(base_batch), int(batch),
                                      ctypes.byref(out)), "lamb_sqrt_scaled_lr")
    return out.value


def lamb_plan_set_timing(plan: Plan, max_steps: int, every: int = 1) -> None:
    _check(load().lamb_plan_set_timing(_vp(plan.handle), int(max_steps), int(every)),
           "lamb_plan_set_timing")


def lamb_plan_timing(plan: Plan) -> Tuple[Tuple[float, float, float, float, float], int]:
    """Summed (moments, finalize, apply, single-pass, finiteness-check) kernel
    milliseconds and the step count."""
    ms = (ctypes.c_double * 5)()
    steps = ctypes.c_int64()
    _check(load().lamb_plan_timing(_vp(plan.handle), ms, ctypes.byref(steps)),
           "lamb_plan_timing")
    return tuple(ms[k] for k in range(5)), steps.value


def lamb_plan_set_path(plan: Plan, path="auto") -> None:
    """``path``: "auto" (single pass where a layer fits) or "two-pass"."""
    code = PATHS[path] if isinstance(path, str) else int(path)
    _check(load().lamb_plan_set_path(_vp(plan.handle), code), "lamb_plan_set_path")


def lamb_plan_tiles(plan: Plan, with_elems: bool = False):
    """(tiles per tensor on the single pass, total single-pass tiles, tile shape
    in float4 groups per thread: 8 or 10), and with ``with_elems`` also the
    elements of each tensor on the single pass (the rest of a layer larger
    than one round takes the two-pass kernels)."""
    n = lamb_plan_info(plan)[0]
    per = (ctypes.c_int32 * n)()
    elems = (ctypes.c_int64 * n)()
    total, groups = ctypes.c_int32(), ctypes.c_int32()
    _check(load().lamb_plan_tiles(_vp(plan.handle), per, ctypes.byref(total),
                                  ctypes.byref(groups), elems), "lamb_plan_tiles")
    if with_elems:
        return list(per), total.value, groups.value, list(elems)
    return list(per), total.value, groups.value


def lamb_tile_schedule(numel: Sequence[int], max_round: int, tile_groups: int = 0):
    """The single-pass schedule (host only): (entry_tensor, entry_start,
    entry_len, first_tile, tiles, round, groups) with lists for the first
    five; entry_tensor -1 marks an empty entry, ``round`` is the grid width,
    ``groups`` the tile shape (``tile_groups`` 0: a plan's choice)."""
    n = len(numel)
    arr = (ctypes.c_int64 * n)(*[int(v) for v in numel])
    first = (ctypes.c_int32 * n)()
    tiles = (ctypes.c_int32 * n)()
    count, width, groups = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    lib = load()
    _check(lib.lamb_tile_schedule(arr, n, int(max_round), int(tile_groups), 0, None, None, None,
                                  first, tiles, ctypes.byref(count), ctypes.byref(width),
                                  ctypes.byref(groups)), "lamb_tile_schedule")
    k = count.value
    et, es, el = (ctypes.c_int32 * k)(), (ctypes.c_int64 * k)(), (ctypes.c_int32 * k)()
    _check(lib.lamb_tile_schedule(arr, n, int(max_round), groups.value, k, et, es, el, first,
                                  tiles, ctypes.byref(count), ctypes.byref(width), None),
           "lamb_tile_schedule")
    return list(et), list(es), list(el), list(first), list(tiles), width.value, groups.value


def lamb_plan_check(plan: Plan, stream: int = 0) -> None:
    """Synchronise `stream`; raise LambError (LAMB_ESYNC) if a single-pass step
    of the plan abandoned a wait."""
    _check(load().lamb_plan_check(_vp(plan.handle), _vp(stream)), "lamb_plan_check")


def lamb_step_partials(plan: Plan, hp: lamb_hparams, stream: int = 0, totals: int = 0) -> None:
    """First half of a split step: the moment pass over the plan's blocks and
    each block's partial norms into ``totals`` (device, 2 n + 1 doubles)."""
    _check(load().lamb_step_partials(_vp(plan.handle), ctypes.byref(hp), _vp(stream),
                                     _vp(totals)), "lamb_step_partials")


def lamb_step_finish(plan: Plan, hp: lamb_hparams, stream: int = 0, totals: int = 0,
                     ratio_out: int = 0, norms_out: int = 0, nonfinite_out: int = 0) -> None:
    """Second half of a split step, from the shards' combined ``totals``."""
    _check(load().lamb_step_finish(_vp(plan.handle), ctypes.byref(hp), _vp(stream), _vp(totals),
                                   _vp(ratio_out), _vp(norms_out), _vp(nonfinite_out)),
           "lamb_step_finish")


def lamb_plan_set_u_check(plan: Plan, enable: bool) -> None:
    _check(load().lamb_plan_set_u_check(_vp(plan.handle), int(bool(enable))),
           "lamb_plan_set_u_check")


def lamb_plan_u_partials(plan: Plan, stream: int = 0):
    """(moment, apply) per-chunk partial norms of the last checked step, each
    an (n, 2) float64 array of {x, u} pairs (n = 0 when none was checked)."""
    lib = load()
    n = ctypes.c_int32()
    # the count first: capacity 0 fails with LAMB_EINVAL but still sets it
    status = lib.lamb_plan_u_partials(_vp(plan.handle), _vp(stream), 0, None, None,
                                      ctypes.byref(n))
    if status not in (LAMB_OK, LAMB_EINVAL):
        _check(status, "lamb_plan_u_partials")
    k = n.value
    moment = np.zeros((k, 2), np.float64)
    apply = np.zeros((k, 2), np.float64)
    if k:
        _check(lib.lamb_plan_u_partials(_vp(plan.handle), _vp(stream), k,
                                        ctypes.c_void_p(moment.ctypes.data),
                                        ctypes.c_void_p(apply.ctypes.data), ctypes.byref(n)),
               "lamb_plan_u_partials")
    return moment, apply


def lamb_step_static(tensors: Sequence[Tuple[int, int, int, int, int, int]], g_dtype: int,
                     hp: lamb_hparams, chunk_elems: int = 0, stream: int = 0, ratio_out: int = 0,
                     norms_out: int = 0, nonfinite_out: int = 0) -> None:
    """A step without a plan (the library's fixed device array holds its
    tables): tensors as for lamb_plan_create, (x, g, m, v, numel, wd) device
    pointers per block."""
    n = len(tensors)
    arr = (lamb_tensor * max(n, 1))()
    for i, (x, g, m, v, numel, wd) in enumerate(tensors):
        arr[i] = lamb_tensor(int(x) or None, int(g) or None, int(m) or None,
                             int(v) if v else None, int(numel), int(wd), 0)
    _check(load().lamb_step_static(arr, n, int(g_dtype), int(chunk_elems), ctypes.byref(hp),
                                   _vp(stream), _vp(ratio_out), _vp(norms_out),
                                   _vp(nonfinite_out)), "lamb_step_static")


def lamb_plan_set_trace(plan: Plan, trace: int = 0) -> None:
    """Per-tile clock stamps of later single-pass steps into ``trace`` (device
    pointer to 4 x n_tiles uint64), or off (0)."""
    _check(load().lamb_plan_set_trace(_vp(plan.handle), _vp(trace)), "lamb_plan_set_trace")
