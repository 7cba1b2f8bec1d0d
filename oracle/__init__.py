"""CPU oracle of the LAMB (Algorithm 2), N-LAMB / NN-LAMB (Algorithms 3 and
4) and LARS (Algorithm 1) steps.

TEST INFRASTRUCTURE ONLY: the test suite, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` are the only users. It imports nothing from
the HIP library package and shares no code with it. The arithmetic lives in
``lamb_oracle.c`` (plain C, double); this module only marshals numpy arrays.

Inputs are lists of per-tensor numpy arrays: x, m, v are float32 and updated
in place; g is float32, or uint16 holding bf16 bit patterns. Every step takes
``grad_scale`` (g_t = grad_scale * g), ``norm`` ("l2", "l1" or "linf", the
layer norm of Appendix F) and ``skip_nonfinite``: when set and any scaled
gradient element of any tensor is NaN or infinite, the step changes nothing
and returns NaN ratios and norms.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "lamb_oracle.c")
LIBRARY = os.path.join(HERE, "liblamb_oracle.so")

CFLAGS = ["-O2", "-std=c11", "-fno-fast-math", "-ffp-contract=off", "-fPIC", "-shared"]


def build(source: str = SOURCE, output: str = LIBRARY) -> str:
    """Compile the oracle with gcc (single-threaded, no fast-math, no FMA contraction)."""
    tmp = output + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", *CFLAGS, source, "-o", tmp, "-lm"])
    os.replace(tmp, output)
    return output


_DP = ctypes.POINTER(ctypes.c_double)
NORMS = {"l2": 0, "l1": 1, "linf": 2}


def _ptr(a: np.ndarray) -> ctypes.c_void_p:
    return ctypes.c_void_p(a.ctypes.data)


def _check_state(a: np.ndarray, n: int, what: str) -> None:
    if a.dtype != np.float32 or not a.flags.c_contiguous or not a.flags.writeable:
        raise TypeError("%s must be a writeable contiguous float32 array" % what)
    if a.size != n:
        raise ValueError("%s has %d elements, expected %d" % (what, a.size, n))


def _grad_kind(g: np.ndarray, n: int) -> int:
    if not g.flags.c_contiguous or g.size != n:
        raise ValueError("gradient must be contiguous with %d elements" % n)
    if g.dtype == np.float32:
        return 0
    if g.dtype == np.uint16:
        return 1
    raise TypeError("gradient dtype must be float32 or uint16 (bf16 bits)")


class Oracle:
    """Handle on one compiled oracle library (the default one, or a test variant)."""

    def __init__(self, path: str = LIBRARY):
        self.path = path
        lib = ctypes.CDLL(path)
        lib.oracle_lamb_layer.restype = ctypes.c_int
        lib.oracle_lamb_layer.argtypes = [
            ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
            ctypes.c_void_p, ctypes.c_void_p,
            ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_double,
            ctypes.c_double, ctypes.c_int, ctypes.c_double, ctypes.c_double,
            ctypes.c_int64, ctypes.c_int, ctypes.c_double, ctypes.c_int, _DP]
        lib.oracle_nlamb_layer.restype = ctypes.c_int
        lib.oracle_nlamb_layer.argtypes = [
            ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
            ctypes.c_void_p, ctypes.c_void_p,
            ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_double,
            ctypes.c_double, ctypes.c_int, ctypes.c_double, ctypes.c_double,
            ctypes.c_int64, ctypes.c_int, ctypes.c_double, ctypes.c_int, _DP]
        lib.oracle_lars_layer.restype = ctypes.c_int
        lib.oracle_lars_layer.argtypes = [
            ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
            ctypes.c_void_p, ctypes.c_double, ctypes.c_double, ctypes.c_double,
            ctypes.c_int, ctypes.c_double, ctypes.c_double, ctypes.c_double,
            ctypes.c_double, ctypes.c_int, _DP]
        lib.oracle_round_bf16.restype = None
        lib.oracle_round_bf16.argtypes = [ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
        lib.oracle_gradient_finite.restype = ctypes.c_int
        lib.oracle_gradient_finite.argtypes = [ctypes.c_int64, ctypes.c_void_p, ctypes.c_int,
                                               ctypes.c_double]
        self._lib = lib

    def gradients_finite(self, gs: Sequence[np.ndarray], grad_scale: float = 1.0) -> bool:
        """True unless some fp32(g_j) * fp32(grad_scale) of some tensor is NaN or infinite."""
        for g in gs:
            kind = _grad_kind(g, g.size)
            if not self._lib.oracle_gradient_finite(g.size, _ptr(g), kind, grad_scale):
                return False
        return True

    def round_bf16(self, x: np.ndarray) -> np.ndarray:
        """bf16 bit patterns (uint16) of fp32 ``x``, round to nearest even."""
        x = np.ascontiguousarray(x, dtype=np.float32)
        out = np.empty(x.size, dtype=np.uint16)
        self._lib.oracle_round_bf16(x.size, _ptr(x), _ptr(out))
        return out

    def _skipped(self, gs, grad_scale, skip_nonfinite):
        if skip_nonfinite and not self.gradients_finite(gs, grad_scale):
            return np.full((len(gs), 3), np.nan)
        return None

    def lamb_step(self, xs: Sequence[np.ndarray], gs: Sequence[np.ndarray],
                  ms: Sequence[np.ndarray], vs: Sequence[np.ndarray],
                  wd_mask: Sequence[bool], *, lr: float, beta1: float, beta2: float,
                  eps: float, weight_decay: float, gamma_l: float, gamma_u: float,
                  step: int, bias_correction: bool = True, grad_scale: float = 1.0,
                  norm: str = "l2", skip_nonfinite: bool = False) -> np.ndarray:
        """One LAMB step over every block; returns (n, 3) [ratio, ||x||, ||u||]."""
        skipped = self._skipped(gs, grad_scale, skip_nonfinite)
        if skipped is not None:
            return skipped
        n = len(xs)
        out = np.zeros((n, 3), dtype=np.float64)
        for i in range(n):
            d = xs[i].size
            _check_state(xs[i], d, "x[%d]" % i)
            _check_state(ms[i], d, "m[%d]" % i)
            _check_state(vs[i], d, "v[%d]" % i)
            kind = _grad_kind(gs[i], d)
            res = out[i]
            rc = self._lib.oracle_lamb_layer(
                d, _ptr(xs[i]), _ptr(gs[i]), kind, _ptr(ms[i]), _ptr(vs[i]),
                lr, beta1, beta2, eps, weight_decay, int(bool(wd_mask[i])),
                gamma_l, gamma_u, int(step), int(bool(bias_correction)), grad_scale,
                NORMS[norm], res.ctypes.data_as(_DP))
            if rc != 0:
                raise RuntimeError("oracle_lamb_layer failed on tensor %d (%d)" % (i, rc))
        return out

    def nlamb_step(self, xs: Sequence[np.ndarray], gs: Sequence[np.ndarray],
                   ms: Sequence[np.ndarray], vs: Sequence[np.ndarray],
                   wd_mask: Sequence[bool], *, lr: float, beta1: float, beta2: float,
                   eps: float, weight_decay: float, gamma_l: float, gamma_u: float,
                   step: int, nesterov_v: bool = False, grad_scale: float = 1.0,
                   norm: str = "l2", skip_nonfinite: bool = False) -> np.ndarray:
        """One N-LAMB (Algorithm 3) or NN-LAMB (Algorithm 4, nesterov_v) step;
        returns (n, 3) [ratio, ||x||, ||u||]."""
        skipped = self._skipped(gs, grad_scale, skip_nonfinite)
        if skipped is not None:
            return skipped
        n = len(xs)
        out = np.zeros((n, 3), dtype=np.float64)
        for i in range(n):
            d = xs[i].size
            _check_state(xs[i], d, "x[%d]" % i)
            _check_state(ms[i], d, "m[%d]" % i)
            _check_state(vs[i], d, "v[%d]" % i)
            kind = _grad_kind(gs[i], d)
            res = out[i]
            rc = self._lib.oracle_nlamb_layer(
                d, _ptr(xs[i]), _ptr(gs[i]), kind, _ptr(ms[i]), _ptr(vs[i]),
                lr, beta1, beta2, eps, weight_decay, int(bool(wd_mask[i])),
                gamma_l, gamma_u, int(step), int(bool(nesterov_v)), grad_scale,
                NORMS[norm], res.ctypes.data_as(_DP))
            if rc != 0:
                raise RuntimeError("oracle_nlamb_layer failed on tensor %d (%d)" % (i, rc))
        return out

    def lars_step(self, xs: Sequence[np.ndarray], gs: Sequence[np.ndarray],
                  ms: Sequence[np.ndarray], wd_mask: Sequence[bool], *, lr: float,
                  momentum: float, weight_decay: float, gamma_l: float, gamma_u: float,
                  trust_coef: float, grad_scale: float = 1.0, norm: str = "l2",
                  skip_nonfinite: bool = False) -> np.ndarray:
        """One LARS step over every block; returns (n, 3) [ratio, ||x||, ||m||]."""
        skipped = self._skipped(gs, grad_scale, skip_nonfinite)
        if skipped is not None:
            return skipped
        n = len(xs)
        out = np.zeros((n, 3), dtype=np.float64)
        for i in range(n):
            d = xs[i].size
            _check_state(xs[i], d, "x[%d]" % i)
            _check_state(ms[i], d, "m[%d]" % i)
            kind = _grad_kind(gs[i], d)
            res = out[i]
            rc = self._lib.oracle_lars_layer(
                d, _ptr(xs[i]), _ptr(gs[i]), kind, _ptr(ms[i]), lr, momentum,
                weight_decay, int(bool(wd_mask[i])), gamma_l, gamma_u, trust_coef,
                grad_scale, NORMS[norm], res.ctypes.data_as(_DP))
            if rc != 0:
                raise RuntimeError("oracle_lars_layer failed on tensor %d (%d)" % (i, rc))
        return out


_default: Optional[Oracle] = None


def load() -> Oracle:
    """The oracle built from ``lamb_oracle.c`` (compiled here first if missing or stale)."""
    global _default
    if _default is None:
        if (not os.path.exists(LIBRARY)
                or os.path.getmtime(LIBRARY) < os.path.getmtime(SOURCE)):
            build()
        _default = Oracle(LIBRARY)
    return _default
