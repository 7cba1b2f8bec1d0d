"""Run the HIP step and the CPU oracle side by side on identical inputs.

Comparison rule for fp32 state (x, m, v), per tensor and per step:
    err_j = |gpu_j - ref_j| / max(|ref_j|, rms(ref))
must stay <= 1e-5, where rms(ref) is the oracle's root-mean-square of that
quantity over the tensor. The RMS floor keeps the relative test meaningful
for elements that land near zero (a step of ~1e-5 moving x through 0 makes a
pure relative error ill-posed there). NaN positions must match exactly.
Trust ratios (and the norms behind them) must agree to 1e-6 relative, and be
exactly 0 wherever the oracle reports 0. For a tensor of a few elements the
update norm can rest on one element whose u cancels (m_hat a difference of
two terms, or r + lambda x with opposite signs); there the ratio tolerance
is raised to twice the first-order bound on the relative error that fp32
evaluation of u can reach (``update_norm_bound``), when that exceeds 1e-6.
"""

from __future__ import annotations

import dataclasses
import os
from typing import List, Optional, Sequence

import numpy as np
import pytest

import oracle
from paper_1904_00962_amd import _lib, paramsets

STATE_TOL = 1e-5
RATIO_TOL = 1e-6


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch


def log(msg: str) -> None:
    print(msg, flush=True)


@dataclasses.dataclass
class Report:
    max_err: float = 0.0
    max_abs: float = 0.0
    max_rel: float = 0.0
    n_rel_over: int = 0
    max_ratio: float = 0.0  # worst relative error of a trust ratio or norm

    def merge(self, other: "Report") -> None:
        self.max_err = max(self.max_err, other.max_err)
        self.max_abs = max(self.max_abs, other.max_abs)
        self.max_rel = max(self.max_rel, other.max_rel)
        self.n_rel_over += other.n_rel_over
        self.max_ratio = max(self.max_ratio, other.max_ratio)


def compare_state(gpu: np.ndarray, ref: np.ndarray, what: str, tol: float = STATE_TOL) -> Report:
    a = gpu.astype(np.float64)
    b = ref.astype(np.float64)
    nan_a, nan_b = np.isnan(a), np.isnan(b)
    if not np.array_equal(nan_a, nan_b):
        raise AssertionError("%s: NaN positions differ (%d vs %d)"
                             % (what, int(nan_a.sum()), int(nan_b.sum())))
    ok = ~nan_b
    a, b = a[ok], b[ok]
    if a.size == 0:
        return Report()
    inf_b = np.isinf(b)
    if np.any(inf_b):
        if not np.array_equal(a[inf_b], b[inf_b]):
            raise AssertionError("%s: infinite values differ" % what)
        a, b = a[~inf_b], b[~inf_b]
        if a.size == 0:
            return Report()
    rms = float(np.sqrt(np.mean(b * b)))
    floor = max(rms, np.finfo(np.float32).tiny)
    diff = np.abs(a - b)
    err = diff / np.maximum(np.abs(b), floor)
    with np.errstate(divide="ignore", invalid="ignore"):
        rel = np.where(b != 0, diff / np.abs(b), np.where(diff == 0, 0.0, np.inf))
    r = Report(float(err.max()), float(diff.max()), float(rel.max()), int((rel > tol).sum()))
    if r.max_err > tol:
        j = int(np.argmax(err))
        raise AssertionError("%s: error %.3e > %.1e at element %d (gpu %r, oracle %r, rms %.3e)"
                             % (what, r.max_err, tol, j, a[j], b[j], rms))
    return r


def compare_state_device(gpu, ref: np.ndarray, what: str, tol: float = STATE_TOL) -> Report:
    """compare_state with the arithmetic on the GPU (the oracle's values are
    uploaded): the same rule, fast enough for whole models."""
    import torch
    a = gpu.reshape(-1).double()
    b = torch.from_numpy(np.ascontiguousarray(ref).reshape(-1)).to(gpu.device).double()
    nan_a, nan_b = torch.isnan(a), torch.isnan(b)
    if not torch.equal(nan_a, nan_b):
        raise AssertionError("%s: NaN positions differ (%d vs %d)"
                             % (what, int(nan_a.sum()), int(nan_b.sum())))
    if bool(nan_b.any()):
        a, b = a[~nan_b], b[~nan_b]
    inf_b = torch.isinf(b)
    if bool(inf_b.any()):
        if not torch.equal(a[inf_b], b[inf_b]):
            raise AssertionError("%s: infinite values differ" % what)
        a, b = a[~inf_b], b[~inf_b]
    if a.numel() == 0:
        return Report()
    rms = float(torch.sqrt(torch.mean(b * b)))
    floor = max(rms, float(np.finfo(np.float32).tiny))
    diff = torch.abs(a - b)
    err = diff / torch.clamp(torch.abs(b), min=floor)
    rel = torch.where(b != 0, diff / torch.abs(b),
                      torch.where(diff == 0, torch.zeros_like(diff),
                                  torch.full_like(diff, float("inf"))))
    j = int(torch.argmax(err))
    r = Report(float(err[j]), float(diff.max()), float(rel.max()), int((rel > tol).sum()))
    if r.max_err > tol:
        raise AssertionError("%s: error %.3e > %.1e at element %d (gpu %r, oracle %r, rms %.3e)"
                             % (what, r.max_err, tol, j, float(a[j]), float(b[j]), rms))
    return r


def compare_ratios(gpu: np.ndarray, ref: np.ndarray, what: str, tol=RATIO_TOL) -> float:
    """Relative agreement per entry; ``tol`` is one bound or one per entry."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    tol = np.broadcast_to(np.asarray(tol, np.float64), ref.shape)
    if not np.array_equal(np.isnan(gpu), np.isnan(ref)):
        raise AssertionError("%s: NaN positions differ" % what)
    ok = ~np.isnan(ref)
    g, r, t = gpu[ok], ref[ok], tol[ok]
    zero = r == 0
    if not np.all(g[zero] == 0):
        raise AssertionError("%s: GPU reports a nonzero value where the oracle has 0" % what)
    if np.any(~zero):
        rel = np.abs(g[~zero] - r[~zero]) / np.abs(r[~zero])
        over = rel / t[~zero]
        k = int(np.argmax(over))
        if over[k] > 1.0:
            raise AssertionError("%s: relative error %.3e > %.1e (gpu %r, oracle %r)"
                                 % (what, rel[k], t[~zero][k], g[~zero][k], r[~zero][k]))
        return float(rel.max())
    return 0.0


EPS32 = 2.0 ** -24  # unit roundoff of fp32 round-to-nearest


def _widen(g: np.ndarray) -> np.ndarray:
    if g.dtype == np.uint16:
        return (g.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return g.astype(np.float64)


def update_norm_bound(variant: int, x, g, m, v, wd: bool, *, beta1: float, beta2: float = 0.0,
                      eps: float = 0.0, weight_decay: float = 0.0, step: int = 1,
                      bias_correction: bool = True, grad_scale: float = 1.0,
                      norm: int = 0) -> float:
    """First-order bound on the relative error of ||u|| (||m_t|| for LARS)
    when u is evaluated in fp32 from the fp32 state, as the kernels do, against
    its exact value (the oracle's double), where the state entering the step
    may differ from the oracle's by up to two ulps in x, m and v (it was
    rounded along another path). Per element, a running error bound over the
    formula's roundings, each term counted by its magnitude (eps = 2^-24):
      moments  m_t = b1 m + (1 - b1) g: error <= 5 eps A_m, A_m = |b1 m| + |(1 - b1) g|
      m_hat    c m_t, or a m_t + b g (Nesterov): error <= 8 eps A_hat with
               A_hat = |c| A_m, or |a| A_m + |b g|
      v_hat    a sum of non-negative terms: relative error <= 12 eps, so
               d = sqrt(v_hat) + eps has relative error <= 8 eps
      r        m_hat / d: error <= 8 eps A_hat / d + 9 eps |r|
      u        r + lambda x: error <= err(r) + 3 eps |lambda x| + eps |u|
      LARS     m_t = b1 m + (1 - b1)(g + lambda x): error <= 6 eps A
    then, with err_j those bounds, the first-order error of the norm: L2
    sum u_j du_j / sum u_j^2, L1 sum sign(u_j) du_j / sum |u_j|, L-infinity
    at most max err_j / max |u_j|. For L2 and L1 the sum is bounded twice: in
    the worst case (every |du_j| = err_j, signs aligned), and with err_j split
    into the part every element shares (the fp32 roundings of the step's
    coefficients: 2 eps A_hat / d + 2 eps |r|, or eps A for LARS), summed in
    full, and the rest, independent roundings per element, bounded by
    |sum c_j du_j| <= 6 sqrt(sum c_j^2 err_j^2) (Hoeffding's inequality with
    lambda = 6, failure probability below 3e-8, as in Higham and Mary's
    probabilistic rounding-error analysis, 2019); the bound is the smaller. A
    tensor of a few elements gets the worst case, a large one the
    probabilistic bound, far below 1e-6. Inputs are the state before the step
    (numpy arrays, g as fp32 or bf16 bits)."""
    x = np.asarray(x, np.float64)
    m = np.asarray(m, np.float64)
    gs = grad_scale * _widen(np.asarray(g))
    lam = weight_decay if wd else 0.0
    b1, b2, t = float(beta1), float(beta2), int(step)
    if variant == _lib.LAMB_VARIANT_LARS:
        u = b1 * m + (1.0 - b1) * (gs + lam * x)
        a_all = np.abs(b1 * m) + (1.0 - b1) * (np.abs(gs) + np.abs(lam * x))
        err = 6.0 * EPS32 * a_all
        shared = EPS32 * a_all
    else:
        v = np.asarray(v, np.float64)
        mt = b1 * m + (1.0 - b1) * gs
        a_m = np.abs(b1 * m) + np.abs((1.0 - b1) * gs)
        vt = b2 * v + (1.0 - b2) * gs * gs
        if variant == _lib.LAMB_VARIANT_LAMB:
            c1 = 1.0 - b1 ** t if bias_correction else 1.0
            c2 = 1.0 - b2 ** t if bias_correction else 1.0
            mh, a_h, vh = mt / c1, a_m / c1, vt / c2
        else:
            a, b = b1 / (1.0 - b1 ** (t + 1)), (1.0 - b1) / (1.0 - b1 ** t)
            mh, a_h = a * mt + b * gs, abs(a) * a_m + np.abs(b * gs)
            if variant == _lib.LAMB_VARIANT_NNLAMB:
                vh = b2 * vt / (1.0 - b2 ** (t + 1)) + (1.0 - b2) * gs * gs / (1.0 - b2 ** t)
            else:
                vh = b2 * vt / (1.0 - b2 ** t)
        d = np.sqrt(vh) + eps
        r = mh / d
        u = r + lam * x
        err = EPS32 * (8.0 * a_h / d + 9.0 * np.abs(r) + 3.0 * np.abs(lam * x) + np.abs(u))
        shared = EPS32 * (2.0 * a_h / d + 2.0 * np.abs(r))
    au = np.abs(u)
    if norm == _lib.LAMB_NORM_LINF:
        den = float(au.max())
        return float(err.max()) / den if den > 0 else 0.0
    own = err - shared
    if norm == _lib.LAMB_NORM_L1:
        den = float(au.sum())
        worst = float(err.sum())
        prob = float(shared.sum()) + 6.0 * float(np.sqrt(np.sum(own * own)))
    else:
        den = float(np.sum(au * au))
        worst = float(np.sum(au * err))
        prob = float(np.sum(au * shared)) + 6.0 * float(np.sqrt(np.sum((au * own) ** 2)))
    return min(worst, prob) / den if den > 0 else 0.0


# Environment variable a plan reads for its single-pass tile shape (8 or 10).
TILE_ENV = "LAMB_MI355X_TILE_GROUPS"


def create_plan(rows, g_dtype: int, algo: int, chunk_elems: int, path: str) -> "_lib.Plan":
    """A plan on ``path``: "auto", "two-pass", or "wide", the single pass with
    10-group tiles, forced through the environment override so that small
    layers exercise that kernel."""
    wide = path == "wide"
    saved = os.environ.get(TILE_ENV)
    if wide:
        os.environ[TILE_ENV] = "10"
    try:
        plan = _lib.lamb_plan_create(rows, g_dtype, algo, chunk_elems)
    finally:
        if wide:
            if saved is None:
                del os.environ[TILE_ENV]
            else:
                os.environ[TILE_ENV] = saved
    _lib.lamb_plan_set_path(plan, "auto" if wide else path)
    if wide:
        assert _lib.lamb_plan_tiles(plan)[2] == 10
    return plan


class Pair:
    """Device state + plan for the HIP path, and host state for the oracle."""

    def __init__(self, xs: Sequence, wd: Sequence[bool], g_dtype: str, algo: str,
                 chunk_elems: int = 0, oracle_subset: Optional[Sequence[int]] = None,
                 path: str = "auto"):
        torch = torch_cuda()
        self.torch = torch
        self.algo = algo
        self.n = len(xs)
        self.wd = [bool(w) for w in wd]
        dev = torch.device("cuda")
        gt = torch.bfloat16 if g_dtype == "bf16" else torch.float32
        self.X = [torch.as_tensor(x).to(dev, torch.float32).contiguous() for x in xs]
        self.G = [torch.zeros(x.numel(), dtype=gt, device=dev) for x in self.X]
        self.M = [torch.zeros_like(x) for x in self.X]
        self.V = [torch.zeros_like(x) for x in self.X] if algo != "lars" else None
        self.subset = list(range(self.n)) if oracle_subset is None else list(oracle_subset)
        self.hx = [paramsets.host_array(self.X[i]).copy() for i in self.subset]
        self.hm = [np.zeros(self.X[i].numel(), np.float32) for i in self.subset]
        self.hv = [np.zeros(self.X[i].numel(), np.float32) for i in self.subset]
        self.ratio = torch.zeros(self.n, dtype=torch.float64, device=dev)
        self.norms = torch.zeros(2 * self.n, dtype=torch.float64, device=dev)
        rows = [(self.X[i].data_ptr(), self.G[i].data_ptr(), self.M[i].data_ptr(),
                 self.V[i].data_ptr() if self.V is not None else 0, self.X[i].numel(),
                 int(self.wd[i])) for i in range(self.n)]
        kind = _lib.LAMB_GRAD_BF16 if g_dtype == "bf16" else _lib.LAMB_GRAD_F32
        algo_id = _lib.LAMB_ALGO_LARS if algo == "lars" else _lib.LAMB_ALGO_LAMB
        self.plan = create_plan(rows, kind, algo_id, chunk_elems, path)
        self.path = path
        self.oracle = oracle.load()

    def set_grads(self, grads: Sequence) -> List[np.ndarray]:
        for G, g in zip(self.G, grads):
            G.copy_(self.torch.as_tensor(g).reshape(-1).to(G.device))
        return [paramsets.host_array(self.G[i]).copy() for i in self.subset]

    def gpu_lamb(self, hp: dict, step: int, bias_correction: bool = True) -> None:
        _lib.lamb_step(self.plan, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"],
                       hp["weight_decay"], hp["gamma_l"], hp["gamma_u"], step, bias_correction,
                       self.torch.cuda.current_stream().cuda_stream, self.ratio.data_ptr(),
                       self.norms.data_ptr())

    def gpu_nlamb(self, hp: dict, step: int, nesterov_v: bool) -> None:
        _lib.nlamb_step(self.plan, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"],
                        hp["weight_decay"], hp["gamma_l"], hp["gamma_u"], step, nesterov_v,
                        self.torch.cuda.current_stream().cuda_stream, self.ratio.data_ptr(),
                        self.norms.data_ptr())

    def gpu_lars(self, hp: dict) -> None:
        _lib.lars_step(self.plan, hp["lr"], hp["momentum"], hp["weight_decay"], hp["gamma_l"],
                       hp["gamma_u"], hp["trust_coef"],
                       self.torch.cuda.current_stream().cuda_stream, self.ratio.data_ptr(),
                       self.norms.data_ptr())

    def oracle_lamb(self, hg, hp: dict, step: int, bias_correction: bool = True) -> np.ndarray:
        return self.oracle.lamb_step(self.hx, hg, self.hm, self.hv,
                                     [self.wd[i] for i in self.subset], step=step,
                                     bias_correction=bias_correction, **f32_scalars(hp))

    def oracle_nlamb(self, hg, hp: dict, step: int, nesterov_v: bool) -> np.ndarray:
        return self.oracle.nlamb_step(self.hx, hg, self.hm, self.hv,
                                      [self.wd[i] for i in self.subset], step=step,
                                      nesterov_v=nesterov_v, **f32_scalars(hp))

    def oracle_lars(self, hg, hp: dict) -> np.ndarray:
        return self.oracle.lars_step(self.hx, hg, self.hm, [self.wd[i] for i in self.subset],
                                     **f32_scalars(hp))

    def compare(self, ref: np.ndarray, label: str, ratio_tol=RATIO_TOL) -> Report:
        """Element-wise state and per-tensor ratio/norm comparison for the subset
        (ratios and norms only when the oracle did not skip the step). First
        checks that no single-pass wait of the plan was abandoned.
        ratio_tol: one bound, or one per tensor of the subset (for the trust
        ratio and ||u||; ||x|| is always held to RATIO_TOL)."""
        _lib.lamb_plan_check(self.plan, self.torch.cuda.current_stream().cuda_stream)
        self.torch.cuda.synchronize()
        rep = Report()
        ratio = self.ratio.cpu().numpy()
        norms = self.norms.cpu().numpy().reshape(-1, 2)
        for k, i in enumerate(self.subset):
            rep.merge(compare_state_device(self.X[i], self.hx[k], "%s x[%d]" % (label, i)))
            rep.merge(compare_state_device(self.M[i], self.hm[k], "%s m[%d]" % (label, i)))
            if self.V is not None:
                rep.merge(compare_state_device(self.V[i], self.hv[k], "%s v[%d]" % (label, i)))
        idx = np.asarray(self.subset, dtype=np.int64)
        if idx.size == 0 or np.all(np.isnan(ref)):
            return rep
        rep.max_ratio = max(
            compare_ratios(ratio[idx], ref[:, 0], label + " trust ratio", ratio_tol),
            compare_ratios(norms[idx, 0], ref[:, 1], label + " ||x||", RATIO_TOL),
            compare_ratios(norms[idx, 1], ref[:, 2], label + " ||u||", ratio_tol))
        return rep

    def ratio_tolerances(self, hp, hg) -> np.ndarray:
        """Per-tensor ratio tolerance of a step with hyperparameters ``hp`` (an
        ``_lib.lamb_hparams``) on the current host state (call before the
        oracle step): max(RATIO_TOL, 2 update_norm_bound)."""
        out = np.full(len(self.subset), RATIO_TOL)
        for k, i in enumerate(self.subset):
            with np.errstate(invalid="ignore", over="ignore"):  # a planted NaN or inf
                bound = update_norm_bound(
                    hp.variant, self.hx[k], hg[k], self.hm[k],
                    self.hv[k] if self.V is not None else None, self.wd[i], beta1=hp.beta1,
                    beta2=hp.beta2, eps=hp.eps, weight_decay=hp.weight_decay, step=hp.step,
                    bias_correction=bool(hp.bias_correction), grad_scale=hp.grad_scale,
                    norm=hp.norm)
            out[k] = max(RATIO_TOL, 2.0 * bound)
        return out

    def close(self) -> None:
        self.plan.close()


SCALAR_KEYS = ("lr", "beta1", "beta2", "eps", "weight_decay", "gamma_l", "gamma_u", "momentum",
               "trust_coef")


def f32_scalars(hp: dict) -> dict:
    """The oracle takes the same fp32-rounded scalars the C ABI receives."""
    out = {}
    for k, v in hp.items():
        out[k] = float(np.float32(v)) if k in SCALAR_KEYS else v
    return out


def lamb_hp(ps: paramsets.ParamSet) -> dict:
    return dict(lr=ps.lr, beta1=ps.beta1, beta2=ps.beta2, eps=ps.eps,
                weight_decay=ps.weight_decay, gamma_l=ps.gamma_l, gamma_u=ps.gamma_u)


def nlamb_hp(ps: paramsets.ParamSet) -> dict:
    """N-LAMB / NN-LAMB settings of Appendix D (beta1 0.975, beta2 0.999, eps 1e-8)."""
    return dict(lamb_hp(ps), beta1=0.975, beta2=0.999, eps=1e-8)


def lars_hp(ps: paramsets.ParamSet) -> dict:
    return dict(lr=ps.lars_lr, momentum=ps.lars_momentum, weight_decay=ps.weight_decay,
                gamma_l=ps.gamma_l, gamma_u=ps.gamma_u, trust_coef=ps.lars_trust_coef)


NORM_NAMES = {0: "l2", 1: "l1", 2: "linf"}


def step_ex_both(pair: Pair, hp, hg, nonfinite=None):
    """One ``lamb_step_ex`` with hyperparameters ``hp`` (an ``_lib.lamb_hparams``,
    fp32 fields) on the GPU and the matching oracle step; returns the oracle's
    per-tensor [ratio, ||x||, ||u||] (NaN rows when it skipped the step)."""
    _lib.lamb_step_ex(pair.plan, hp, pair.torch.cuda.current_stream().cuda_stream,
                      pair.ratio.data_ptr(), pair.norms.data_ptr(),
                      nonfinite.data_ptr() if nonfinite is not None else 0)
    return step_ex_both_oracle(pair, hp, hg)


def step_ex_both_oracle(pair: Pair, hp, hg):
    """The oracle's half of step_ex_both: the step with hyperparameters ``hp``
    on the pair's host state; returns [ratio, ||x||, ||u||] per tensor."""
    wd = [pair.wd[i] for i in pair.subset]
    common = dict(lr=hp.lr, weight_decay=hp.weight_decay, gamma_l=hp.gamma_l,
                  gamma_u=hp.gamma_u, grad_scale=hp.grad_scale, norm=NORM_NAMES[hp.norm],
                  skip_nonfinite=bool(hp.skip_nonfinite))
    o = pair.oracle
    if hp.variant == _lib.LAMB_VARIANT_LAMB:
        return o.lamb_step(pair.hx, hg, pair.hm, pair.hv, wd, beta1=hp.beta1, beta2=hp.beta2,
                           eps=hp.eps, step=hp.step, bias_correction=bool(hp.bias_correction),
                           **common)
    if hp.variant in (_lib.LAMB_VARIANT_NLAMB, _lib.LAMB_VARIANT_NNLAMB):
        return o.nlamb_step(pair.hx, hg, pair.hm, pair.hv, wd, beta1=hp.beta1, beta2=hp.beta2,
                            eps=hp.eps, step=hp.step,
                            nesterov_v=hp.variant == _lib.LAMB_VARIANT_NNLAMB, **common)
    return o.lars_step(pair.hx, hg, pair.hm, wd, momentum=hp.beta1, trust_coef=hp.trust_coef,
                       **common)


def step_both(pair: Pair, algo: str, hg, hp: dict, t: int, bias_correction: bool = True):
    """One step of ``algo`` on the GPU and in the oracle; returns the oracle's
    per-tensor [ratio, ||x||, ||u||]."""
    if algo == "lamb":
        pair.gpu_lamb(hp, t, bias_correction)
        return pair.oracle_lamb(hg, hp, t, bias_correction)
    if algo in ("nlamb", "nnlamb"):
        pair.gpu_nlamb(hp, t, algo == "nnlamb")
        return pair.oracle_nlamb(hg, hp, t, algo == "nnlamb")
    pair.gpu_lars(hp)
    return pair.oracle_lars(hg, hp)


def run_config(cfg: int, steps: int, algo: str = "lamb", chunk_elems: int = 0,
               device: str = "cuda", oracle_subset: Optional[Sequence[int]] = None,
               path: str = "auto") -> Report:
    """Parity over ``steps`` steps of a named parameter set, compared every step."""
    ps = paramsets.get(cfg)
    log("parity cfg=%d (%s) algo=%s steps=%d chunk=%d path=%s"
        % (cfg, ps.name, algo, steps, chunk_elems, path))
    pair = Pair(paramsets.draw_params(ps, device=device), ps.wd_mask(), ps.g_dtype, algo,
                chunk_elems, oracle_subset, path)
    per, total, groups, elems = _lib.lamb_plan_tiles(pair.plan, True)
    whole = sum(1 for e, x in zip(elems, pair.X) if e == x.numel())
    log("  single-pass layers %d whole, %d split, of %d; %d tiles of %d groups"
        % (whole, len(per) - whole, len(per), total, groups))
    rep = Report()
    hp = {"lamb": lamb_hp, "lars": lars_hp, "nlamb": nlamb_hp, "nnlamb": nlamb_hp}[algo](ps)
    try:
        for t in range(1, steps + 1):
            hg = pair.set_grads(paramsets.draw_grads(ps, t, device=device))
            ref = step_both(pair, algo, hg, hp, t)
            r = pair.compare(ref, "cfg%d %s step %d" % (cfg, algo, t))
            log("  step %d: max err %.3e, max abs %.3e, max rel %.3e, rel>1e-5: %d, "
                "ratio/norm rel %.3e" % (t, r.max_err, r.max_abs, r.max_rel, r.n_rel_over,
                                         r.max_ratio))
            rep.merge(r)
    finally:
        pair.close()
    return rep
