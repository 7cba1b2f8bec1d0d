"""LAMB and LARS optimizers over lists of torch tensors on an MI355X.

PyTorch supplies device memory and the current stream only; the step itself
is the HIP library (``_lib``). The plan binds the buffers' addresses, so
parameters and gradients must be persistent, contiguous device tensors: write
each step's gradient into the same ``grads`` tensors (e.g. ``g.copy_(...)``).

Defaults follow the paper: beta1 = 0.9, beta2 = 0.999, eps = 1e-6,
lambda = 0.01 (Section 4 and Appendix H); phi clamps to [0, 10].

Failure handling. A single-pass step that gives up a wait (its layer's tiles
were not all resident) leaves the plan inert: no later step moves anything.
The optimizer reads the plan's fault word every ``check_every`` steps and in
``state_dict()`` and raises ``LambError`` (status LAMB_ESYNC) once it is set.
Recover by restoring x, m and v from a checkpoint (``load_state_dict``) and
calling ``rebuild()``, on ``path="two-pass"`` if the device cannot be given to
the single pass alone.

Step count. ``t`` counts the steps that ran: with ``skip_nonfinite``, a step
skipped for a non-finite gradient does not advance it (nor the bias correction
or the learning-rate schedule). The verdict of a step is read, through pinned
host memory, when the next step starts (or when ``t`` is read), waiting only
for the optimizer's own previous step.
"""

from __future__ import annotations

from typing import Optional, Sequence, Tuple

from . import _lib


def _torch():
    import torch
    return torch


def _check_tensors(params, grads):
    torch = _torch()
    if len(params) == 0 or len(params) != len(grads):
        raise ValueError("need one gradient per parameter tensor (got %d and %d)"
                         % (len(params), len(grads)))
    g_dtype = grads[0].dtype
    if g_dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("gradients must be float32 or bfloat16")
    device = params[0].device
    if device.type != "cuda":
        raise ValueError("parameters must live on a GPU")
    for i, (p, g) in enumerate(zip(params, grads)):
        if p.dtype != torch.float32:
            raise TypeError("parameter %d is %s; the step keeps fp32 master weights" % (i, p.dtype))
        if g.dtype != g_dtype:
            raise TypeError("all gradients must share one dtype")
        if p.device != device or g.device != device:
            raise ValueError("tensor %d is on another device" % i)
        if not p.is_contiguous() or not g.is_contiguous():
            raise ValueError("tensor %d is not contiguous" % i)
        if p.numel() != g.numel() or p.numel() == 0:
            raise ValueError("tensor %d: parameter and gradient sizes differ or are empty" % i)
    return g_dtype, device


def _check_state(state, buffers) -> None:
    """A saved state must hold one tensor of the right size per parameter for
    every buffer, and a step count >= 0."""
    if int(state["step"]) < 0:
        raise ValueError("step must be >= 0")
    for name, dst in buffers.items():
        src = state[name]
        if len(src) != len(dst):
            raise ValueError("state %r has %d tensors, the optimizer %d" % (name, len(src), len(dst)))
        for i, (d, t) in enumerate(zip(dst, src)):
            if t.numel() != d.numel():
                raise ValueError("state %r tensor %d has %d elements, need %d"
                                 % (name, i, t.numel(), d.numel()))


class _LayerwiseOptimizer:
    algo = _lib.LAMB_ALGO_LAMB

    def __init__(self, params: Sequence, grads: Sequence, lr: float, weight_decay: float,
                 clamp: Tuple[float, float], wd_mask: Optional[Sequence[bool]],
                 chunk_elems: int, with_v: bool, norm: str = "l2", grad_scale: float = 1.0,
                 skip_nonfinite: bool = False, schedule=None, path: str = "auto",
                 check_every: int = 100):
        torch = _torch()
        if path not in _lib.PATHS:
            raise ValueError("path must be one of %s" % (tuple(_lib.PATHS),))
        if int(check_every) < 0:
            raise ValueError("check_every must be >= 0 (0: never)")
        self.check_every = int(check_every)
        self.params = list(params)
        self.grads = list(grads)
        g_dtype, self.device = _check_tensors(self.params, self.grads)
        self.lr = float(lr)
        self.weight_decay = float(weight_decay)
        self.gamma_l, self.gamma_u = float(clamp[0]), float(clamp[1])
        if wd_mask is None:
            wd_mask = [p.dim() > 1 for p in self.params]
        self.wd_mask = [bool(w) for w in wd_mask]
        if len(self.wd_mask) != len(self.params):
            raise ValueError("wd_mask needs one entry per tensor")
        self.m = [torch.zeros_like(p) for p in self.params]
        self.v = [torch.zeros_like(p) for p in self.params] if with_v else None
        n = len(self.params)
        self.ratios = torch.zeros(n, dtype=torch.float64, device=self.device)
        self.norms = torch.zeros(2 * n, dtype=torch.float64, device=self.device)
        if norm not in _lib.NORMS:
            raise ValueError("norm must be one of %s" % (tuple(_lib.NORMS),))
        self.norm = norm
        self.grad_scale = float(grad_scale)
        self.skip_nonfinite = bool(skip_nonfinite)
        # 1 after a step skipped for a non-finite gradient (device int32)
        self.found_nonfinite = torch.zeros(1, dtype=torch.int32, device=self.device)
        self.bf16_copies = None
        # (steps, warmup_steps, peak_lr, power) stages: the lr of step t comes
        # from lamb_lr_at (Section 4) unless step() is given one
        self.schedule = [tuple(s) for s in schedule] if schedule else None
        self._g_kind = _lib.LAMB_GRAD_BF16 if g_dtype == torch.bfloat16 else _lib.LAMB_GRAD_F32
        self._chunk_elems = int(chunk_elems)
        self.plan = None
        self.path = path
        self._build_plan()
        self._t = 0
        self._launched = 0
        # The last step's skip verdict, copied to pinned host memory behind an
        # event; resolved before the next step picks its t.
        self._verdict_host = (torch.zeros(1, dtype=torch.int32, pin_memory=True)
                              if self.skip_nonfinite else None)
        self._verdict_event = None

    def _build_plan(self) -> None:
        torch = _torch()
        rows = []
        for i, (p, g) in enumerate(zip(self.params, self.grads)):
            v = self.v[i].data_ptr() if self.v is not None else 0
            rows.append((p.data_ptr(), g.data_ptr(), self.m[i].data_ptr(), v, p.numel(),
                         int(self.wd_mask[i])))
        with torch.cuda.device(self.device):
            plan = _lib.lamb_plan_create(rows, self._g_kind, self.algo, self._chunk_elems)
        _lib.lamb_plan_set_path(plan, self.path)
        if self.bf16_copies is not None:
            _lib.lamb_plan_set_bf16_copies(plan, [c.data_ptr() if c is not None else 0
                                                  for c in self.bf16_copies])
        old, self.plan = self.plan, plan
        if old is not None:
            old.close()

    def rebuild(self, path: Optional[str] = None) -> None:
        """Replace the plan by a new one over the same buffers (after a give-up,
        once the state is restored); ``path`` optionally switches the path."""
        if path is not None:
            if path not in _lib.PATHS:
                raise ValueError("path must be one of %s" % (tuple(_lib.PATHS),))
            self.path = path
        _torch().cuda.synchronize(self.device)
        self._build_plan()

    @property
    def t(self) -> int:
        """Steps that ran (a skipped step does not count)."""
        self._resolve_verdict()
        return self._t

    def _resolve_verdict(self) -> None:
        if self._verdict_event is not None:
            self._verdict_event.synchronize()
            self._verdict_event = None
            if int(self._verdict_host[0]) != 0:
                self._t -= 1

    def _next_t(self) -> int:
        """t of the step about to run: one past the steps that ran."""
        self._resolve_verdict()
        self._t += 1
        return self._t

    def _stream(self) -> int:
        return _torch().cuda.current_stream(self.device).cuda_stream

    def _lr(self, lr: Optional[float], t: int) -> float:
        if lr is not None:
            return float(lr)
        if self.schedule:
            return _lib.lamb_lr_at(self.schedule, t)
        return self.lr

    def _run(self, hp) -> None:
        torch = _torch()
        hp.norm = _lib.NORMS[self.norm]
        hp.skip_nonfinite = int(self.skip_nonfinite)
        stream = self._stream()
        _lib.lamb_step_ex(self.plan, hp, stream, self.ratios.data_ptr(), self.norms.data_ptr(),
                          self.found_nonfinite.data_ptr() if self.skip_nonfinite else 0)
        if self.skip_nonfinite:
            self._verdict_host.copy_(self.found_nonfinite, non_blocking=True)
            self._verdict_event = torch.cuda.Event()
            self._verdict_event.record(torch.cuda.current_stream(self.device))
        self._launched += 1
        if self.check_every and self._launched % self.check_every == 0:
            self.check()

    def attach_bf16_copies(self, copies="allocate"):
        """Have every later step also write bf16(x) (round to nearest even) into
        ``copies``: one contiguous bf16 tensor per parameter with the same
        numel, or "allocate" to create them, or None to detach. Returns the
        attached list (``self.bf16_copies``)."""
        torch = _torch()
        if copies is None:
            _lib.lamb_plan_set_bf16_copies(self.plan, None)
            self.bf16_copies = None
            return None
        if isinstance(copies, str) and copies == "allocate":
            copies = [torch.empty(p.numel(), dtype=torch.bfloat16, device=self.device)
                      for p in self.params]
        copies = list(copies)
        if len(copies) != len(self.params):
            raise ValueError("need one copy per parameter tensor")
        for i, (c, p) in enumerate(zip(copies, self.params)):
            if c is None:
                continue
            if c.dtype != torch.bfloat16 or c.device != self.device or not c.is_contiguous():
                raise TypeError("copy %d must be a contiguous bf16 tensor on %s" % (i, self.device))
            if c.numel() != p.numel():
                raise ValueError("copy %d has %d elements, parameter %d" % (i, c.numel(), p.numel()))
        _lib.lamb_plan_set_bf16_copies(self.plan, [c.data_ptr() if c is not None else 0
                                                   for c in copies])
        self.bf16_copies = copies
        return copies

    def check(self) -> None:
        """Wait for the current stream and raise ``LambError`` (LAMB_ESYNC) if a
        single-pass step gave up a wait: the plan is then inert. Restore the
        state from a checkpoint and call ``rebuild()``."""
        _lib.lamb_plan_check(self.plan, self._stream())

    def close(self) -> None:
        self.plan.close()


class LAMB(_LayerwiseOptimizer):
    """Algorithm 2: Adam moments with bias correction, then a per-layer trust ratio."""

    algo = _lib.LAMB_ALGO_LAMB

    VARIANTS = ("lamb", "n-lamb", "nn-lamb")

    def __init__(self, params, grads, lr: float = 1e-3, betas=(0.9, 0.999), eps: float = 1e-6,
                 weight_decay: float = 0.01, clamp=(0.0, 10.0), wd_mask=None,
                 bias_correction: bool = True, chunk_elems: int = 0, variant: str = "lamb",
                 norm: str = "l2", grad_scale: float = 1.0, skip_nonfinite: bool = False,
                 schedule=None, path: str = "auto", check_every: int = 100):
        """``variant``: "lamb" (Algorithm 2), "n-lamb" (Algorithm 3) or "nn-lamb"
        (Algorithm 4; the paper pairs both with betas=(0.975, 0.999), eps=1e-8).
        ``norm``: "l2" (default), "l1" or "linf" (Appendix F). ``grad_scale``
        multiplies every gradient element (e.g. 1/N for a summed gradient, or a
        loss-scale inverse). ``skip_nonfinite``: a step whose scaled gradient
        holds a NaN or infinity changes nothing and sets ``found_nonfinite``.
        ``schedule``: stages (steps, warmup_steps, peak_lr, power) that set the
        learning rate of each step (warmup, then polynomial decay, Section 4).
        ``path``: "auto" (layers of up to 8.4M elements, or 10.5M where the
        plan takes the wider tile, take the single-pass kernel) or
        "two-pass". ``check_every``: read the plan's fault word every that many
        steps (0: only in ``check()`` and ``state_dict()``)."""
        if variant not in self.VARIANTS:
            raise ValueError("variant must be one of %s" % (self.VARIANTS,))
        if variant != "lamb" and not bias_correction:
            raise ValueError("N-LAMB and NN-LAMB carry their own bias correction")
        super().__init__(params, grads, lr, weight_decay, clamp, wd_mask, chunk_elems, True,
                         norm, grad_scale, skip_nonfinite, schedule, path, check_every)
        self.beta1, self.beta2 = float(betas[0]), float(betas[1])
        self.eps = float(eps)
        self.bias_correction = bool(bias_correction)
        self.variant = variant

    def step(self, lr: Optional[float] = None) -> None:
        """Apply one step at t = (steps that ran) + 1; per-tensor ratios and
        norms land in ``self.ratios`` and ``self.norms`` (device, float64)."""
        t = self._next_t()
        self._run(_lib.lamb_hparams_init(
            self.variant, step=t, lr=self._lr(lr, t),
            beta1=self.beta1, beta2=self.beta2, eps=self.eps, weight_decay=self.weight_decay,
            gamma_l=self.gamma_l, gamma_u=self.gamma_u, grad_scale=self.grad_scale,
            bias_correction=int(self.bias_correction)))

    def state_dict(self):
        """Step count and moments (after checking that no wait was given up)."""
        self.check()
        return {"step": self.t, "m": [m.clone() for m in self.m], "v": [v.clone() for v in self.v]}

    def load_state_dict(self, state) -> None:
        _check_state(state, {"m": self.m, "v": self.v})
        self._resolve_verdict()
        self._t = int(state["step"])
        for dst, src in zip(self.m, state["m"]):
            dst.copy_(src)
        for dst, src in zip(self.v, state["v"]):
            dst.copy_(src)


class LARS(_LayerwiseOptimizer):
    """Algorithm 1: momentum with weight decay, then a per-layer trust ratio."""

    algo = _lib.LAMB_ALGO_LARS

    def __init__(self, params, grads, lr: float = 1e-3, momentum: float = 0.9,
                 weight_decay: float = 0.01, clamp=(0.0, 10.0), trust_coef: float = 1e-3,
                 wd_mask=None, chunk_elems: int = 0, norm: str = "l2", grad_scale: float = 1.0,
                 skip_nonfinite: bool = False, schedule=None, path: str = "auto",
                 check_every: int = 100):
        super().__init__(params, grads, lr, weight_decay, clamp, wd_mask, chunk_elems, False,
                         norm, grad_scale, skip_nonfinite, schedule, path, check_every)
        self.momentum = float(momentum)
        self.trust_coef = float(trust_coef)

    def step(self, lr: Optional[float] = None) -> None:
        t = self._next_t()
        self._run(_lib.lamb_hparams_init(
            "lars", lr=self._lr(lr, t), beta1=self.momentum,
            weight_decay=self.weight_decay, gamma_l=self.gamma_l, gamma_u=self.gamma_u,
            trust_coef=self.trust_coef, grad_scale=self.grad_scale))

    def state_dict(self):
        """Step count and momentum (after checking that no wait was given up)."""
        self.check()
        return {"step": self.t, "m": [m.clone() for m in self.m]}

    def load_state_dict(self, state) -> None:
        _check_state(state, {"m": self.m})
        self._resolve_verdict()
        self._t = int(state["step"])
        for dst, src in zip(self.m, state["m"]):
            dst.copy_(src)
