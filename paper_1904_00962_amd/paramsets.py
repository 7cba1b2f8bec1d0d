"""Seeded synthetic parameter sets shaped like the paper's workloads.

This module only draws inputs: tensor shapes, weight-decay masks, initial
parameters x and gradients g. It holds none of the optimizer's arithmetic and
imports nothing from the HIP library or from the oracle, so both sides of a
parity test can take their inputs from it.

The paper trains BERT (Section 4.1) and ResNet-50 on ImageNet (Section 4.2);
an optimizer step only reads parameter, gradient and state tensors, so these
sets keep the models' parameter shapes and replace values with i.i.d.
Gaussians: x ~ N(0, sigma_x) and g ~ N(0, 1e-3) (second argument = standard
deviation). Moments start at zero, as Algorithms 1 and 2 set m_0 = v_0 = 0.

Seeds: x uses ``1000 * cfg``; the gradient of step t uses ``1000 * cfg + t``.
Values are drawn tensor by tensor in canonical order with a seeded torch
generator in fp32 (on the CPU, or on the GPU for the large sets); bf16
gradients are the round-to-nearest-even cast of the fp32 draw. The oracle
side receives the same bits through ``host_array``.
"""

from __future__ import annotations

import dataclasses
from typing import List, Sequence, Tuple

import numpy as np

Shape = Tuple[int, ...]


@dataclasses.dataclass(frozen=True)
class TensorSpec:
    name: str
    shape: Shape
    wd: bool  # decoupled weight decay applies (False for biases and norms)

    @property
    def numel(self) -> int:
        n = 1
        for s in self.shape:
            n *= s
        return n


@dataclasses.dataclass(frozen=True)
class ParamSet:
    cfg: int
    name: str
    tensors: Tuple[TensorSpec, ...]
    sigma_x: float
    sigma_g: float
    g_dtype: str  # "f32" or "bf16"
    # LAMB hyperparameters (defaults follow Section 4 / Appendix H)
    lr: float
    beta1: float
    beta2: float
    eps: float
    weight_decay: float
    gamma_l: float
    gamma_u: float
    # LARS hyperparameters (used where the workload is run with LARS)
    lars_lr: float = 1e-3
    lars_momentum: float = 0.9
    lars_trust_coef: float = 1e-3

    @property
    def numel(self) -> int:
        return sum(t.numel for t in self.tensors)

    @property
    def n_tensors(self) -> int:
        return len(self.tensors)

    def numels(self) -> List[int]:
        return [t.numel for t in self.tensors]

    def wd_mask(self) -> List[bool]:
        return [t.wd for t in self.tensors]


def _linear(prefix: str, out_f: int, in_f: int, bias: bool = True) -> List[TensorSpec]:
    specs = [TensorSpec(prefix + ".weight", (out_f, in_f), True)]
    if bias:
        specs.append(TensorSpec(prefix + ".bias", (out_f,), False))
    return specs


def _norm(prefix: str, width: int) -> List[TensorSpec]:
    return [TensorSpec(prefix + ".gamma", (width,), False),
            TensorSpec(prefix + ".beta", (width,), False)]


def tiny_tensors() -> List[TensorSpec]:
    shapes = [(256, 256), (256,), (256, 1024), (1024,), (1024, 256), (256,), (64, 256), (256,)]
    return [TensorSpec("t%d" % i, s, len(s) > 1) for i, s in enumerate(shapes)]


def bert_tensors(hidden: int, ffn: int, layers: int, vocab: int = 30522,
                 positions: int = 512, types: int = 2) -> List[TensorSpec]:
    """BERT encoder parameter list: embeddings, encoder layers, pooler."""
    t: List[TensorSpec] = [
        TensorSpec("emb.token", (vocab, hidden), True),
        TensorSpec("emb.position", (positions, hidden), True),
        TensorSpec("emb.type", (types, hidden), True),
    ]
    t += _norm("emb.ln", hidden)
    for i in range(layers):
        p = "layer%d." % i
        for proj in ("q", "k", "v", "o"):
            t += _linear(p + proj, hidden, hidden)
        t += _norm(p + "ln1", hidden)
        t.append(TensorSpec(p + "ffn_in.weight", (hidden, ffn), True))
        t.append(TensorSpec(p + "ffn_in.bias", (ffn,), False))
        t.append(TensorSpec(p + "ffn_out.weight", (ffn, hidden), True))
        t.append(TensorSpec(p + "ffn_out.bias", (hidden,), False))
        t += _norm(p + "ln2", hidden)
    t += _linear("pooler", hidden, hidden)
    return t


def resnet50_tensors() -> List[TensorSpec]:
    """ResNet-50 (bottleneck v1) convolution, batch-norm and classifier tensors."""
    t: List[TensorSpec] = [TensorSpec("stem.conv", (64, 3, 7, 7), True)]
    t += _norm("stem.bn", 64)
    c_in = 64
    for s, (w, n) in enumerate([(64, 3), (128, 4), (256, 6), (512, 3)]):
        for b in range(n):
            p = "stage%d.block%d." % (s + 1, b)
            t.append(TensorSpec(p + "conv1", (w, c_in, 1, 1), True))
            t += _norm(p + "bn1", w)
            t.append(TensorSpec(p + "conv2", (w, w, 3, 3), True))
            t += _norm(p + "bn2", w)
            t.append(TensorSpec(p + "conv3", (4 * w, w, 1, 1), True))
            t += _norm(p + "bn3", 4 * w)
            if b == 0:
                t.append(TensorSpec(p + "proj", (4 * w, c_in, 1, 1), True))
                t += _norm(p + "proj_bn", 4 * w)
            c_in = 4 * w
    t += _linear("fc", 1000, 2048)
    return t


def gpt_tensors(hidden: int = 1600, ffn: int = 6400, layers: int = 48,
                vocab: int = 50257, positions: int = 1024) -> List[TensorSpec]:
    """Decoder-only transformer with a fused QKV projection (1.5B at defaults)."""
    t: List[TensorSpec] = [
        TensorSpec("emb.token", (vocab, hidden), True),
        TensorSpec("emb.position", (positions, hidden), True),
    ]
    for i in range(layers):
        p = "layer%d." % i
        t += _norm(p + "ln1", hidden)
        t.append(TensorSpec(p + "qkv.weight", (hidden, 3 * hidden), True))
        t.append(TensorSpec(p + "qkv.bias", (3 * hidden,), False))
        t += _linear(p + "o", hidden, hidden)
        t += _norm(p + "ln2", hidden)
        t.append(TensorSpec(p + "ffn_in.weight", (hidden, ffn), True))
        t.append(TensorSpec(p + "ffn_in.bias", (ffn,), False))
        t.append(TensorSpec(p + "ffn_out.weight", (ffn, hidden), True))
        t.append(TensorSpec(p + "ffn_out.bias", (hidden,), False))
    t += _norm("final_ln", hidden)
    return t


_COMMON = dict(beta1=0.9, beta2=0.999, eps=1e-6, weight_decay=0.01, gamma_l=0.0, gamma_u=10.0)

CONFIGS = {
    0: ParamSet(0, "tiny", tuple(tiny_tensors()), 0.02, 1e-3, "f32", lr=1e-3, **_COMMON),
    1: ParamSet(1, "bert-base", tuple(bert_tensors(768, 3072, 12)), 0.02, 1e-3, "f32",
                lr=1e-3, **_COMMON),
    2: ParamSet(2, "bert-large", tuple(bert_tensors(1024, 4096, 24)), 0.02, 1e-3, "bf16",
                lr=6e-3, **_COMMON),
    3: ParamSet(3, "resnet50", tuple(resnet50_tensors()), 0.05, 1e-3, "f32", lr=1e-3,
                lars_lr=1e-3, lars_momentum=0.9, lars_trust_coef=1e-3, **_COMMON),
    4: ParamSet(4, "gpt-1.5b", tuple(gpt_tensors()), 0.02, 1e-3, "bf16", lr=6e-3, **_COMMON),
}


def get(cfg: int) -> ParamSet:
    return CONFIGS[cfg]


def _torch():
    import torch  # local import: shape queries need no torch
    return torch


def _generator(seed: int, device):
    torch = _torch()
    return torch.Generator(device=torch.device(device)).manual_seed(seed)


def draw_params(ps: ParamSet, indices: Sequence[int] | None = None, device="cpu") -> list:
    """Initial x (fp32 torch tensors, flat) for every tensor or the listed ones.

    Seed ``1000 * cfg`` on a torch generator of ``device``. Tensors are always
    drawn in canonical order from that one generator, so a tensor's values do
    not depend on which subset is requested. CPU and GPU generators give
    different (equally valid) draws; a parity test draws once and hands the
    same bits to both sides.
    """
    torch = _torch()
    gen = _generator(1000 * ps.cfg, device)
    want = set(range(ps.n_tensors)) if indices is None else set(indices)
    out = []
    for i, spec in enumerate(ps.tensors):
        a = torch.randn(spec.numel, generator=gen, dtype=torch.float32, device=device)
        if i in want:
            out.append(a.mul_(ps.sigma_x))
    return out


def draw_grads(ps: ParamSet, step: int, indices: Sequence[int] | None = None,
               device="cpu") -> list:
    """Gradient of step ``step`` (>= 1), seed ``1000 * cfg + step``: flat fp32
    tensors, or bf16 tensors rounded to nearest even from the fp32 draw."""
    torch = _torch()
    gen = _generator(1000 * ps.cfg + step, device)
    want = set(range(ps.n_tensors)) if indices is None else set(indices)
    out = []
    for i, spec in enumerate(ps.tensors):
        a = torch.randn(spec.numel, generator=gen, dtype=torch.float32, device=device)
        if i in want:
            a.mul_(ps.sigma_g)
            out.append(a.to(torch.bfloat16) if ps.g_dtype == "bf16" else a)
    return out


def host_array(t) -> np.ndarray:
    """A torch tensor's bits as a host numpy array (bf16 as uint16 patterns)."""
    torch = _torch()
    t = t.detach().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()

