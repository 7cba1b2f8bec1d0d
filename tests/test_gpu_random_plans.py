"""Seeded random plans against the oracle: tensor counts and sizes (many of
them on chunk, block and tile boundaries), chunk sizes, paths, algorithms,
gradient dtypes, layer norms, the non-finite skip mode and hyperparameters
drawn from their documented ranges; two steps each, compared element by
element with the parity tolerances."""

import math

import numpy as np
import pytest

import gpu_harness as H
from paper_1904_00962_amd import _lib

pytestmark = pytest.mark.gpu

ALGOS = ["lamb", "n-lamb", "nn-lamb", "lars"]
CHUNKS = [0, 8, 64, 256, 520, 1024, 4096]
PATHS = ["auto", "wide", "two-pass"]
BOUNDARY = [1, 3, 4, 255, 256, 257, 1023, 1024, 1025, 8191, 8192, 8193, 10239, 10240, 10241]


def _case(seed):
    rng = np.random.default_rng(seed)
    sizes = []
    for _ in range(int(rng.integers(1, 13))):
        if rng.random() < 0.4:
            sizes.append(int(rng.choice(BOUNDARY)) * int(rng.integers(1, 4)))
        else:
            sizes.append(max(1, int(math.exp(rng.uniform(0.0, math.log(3e5))))))
    algo = ALGOS[int(rng.integers(len(ALGOS)))]
    fields = dict(lr=float(10 ** rng.uniform(-4, -1)),
                  weight_decay=float(0.0 if rng.random() < 0.3 else 10 ** rng.uniform(-4, -1)),
                  norm=["l2", "l1", "linf"][int(rng.integers(3))],
                  grad_scale=float(rng.choice([1.0, 0.5, 2.0 ** -8, 3.0])),
                  skip_nonfinite=int(rng.random() < 0.3))
    gamma_l = 0.0 if rng.random() < 0.6 else float(rng.uniform(0.0, 0.5))
    fields.update(gamma_l=gamma_l,
                  gamma_u=float(math.inf if rng.random() < 0.2 else gamma_l + rng.uniform(0.1, 20)))
    if algo == "lars":
        fields.update(beta1=float(rng.uniform(0.0, 0.99)),
                      trust_coef=float(10 ** rng.uniform(-3, 0)))
    else:
        fields.update(beta1=float(rng.uniform(0.5, 0.99)), beta2=float(rng.uniform(0.9, 0.9999)),
                      eps=float(10 ** rng.uniform(-8, -4)))
        if algo == "lamb":
            fields.update(bias_correction=int(rng.random() < 0.8))
    return dict(sizes=sizes, algo=algo, fields=fields,
                g_dtype="bf16" if rng.random() < 0.5 else "f32",
                chunk=int(rng.choice(CHUNKS)), path=PATHS[int(rng.integers(len(PATHS)))],
                rng=rng)


@pytest.mark.parametrize("seed", range(64))
def test_random_plan(seed):
    import torch
    H.torch_cuda()
    c = _case(5000 + seed)
    rng = c["rng"]
    H.log("random plan %d: %s %s chunk=%d path=%s tensors=%s %s"
          % (seed, c["algo"], c["g_dtype"], c["chunk"], c["path"], c["sizes"], c["fields"]))
    xs = [(rng.standard_normal(n) * rng.uniform(0.01, 1.0)).astype(np.float32)
          for n in c["sizes"]]
    wd = [bool(rng.random() < 0.7) for _ in c["sizes"]]
    pair = H.Pair(xs, wd, c["g_dtype"], "lars" if c["algo"] == "lars" else "lamb", c["chunk"],
                  path=c["path"])
    try:
        for t in (1, 2):
            gs = []
            for n in c["sizes"]:
                g = torch.from_numpy((rng.standard_normal(n) * 1e-3).astype(np.float32))
                gs.append(g.to(torch.bfloat16) if c["g_dtype"] == "bf16" else g)
            hg = pair.set_grads(gs)
            hp = _lib.lamb_hparams_init(c["algo"], step=t, **c["fields"])
            ref = H.step_ex_both(pair, hp, hg)
            pair.compare(ref, "random plan %d step %d" % (seed, t))
    finally:
        pair.close()
