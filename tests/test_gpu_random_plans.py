"""Seeded random plans against the oracle: tensor counts and sizes (many of
them on chunk, block and tile boundaries), chunk sizes, paths, algorithms,
gradient dtypes, layer norms, the non-finite skip mode, bf16 copies of x and
hyperparameters drawn from their documented ranges; two steps each, compared
element by element with the parity tolerances.

Trust ratios and ||u|| are held to 1e-6 relative, or, for a tensor whose
update norm rests on a few elements of u that cancel, to twice the derived
bound on what fp32 evaluation of u can reach (``gpu_harness.update_norm_bound``),
whichever is larger. With random moments and gradients, one element's m_hat
(a sum of two terms of either sign for N-LAMB and NN-LAMB) or its r + lambda x
can cancel to a small fraction of its terms; in a tensor of one or a few
elements that element sets ||u|| and the ratio phi / ||u||. Random plan 0 of
the skip test, a one-element N-LAMB tensor, cancels m_hat twentyfold at step
3 and its ratio differs from the oracle's by 2.3e-6 relative, within that
tensor's bound.
"""

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
    # bf16 copies of x on some tensors of some plans (their own draws)
    crng = np.random.default_rng(9000 + seed)
    copies = [None] * len(xs)
    if crng.random() < 0.4:
        copies = [torch.full((n,), 12345, dtype=torch.int16, device="cuda").view(torch.bfloat16)
                  if crng.random() < 0.7 else None for n in c["sizes"]]
        _lib.lamb_plan_set_bf16_copies(pair.plan, [b.data_ptr() if b is not None else 0
                                                   for b in copies])
    try:
        for t in (1, 2):
            gs = []
            for n in c["sizes"]:
                g = torch.from_numpy((rng.standard_normal(n) * 1e-3).astype(np.float32))
                gs.append(g.to(torch.bfloat16) if c["g_dtype"] == "bf16" else g)
            hg = pair.set_grads(gs)
            hp = _lib.lamb_hparams_init(c["algo"], step=t, **c["fields"])
            tol = pair.ratio_tolerances(hp, hg)
            ref = H.step_ex_both(pair, hp, hg)
            pair.compare(ref, "random plan %d step %d" % (seed, t), ratio_tol=tol)
            for i, b in enumerate(copies):
                if b is None:
                    continue
                # torch's cast of the GPU's own x, bit for bit; within one bf16
                # step of the oracle's rounding of the oracle's x wherever
                # |x| >= rms/256: there a bf16 step (>= |x| 2^-8) exceeds the
                # x tolerance of 1e-5 rms, below it the tolerance can exceed it
                got = b.view(torch.int16).cpu().numpy()
                assert np.array_equal(got, pair.X[i].to(torch.bfloat16).view(torch.int16)
                                      .cpu().numpy()), (t, i)
                hx = pair.hx[i]
                rms = float(np.sqrt(np.mean(hx.astype(np.float64) ** 2)))
                far = np.abs(hx) >= rms / 256
                want = pair.oracle.round_bf16(hx).view(np.int16)
                diff = np.abs(got.astype(np.int32) - want.astype(np.int32))
                assert np.all(diff[far] <= 1), (t, i)
    finally:
        pair.close()


@pytest.mark.parametrize("seed", range(32))
def test_random_plan_skips_a_nonfinite_step(seed):
    """Random plans in skip mode: a step whose gradient holds one NaN or
    infinity at a random place changes nothing (bit for bit) and reports 1;
    the finite steps around it follow the oracle."""
    import torch
    H.torch_cuda()
    c = _case(7000 + seed)
    rng = c["rng"]
    c["fields"]["skip_nonfinite"] = 1
    bad_tensor = int(rng.integers(len(c["sizes"])))
    bad_at = int(rng.integers(c["sizes"][bad_tensor]))
    bad_value = float(rng.choice([math.inf, -math.inf, math.nan]))
    H.log("random skip plan %d: %s %s chunk=%d path=%s tensors=%s, %r at %d of tensor %d"
          % (seed, c["algo"], c["g_dtype"], c["chunk"], c["path"], c["sizes"], bad_value,
             bad_at, bad_tensor))
    xs = [(rng.standard_normal(n) * rng.uniform(0.01, 1.0)).astype(np.float32)
          for n in c["sizes"]]
    wd = [bool(rng.random() < 0.7) for _ in c["sizes"]]
    pair = H.Pair(xs, wd, c["g_dtype"], "lars" if c["algo"] == "lars" else "lamb", c["chunk"],
                  path=c["path"])
    flag = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    try:
        for t in (1, 2, 3):
            gs = []
            for i, n in enumerate(c["sizes"]):
                g = torch.from_numpy((rng.standard_normal(n) * 1e-3).astype(np.float32))
                if t == 2 and i == bad_tensor:
                    g[bad_at] = bad_value
                gs.append(g.to(torch.bfloat16) if c["g_dtype"] == "bf16" else g)
            hg = pair.set_grads(gs)
            before = [x.clone() for x in pair.X] + [m.clone() for m in pair.M]
            hp = _lib.lamb_hparams_init(c["algo"], step=t, **c["fields"])
            tol = pair.ratio_tolerances(hp, hg)
            ref = H.step_ex_both(pair, hp, hg, flag)
            pair.compare(ref, "random skip plan %d step %d" % (seed, t), ratio_tol=tol)
            torch.cuda.synchronize()
            assert int(flag) == (1 if t == 2 else 0), (t, int(flag))
            if t == 2:
                assert bool(np.all(np.isnan(ref)))
                assert all(torch.equal(a, b) for a, b in
                           zip(before, [x for x in pair.X] + [m for m in pair.M]))
    finally:
        pair.close()
