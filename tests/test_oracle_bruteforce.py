"""The oracle's double arithmetic against 50-digit decimal arithmetic.

Tiny random cases (up to 3 blocks of up to 9 elements, 3 steps, eps > 0,
lambda > 0, mixed masks, clamps active). Both sides start every step from the
same fp32 state and round the new state to fp32, so x, m, v must agree to one
fp32 rounding and the trust ratios to ~1e-13. This guards the floating-point
evaluation (powers, square roots, accumulation), not the reading of the
algorithm, which the pins in ``oracle_pins`` fix.
"""

import decimal
from decimal import Decimal as D

import numpy as np
import pytest

import oracle

decimal.getcontext().prec = 50


def _dec(a):
    return D(float(a))


def _phi(z, gl, gu):
    return min(max(z, gl), gu)


def _lamb_block(x, g, m, v, lam, hp, t):
    b1, b2, eps, lr = (_dec(hp[k]) for k in ("beta1", "beta2", "eps", "lr"))
    c1, c2 = 1 - b1 ** t, 1 - b2 ** t
    u, mo, vo = [], [], []
    for xj, gj, mj, vj in zip(x, g, m, v):
        M = b1 * _dec(mj) + (1 - b1) * _dec(gj)
        V = b2 * _dec(vj) + (1 - b2) * _dec(gj) ** 2
        r = (M / c1) / ((V / c2).sqrt() + eps)
        u.append(r + lam * _dec(xj))
        mo.append(M)
        vo.append(V)
    nx = sum(_dec(a) ** 2 for a in x).sqrt()
    nu = sum(a * a for a in u).sqrt()
    ratio = D(0) if nu == 0 else _phi(nx, _dec(hp["gamma_l"]), _dec(hp["gamma_u"])) / nu
    xo = [_dec(a) - lr * ratio * b for a, b in zip(x, u)]
    return xo, mo, vo, ratio


def _lars_block(x, g, m, lam, hp):
    b1, lr, k = (_dec(hp[q]) for q in ("momentum", "lr", "trust_coef"))
    M = [b1 * _dec(mj) + (1 - b1) * (_dec(gj) + lam * _dec(xj)) for xj, gj, mj in zip(x, g, m)]
    nx = sum(_dec(a) ** 2 for a in x).sqrt()
    nm = sum(a * a for a in M).sqrt()
    ratio = D(0) if nm == 0 else k * _phi(nx, _dec(hp["gamma_l"]), _dec(hp["gamma_u"])) / nm
    return [_dec(a) - lr * ratio * b for a, b in zip(x, M)], M, ratio


def _f32(vals):
    return np.array([float(a) for a in vals], dtype=np.float32)


@pytest.mark.parametrize("seed", range(12))
def test_lamb_bruteforce(seed):
    o = oracle.load()
    rng = np.random.default_rng(seed)
    nb = int(rng.integers(1, 4))
    sizes = [int(rng.integers(1, 10)) for _ in range(nb)]
    xs = [(rng.standard_normal(n) * rng.choice([0.05, 1.0, 5.0])).astype(np.float32) for n in sizes]
    ms = [np.zeros(n, np.float32) for n in sizes]
    vs = [np.zeros(n, np.float32) for n in sizes]
    wd = [bool(rng.integers(0, 2)) for _ in sizes]
    hp = dict(lr=0.01, beta1=float(rng.uniform(0.5, 0.95)), beta2=float(rng.uniform(0.9, 0.9999)),
              eps=float(10 ** rng.uniform(-5, -2)), weight_decay=0.05, gamma_l=0.1, gamma_u=10.0)
    for t in (1, 2, 3):
        gs = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for n in sizes]
        expect = [_lamb_block(x, g, m, v, _dec(hp["weight_decay"]) if w else D(0), hp, t)
                  for x, g, m, v, w in zip(xs, gs, ms, vs, wd)]
        out = o.lamb_step(xs, gs, ms, vs, wd, step=t, **hp)
        for i, (xo, mo, vo, ratio) in enumerate(expect):
            np.testing.assert_allclose(out[i, 0], float(ratio), rtol=1e-13)
            np.testing.assert_allclose(xs[i], _f32(xo), rtol=1.2e-7, atol=1e-30)
            np.testing.assert_allclose(ms[i], _f32(mo), rtol=1.2e-7, atol=1e-30)
            np.testing.assert_allclose(vs[i], _f32(vo), rtol=1.2e-7, atol=1e-30)


@pytest.mark.parametrize("seed", range(6))
def test_lars_bruteforce(seed):
    o = oracle.load()
    rng = np.random.default_rng(100 + seed)
    sizes = [int(rng.integers(1, 10)) for _ in range(int(rng.integers(1, 4)))]
    xs = [(rng.standard_normal(n) * rng.choice([0.05, 1.0, 5.0])).astype(np.float32) for n in sizes]
    ms = [np.zeros(n, np.float32) for n in sizes]
    wd = [bool(rng.integers(0, 2)) for _ in sizes]
    hp = dict(lr=0.01, momentum=float(rng.uniform(0.5, 0.95)), weight_decay=0.05, gamma_l=0.1,
              gamma_u=10.0, trust_coef=0.01)
    for _ in range(3):
        gs = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for n in sizes]
        expect = [_lars_block(x, g, m, _dec(hp["weight_decay"]) if w else D(0), hp)
                  for x, g, m, w in zip(xs, gs, ms, wd)]
        out = o.lars_step(xs, gs, ms, wd, **hp)
        for i, (xo, mo, ratio) in enumerate(expect):
            np.testing.assert_allclose(out[i, 0], float(ratio), rtol=1e-13)
            np.testing.assert_allclose(xs[i], _f32(xo), rtol=1.2e-7, atol=1e-30)
            np.testing.assert_allclose(ms[i], _f32(mo), rtol=1.2e-7, atol=1e-30)
