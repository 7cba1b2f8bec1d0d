"""Pins of the CPU oracle: facts fixed by the paper and by mathematics.

Every function takes an oracle handle ``o`` (``oracle.Oracle``) and raises
AssertionError when the oracle disagrees with the fact it checks. None of them
restates the oracle's arithmetic: each checks a hand-worked example, a closed
form, an invariant or a special case named in its docstring, so that a slip
anywhere in the oracle (a dropped term, a wrong sign, index or coefficient,
swapped operands) breaks at least one of them. ``test_oracle_mutants`` plants
such slips in a copy of the oracle and checks that each one is caught.

Sources: Algorithm 1 (LARS), Algorithm 2 (LAMB) and Algorithms 3 and 4
(N-LAMB, NN-LAMB, Appendix D) of You et al., the scaling function phi of
Section 3, the sign-SGD remark of Section 3.2, the bound on ||r|| used in the
proof of Theorem 3 (Appendix B) and the bias correction remark of Appendix E.
"""

from __future__ import annotations

import configparser
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hand_cases.ini")

LAMB_DEFAULTS = dict(lr=0.01, beta1=0.9, beta2=0.999, eps=0.0, weight_decay=0.0,
                     gamma_l=0.0, gamma_u=10.0)
LARS_DEFAULTS = dict(lr=0.01, momentum=0.9, weight_decay=0.0, gamma_l=0.0, gamma_u=10.0,
                     trust_coef=1.0)


def _f32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def _zeros_like(xs):
    return [np.zeros_like(x) for x in xs]


def _lamb(o, xs, gs, ms, vs, wd, step, **hp):
    kw = dict(LAMB_DEFAULTS)
    kw.update(hp)
    return o.lamb_step(xs, gs, ms, vs, wd, step=step, **kw)


def _lars(o, xs, gs, ms, wd, **hp):
    kw = dict(LARS_DEFAULTS)
    kw.update(hp)
    return o.lars_step(xs, gs, ms, wd, **kw)


def _phi(z, gl, gu):
    return min(max(z, gl), gu)


def _close(a, b, rtol, atol=0.0, what=""):
    np.testing.assert_allclose(np.asarray(a, np.float64), np.asarray(b, np.float64),
                               rtol=rtol, atol=atol, err_msg=what)


# ---------------------------------------------------------------------------
# Hand-worked examples (tests/golden/hand_cases.ini)
# ---------------------------------------------------------------------------

def _golden():
    cp = configparser.ConfigParser(inline_comment_prefixes=("#",))
    cp.read(GOLDEN)
    return cp


def _vec(s):
    return [float(t) for t in s.split()]


def pin_hand_cases(o):
    """Exact-rational single steps H1A, H1B (two steps), H2 (clamp), H3A/H3B (LARS)."""
    cp = _golden()
    assert cp.sections(), "golden hand cases missing"
    for name in cp.sections():
        c = cp[name]
        x = [_f32(_vec(c["x"]))]
        g = [_f32(_vec(c["g"]))]
        m = _zeros_like(x)
        wd = [c.getint("wd") == 1]
        lam = c.getfloat("weight_decay")
        if c["algo"] == "lamb":
            v = _zeros_like(x)
            out = _lamb(o, x, g, m, v, wd, 1, weight_decay=lam)
            _close(v[0], _vec(c["v_out"]), 1.2e-7, what=name + " v")
        else:
            out = _lars(o, x, g, m, wd, weight_decay=lam, trust_coef=c.getfloat("trust_coef"))
        _close(m[0], _vec(c["m_out"]), 1.2e-7, what=name + " m")
        _close(out[0, 0], c.getfloat("ratio"), 1e-12, what=name + " ratio")
        _close(out[0, 1], c.getfloat("norm_x"), 1e-12, what=name + " ||x||")
        _close(out[0, 2], c.getfloat("norm_u"), 1e-12, what=name + " ||u||")
        _close(x[0], _vec(c["x_out"]), 1.2e-7, what=name + " x")
        if "x_out2" in c:
            out = _lamb(o, x, g, m, v, wd, 2, weight_decay=lam)
            _close(m[0], _vec(c["m_out2"]), 2.5e-7, what=name + " m step 2")
            _close(v[0], _vec(c["v_out2"]), 2.5e-7, what=name + " v step 2")
            _close(out[0, 0], c.getfloat("ratio2"), 5e-8, what=name + " ratio step 2")
            _close(out[0, 1], c.getfloat("norm_x2"), 5e-8, what=name + " ||x|| step 2")
            _close(out[0, 2], c.getfloat("norm_u2"), 5e-8, what=name + " ||u|| step 2")
            _close(x[0], _vec(c["x_out2"]), 2.5e-7, what=name + " x step 2")


# ---------------------------------------------------------------------------
# LAMB closed forms and invariants
# ---------------------------------------------------------------------------

def _three_blocks(rng):
    """Blocks that exercise phi's upper clamp, the middle branch and the lower clamp."""
    sizes = (200, 30, 20)
    scales = (1.0, 0.4, 0.05)      # ||x|| ~ 14 (> 10), ~ 2.2, ~ 0.22 (< gamma_l = 1)
    xs = [_f32(rng.standard_normal(n) * s) for n, s in zip(sizes, scales)]
    return xs, [True, True, False]


def pin_constant_gradient(o):
    """Constant g_t = g from zero moments: m_t = (1 - b1^t) g and v_t = (1 - b2^t) g^2
    (geometric series), so m_hat = g and v_hat = g^2 at every t and
    u = g / (|g| + eps) + lambda_i x_t; the step is x_t - eta phi(||x_t||) u / ||u||.

    The stored moments stay uncorrected; eps sits after the square root of the
    bias-corrected v_hat; the mask removes lambda from the third block.
    """
    rng = np.random.default_rng(11)
    xs, wd = _three_blocks(rng)
    gs = [_f32(rng.standard_normal(x.size) * 1e-3) for x in xs]
    ms, vs = _zeros_like(xs), _zeros_like(xs)
    b1, b2, eps, lam, lr, gl, gu = 0.8, 0.95, 3e-4, 0.05, 0.05, 1.0, 10.0
    for t in range(1, 7):
        x_old = [x.astype(np.float64) for x in xs]
        out = _lamb(o, xs, gs, ms, vs, wd, t, lr=lr, beta1=b1, beta2=b2, eps=eps,
                    weight_decay=lam, gamma_l=gl, gamma_u=gu)
        for i, (g, xo) in enumerate(zip(gs, x_old)):
            gd = g.astype(np.float64)
            _close(ms[i], (1 - b1 ** t) * gd, 1e-6, what="m_t closed form, t=%d" % t)
            _close(vs[i], (1 - b2 ** t) * gd * gd, 1e-6, what="v_t closed form, t=%d" % t)
            u = gd / (np.abs(gd) + eps) + (lam if wd[i] else 0.0) * xo
            nx, nu = np.linalg.norm(xo), np.linalg.norm(u)
            _close(out[i, 1], nx, 1e-12, what="||x||")
            _close(out[i, 2], nu, 1e-6, what="||u||, t=%d block %d" % (t, i))
            _close(out[i, 0], _phi(nx, gl, gu) / nu, 1e-6, what="trust ratio t=%d" % t)
            expect = xo - lr * _phi(nx, gl, gu) * u / nu
            step = np.max(np.abs(expect - xo))
            _close(xs[i], expect, 0, atol=2e-7 * np.max(np.abs(xo)) + 1e-6 * step,
                   what="x_{t+1} closed form, t=%d block %d" % (t, i))


def pin_step_length(o):
    """Section 3: the per-layer step has length eta * phi(||x_t||) whenever u != 0
    (the update is normalised to unit norm, then scaled)."""
    rng = np.random.default_rng(12)
    xs, wd = _three_blocks(rng)
    ms, vs = _zeros_like(xs), _zeros_like(xs)
    lr, gl, gu = 0.05, 1.0, 10.0
    for t in range(1, 5):
        gs = [_f32(rng.standard_normal(x.size) * 1e-3) for x in xs]
        x_old = [x.astype(np.float64) for x in xs]
        _lamb(o, xs, gs, ms, vs, wd, t, lr=lr, beta1=0.9, beta2=0.999, eps=1e-6,
              weight_decay=0.1, gamma_l=gl, gamma_u=gu)
        for i, xo in enumerate(x_old):
            length = np.linalg.norm(xs[i].astype(np.float64) - xo)
            _close(length, lr * _phi(np.linalg.norm(xo), gl, gu), 2e-5,
                   what="step length t=%d block %d" % (t, i))


def pin_sign_sgd(o):
    """Section 3.2: with beta1 = beta2 = 0 (and eps = lambda = 0) LAMB is sign-SGD
    scaled by the square root of the layer dimension:
    x_{t+1} = x_t - eta phi(||x_t||) sign(g_t) / sqrt(d_i)."""
    rng = np.random.default_rng(13)
    xs = [_f32(rng.standard_normal(n) * s) for n, s in ((64, 2.0), (9, 0.3))]
    ms, vs = _zeros_like(xs), _zeros_like(xs)
    lr = 0.1
    for t in (1, 2, 3):
        gs = [_f32(rng.standard_normal(x.size)) for x in xs]
        x_old = [x.astype(np.float64) for x in xs]
        _lamb(o, xs, gs, ms, vs, [True, True], t, lr=lr, beta1=0.0, beta2=0.0)
        for i, xo in enumerate(x_old):
            d = xo.size
            expect = xo - lr * _phi(np.linalg.norm(xo), 0.0, 10.0) * np.sign(gs[i]) / math.sqrt(d)
            _close(xs[i], expect, 2e-7, atol=1e-9, what="sign-SGD t=%d" % t)


def pin_scalar_sign(o):
    """A single scalar block with phi == 1 (gamma_l = gamma_u = 1) moves by exactly
    eta * sign(u); with lambda = 0, u has the sign of g."""
    rng = np.random.default_rng(14)
    x = [_f32([0.7])]
    m, v = _zeros_like(x), _zeros_like(x)
    for t in range(1, 6):
        g = [_f32([rng.standard_normal()])]
        before = float(x[0][0])
        _lamb(o, x, g, m, v, [True], t, lr=0.125, eps=1e-6, gamma_l=1.0, gamma_u=1.0)
        _close(float(x[0][0]) - before, -0.125 * np.sign(m[0][0]), 0, atol=1e-7,
               what="scalar step t=%d" % t)


def pin_first_step(o):
    """Step 1 from m_0 = v_0 = 0: m_hat = g and v_hat = g^2 exactly, so with
    eps = lambda = 0 each u_j = sign(g_j) and ||u|| = sqrt(d); the stored moments
    are (1 - beta1) g and (1 - beta2) g^2. Holds for any betas."""
    rng = np.random.default_rng(15)
    for b1, b2 in ((0.8, 0.95), (0.5, 0.75), (0.9, 0.999)):
        x = [_f32(rng.standard_normal(37))]
        g = [_f32(rng.standard_normal(37) * 1e-2)]
        m, v = _zeros_like(x), _zeros_like(x)
        out = _lamb(o, x, g, m, v, [True], 1, beta1=b1, beta2=b2)
        gd = g[0].astype(np.float64)
        _close(out[0, 2], math.sqrt(37), 1e-12, what="||u|| at t=1")
        _close(m[0], (1 - b1) * gd, 1.2e-7, what="m_1")
        _close(v[0], (1 - b2) * gd * gd, 1.2e-7, what="v_1")


def pin_bias_correction_factor(o):
    """Bias correction multiplies u by sqrt(1 - beta2^t) / (1 - beta1^t) when
    eps = lambda = 0 (Appendix E describes it as a learning-rate factor); the
    normalisation then cancels it, so the trust ratios with and without the
    correction differ by exactly that factor and x moves identically."""
    rng = np.random.default_rng(16)
    b1, b2 = 0.85, 0.97
    x = [_f32(rng.standard_normal(50))]
    m, v = _zeros_like(x), _zeros_like(x)
    for t in range(1, 6):
        g = [_f32(rng.standard_normal(50) * 1e-3)]
        runs = []
        for bc in (True, False):
            xx, mm, vv = [x[0].copy()], [m[0].copy()], [v[0].copy()]
            out = _lamb(o, xx, g, mm, vv, [True], t, lr=0.05, beta1=b1, beta2=b2,
                        bias_correction=bc)
            runs.append((out, xx[0], mm[0], vv[0]))
        (on, x_on, m_on, v_on), (off, x_off, m_off, v_off) = runs
        factor = (1 - b1 ** t) / math.sqrt(1 - b2 ** t)
        _close(on[0, 0], off[0, 0] * factor, 1e-12, what="ratio factor t=%d" % t)
        assert np.array_equal(m_on, m_off) and np.array_equal(v_on, v_off)
        _close(x_on, x_off, 1e-7, what="x with/without correction t=%d" % t)
        x, m, v = [x_on], [m_on], [v_on]


def pin_no_correction_first_step(o):
    """Without bias correction (Appendix E), step 1 uses m_1 = (1 - b1) g and
    v_1 = (1 - b2) g^2 directly: u_j = (1 - b1) g_j / (sqrt(1 - b2) |g_j| + eps)."""
    rng = np.random.default_rng(17)
    b1, b2, eps = 0.9, 0.99, 2e-4
    x = [_f32(rng.standard_normal(40))]
    g = [_f32(rng.standard_normal(40) * 1e-3)]
    m, v = _zeros_like(x), _zeros_like(x)
    out = _lamb(o, x, g, m, v, [True], 1, beta1=b1, beta2=b2, eps=eps, bias_correction=False)
    gd = g[0].astype(np.float64)
    u = (1 - b1) * gd / (math.sqrt(1 - b2) * np.abs(gd) + eps)
    _close(out[0, 2], np.linalg.norm(u), 1e-12, what="||u|| without correction")


def pin_ratio_bound(o):
    """Appendix B bounds the Adam ratio: with beta1 = 0, lambda = eps = 0,
    |r_j| <= sqrt((1 - beta2^t) / (1 - beta2)) under bias correction, hence
    ||u|| <= sqrt(d (1 - beta2^t) / (1 - beta2)), with equality at t = 1."""
    rng = np.random.default_rng(18)
    b2, d = 0.9, 64
    x = [_f32(rng.standard_normal(d))]
    m, v = _zeros_like(x), _zeros_like(x)
    for t in range(1, 9):
        g = [_f32(rng.standard_normal(d) * 10.0 ** rng.uniform(-4, -1))]
        out = _lamb(o, x, g, m, v, [True], t, beta1=0.0, beta2=b2)
        bound = math.sqrt(d * (1 - b2 ** t) / (1 - b2))
        assert out[0, 2] <= bound * (1 + 1e-12), "||r|| above the bound at t=%d" % t
        if t == 1:
            _close(out[0, 2], bound, 1e-12, what="bound attained at t=1")


def pin_mask(o):
    """A block whose mask is 0 steps exactly like the same block with lambda = 0."""
    rng = np.random.default_rng(19)
    x = _f32(rng.standard_normal(33))
    res = []
    for wd, lam in ((False, 0.3), (True, 0.0)):
        xs, ms, vs = [x.copy()], [np.zeros(33, np.float32)], [np.zeros(33, np.float32)]
        outs = []
        for t in (1, 2):
            g = [_f32(np.random.default_rng(100 + t).standard_normal(33) * 1e-3)]
            outs.append(_lamb(o, xs, g, ms, vs, [wd], t, weight_decay=lam, eps=1e-6))
        res.append((xs[0], ms[0], vs[0], outs))
    assert np.array_equal(res[0][0], res[1][0]) and np.array_equal(res[0][1], res[1][1])
    assert all(np.array_equal(a, b) for a, b in zip(res[0][3], res[1][3]))
    # and lambda does act when the mask is on
    xs, ms, vs = [x.copy()], [np.zeros(33, np.float32)], [np.zeros(33, np.float32)]
    g = [_f32(np.random.default_rng(101).standard_normal(33) * 1e-3)]
    out = _lamb(o, xs, g, ms, vs, [True], 1, weight_decay=0.3, eps=1e-6)
    assert abs(out[0, 2] - res[0][3][0][0, 2]) > 1e-3


def pin_scale_invariance(o):
    """With lambda = eps = 0 the Adam ratio is 0-homogeneous in g: scaling every
    g_t by 2 scales m by 2 and v by 4 exactly and leaves x bit for bit unchanged."""
    rng = np.random.default_rng(20)
    x0 = _f32(rng.standard_normal(48))
    grads = [_f32(rng.standard_normal(48) * 1e-3) for _ in range(3)]
    res = []
    for c in (1.0, 2.0):
        xs, ms, vs = [x0.copy()], [np.zeros(48, np.float32)], [np.zeros(48, np.float32)]
        for t, g in enumerate(grads, 1):
            _lamb(o, xs, [_f32(g * c)], ms, vs, [True], t, beta1=0.9, beta2=0.99)
        res.append((xs[0], ms[0], vs[0]))
    assert np.array_equal(res[0][0], res[1][0])
    assert np.array_equal(res[0][1] * 2, res[1][1])
    assert np.array_equal(res[0][2] * 4, res[1][2])


def pin_zero_block(o):
    """phi(0) = gamma_l: a zero block stays put when gamma_l = 0 and moves by
    eta * gamma_l otherwise."""
    g = [_f32(np.linspace(-1e-3, 1e-3, 16) + 1e-5)]
    for gl in (0.0, 0.5):
        x = [np.zeros(16, np.float32)]
        m, v = _zeros_like(x), _zeros_like(x)
        _lamb(o, x, g, m, v, [True], 1, lr=0.1, gamma_l=gl, eps=1e-6)
        _close(np.linalg.norm(x[0].astype(np.float64)), 0.1 * gl, 1e-6, what="zero block")


def pin_zero_update(o):
    """g = 0 and lambda = 0 give u = 0: the step is exactly zero, the reported
    ratio is 0 and nothing becomes NaN (LAMB and LARS)."""
    x = [_f32(np.arange(1, 10) * 0.1)]
    x0 = x[0].copy()
    g = [np.zeros(9, np.float32)]
    m, v = _zeros_like(x), _zeros_like(x)
    out = _lamb(o, x, g, m, v, [True], 1, eps=1e-6)
    assert np.array_equal(x[0], x0) and out[0, 0] == 0.0 and out[0, 2] == 0.0
    out = _lars(o, x, g, m, [True])
    assert np.array_equal(x[0], x0) and out[0, 0] == 0.0 and out[0, 2] == 0.0


def pin_permutation(o):
    """Norms are symmetric: permuting the elements of a block permutes its
    outputs and keeps its trust ratio."""
    rng = np.random.default_rng(21)
    x = _f32(rng.standard_normal(29))
    g = _f32(rng.standard_normal(29) * 1e-3)
    perm = rng.permutation(29)
    a = [x.copy()], [g], [np.zeros(29, np.float32)], [np.zeros(29, np.float32)]
    b = [x[perm].copy()], [g[perm].copy()], [np.zeros(29, np.float32)], [np.zeros(29, np.float32)]
    oa = _lamb(o, *a, [True], 1, weight_decay=0.01, eps=1e-6)
    ob = _lamb(o, *b, [True], 1, weight_decay=0.01, eps=1e-6)
    _close(oa[0], ob[0], 1e-14)
    _close(a[0][0][perm], b[0][0], 1.2e-7)
    assert np.array_equal(a[2][0][perm], b[2][0]) and np.array_equal(a[3][0][perm], b[3][0])


def pin_bf16_gradient(o):
    """A bf16 gradient means the value it encodes: the step equals the step with
    that value given in fp32 (widened by torch's own bf16 conversion)."""
    import torch
    rng = np.random.default_rng(22)
    x = _f32(rng.standard_normal(40) * 0.02)
    g32 = torch.from_numpy(rng.standard_normal(40).astype(np.float32) * 1e-3)
    bits = g32.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()
    widened = g32.to(torch.bfloat16).to(torch.float32).numpy().copy()
    res = []
    for g in (bits, widened):
        xs, ms, vs = [x.copy()], [np.zeros(40, np.float32)], [np.zeros(40, np.float32)]
        out = _lamb(o, xs, [g], ms, vs, [True], 1, weight_decay=0.01, eps=1e-6)
        res.append((xs[0], ms[0], vs[0], out))
    for a, b in zip(res[0], res[1]):
        assert np.array_equal(a, b)
    xs, ms = [x.copy()], [np.zeros(40, np.float32)]
    o1 = _lars(o, xs, [bits], ms, [True], weight_decay=0.01)
    xs2, ms2 = [x.copy()], [np.zeros(40, np.float32)]
    o2 = _lars(o, xs2, [widened], ms2, [True], weight_decay=0.01)
    assert np.array_equal(xs[0], xs2[0]) and np.array_equal(o1, o2)


# ---------------------------------------------------------------------------
# LARS closed forms and invariants
# ---------------------------------------------------------------------------

def pin_lars_normalized_sgd(o):
    """Section 3: LARS with beta1 = 0 and lambda = 0 is layerwise normalised SGD,
    x_{t+1} = x_t - eta kappa phi(||x_t||) g / ||g||, with m_t = g_t."""
    rng = np.random.default_rng(31)
    xs = [_f32(rng.standard_normal(n) * s) for n, s in ((100, 2.0), (12, 0.1))]
    ms = _zeros_like(xs)
    gl, gu, lr, kappa = 0.5, 10.0, 0.1, 0.7
    for _ in range(3):
        gs = [_f32(rng.standard_normal(x.size) * 1e-3) for x in xs]
        x_old = [x.astype(np.float64) for x in xs]
        out = _lars(o, xs, gs, ms, [True, False], lr=lr, momentum=0.0, gamma_l=gl,
                    gamma_u=gu, trust_coef=kappa)
        for i, xo in enumerate(x_old):
            gd = gs[i].astype(np.float64)
            ph = _phi(np.linalg.norm(xo), gl, gu)
            assert np.array_equal(ms[i], gs[i])
            _close(out[i, 0], kappa * ph / np.linalg.norm(gd), 1e-12)
            _close(xs[i], xo - lr * kappa * ph * gd / np.linalg.norm(gd), 2e-7, atol=1e-9)


def pin_lars_constant_gradient(o):
    """Constant g with lambda = 0 from m_0 = 0: m_t = (1 - beta1^t) g (geometric
    series with the (1 - beta1) dampening), the step follows -g / ||g|| with
    length eta kappa phi(||x_t||)."""
    rng = np.random.default_rng(32)
    xs = [_f32(rng.standard_normal(60) * 3.0)]
    gs = [_f32(rng.standard_normal(60) * 1e-3)]
    ms = _zeros_like(xs)
    b1, lr, kappa = 0.8, 0.05, 0.5
    gd = gs[0].astype(np.float64)
    for t in range(1, 6):
        xo = xs[0].astype(np.float64)
        out = _lars(o, xs, gs, ms, [True], lr=lr, momentum=b1, trust_coef=kappa)
        _close(ms[0], (1 - b1 ** t) * gd, 1e-6, what="LARS m_t t=%d" % t)
        _close(out[0, 2], (1 - b1 ** t) * np.linalg.norm(gd), 1e-6)
        ph = _phi(np.linalg.norm(xo), 0.0, 10.0)
        _close(xs[0], xo - lr * kappa * ph * gd / np.linalg.norm(gd), 2e-6, atol=1e-8)


def pin_lars_weight_decay(o):
    """LARS with beta1 = 0: m_t = g_t + lambda_i x_t (Algorithm 1 adds the decay
    before the momentum); the mask removes it."""
    rng = np.random.default_rng(33)
    xs = [_f32(rng.standard_normal(n)) for n in (25, 7)]
    gs = [_f32(rng.standard_normal(x.size) * 1e-2) for x in xs]
    ms = _zeros_like(xs)
    x_old = [x.astype(np.float64) for x in xs]
    _lars(o, xs, gs, ms, [True, False], momentum=0.0, weight_decay=0.1)
    _close(ms[0], gs[0].astype(np.float64) + 0.1 * x_old[0], 1.2e-7)
    assert np.array_equal(ms[1], gs[1])


def pin_lars_step_length(o):
    """LARS steps have length eta kappa phi(||x_t||) whenever m_t != 0."""
    rng = np.random.default_rng(34)
    xs = [_f32(rng.standard_normal(n) * s) for n, s in ((150, 1.5), (30, 0.5), (10, 0.02))]
    ms = _zeros_like(xs)
    lr, kappa, gl, gu = 0.05, 0.3, 0.1, 10.0
    for _ in range(4):
        gs = [_f32(rng.standard_normal(x.size) * 1e-3) for x in xs]
        x_old = [x.astype(np.float64) for x in xs]
        _lars(o, xs, gs, ms, [True, True, False], lr=lr, momentum=0.9, weight_decay=0.05,
              gamma_l=gl, gamma_u=gu, trust_coef=kappa)
        for i, xo in enumerate(x_old):
            length = np.linalg.norm(xs[i].astype(np.float64) - xo)
            _close(length, lr * kappa * _phi(np.linalg.norm(xo), gl, gu), 2e-5)


# ---------------------------------------------------------------------------
# N-LAMB (Algorithm 3) and NN-LAMB (Algorithm 4)
# ---------------------------------------------------------------------------

def _nlamb(o, xs, gs, ms, vs, wd, step, nesterov_v, **hp):
    kw = dict(LAMB_DEFAULTS)
    kw.update(hp)
    return o.nlamb_step(xs, gs, ms, vs, wd, step=step, nesterov_v=nesterov_v, **kw)


def _nesterov_factor(beta, t):
    """Coefficient of g in the Nesterov-corrected moment when g_t is constant:
    beta (1 - beta^t) / (1 - beta^(t+1)) + (1 - beta) / (1 - beta^t)."""
    return beta * (1 - beta ** t) / (1 - beta ** (t + 1)) + (1 - beta) / (1 - beta ** t)


def pin_nlamb_constant_gradient(o):
    """Constant g from zero moments: m_t = (1 - b1^t) g and v_t = (1 - b2^t) g^2
    (geometric series). Substituted into Algorithms 3 and 4, m_hat = c_m(t) g
    with c_m the Nesterov factor of b1; v_hat = b2 g^2 (N-LAMB) or c_v(t) g^2
    with the factor of b2 (NN-LAMB). So u = c_m g / (sqrt(c_v) |g| + eps) +
    lambda_i x_t, at every t."""
    rng = np.random.default_rng(41)
    b1, b2, eps, lam, lr = 0.7, 0.9, 2e-4, 0.05, 0.05
    for nesterov_v in (False, True):
        xs, wd = _three_blocks(rng)
        gs = [_f32(rng.standard_normal(x.size) * 1e-3) for x in xs]
        ms, vs = _zeros_like(xs), _zeros_like(xs)
        for t in range(1, 7):
            x_old = [x.astype(np.float64) for x in xs]
            out = _nlamb(o, xs, gs, ms, vs, wd, t, nesterov_v, lr=lr, beta1=b1, beta2=b2,
                         eps=eps, weight_decay=lam, gamma_l=1.0, gamma_u=10.0)
            cm = _nesterov_factor(b1, t)
            cv = _nesterov_factor(b2, t) if nesterov_v else b2
            for i, (g, xo) in enumerate(zip(gs, x_old)):
                gd = g.astype(np.float64)
                _close(ms[i], (1 - b1 ** t) * gd, 1e-6, what="N-LAMB m_t")
                _close(vs[i], (1 - b2 ** t) * gd * gd, 1e-6, what="N-LAMB v_t")
                u = cm * gd / (math.sqrt(cv) * np.abs(gd) + eps) + (lam if wd[i] else 0.0) * xo
                nx, nu = np.linalg.norm(xo), np.linalg.norm(u)
                what = "%s t=%d block %d" % ("NN-LAMB" if nesterov_v else "N-LAMB", t, i)
                _close(out[i, 2], nu, 1e-6, what=what + " ||u||")
                _close(out[i, 0], _phi(nx, 1.0, 10.0) / nu, 1e-6, what=what + " ratio")
                expect = xo - lr * _phi(nx, 1.0, 10.0) * u / nu
                step = np.max(np.abs(expect - xo))
                _close(xs[i], expect, 0, atol=2e-7 * np.max(np.abs(xo)) + 1e-6 * step, what=what)


def pin_nnlamb_lookahead(o):
    """Nesterov's look-ahead: once the bias corrections have decayed (large t),
    NN-LAMB's m_hat and v_hat are the moments one further update with the same
    gradient would give. Its step from (m, v) therefore equals the uncorrected
    LAMB step (Appendix E) taken from the moments after one LAMB update."""
    rng = np.random.default_rng(42)
    b1, b2, t = 0.6, 0.7, 4000          # b^t underflows: corrections are exactly 1
    x0 = _f32(rng.standard_normal(50))
    m0 = _f32(rng.standard_normal(50) * 1e-3)
    v0 = _f32(np.abs(rng.standard_normal(50)) * 1e-6)
    g = [_f32(rng.standard_normal(50) * 1e-3)]
    xa, ma, va = [x0.copy()], [m0.copy()], [v0.copy()]
    oa = _nlamb(o, xa, g, ma, va, [True], t, True, beta1=b1, beta2=b2, eps=1e-6,
                weight_decay=0.02)
    # advance the moments once with the same gradient, then an uncorrected LAMB step
    xb, mb, vb = [x0.copy()], [m0.copy()], [v0.copy()]
    _lamb(o, [x0.copy()], g, mb, vb, [True], 1, beta1=b1, beta2=b2, bias_correction=False)
    ob = _lamb(o, xb, g, mb, vb, [True], 1, beta1=b1, beta2=b2, eps=1e-6, weight_decay=0.02,
               bias_correction=False)
    _close(oa[0], ob[0], 1e-6, what="look-ahead ratio/norms")
    _close(xa[0], xb[0], 1e-7, what="look-ahead x")


LAMB_PINS = [pin_hand_cases, pin_constant_gradient, pin_step_length, pin_sign_sgd,
             pin_scalar_sign, pin_first_step, pin_bias_correction_factor,
             pin_no_correction_first_step, pin_ratio_bound, pin_mask, pin_scale_invariance,
             pin_zero_block, pin_zero_update, pin_permutation, pin_bf16_gradient]
# ---------------------------------------------------------------------------
# Gradient scaling, other layer norms (Appendix F), skipping non-finite steps
# ---------------------------------------------------------------------------

def pin_grad_scale(o):
    """g_t is the scaled gradient: a step on (g, s = 2^k) is bit for bit the step
    on (2^k g, 1) for every algorithm; for LARS with beta1 = 0 the momentum is
    s g + lambda x (the scale never touches the decay term)."""
    rng = np.random.default_rng(51)
    x0 = _f32(rng.standard_normal(37))
    g = _f32(rng.standard_normal(37) * 1e-3)
    for algo in ("lamb", "nlamb", "lars"):
        res = []
        for gg, sc in ((g, 0.25), (_f32(g * 0.25), 1.0)):
            xs, ms, vs = [x0.copy()], [np.zeros(37, np.float32)], [np.zeros(37, np.float32)]
            for t in (1, 2):
                if algo == "lamb":
                    out = _lamb(o, xs, [gg], ms, vs, [True], t, eps=1e-6, weight_decay=0.02,
                                grad_scale=sc)
                elif algo == "nlamb":
                    out = _nlamb(o, xs, [gg], ms, vs, [True], t, True, eps=1e-6,
                                 weight_decay=0.02, grad_scale=sc)
                else:
                    out = _lars(o, xs, [gg], ms, [True], weight_decay=0.02, grad_scale=sc)
            res.append((xs[0], ms[0], vs[0], out))
        for a, b in zip(*res):
            assert np.array_equal(a, b), algo
    xs, ms = [x0.copy()], [np.zeros(37, np.float32)]
    _lars(o, xs, [g], ms, [True], momentum=0.0, weight_decay=0.1, grad_scale=0.37)
    _close(ms[0], 0.37 * g.astype(np.float64) + 0.1 * x0.astype(np.float64), 1.2e-7)


def _pnorm(a, norm):
    a = np.abs(np.asarray(a, np.float64))
    return {"l2": np.sqrt(np.sum(a * a)), "l1": np.sum(a), "linf": np.max(a)}[norm]


def pin_other_norms(o):
    """Appendix F swaps the layer norm: with the L1 or L-infinity norm the
    reported ||x|| is sum|x| or max|x|, and u / ||u|| has unit norm in that
    norm, so the step has that norm's length eta * phi(||x||) (LAMB, N-LAMB)
    or eta * kappa * phi(||x||) (LARS). With beta1 = beta2 = eps = lambda = 0,
    u = sign(g): the L-infinity step is eta phi sign(g) and the L1 step is
    eta phi sign(g) / d."""
    rng = np.random.default_rng(52)
    lr, gl, gu, kappa = 0.05, 0.5, 10.0, 0.3
    for norm in ("l1", "linf"):
        xs = [_f32(rng.standard_normal(n) * sc) for n, sc in ((120, 1.0), (40, 0.02))]
        ms, vs = _zeros_like(xs), _zeros_like(xs)
        for algo in ("lamb", "nlamb", "lars"):
            for t in (1, 2):
                gs = [_f32(rng.standard_normal(x.size) * 1e-3) for x in xs]
                x_old = [x.astype(np.float64) for x in xs]
                if algo == "lamb":
                    out = _lamb(o, xs, gs, ms, vs, [True, False], t, lr=lr, eps=1e-6,
                                weight_decay=0.05, gamma_l=gl, gamma_u=gu, norm=norm)
                    k = 1.0
                elif algo == "nlamb":
                    out = _nlamb(o, xs, gs, ms, vs, [True, False], t, False, lr=lr, eps=1e-6,
                                 weight_decay=0.05, gamma_l=gl, gamma_u=gu, norm=norm)
                    k = 1.0
                else:
                    out = _lars(o, xs, gs, ms, [True, False], lr=lr, weight_decay=0.05,
                                gamma_l=gl, gamma_u=gu, trust_coef=kappa, norm=norm)
                    k = kappa
                for i, xo in enumerate(x_old):
                    _close(out[i, 1], _pnorm(xo, norm), 1e-12, what=norm + " ||x||")
                    length = _pnorm(xs[i].astype(np.float64) - xo, norm)
                    _close(length, lr * k * _phi(_pnorm(xo, norm), gl, gu), 2e-5,
                           what="%s %s step length" % (norm, algo))
        x = [_f32(rng.standard_normal(30) * 0.3)]
        g = [_f32(rng.standard_normal(30))]
        m, v = _zeros_like(x), _zeros_like(x)
        xo = x[0].astype(np.float64)
        _lamb(o, x, g, m, v, [True], 1, lr=0.1, beta1=0.0, beta2=0.0, norm=norm)
        div = 30.0 if norm == "l1" else 1.0
        expect = xo - 0.1 * _phi(_pnorm(xo, norm), 0.0, 10.0) * np.sign(g[0]) / div
        _close(x[0], expect, 2e-7, atol=1e-9, what=norm + " sign-SGD")


def pin_skip_nonfinite(o):
    """A step with any NaN or infinite scaled gradient, in any tensor, changes
    nothing when skipping is asked for; finiteness is decided on the fp32
    product (3e38 * 10 overflows fp32 though not double)."""
    rng = np.random.default_rng(53)
    base_x = [_f32(rng.standard_normal(n)) for n in (20, 9)]
    for bad, scale in ((np.inf, 1.0), (np.nan, 1.0), (3e38, 10.0)):
        gs = [_f32(rng.standard_normal(20) * 1e-3), _f32(rng.standard_normal(9) * 1e-3)]
        gs[1][4] = bad
        for algo in ("lamb", "nlamb", "lars"):
            xs = [x.copy() for x in base_x]
            ms = [np.full(x.size, 0.5, np.float32) for x in xs]
            vs = [np.full(x.size, 0.25, np.float32) for x in xs]
            kw = dict(grad_scale=scale, skip_nonfinite=True)
            if algo == "lamb":
                out = _lamb(o, xs, gs, ms, vs, [True, True], 3, **kw)
            elif algo == "nlamb":
                out = _nlamb(o, xs, gs, ms, vs, [True, True], 3, False, **kw)
            else:
                out = _lars(o, xs, gs, ms, [True, True], **kw)
            assert np.all(np.isnan(out))
            for a, b in zip(xs, base_x):
                assert np.array_equal(a, b)
            assert all(np.all(m == 0.5) for m in ms) and all(np.all(v == 0.25) for v in vs)
        assert not o.gradients_finite(gs, scale)
    gs = [_f32(rng.standard_normal(20) * 1e-3), _f32([3e38] * 9)]
    assert o.gradients_finite(gs, 1.0)
    xs = [x.copy() for x in base_x]
    out = _lamb(o, xs, gs, _zeros_like(xs), _zeros_like(xs), [True, True], 1, skip_nonfinite=True)
    assert np.all(np.isfinite(out)) and not np.array_equal(xs[0], base_x[0])


def pin_bf16_copy_rounding(o):
    """The bf16 working copy is round-to-nearest-even of fp32 x, bit for bit
    torch's own conversion: random values, exact ties (both parities),
    subnormals, +-inf, the largest finite fp32 (rounds to inf), NaN."""
    import torch
    rng = np.random.default_rng(54)
    vals = [rng.standard_normal(4000).astype(np.float32) * 10.0 ** rng.uniform(-30, 30, 4000)]
    base = rng.integers(0, 1 << 15, size=200).astype(np.uint32) << 16
    ties = (base | 0x8000).view(np.float32)                     # halfway: round to even
    near = (base | 0x7FFF).view(np.float32)
    above = (base | 0x8001).view(np.float32)
    special = np.array([0.0, -0.0, 1e-45, -1e-40, np.inf, -np.inf, 3.4028235e38, -3.4028235e38,
                        1.0, 1.00390625, 1.01171875], dtype=np.float32)
    x = np.concatenate(vals + [ties, near, above, special]).astype(np.float32)
    ours = o.round_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    nan = o.round_bf16(np.array([np.nan, -np.nan], dtype=np.float32))
    assert np.all(nan == 0x7FC0)


NLAMB_PINS = [pin_nlamb_constant_gradient, pin_nnlamb_lookahead]
EXTENSION_PINS = [pin_grad_scale, pin_other_norms, pin_skip_nonfinite, pin_bf16_copy_rounding]
LARS_PINS = [pin_lars_normalized_sgd, pin_lars_constant_gradient, pin_lars_weight_decay,
             pin_lars_step_length]
ALL_PINS = LAMB_PINS + NLAMB_PINS + EXTENSION_PINS + LARS_PINS
