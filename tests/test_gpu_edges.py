"""Edge cases of the HIP step against the oracle: ragged sizes around every
tile boundary, degenerate blocks, special values, flags and validation."""

import math

import numpy as np
import pytest

import gpu_harness as H
from paper_1904_00962_amd import _lib

pytestmark = pytest.mark.gpu

DEFAULT = dict(lr=1e-2, beta1=0.9, beta2=0.999, eps=1e-6, weight_decay=0.01, gamma_l=0.0,
               gamma_u=10.0)
LARS = dict(lr=1e-2, momentum=0.9, weight_decay=0.01, gamma_l=0.0, gamma_u=10.0, trust_coef=0.01)


def _xs(rng, sizes, scale=0.5):
    return [(rng.standard_normal(n) * scale).astype(np.float32) for n in sizes]


def _gs(rng, sizes, g_dtype="f32", scale=1e-3):
    import torch
    out = []
    for n in sizes:
        t = torch.from_numpy((rng.standard_normal(n) * scale).astype(np.float32))
        out.append(t.to(torch.bfloat16) if g_dtype == "bf16" else t)
    return out


PATHS = ["auto", "wide", "two-pass"]


def _run(xs, wd, g_dtype, algo, chunk, steps, hp, rng, grads=None, bias_correction=True,
         ratio_tol=H.RATIO_TOL, path="auto"):
    pair = H.Pair(xs, wd, g_dtype, algo, chunk, path=path)
    try:
        for t in range(1, steps + 1):
            gs = grads(t) if grads else _gs(rng, [x.size for x in xs], g_dtype)
            hg = pair.set_grads(gs)
            ref = H.step_both(pair, algo, hg, hp, t, bias_correction)
            pair.compare(ref, "%s %s chunk=%d %s step %d" % (algo, g_dtype, chunk, path, t),
                         ratio_tol)
        return pair
    finally:
        pair.close()


RAGGED = [1, 2, 3, 4, 5, 7, 8, 9, 15, 16, 17, 255, 256, 257, 1023, 1024, 1025, 1031, 2047,
          2048, 2049, 4095, 4096, 4097, 8191, 8193]


NLAMB = dict(DEFAULT, beta1=0.975, eps=1e-8)


@pytest.mark.parametrize("algo,g_dtype", [("lamb", "f32"), ("lamb", "bf16"), ("lars", "f32"),
                                          ("lars", "bf16"), ("nlamb", "bf16"),
                                          ("nnlamb", "f32")])
@pytest.mark.parametrize("chunk,path", [(8, "two-pass"), (64, "two-pass"), (520, "two-pass"),
                                        (1024, "two-pass"), (0, "two-pass"), (0, "auto"),
                                        (0, "wide")])
def test_ragged_sizes(algo, g_dtype, chunk, path):
    """Every tensor length around the 4-element group, the workgroup's span
    (one to four waves, by chunk size), the unrolled loop trip and the chunk
    boundary; on the single pass, around
    the 8192- and 10240-element tiles and their multiples (layers of several
    tiles)."""
    rng = np.random.default_rng(1000 + chunk)
    sizes = list(RAGGED)
    if chunk:
        sizes += [chunk - 1, chunk, chunk + 1, 4 * chunk + 5]
    else:
        sizes += [32767, 32768, 32769, 4 * 32768 + 5]
    if path in ("auto", "wide"):
        sizes += [8191, 8192, 8193, 2 * 8192 - 3, 3 * 8192, 5 * 8192 + 7]
        sizes += [10239, 10240, 10241, 3 * 10240 + 11]
    xs = _xs(rng, sizes)
    wd = [i % 3 != 0 for i in range(len(sizes))]
    hp = {"lamb": DEFAULT, "lars": LARS, "nlamb": NLAMB, "nnlamb": NLAMB}[algo]
    H.log("ragged algo=%s g=%s chunk=%d path=%s tensors=%d"
          % (algo, g_dtype, chunk, path, len(sizes)))
    _run(xs, wd, g_dtype, algo, chunk, 3, hp, rng, path=path)


@pytest.mark.parametrize("path", PATHS)
def test_zero_gradient_block_does_not_move(path):
    """||u|| = 0: ratio exactly 0, x bit for bit unchanged, no NaN."""
    torch = H.torch_cuda()
    rng = np.random.default_rng(5)
    xs = _xs(rng, [100, 37])
    pair = H.Pair(xs, [False, True], "f32", "lamb", path=path)
    try:
        hg = pair.set_grads([torch.zeros(100), torch.from_numpy(rng.standard_normal(37).astype(np.float32) * 1e-3)])
        x0 = pair.X[0].clone()
        pair.gpu_lamb(DEFAULT, 1)
        ref = pair.oracle_lamb(hg, DEFAULT, 1)
        pair.compare(ref, "zero grad")
        assert torch.equal(pair.X[0], x0)
        assert float(pair.ratio[0]) == 0.0 and ref[0, 0] == 0.0
    finally:
        pair.close()


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("gamma_l", [0.0, 0.25])
def test_zero_parameter_block(gamma_l, path):
    """phi(0) = gamma_l: a zero block stays put at gamma_l = 0, else moves."""
    rng = np.random.default_rng(6)
    xs = [np.zeros(513, np.float32), _xs(rng, [300])[0]]
    hp = dict(DEFAULT, gamma_l=gamma_l)
    _run(xs, [True, True], "f32", "lamb", 0, 2, hp, rng, path=path)
    _run(xs, [True, True], "f32", "lars", 0, 2, dict(LARS, gamma_l=gamma_l), rng, path=path)


@pytest.mark.parametrize("path", PATHS)
def test_nan_gradient_propagates_like_the_oracle(path):
    torch = H.torch_cuda()
    rng = np.random.default_rng(7)
    xs = _xs(rng, [64, 65, 3 * 8192 + 1])
    g0 = torch.from_numpy((rng.standard_normal(64) * 1e-3).astype(np.float32))
    g0[17] = float("nan")
    g1 = torch.from_numpy((rng.standard_normal(65) * 1e-3).astype(np.float32))
    g2 = torch.from_numpy((rng.standard_normal(3 * 8192 + 1) * 1e-3).astype(np.float32))
    g2[2 * 8192 + 5] = float("inf")  # in the third tile of a three-tile layer
    pair = H.Pair(xs, [True, True, False], "f32", "lamb", path=path)
    try:
        hg = pair.set_grads([g0, g1, g2])
        pair.gpu_lamb(DEFAULT, 1)
        ref = pair.oracle_lamb(hg, DEFAULT, 1)
        pair.compare(ref, "nan grad")
        assert np.isnan(ref[0, 0]) and math.isnan(float(pair.ratio[0]))
        assert np.isnan(ref[2, 0]) and math.isnan(float(pair.ratio[2]))
    finally:
        pair.close()


@pytest.mark.parametrize("hp", [
    dict(DEFAULT, gamma_u=float("inf")),
    dict(DEFAULT, gamma_l=5.0, gamma_u=5.0),
    dict(DEFAULT, beta1=0.0, beta2=0.0, eps=0.0, weight_decay=0.0),
    dict(DEFAULT, eps=0.0),
    dict(DEFAULT, weight_decay=0.5, lr=0.3),
], ids=["no-upper-clamp", "phi-const", "sign-sgd", "eps0", "big-lr-wd"])
@pytest.mark.parametrize("path", PATHS)
def test_scalar_settings(hp, path):
    rng = np.random.default_rng(8)
    xs = _xs(rng, [4096, 333, 9, 1, 20000], scale=2.0)
    _run(xs, [True, False, True, True, False], "f32", "lamb", 1024, 4, hp, rng, path=path)


@pytest.mark.parametrize("path", PATHS)
def test_without_bias_correction(path):
    rng = np.random.default_rng(9)
    xs = _xs(rng, [5000, 77, 17000])
    _run(xs, [True, False, True], "bf16", "lamb", 2048, 4, DEFAULT, rng, bias_correction=False,
         path=path)


@pytest.mark.parametrize("path", PATHS)
def test_lars_trust_coefficient_one_and_no_momentum(path):
    rng = np.random.default_rng(10)
    xs = _xs(rng, [3000, 5, 9000])
    _run(xs, [True, False, True], "f32", "lars", 0, 3,
         dict(LARS, trust_coef=1.0, momentum=0.0), rng, path=path)


@pytest.mark.parametrize("path", PATHS)
def test_guard_bands_untouched(path):
    """Tensors carved out of one buffer with canary gaps between them: no
    kernel writes outside its tensors."""
    torch = H.torch_cuda()
    sizes = [1, 7, 1000, 4097, 33, 20001]
    gap = 64
    total = sum(sizes) + gap * (len(sizes) + 1)
    bufs = {k: torch.full((total,), -7.25, device="cuda") for k in "xgmv"}
    views = {k: [] for k in "xgmv"}
    off = gap
    rng = np.random.default_rng(11)
    for n in sizes:
        for k in "xgmv":
            views[k].append(bufs[k][off:off + n])
        views["x"][-1].copy_(torch.from_numpy(rng.standard_normal(n).astype(np.float32)))
        views["g"][-1].copy_(torch.from_numpy(rng.standard_normal(n).astype(np.float32) * 1e-3))
        views["m"][-1].zero_()
        views["v"][-1].zero_()
        off += n + gap
        off = (off + 3) // 4 * 4  # keep every tensor 16-byte aligned
    canary = {k: bufs[k].clone() for k in "xgmv"}
    mask = torch.ones(total, dtype=torch.bool, device="cuda")
    for k in "xgmv":
        for v in views[k]:
            start = (v.data_ptr() - bufs[k].data_ptr()) // 4
            mask[start:start + v.numel()] = False
    rows = [(views["x"][i].data_ptr(), views["g"][i].data_ptr(), views["m"][i].data_ptr(),
             views["v"][i].data_ptr(), sizes[i], 1) for i in range(len(sizes))]
    with H.create_plan(rows, _lib.LAMB_GRAD_F32, _lib.LAMB_ALGO_LAMB, 8, path) as plan:
        for t in range(1, 4):
            _lib.lamb_step(plan, 0.01, 0.9, 0.999, 1e-6, 0.01, 0.0, 10.0, t, True,
                           torch.cuda.current_stream().cuda_stream)
        _lib.lamb_plan_check(plan)
        torch.cuda.synchronize()
    for k in "xgmv":
        assert torch.equal(bufs[k][mask], canary[k][mask]), "canary overwritten in " + k
    assert not torch.equal(bufs["x"], canary["x"])


def test_validation_leaves_state_untouched():
    torch = H.torch_cuda()
    rng = np.random.default_rng(12)
    pair = H.Pair(_xs(rng, [100]), [True], "f32", "lamb")
    lars = H.Pair(_xs(rng, [100]), [True], "f32", "lars")
    try:
        pair.set_grads(_gs(rng, [100]))
        x0 = pair.X[0].clone()
        s = torch.cuda.current_stream().cuda_stream
        bad = [
            dict(step=0), dict(beta1=1.0), dict(beta2=-0.1), dict(eps=-1e-6),
            dict(lr=float("nan")), dict(weight_decay=float("inf")), dict(gamma_l=2.0, gamma_u=1.0),
            dict(gamma_l=-1.0), dict(gamma_u=float("nan")), dict(bias_correction=2),
        ]
        for b in bad:
            a = dict(DEFAULT, step=1, bias_correction=1)
            a.update(b)
            with pytest.raises(_lib.LambError) as e:
                _lib.load()
                st = _lib.load().lamb_step(_lib._vp(pair.plan.handle), a["lr"], a["beta1"],
                                          a["beta2"], a["eps"], a["weight_decay"], a["gamma_l"],
                                          a["gamma_u"], a["step"], a["bias_correction"],
                                          _lib._vp(s), None, None)
                _lib._check(st, "lamb_step")
            assert e.value.status == _lib.LAMB_EINVAL, b
        with pytest.raises(_lib.LambError) as e:
            _lib.lars_step(pair.plan, 0.01, 0.9, 0.01, 0.0, 10.0, 0.01, s)
        assert e.value.status == _lib.LAMB_EPLAN
        with pytest.raises(_lib.LambError) as e:
            _lib.lamb_step(lars.plan, 0.01, 0.9, 0.999, 1e-6, 0.01, 0.0, 10.0, 1, True, s)
        assert e.value.status == _lib.LAMB_EPLAN
        with pytest.raises(_lib.LambError) as e:
            _lib.nlamb_step(lars.plan, 0.01, 0.975, 0.999, 1e-8, 0.01, 0.0, 10.0, 1, True, s)
        assert e.value.status == _lib.LAMB_EPLAN
        with pytest.raises(_lib.LambError) as e:
            _lib.nlamb_step(pair.plan, 0.01, 0.975, 0.999, 1e-8, 0.01, 0.0, 10.0, 0, True, s)
        assert e.value.status == _lib.LAMB_EINVAL
        with pytest.raises(_lib.LambError) as e:
            _lib.lars_step(lars.plan, 0.01, 1.5, 0.01, 0.0, 10.0, 0.01, s)
        assert e.value.status == _lib.LAMB_EINVAL
        torch.cuda.synchronize()
        assert torch.equal(pair.X[0], x0)
        assert not torch.any(pair.M[0] != 0)
    finally:
        pair.close()
        lars.close()


def test_tensor_beyond_int32_elements():
    """One tensor of 2^31 + 1029 elements (8 GiB per fp32 array), so chunk
    starts pass 2^31. With constant x = c and g = a, every u_j equals the
    same value, so ||x|| = |c| sqrt(d), ||u|| = |u| sqrt(d) and the step is
    x - lr * phi / sqrt(d) * sign(u) for every element; each element of x,
    m, v is checked against that closed form (Algorithm 2), which also
    shows every element was updated exactly once."""
    torch = H.torch_cuda()
    d = (1 << 31) + 1029
    c, a = 0.02, 1e-3
    lr, b1, b2, eps, lam = 6e-3, 0.9, 0.999, 1e-6, 0.01
    H.log("int64 tensor: %d elements" % d)
    x = torch.full((d,), c, dtype=torch.float32, device="cuda")
    g = torch.full((d,), a, dtype=torch.bfloat16, device="cuda")
    m = torch.zeros_like(x)
    v = torch.zeros_like(x)
    ratio = torch.zeros(1, dtype=torch.float64, device="cuda")
    norms = torch.zeros(2, dtype=torch.float64, device="cuda")
    rows = [(x.data_ptr(), g.data_ptr(), m.data_ptr(), v.data_ptr(), d, 1)]
    with _lib.lamb_plan_create(rows, _lib.LAMB_GRAD_BF16, _lib.LAMB_ALGO_LAMB, 0) as plan:
        _lib.lamb_step(plan, lr, b1, b2, eps, lam, 0.0, 10.0, 1, True,
                       torch.cuda.current_stream().cuda_stream, ratio.data_ptr(), norms.data_ptr())
        torch.cuda.synchronize()
    f = lambda z: float(np.float32(z))  # noqa: E731  (scalars as the ABI receives them)
    X, G = f(c), float(torch.tensor(a, dtype=torch.bfloat16).float())
    M, V = (1 - f(b1)) * G, (1 - f(b2)) * G * G          # step 1 from zero moments
    u = (M / (1 - f(b1))) / (np.sqrt(V / (1 - f(b2))) + f(eps)) + f(lam) * X
    phi = min(abs(X) * np.sqrt(d), 10.0)
    want_ratio = phi / (abs(u) * np.sqrt(d))
    assert abs(float(ratio) - want_ratio) <= 1e-6 * want_ratio
    assert abs(float(norms[0]) - abs(X) * np.sqrt(d)) <= 1e-9 * abs(X) * np.sqrt(d)
    want_x = X - f(lr) * want_ratio * u
    for name, t, want in (("x", x, want_x), ("m", m, M), ("v", v, V)):
        lo, hi = float(t.min()), float(t.max())
        assert abs(lo - want) <= 1e-6 * abs(want) and abs(hi - want) <= 1e-6 * abs(want), \
            (name, lo, hi, want)
    del x, g, m, v
    torch.cuda.empty_cache()


def test_subnormal_and_zero_gradients():
    """bf16 and fp32 gradients that are subnormal or exactly zero (with the
    paper's eps > 0): the step stays finite and matches the oracle.

    The second tensor's first moment m_t = (1 - beta1) g ~ 3e-40 is an fp32
    subnormal: the kernel derives u from the stored fp32 m_t, whose spacing
    there is 2^-149, so the per-tensor ratio may move by half that spacing
    relative to |m_t| on top of the usual bound."""
    torch = H.torch_cuda()
    rng = np.random.default_rng(13)
    for g_dtype in ("f32", "bf16"):
        xs = _xs(rng, [300, 64])
        g0 = torch.from_numpy((rng.standard_normal(300) * 1e-3).astype(np.float32))
        g0[::7] = 0.0
        g0[1::7] = 1e-40          # fp32 subnormal (bf16 keeps its top half)
        g1 = torch.full((64,), 3e-39)
        gs = [g0, g1] if g_dtype == "f32" else [g0.to(torch.bfloat16), g1.to(torch.bfloat16)]
        tol = H.RATIO_TOL + 2.0 ** -150 / (0.1 * float(gs[1][0].float()))
        _run(xs, [True, False], g_dtype, "lamb", 64, 3, DEFAULT, rng, grads=lambda t: gs,
             ratio_tol=tol)


@pytest.mark.parametrize("groups", [8, 10])
def test_single_pass_layout_and_rounds(groups):
    """The single pass runs in rounds of one workgroup per tile, four per CU.
    A layer of exactly one round of tiles takes it whole; a layer of one
    element more than a round of the wider tile puts its last round (from a
    multiple of 1024 elements) on it and its head on the two-pass kernels; layers
    that leave a gap in a round (padded with empty entries) and a layer that
    fills the last round still match the oracle on every element. With a
    layer that only the 10240-element tile fits in a round, the plan picks
    that tile; without one it keeps the 8192-element tile."""
    torch = H.torch_cuda()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    R, T, W = 4 * cus, 1024 * groups, 10240
    sizes = [R * T, R * W + 1, int(0.68 * R) * T - 3, int(0.39 * R) * T + 5, int(0.29 * R) * T,
             30 * T - 1, 100, 7]
    if groups == 10:
        sizes.append(R * 8192 + 1)  # fits a round of the wide tile only
    rng = np.random.default_rng(21)
    xs = _xs(rng, sizes)
    wd = [i % 2 == 0 for i in range(len(sizes))]
    H.log("single-pass rounds: R=%d groups=%d sizes=%s" % (R, groups, sizes))
    pair = H.Pair(xs, wd, "bf16", "lamb", path="auto")
    try:
        per, total, got, elems = _lib.lamb_plan_tiles(pair.plan, True)
        assert got == groups
        head = -(-(sizes[1] - R * T) // 1024) * 1024
        want_elems = list(sizes)
        want_elems[1] = sizes[1] - head
        assert elems == want_elems and 0 < want_elems[1] <= R * T
        want = [(n + T - 1) // T for n in want_elems]
        assert per == want
        assert total >= sum(want)
        for t in range(1, 3):
            gs = _gs(rng, sizes, "bf16")
            hg = pair.set_grads(gs)
            ref = H.step_both(pair, "lamb", hg, DEFAULT, t)
            pair.compare(ref, "rounds groups %d step %d" % (groups, t))
    finally:
        pair.close()


@pytest.mark.parametrize("path", PATHS)
def test_many_small_layers(path):
    """3000 layers of 1 to 300 elements plus two multi-tile layers: rounds
    filled mostly with one-tile layers, against the oracle on every
    element."""
    rng = np.random.default_rng(41)
    sizes = [int(v) for v in rng.integers(1, 301, size=3000)] + [5 * 8192 + 11, 2 * 8192]
    xs = _xs(rng, sizes)
    wd = [bool(v) for v in rng.integers(0, 2, size=len(sizes))]
    H.log("many small layers: %d layers, path %s" % (len(sizes), path))
    _run(xs, wd, "bf16", "lamb", 0, 2, DEFAULT, rng, path=path)
