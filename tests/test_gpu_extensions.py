"""lamb_step_ex against the oracle: the layer norms of Appendix F, gradient
scaling (the 1/|S_t| of Algorithms 1-2, or a loss scale), and the deferred
mode that skips a step whose scaled gradient is not finite."""

import numpy as np
import pytest

import gpu_harness as H
from paper_1904_00962_amd import _lib, paramsets

pytestmark = pytest.mark.gpu

ALGOS = ["lamb", "n-lamb", "nn-lamb", "lars"]


def _hp(algo, **kw):
    base = dict(lr=1e-2, weight_decay=0.01, gamma_l=0.0, gamma_u=10.0)
    if algo == "lars":
        base.update(trust_coef=0.01)
    base.update(kw)
    return _lib.lamb_hparams_init(algo, **base)


def _pair(xs, wd, g_dtype, algo, chunk=0, path="auto"):
    return H.Pair(xs, wd, g_dtype, "lars" if algo == "lars" else "lamb", chunk, path=path)


def _grads(rng, xs, g_dtype, scale=1e-3):
    import torch
    out = []
    for x in xs:
        t = torch.from_numpy((rng.standard_normal(len(x)) * scale).astype(np.float32))
        out.append(t.to(torch.bfloat16) if g_dtype == "bf16" else t)
    return out


@pytest.mark.parametrize("algo", ALGOS)
@pytest.mark.parametrize("norm", ["l1", "linf"])
def test_other_norms(algo, norm):
    """Tiny set and ragged sizes with the L1 and L-infinity layer norms."""
    ps = paramsets.get(0)
    rng = np.random.default_rng(7)
    ragged = [(rng.standard_normal(n) * 0.3).astype(np.float32)
              for n in (1, 3, 5, 64, 257, 1023, 2049, 4097, 3 * 8192 + 3)]
    rwd = [i % 2 == 0 for i in range(len(ragged))]
    for xs, wd, g_dtype, chunk, path in ((paramsets.draw_params(ps), ps.wd_mask(), "f32", 0, "auto"),
                                         (ragged, rwd, "bf16", 64, "two-pass"),
                                         (ragged, rwd, "bf16", 0, "auto"),
                                         (ragged, rwd, "f32", 0, "wide")):
        H.log("norm=%s algo=%s tensors=%d chunk=%d path=%s" % (norm, algo, len(xs), chunk, path))
        pair = _pair(xs, wd, g_dtype, algo, chunk, path)
        try:
            for t in range(1, 4):
                hg = pair.set_grads(_grads(rng, pair.X, g_dtype))
                ref = H.step_ex_both(pair, _hp(algo, step=t, norm=norm), hg)
                pair.compare(ref, "%s %s step %d" % (norm, algo, t))
        finally:
            pair.close()


@pytest.mark.parametrize("algo", ["lamb", "nn-lamb", "lars"])
@pytest.mark.parametrize("scale,g_mult", [(0.125, 1.0), (0.37, 1.0), (1.0 / 65536, 65536.0)])
def test_grad_scale(algo, scale, g_mult):
    """g_t = grad_scale * g: a mean over summed gradients (0.125), an arbitrary
    factor, and a loss scale of 2^16 undone by grad_scale."""
    ps = paramsets.get(3)
    rng = np.random.default_rng(8)
    sample = [0, 1, 2, 10, 11, ps.n_tensors - 2, ps.n_tensors - 1]
    xs = paramsets.draw_params(ps, indices=sample)
    wd = [ps.wd_mask()[i] for i in sample]
    pair = _pair(xs, wd, "bf16", algo)
    try:
        for t in range(1, 4):
            hg = pair.set_grads(_grads(rng, pair.X, "bf16", 1e-3 * g_mult))
            ref = H.step_ex_both(pair, _hp(algo, step=t, grad_scale=scale), hg)
            pair.compare(ref, "scale %g %s step %d" % (scale, algo, t))
    finally:
        pair.close()


@pytest.mark.parametrize("algo", ALGOS)
def test_deferred_mode_equals_direct_mode(algo):
    """With finite gradients, the deferred mode (moment pass over chunks 8x as
    large, moments written by the apply pass) gives bit for bit the x, m, v
    and ratios of the direct mode on a plan with 8x larger chunks."""
    torch = H.torch_cuda()
    ps = paramsets.get(3)
    xs = paramsets.draw_params(ps, device="cuda")
    runs = []
    for skip, chunk in ((0, 2048), (1, 256)):
        pair = _pair([x.clone() for x in xs], ps.wd_mask(), "f32", algo, chunk, "two-pass")
        pair.subset = []
        flag = torch.zeros(1, dtype=torch.int32, device="cuda")
        for t in range(1, 4):
            for G, g in zip(pair.G, paramsets.draw_grads(ps, t, device="cuda")):
                G.copy_(g)
            _lib.lamb_step_ex(pair.plan, _hp(algo, step=t, skip_nonfinite=skip),
                              torch.cuda.current_stream().cuda_stream, pair.ratio.data_ptr(),
                              pair.norms.data_ptr(), flag.data_ptr() if skip else 0)
        torch.cuda.synchronize()
        runs.append(([x.clone() for x in pair.X], [m.clone() for m in pair.M],
                     [v.clone() for v in pair.V] if pair.V else [], pair.ratio.clone(), int(flag)))
        pair.close()
    (x0, m0, v0, r0, _), (x1, m1, v1, r1, f1) = runs
    assert f1 == 0
    assert all(torch.equal(a, b) for a, b in zip(x0 + m0 + v0, x1 + m1 + v1))
    assert torch.equal(r0, r1)


@pytest.mark.parametrize("path", ["auto", "wide", "two-pass"])
@pytest.mark.parametrize("algo", ALGOS)
@pytest.mark.parametrize("g_dtype", ["f32", "bf16"])
def test_skip_nonfinite_sequence(algo, g_dtype, path):
    """Finite and non-finite steps interleaved: a skipped step changes nothing
    (bit for bit) and reports 1; the next finite step proceeds as the oracle
    does. Covers +inf, NaN and an fp32 overflow caused by grad_scale. On the
    single pass the verdict comes from a read-only check of g; on the
    two-pass path from the deferred moment pass. The last layer has three
    tiles, so its tiles meet through the slots, which a skipped step must
    leave ready for the next one."""
    torch = H.torch_cuda()
    rng = np.random.default_rng(9)
    xs = [(rng.standard_normal(n) * 0.2).astype(np.float32)
          for n in (700, 33, 4096, 5, 3 * 8192 + 77)]
    pair = _pair(xs, [True, False, True, True, True], g_dtype, algo, chunk=256, path=path)
    flag = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    plan_steps = [("ok", 1.0), ("inf", 1.0), ("ok", 1.0), ("nan", 1.0), ("ok", 1.0),
                  ("overflow", 3e38), ("overflow", 3e38), ("ok", 1.0)]
    t = 0
    try:
        for k, (kind, scale) in enumerate(plan_steps):
            gs = _grads(rng, pair.X, g_dtype)
            if kind == "inf":
                gs[2][1234] = float("inf")
            elif kind == "nan":
                gs[0][0] = float("nan")
            elif kind == "overflow":  # finite values whose fp32 product with scale overflows
                gs[3][2] = 2.0
            hg = pair.set_grads(gs)
            before = [x.clone() for x in pair.X] + [m.clone() for m in pair.M]
            t += 1
            ref = H.step_ex_both(pair, _hp(algo, step=t, grad_scale=scale, skip_nonfinite=1),
                                 hg, flag)
            pair.compare(ref, "%s %s step %d (%s)" % (algo, g_dtype, k, kind))
            torch.cuda.synchronize()
            skipped = bool(np.all(np.isnan(ref)))
            assert int(flag) == int(skipped), (k, kind, int(flag))
            after = [x for x in pair.X] + [m for m in pair.M]
            if skipped:
                assert all(torch.equal(a, b) for a, b in zip(before, after))
            assert skipped == (kind != "ok")
    finally:
        pair.close()


@pytest.mark.parametrize("path", ["auto", "wide"])
def test_skip_nonfinite_with_two_pass_layer(path):
    """The single-pass skip mode with a layer larger than one round (with
    either tile): its head takes a moment pass before the single pass and an
    apply pass after it, and the check's verdict stops both, the apply pass
    through the copy the totals kernel takes (the single pass rewrites the
    epoch's verdict words as it ends)."""
    torch = H.torch_cuda()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    big = 4 * cus * 10240 + 1029
    rng = np.random.default_rng(19)
    xs = [(rng.standard_normal(n) * 0.2).astype(np.float32) for n in (big, 3000, 7)]
    pair = _pair(xs, [True, True, False], "bf16", "lamb", path=path)
    flag = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    try:
        per, _, _, elems = _lib.lamb_plan_tiles(pair.plan, True)
        assert 0 < elems[0] < big and elems[1:] == [3000, 7] and min(per) > 0
        for t, kind in enumerate(["ok", "nan_big", "ok", "inf_small", "ok"], start=1):
            gs = _grads(rng, pair.X, "bf16")
            if kind == "nan_big":
                gs[0][big - 3] = float("nan")
            elif kind == "inf_small":
                gs[2][6] = float("inf")
            hg = pair.set_grads(gs)
            before = [x.clone() for x in pair.X + pair.M + pair.V]
            ref = H.step_ex_both(pair, _hp("lamb", step=t, skip_nonfinite=1), hg, flag)
            pair.compare(ref, "skip with a two-pass layer, step %d (%s)" % (t, kind))
            torch.cuda.synchronize()
            assert int(flag) == int(kind != "ok")
            if kind != "ok":
                after = pair.X + pair.M + pair.V
                assert all(torch.equal(a, b) for a, b in zip(before, after))
    finally:
        pair.close()


@pytest.mark.parametrize("algo", ["lamb", "nn-lamb", "lars"])
def test_checked_skip_mode_equals_direct_mode(algo):
    """With finite gradients, a skip_nonfinite step on the single pass runs
    the direct kernels after the check: bit for bit the direct step."""
    torch = H.torch_cuda()
    ps = paramsets.get(3)
    xs = paramsets.draw_params(ps, device="cuda")
    runs = []
    for skip in (0, 1):
        pair = _pair([x.clone() for x in xs], ps.wd_mask(), "f32", algo, 0, "auto")
        pair.subset = []
        flag = torch.zeros(1, dtype=torch.int32, device="cuda")
        for t in range(1, 4):
            for G, g in zip(pair.G, paramsets.draw_grads(ps, t, device="cuda")):
                G.copy_(g)
            _lib.lamb_step_ex(pair.plan, _hp(algo, step=t, skip_nonfinite=skip),
                              torch.cuda.current_stream().cuda_stream, pair.ratio.data_ptr(),
                              pair.norms.data_ptr(), flag.data_ptr() if skip else 0)
        _lib.lamb_plan_check(pair.plan)
        runs.append(([x.clone() for x in pair.X], [m.clone() for m in pair.M],
                     [v.clone() for v in pair.V] if pair.V else [], pair.ratio.clone(), int(flag)))
        pair.close()
    (x0, m0, v0, r0, _), (x1, m1, v1, r1, f1) = runs
    assert f1 == 0
    assert all(torch.equal(a, b) for a, b in zip(x0 + m0 + v0, x1 + m1 + v1))
    assert torch.equal(r0, r1)


def _with(hp, **fields):
    for k, v in fields.items():
        setattr(hp, k, v)
    return hp


def test_step_ex_validation():
    torch = H.torch_cuda()
    rng = np.random.default_rng(10)
    lamb = _pair([rng.standard_normal(64).astype(np.float32)], [True], "f32", "lamb")
    lars = _pair([rng.standard_normal(64).astype(np.float32)], [True], "f32", "lars")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    try:
        x0 = lamb.X[0].clone()
        cases = [
            (lamb, _hp("lars"), 0, _lib.LAMB_EPLAN),
            (lars, _hp("lamb"), 0, _lib.LAMB_EPLAN),
            (lamb, _hp("lamb", norm=3), 0, _lib.LAMB_EINVAL),
            (lamb, _with(_hp("lamb"), variant=7), 0, _lib.LAMB_EINVAL),
            (lamb, _hp("lamb", reserved=1), 0, _lib.LAMB_EINVAL),
            (lamb, _hp("lamb", grad_scale=float("inf")), 0, _lib.LAMB_EINVAL),
            (lamb, _hp("lamb"), flag.data_ptr(), _lib.LAMB_EINVAL),  # flag without skip
            (lamb, _hp("lamb", skip_nonfinite=2), 0, _lib.LAMB_EINVAL),
            (lamb, _hp("n-lamb", bias_correction=0), 0, _lib.LAMB_EINVAL),
            (lamb, _hp("lamb", step=0), 0, _lib.LAMB_EINVAL),
            (lars, _hp("lars", beta1=1.0), 0, _lib.LAMB_EINVAL),
            (lars, _hp("lars", trust_coef=float("nan")), 0, _lib.LAMB_EINVAL),
        ]
        for pair, hp, out, status in cases:
            with pytest.raises(_lib.LambError) as e:
                _lib.lamb_step_ex(pair.plan, hp, s, 0, 0, out)
            assert e.value.status == status
        torch.cuda.synchronize()
        assert torch.equal(lamb.X[0], x0)
    finally:
        lamb.close()
        lars.close()


def _bf16_bits(t):
    import torch
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("algo,skip,g_dtype,path", [
    ("lamb", 0, "bf16", "auto"), ("lamb", 0, "bf16", "two-pass"), ("nn-lamb", 0, "f32", "auto"),
    ("lars", 0, "f32", "auto"), ("lars", 1, "bf16", "auto"), ("lamb", 1, "f32", "auto"),
    ("lamb", 0, "bf16", "wide"), ("lars", 1, "f32", "wide")])
def test_bf16_copies(algo, skip, g_dtype, path):
    """The apply pass writes bf16(x_{t+1}): bit for bit torch's cast of the
    GPU's own x, within one bf16 ulp of the oracle's rounding of the oracle's
    x; a tensor without a copy is unaffected; x, m, v still match the oracle."""
    torch = H.torch_cuda()
    rng = np.random.default_rng(11)
    sizes = [1, 3, 8, 255, 513, 1029, 4097, 70000]
    xs = [(rng.standard_normal(n) * 0.5).astype(np.float32) for n in sizes]
    pair = _pair(xs, [i % 2 == 0 for i in range(len(sizes))], g_dtype, algo, 256, path)
    copies = [torch.full((n,), 12345, dtype=torch.int16, device="cuda").view(torch.bfloat16)
              for n in sizes]
    copies[2] = None
    _lib.lamb_plan_set_bf16_copies(pair.plan, [c.data_ptr() if c is not None else 0
                                               for c in copies])
    try:
        for t in range(1, 4):
            hg = pair.set_grads(_grads(rng, pair.X, g_dtype))
            ref = H.step_ex_both(pair, _hp(algo, step=t, skip_nonfinite=skip), hg)
            pair.compare(ref, "bf16 copy %s step %d" % (algo, t))
            for i, c in enumerate(copies):
                if c is None:
                    continue
                got = _bf16_bits(c)
                assert np.array_equal(got, _bf16_bits(pair.X[i].to(torch.bfloat16)))
                want = pair.oracle.round_bf16(pair.hx[i])
                assert np.all(np.abs(got.astype(np.int32) - want.astype(np.int32)) <= 1)
    finally:
        pair.close()


@pytest.mark.parametrize("path", ["auto", "wide", "two-pass"])
def test_bf16_copy_guard_bands_and_detach(path):
    torch = H.torch_cuda()
    rng = np.random.default_rng(12)
    sizes = [5, 1000, 33]
    xs = [(rng.standard_normal(n)).astype(np.float32) for n in sizes]
    pair = _pair(xs, [True] * 3, "f32", "lamb", 64, path)
    gap = 64
    buf = torch.full((sum(sizes) + gap * 4,), -3, dtype=torch.int16, device="cuda")
    views, off = [], gap
    for n in sizes:
        views.append(buf[off:off + n].view(torch.bfloat16))
        off = (off + n + gap + 7) // 8 * 8
    mask = torch.ones(buf.numel(), dtype=torch.bool, device="cuda")
    for v in views:
        k = (v.data_ptr() - buf.data_ptr()) // 2
        mask[k:k + v.numel()] = False
    before = buf.clone()
    try:
        _lib.lamb_plan_set_bf16_copies(pair.plan, [v.data_ptr() for v in views])
        pair.set_grads(_grads(rng, pair.X, "f32"))
        H.step_ex_both(pair, _hp("lamb", step=1), [paramsets.host_array(g) for g in pair.G])
        torch.cuda.synchronize()
        assert torch.equal(buf[mask], before[mask])
        assert not torch.equal(buf[~mask], before[~mask])
        _lib.lamb_plan_set_bf16_copies(pair.plan, None)
        snap = buf.clone()
        H.step_ex_both(pair, _hp("lamb", step=2), [paramsets.host_array(g) for g in pair.G])
        torch.cuda.synchronize()
        assert torch.equal(buf, snap)
        with pytest.raises(_lib.LambError) as e:  # misaligned
            _lib.lamb_plan_set_bf16_copies(pair.plan, [views[0].data_ptr() + 2, 0, 0])
        assert e.value.status == _lib.LAMB_EALIGN
        with pytest.raises(_lib.LambError) as e:  # copy over x
            _lib.lamb_plan_set_bf16_copies(pair.plan, [pair.X[1].data_ptr(), 0, 0])
        assert e.value.status == _lib.LAMB_EOVERLAP
        with pytest.raises(_lib.LambError) as e:  # two copies share memory
            _lib.lamb_plan_set_bf16_copies(pair.plan, [views[1].data_ptr(), views[1].data_ptr(), 0])
        assert e.value.status == _lib.LAMB_EOVERLAP
    finally:
        pair.close()
