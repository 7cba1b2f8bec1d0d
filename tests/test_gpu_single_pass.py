"""The single-pass kernel beside the two-pass kernels and its failure path.

m and v are elementwise, so both paths give them bit for bit; the layer norms
are summed in a different order, so x and the ratios agree to rounding. A
wait that runs out of polls must be reported and must leave later steps
inert; the poll budget is cut to one from the host so that the give-up
happens at once, with every wait still bounded."""

import numpy as np
import pytest

import gpu_harness as H
from paper_1904_00962_amd import _lib, paramsets

pytestmark = pytest.mark.gpu


def _run_path(cfg, path, steps=2):
    ps = paramsets.get(cfg)
    pair = H.Pair(paramsets.draw_params(ps, device="cuda"), ps.wd_mask(), ps.g_dtype, "lamb",
                  oracle_subset=[], path=path)
    hp = H.lamb_hp(ps)
    for t in range(1, steps + 1):
        pair.set_grads(paramsets.draw_grads(ps, t, device="cuda"))
        pair.gpu_lamb(hp, t)
    _lib.lamb_plan_check(pair.plan)
    state = ([x.clone() for x in pair.X], [m.clone() for m in pair.M],
             [v.clone() for v in pair.V], pair.ratio.clone(), pair.norms.clone())
    pair.close()
    return state


@pytest.mark.parametrize("path", ["auto", "wide"])
def test_single_pass_agrees_with_two_pass(path):
    """BERT-Base: 198 layers on the single pass (with either tile) and the
    token embedding split between the two paths, against the two-pass path
    for everything."""
    torch = H.torch_cuda()
    x1, m1, v1, r1, n1 = _run_path(1, path)
    x2, m2, v2, r2, n2 = _run_path(1, "two-pass")
    assert all(torch.equal(a, b) for a, b in zip(m1 + v1, m2 + v2))
    for k, (a, b) in enumerate(zip(x1, x2)):
        H.compare_state(a.cpu().numpy(), b.cpu().numpy(), "x[%d]" % k)
    H.compare_ratios(r1.cpu().numpy(), r2.cpu().numpy(), "ratio")
    H.compare_ratios(n1.cpu().numpy(), n2.cpu().numpy(), "norms")


def test_abandoned_wait_is_reported(monkeypatch):
    """With a budget of one poll, a tile that finds its layer's scale not yet
    published gives up: the plan reports LAMB_ESYNC and its later steps change
    nothing. A plan built with the normal budget is unaffected."""
    torch = H.torch_cuda()
    rng = np.random.default_rng(31)
    sizes = [200 * 8192, 150 * 8192 + 3, 77]
    xs = [(rng.standard_normal(n) * 0.5).astype(np.float32) for n in sizes]
    monkeypatch.setenv("LAMB_MI355X_SPIN_LIMIT", "1")
    pair = H.Pair(xs, [True, True, False], "f32", "lamb", path="auto")
    monkeypatch.delenv("LAMB_MI355X_SPIN_LIMIT")
    try:
        grads = [torch.from_numpy((rng.standard_normal(n) * 1e-3).astype(np.float32))
                 for n in sizes]
        pair.set_grads(grads)
        pair.gpu_lamb(H.lamb_hp(paramsets.get(0)), 1)
        with pytest.raises(_lib.LambError) as e:
            _lib.lamb_plan_check(pair.plan)
        assert e.value.status == _lib.LAMB_ESYNC
        before = [t.clone() for t in pair.X + pair.M + pair.V]
        pair.gpu_lamb(H.lamb_hp(paramsets.get(0)), 2)
        torch.cuda.synchronize()
        after = pair.X + pair.M + pair.V
        # the single pass does nothing once the plan has given up a wait
        for k in range(2):
            for grp in (0, 3, 6):
                assert torch.equal(before[grp + k], after[grp + k])
    finally:
        pair.close()
    # a fresh plan with the normal budget still steps and matches the oracle
    pair = H.Pair(xs, [True, True, False], "f32", "lamb", path="auto")
    try:
        hg = pair.set_grads(grads)
        ref = H.step_both(pair, "lamb", hg, H.lamb_hp(paramsets.get(0)), 1)
        pair.compare(ref, "after a give-up")
    finally:
        pair.close()


def test_single_pass_beside_other_work():
    """Single-pass steps while another stream keeps the GPU busy with large
    fp32 matrix products. The persistent grid needs every workgroup resident
    at once, which work on another stream can withhold (a library's matrix
    product may itself run as a persistent grid that waits for residency):
    the contract is that every wait ends, and that a step either completes
    and matches the oracle, or gives up, reports LAMB_ESYNC and leaves the
    plan inert, after which a new plan on an idle device matches the
    oracle."""
    torch = H.torch_cuda()
    ps = paramsets.get(1)
    subset = [0, 3, 4, 5, 6, 7, 8, ps.n_tensors - 1]
    pair = H.Pair(paramsets.draw_params(ps, device="cuda"), ps.wd_mask(), ps.g_dtype, "lamb",
                  oracle_subset=subset, path="auto")
    side = torch.cuda.Stream()
    a = torch.randn(4096, 4096, device="cuda")
    b = torch.randn(4096, 4096, device="cuda")
    gave_up = False
    try:
        hp = H.lamb_hp(ps)
        for t in range(1, 4):
            hg = pair.set_grads(paramsets.draw_grads(ps, t, device="cuda"))
            torch.cuda.synchronize()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                for _ in range(6):
                    c = torch.mm(a, b)
            pair.gpu_lamb(hp, t)
            ref = pair.oracle_lamb(hg, hp, t)
            torch.cuda.current_stream().wait_stream(side)
            try:
                pair.compare(ref, "beside other work, step %d" % t)
            except _lib.LambError as e:
                assert e.status == _lib.LAMB_ESYNC, e
                H.log("  step %d gave up a wait beside the matrix products (LAMB_ESYNC)" % t)
                gave_up = True
                before = [x.clone() for x in pair.X + pair.M + pair.V]
                pair.gpu_lamb(hp, t + 1)
                torch.cuda.synchronize()
                assert all(torch.equal(u, w) for u, w in zip(before, pair.X + pair.M + pair.V))
                break
        torch.cuda.synchronize()
        del c
    finally:
        pair.close()
    if gave_up:
        fresh = H.Pair(paramsets.draw_params(ps, device="cuda"), ps.wd_mask(), ps.g_dtype,
                       "lamb", oracle_subset=subset, path="auto")
        try:
            hg = fresh.set_grads(paramsets.draw_grads(ps, 1, device="cuda"))
            fresh.compare(H.step_both(fresh, "lamb", hg, H.lamb_hp(ps), 1), "after a give-up")
        finally:
            fresh.close()


@pytest.mark.parametrize("value", ["9", "8x", "", "-10"])
def test_tile_override_rejects_other_values(monkeypatch, value):
    """The tile override takes 8 or 10; anything else fails plan creation with
    LAMB_EINVAL and a message naming the variable, and creates nothing."""
    torch = H.torch_cuda()
    x = torch.zeros(4096, device="cuda")
    g = torch.zeros(4096, device="cuda")
    m = torch.zeros(4096, device="cuda")
    v = torch.zeros(4096, device="cuda")
    rows = [(x.data_ptr(), g.data_ptr(), m.data_ptr(), v.data_ptr(), 4096, 1)]
    monkeypatch.setenv(H.TILE_ENV, value)
    with pytest.raises(_lib.LambError) as e:
        _lib.lamb_plan_create(rows, _lib.LAMB_GRAD_F32, _lib.LAMB_ALGO_LAMB, 0)
    assert e.value.status == _lib.LAMB_EINVAL
    assert H.TILE_ENV in _lib.last_error()
    for ok, groups in (("8", 8), ("10", 10)):
        monkeypatch.setenv(H.TILE_ENV, ok)
        with _lib.lamb_plan_create(rows, _lib.LAMB_GRAD_F32, _lib.LAMB_ALGO_LAMB, 0) as plan:
            assert _lib.lamb_plan_tiles(plan)[2] == groups


@pytest.mark.parametrize("value", ["abc", "0", "-5", "12 "])
def test_spin_limit_rejects_other_values(monkeypatch, value):
    """The spin limit takes a positive integer; anything else fails plan
    creation with LAMB_EINVAL instead of silently becoming a one-poll budget."""
    torch = H.torch_cuda()
    bufs = [torch.zeros(4096, device="cuda") for _ in range(4)]
    rows = [tuple(b.data_ptr() for b in bufs) + (4096, 1)]
    monkeypatch.setenv("LAMB_MI355X_SPIN_LIMIT", value)
    with pytest.raises(_lib.LambError) as e:
        _lib.lamb_plan_create(rows, _lib.LAMB_GRAD_F32, _lib.LAMB_ALGO_LAMB, 0)
    assert e.value.status == _lib.LAMB_EINVAL
    assert "LAMB_MI355X_SPIN_LIMIT" in _lib.last_error()
    monkeypatch.setenv("LAMB_MI355X_SPIN_LIMIT", "1000")
    with _lib.lamb_plan_create(rows, _lib.LAMB_GRAD_F32, _lib.LAMB_ALGO_LAMB, 0):
        pass


def test_trace_stamps_every_tile_and_changes_nothing():
    """With the trace on, every tile of the schedule gets four ordered stamps,
    and the step's results equal an untraced plan's bit for bit."""
    torch = H.torch_cuda()
    ps = paramsets.get(1)
    xs = paramsets.draw_params(ps, device="cuda")
    pairs = [H.Pair([x.clone() for x in xs], ps.wd_mask(), ps.g_dtype, "lamb", oracle_subset=[])
             for _ in range(2)]
    try:
        per, n_tiles, groups, elems = _lib.lamb_plan_tiles(pairs[1].plan, True)
        cus = torch.cuda.get_device_properties(0).multi_processor_count
        et = _lib.lamb_tile_schedule(elems, 4 * cus, groups)[0]
        stamps = torch.zeros(4 * n_tiles, dtype=torch.int64, device="cuda")
        _lib.lamb_plan_set_trace(pairs[1].plan, stamps.data_ptr())
        for t in (1, 2):
            grads = paramsets.draw_grads(ps, t, device="cuda")
            for p in pairs:
                p.set_grads(grads)
                p.gpu_lamb(H.lamb_hp(ps), t)
        _lib.lamb_plan_set_trace(pairs[1].plan, 0)
        torch.cuda.synchronize()
        for a, b in zip(pairs[0].X + pairs[0].M + pairs[0].V, pairs[1].X + pairs[1].M + pairs[1].V):
            assert torch.equal(a, b)
        assert torch.equal(pairs[0].ratio, pairs[1].ratio)
        s = stamps.cpu().numpy().reshape(-1, 4)
        real = np.asarray(et) >= 0
        assert np.all(s[real] > 0) and np.all(s[~real] == 0)
        assert np.all(np.diff(s[real], axis=1) >= 0)
        # one step's stamps lie within a second
        assert s[real].max() - s[real].min() < 100_000_000
    finally:
        for p in pairs:
            p.close()
