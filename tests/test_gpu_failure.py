"""Failure handling through the optimizer facade.

A single-pass wait that gives up is forced from the host (a poll budget of
one, read at plan creation), so every kernel still exits normally. The
facade must surface it (LAMB_ESYNC) within check_every steps and in
state_dict(); after it no layer may move, the two-pass ones included; a
restored state and a rebuilt plan must continue like the oracle. A step
skipped for a non-finite gradient must not advance the step count, so the
next step's bias correction is the oracle's for the steps that ran."""

import math

import numpy as np
import pytest

import gpu_harness as H
import oracle
from paper_1904_00962_amd import _lib, paramsets

pytestmark = pytest.mark.gpu

# two layers on the single pass (multi-tile), one larger than a round of
# either tile shape (its head takes the two-pass kernels), one tiny
SIZES = [200 * 8192, 150 * 8192 + 3, 11_000_000 + 5, 77]
WD = [True, True, True, False]


def _tensors(torch, seed):
    rng = np.random.default_rng(seed)
    xs = [torch.from_numpy((rng.standard_normal(n) * 0.5).astype(np.float32)).cuda()
          for n in SIZES]
    return rng, xs


def _grads(torch, rng):
    return [torch.from_numpy((rng.standard_normal(n) * 1e-3).astype(np.float32)).cuda()
            for n in SIZES]


def test_facade_reports_a_give_up_and_recovers(monkeypatch):
    torch = H.torch_cuda()
    from paper_1904_00962_amd.optim import LAMB
    rng, xs = _tensors(torch, 41)
    grads = [torch.zeros_like(x) for x in xs]
    opt = LAMB(xs, grads, lr=1e-3, wd_mask=WD, check_every=1)
    try:
        per, _, _, elems = _lib.lamb_plan_tiles(opt.plan, True)
        assert per[0] > 1 and per[1] > 1 and elems[2] < SIZES[2]  # a head on the two-pass kernels
        # one good step, then a checkpoint
        for g, d in zip(grads, _grads(torch, rng)):
            g.copy_(d)
        opt.step()
        saved_x = [x.clone() for x in xs]
        saved = opt.state_dict()
        assert saved["step"] == 1
        # a plan whose waits give up at once
        monkeypatch.setenv("LAMB_MI355X_SPIN_LIMIT", "1")
        opt.rebuild()
        monkeypatch.delenv("LAMB_MI355X_SPIN_LIMIT")
        for g, d in zip(grads, _grads(torch, rng)):
            g.copy_(d)
        with pytest.raises(_lib.LambError) as e:
            opt.step()  # check_every = 1: the fault is read after this step
        assert e.value.status == _lib.LAMB_ESYNC
        # the plan is inert: no layer moves, the two-pass one included
        before = [a.clone() for a in xs + opt.m + opt.v]
        opt.check_every = 0
        opt.step()
        torch.cuda.synchronize()
        for a, b in zip(before, xs + opt.m + opt.v):
            assert torch.equal(a, b)
        with pytest.raises(_lib.LambError):
            opt.state_dict()
        # recovery: restore the checkpoint, rebuild the plan, step again
        for x, s in zip(xs, saved_x):
            x.copy_(s)
        opt.load_state_dict(saved)
        opt.rebuild()
        hx = [paramsets.host_array(x).copy() for x in xs]
        hm = [paramsets.host_array(m).copy() for m in opt.m]
        hv = [paramsets.host_array(v).copy() for v in opt.v]
        hg = [paramsets.host_array(g).copy() for g in grads]
        opt.step()
        opt.check()
        f = lambda a: float(np.float32(a))  # noqa: E731
        ref = oracle.load().lamb_step(hx, hg, hm, hv, WD, lr=f(1e-3), beta1=f(0.9),
                                      beta2=f(0.999), eps=f(1e-6), weight_decay=f(0.01),
                                      gamma_l=0.0, gamma_u=10.0, step=2)
        for i in range(len(xs)):
            H.compare_state_device(xs[i], hx[i], "x[%d] after recovery" % i)
            H.compare_state_device(opt.m[i], hm[i], "m[%d] after recovery" % i)
            H.compare_state_device(opt.v[i], hv[i], "v[%d] after recovery" % i)
        H.compare_ratios(opt.ratios.cpu().numpy(), ref[:, 0], "ratio after recovery")
        assert opt.t == 2
    finally:
        opt.close()


@pytest.mark.parametrize("path", ["auto", "two-pass"])
def test_a_skipped_step_does_not_advance_t(path):
    """Steps 1 and 3 run, step 2 is skipped: the third call runs at t = 2, and
    x, m, v match the oracle's two steps at t = 1 and t = 2."""
    torch = H.torch_cuda()
    from paper_1904_00962_amd.optim import LAMB
    rng, xs = _tensors(torch, 43)
    grads = [torch.zeros_like(x) for x in xs]
    opt = LAMB(xs, grads, lr=1e-3, wd_mask=WD, skip_nonfinite=True, path=path)
    o = oracle.load()
    hx = [paramsets.host_array(x).copy() for x in xs]
    hm = [np.zeros_like(h) for h in hx]
    hv = [np.zeros_like(h) for h in hx]
    f = lambda a: float(np.float32(a))  # noqa: E731
    try:
        for call, t_oracle in ((1, 1), (2, None), (3, 2)):
            gs = _grads(torch, rng)
            if call == 2:
                gs[1][12345] = math.nan
            for g, d in zip(grads, gs):
                g.copy_(d)
            opt.step()
            if t_oracle is not None:
                hg = [paramsets.host_array(g).copy() for g in grads]
                o.lamb_step(hx, hg, hm, hv, WD, lr=f(1e-3), beta1=f(0.9), beta2=f(0.999),
                            eps=f(1e-6), weight_decay=f(0.01), gamma_l=0.0, gamma_u=10.0,
                            step=t_oracle)
            assert opt.t == (1 if call < 3 else 2), (call, opt.t)
            assert int(opt.found_nonfinite) == (1 if call == 2 else 0)
        opt.check()
        for i in range(len(xs)):
            H.compare_state_device(xs[i], hx[i], "x[%d]" % i)
            H.compare_state_device(opt.m[i], hm[i], "m[%d]" % i)
            H.compare_state_device(opt.v[i], hv[i], "v[%d]" % i)
        assert opt.state_dict()["step"] == 2
    finally:
        opt.close()
