"""Properties of the HIP step that need no oracle: bitwise determinism,
chunk-size invariance, per-layer independence, resume, timing hooks and
the optimizer facade."""

import numpy as np
import pytest

import gpu_harness as H
from paper_1904_00962_amd import _lib, paramsets

pytestmark = pytest.mark.gpu


def _state(pair):
    out = [x.clone() for x in pair.X] + [m.clone() for m in pair.M]
    if pair.V is not None:
        out += [v.clone() for v in pair.V]
    return out + [pair.ratio.clone()]


def _steps(cfg, algo, chunk, steps, device="cuda", subset=None, path="auto"):
    ps = paramsets.get(cfg)
    xs = paramsets.draw_params(ps, indices=subset, device=device)
    wd = ps.wd_mask() if subset is None else [ps.wd_mask()[i] for i in subset]
    pair = H.Pair(xs, wd, ps.g_dtype, algo, chunk, oracle_subset=[], path=path)
    hp = H.lamb_hp(ps) if algo == "lamb" else H.lars_hp(ps)
    for t in range(1, steps + 1):
        pair.set_grads(paramsets.draw_grads(ps, t, indices=subset, device=device))
        if algo == "lamb":
            pair.gpu_lamb(hp, t)
        else:
            pair.gpu_lars(hp)
    return pair


@pytest.mark.parametrize("path", ["auto", "wide", "two-pass"])
@pytest.mark.parametrize("cfg,algo", [(2, "lamb"), (3, "lars")])
def test_bitwise_deterministic(cfg, algo, path):
    torch = H.torch_cuda()
    runs = []
    for _ in range(2):
        pair = _steps(cfg, algo, 0, 2, path=path)
        runs.append(_state(pair))
        pair.close()
    for a, b in zip(*runs):
        assert torch.equal(a, b)


def test_chunk_size_invariance():
    """m and v are elementwise, so they do not depend on the chunking or on
    the path at all; x and the ratios agree to rounding of the reduction
    order. The first runs are the single pass with either tile."""
    torch = H.torch_cuda()
    runs = [_state(_steps(1, "lamb", 0, 2))]
    runs += [_state(_steps(1, "lamb", 0, 2, path="wide"))]
    runs += [_state(_steps(1, "lamb", c, 2, path="two-pass")) for c in (0, 4096, 65536)]
    n = paramsets.get(1).n_tensors
    for other in runs[1:]:
        for k in range(n, 3 * n):
            assert torch.equal(runs[0][k], other[k])
        for k in range(n):
            H.compare_state(other[k].cpu().numpy(), runs[0][k].cpu().numpy(), "x[%d]" % k)
        H.compare_ratios(other[-1].cpu().numpy(), runs[0][-1].cpu().numpy(), "ratio")


@pytest.mark.parametrize("path,chunk", [("two-pass", 1024), ("auto", 0), ("wide", 0)])
def test_layer_independence(path, chunk):
    """A step on {A, B} equals a step on {A} and a step on {B}, bit for bit
    (on the single pass, wherever the packing puts each layer)."""
    torch = H.torch_cuda()
    ps = paramsets.get(0)
    joint = _steps(0, "lamb", chunk, 3, path=path)
    parts = [_steps(0, "lamb", chunk, 3, subset=[i], path=path) for i in range(ps.n_tensors)]
    for i, p in enumerate(parts):
        assert torch.equal(joint.X[i], p.X[0])
        assert torch.equal(joint.M[i], p.M[0])
        assert torch.equal(joint.V[i], p.V[0])
        assert torch.equal(joint.ratio[i], p.ratio[0])


def test_resume_is_bitwise():
    """The caller owns x, m, v and t: 6 steps equal 3 steps, a copy out and
    into a fresh optimizer, and 3 more. A state that does not fit the
    optimizer's tensors is refused and changes nothing."""
    torch = H.torch_cuda()
    from paper_1904_00962_amd.optim import LAMB
    ps = paramsets.get(3)
    x0 = paramsets.draw_params(ps, device="cuda")
    grads = [torch.zeros(x.numel(), device="cuda") for x in x0]

    def run(opt, t0, t1):
        for t in range(t0, t1):
            for g, d in zip(grads, paramsets.draw_grads(ps, t, device="cuda")):
                g.copy_(d)
            opt.step()

    mask = ps.wd_mask()
    p1 = [x.clone() for x in x0]
    a = LAMB(p1, grads, lr=ps.lr, wd_mask=mask)
    run(a, 1, 7)
    p2 = [x.clone() for x in x0]
    b = LAMB(p2, grads, lr=ps.lr, wd_mask=mask)
    run(b, 1, 4)
    saved = ([x.clone() for x in p2], b.state_dict())
    b.close()
    p3 = [x.clone() for x in saved[0]]
    c = LAMB(p3, grads, lr=ps.lr, wd_mask=mask)
    # a state of another parameter set is refused before anything is copied
    bad = dict(saved[1], m=saved[1]["m"][:-1])
    with pytest.raises(ValueError):
        c.load_state_dict(bad)
    bad = dict(saved[1], v=[v[:-1] for v in saved[1]["v"]])
    with pytest.raises(ValueError):
        c.load_state_dict(bad)
    assert c.t == 0 and all(int(torch.count_nonzero(m)) == 0 for m in c.m)
    c.load_state_dict(saved[1])
    run(c, 4, 7)
    torch.cuda.synchronize()
    for u, w in zip(p1, p3):
        assert torch.equal(u, w)
    a.close()
    c.close()


@pytest.mark.parametrize("path", ["auto", "two-pass"])
def test_timing_hooks_record_each_kernel(path):
    torch = H.torch_cuda()
    pair = _steps(0, "lamb", 0, 0, path=path)
    ps = paramsets.get(0)
    launched = [3] if path == "auto" else [0, 1, 2]  # the tiny set fits the single pass
    idle = [k for k in range(5) if k not in launched]
    _lib.lamb_plan_set_timing(pair.plan, 8)
    pair.set_grads(paramsets.draw_grads(ps, 1, device="cuda"))
    for t in range(1, 6):
        pair.gpu_lamb(H.lamb_hp(ps), t)
    ms, steps = _lib.lamb_plan_timing(pair.plan)
    assert steps == 5 and all(ms[k] > 0 for k in launched) and all(ms[k] == 0 for k in idle)
    ms2, steps2 = _lib.lamb_plan_timing(pair.plan)
    assert steps2 == 0
    _lib.lamb_plan_set_timing(pair.plan, 3, 4)  # steps 1, 5, 9 of the next 12
    for t in range(6, 18):
        pair.gpu_lamb(H.lamb_hp(ps), t)
    ms, steps = _lib.lamb_plan_timing(pair.plan)
    assert steps == 3 and all(ms[k] > 0 for k in launched)
    with pytest.raises(_lib.LambError):
        _lib.lamb_plan_set_timing(pair.plan, 3, 0)
    _lib.lamb_plan_set_timing(pair.plan, 0)
    pair.close()


def test_facade_matches_oracle():
    torch = H.torch_cuda()
    import oracle
    from paper_1904_00962_amd.optim import LAMB, LARS
    ps = paramsets.get(0)
    for cls in (LAMB, LARS):
        xs = paramsets.draw_params(ps, device="cuda")
        grads = [torch.zeros(x.numel(), device="cuda") for x in xs]
        hx = [paramsets.host_array(x).copy() for x in xs]
        hm = [np.zeros_like(h) for h in hx]
        hv = [np.zeros_like(h) for h in hx]
        # the tensors are flat, so the mask is given (the default reads dim() > 1)
        if cls is LAMB:
            opt = LAMB(xs, grads, lr=ps.lr, wd_mask=ps.wd_mask())
        else:
            opt = LARS(xs, grads, lr=ps.lars_lr, trust_coef=ps.lars_trust_coef,
                       wd_mask=ps.wd_mask())
        for t in (1, 2):
            for g, d in zip(grads, paramsets.draw_grads(ps, t, device="cuda")):
                g.copy_(d)
            hg = [paramsets.host_array(g).copy() for g in grads]
            opt.step()
            if cls is LAMB:
                ref = oracle.load().lamb_step(hx, hg, hm, hv, ps.wd_mask(), step=t,
                                              **H.f32_scalars(H.lamb_hp(ps)))
            else:
                hp = dict(lr=ps.lars_lr, momentum=0.9, weight_decay=0.01, gamma_l=0.0,
                          gamma_u=10.0, trust_coef=ps.lars_trust_coef)
                ref = oracle.load().lars_step(hx, hg, hm, ps.wd_mask(), **H.f32_scalars(hp))
            torch.cuda.synchronize()
            for i in range(ps.n_tensors):
                H.compare_state(paramsets.host_array(xs[i]), hx[i], "facade x")
            H.compare_ratios(opt.ratios.cpu().numpy(), ref[:, 0], "facade ratio")
        opt.close()


def test_facade_schedule_sets_each_steps_lr():
    """A facade step with a schedule equals a plain step given that lr."""
    torch = H.torch_cuda()
    from paper_1904_00962_amd.optim import LAMB
    ps = paramsets.get(0)
    stages = [(5, 2, 1e-2, 1.0), (4, 1, 5e-3, 1.0)]
    xs = paramsets.draw_params(ps, device="cuda")
    grads = [torch.zeros(x.numel(), device="cuda") for x in xs]
    a = LAMB([x.clone() for x in xs], grads, wd_mask=ps.wd_mask(), schedule=stages)
    b = LAMB([x.clone() for x in xs], grads, wd_mask=ps.wd_mask())
    for t in range(1, 10):
        for g, d in zip(grads, paramsets.draw_grads(ps, t, device="cuda")):
            g.copy_(d)
        a.step()
        b.step(lr=_lib.lamb_lr_at(stages, t))
    torch.cuda.synchronize()
    assert all(torch.equal(p, q) for p, q in zip(a.params, b.params))
    a.close()
    b.close()


def test_independent_plans_on_concurrent_streams():
    """Two plans stepped on two streams at once give what each gives alone."""
    torch = H.torch_cuda()
    ps = paramsets.get(3)
    results = []
    for concurrent in (False, True):
        pairs = [_steps(3, algo, 0, 0) for algo in ("lamb", "lars")]
        streams = [torch.cuda.Stream(), torch.cuda.Stream()]
        for p in pairs:
            p.set_grads(paramsets.draw_grads(ps, 1, device="cuda"))
        torch.cuda.synchronize()
        for t in range(1, 4):
            for k, (p, s) in enumerate(zip(pairs, streams)):
                with torch.cuda.stream(s):
                    if k == 0:
                        p.gpu_lamb(H.lamb_hp(ps), t)
                    else:
                        p.gpu_lars(H.lars_hp(ps))
                if not concurrent:
                    torch.cuda.synchronize()
        torch.cuda.synchronize()
        results.append([_state(p) for p in pairs])
        for p in pairs:
            p.close()
    for a, b in zip(results[0], results[1]):
        assert all(torch.equal(u, w) for u, w in zip(a, b))


@pytest.mark.parametrize("path,skip", [("auto", 0), ("two-pass", 0), ("two-pass", 1), ("auto", 1),
                                       ("wide", 0), ("wide", 1)])
def test_graph_capture_replays_match_eager(path, skip):
    """A captured step (fixed scalars, gradients read from the same buffers)
    replayed three times, with eager work between replays, equals three eager
    steps. The single pass keeps its slot epoch on the device; in deferred
    mode the second replay sees a NaN gradient and must skip, and the third
    must not: the non-finite verdict is handed over on the device, not by a
    host counter or a memset."""
    torch = H.torch_cuda()
    ps = paramsets.get(0)
    hp = _lib.lamb_hparams_init("lamb", step=4, lr=ps.lr, skip_nonfinite=skip)
    grads = [paramsets.draw_grads(ps, t, device="cuda") for t in (1, 2, 3)]
    if skip:
        grads[1][2][5] = float("nan")
    runs = []
    for graph in (False, True):
        pair = _steps(0, "lamb", 1024, 0, path=path)
        flag = torch.full((1,), 7, dtype=torch.int32, device="cuda")

        def step():
            _lib.lamb_step_ex(pair.plan, hp, torch.cuda.current_stream().cuda_stream,
                              pair.ratio.data_ptr(), pair.norms.data_ptr(),
                              flag.data_ptr() if skip else 0)

        pair.set_grads(grads[0])
        step()  # one eager step first in both runs
        torch.cuda.synchronize()
        states = []
        if graph:
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                step()
            torch.cuda.synchronize()
            for r in range(3):
                pair.set_grads(grads[r])
                torch.cuda.synchronize()
                g.replay()
                torch.cuda.synchronize()
                scratch = torch.randn(1 << 20, device="cuda").sum()  # eager work between replays
                torch.cuda.synchronize()
                states.append(_state(pair) + [flag.clone()])
            del scratch
        else:
            for r in range(3):
                pair.set_grads(grads[r])
                step()
                torch.cuda.synchronize()
                states.append(_state(pair) + [flag.clone()])
        _lib.lamb_plan_check(pair.plan)
        runs.append(states)
        pair.close()
    if skip:
        assert [int(s[-1]) for s in runs[0]] == [0, 1, 0]
        for a, b in zip(runs[0][0][:-2], runs[0][1][:-2]):
            assert torch.equal(a, b)  # the NaN step left x, m, v alone
    for r, (eager, replay) in enumerate(zip(runs[0], runs[1])):
        for k, (a, b) in enumerate(zip(eager, replay)):
            assert _same_bits(a, b), "replay %d, state entry %d of %d: eager %s, replay %s" % (
                r, k, len(eager), a.flatten()[:4].tolist(), b.flatten()[:4].tolist())


def _same_bits(a, b):
    """Bitwise equality that also holds for equal NaN patterns."""
    torch = H.torch_cuda()
    if a.dtype == torch.float64:
        return torch.equal(a.view(torch.int64), b.view(torch.int64))
    if a.dtype == torch.float32:
        return torch.equal(a.view(torch.int32), b.view(torch.int32))
    return torch.equal(a, b)
