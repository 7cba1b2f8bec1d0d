"""The planless step (lamb_step_static), which allocates nothing and keeps its
tables in the library's fixed device array, against lamb_step_ex on a plan
on the two-pass path with the same chunk size: x, m, v, trust ratios and
norms equal bit for bit, on calls in a row whose second table is smaller
than the first (the array keeps the last call's contents), for LAMB, N-LAMB,
LARS and the skip mode. Tables beyond the array's limits are refused before
any HIP call."""

import math

import pytest

import gpu_harness as H
from paper_1904_00962_amd import _lib, paramsets

pytestmark = pytest.mark.gpu


class Twin:
    """Two copies of one state: one stepped through a plan, one planless."""

    def __init__(self, cfg, algo, g_dtype=None, chunk=0):
        torch = H.torch_cuda()
        self.torch = torch
        self.ps = ps = paramsets.get(cfg)
        self.algo = algo
        self.chunk = chunk
        g_dtype = g_dtype or ps.g_dtype
        gt = torch.bfloat16 if g_dtype == "bf16" else torch.float32
        self.g_kind = _lib.LAMB_GRAD_BF16 if g_dtype == "bf16" else _lib.LAMB_GRAD_F32
        xs = paramsets.draw_params(ps, device="cuda")
        self.sides = []
        for _ in range(2):
            X = [x.clone() for x in xs]
            side = dict(X=X, G=[torch.zeros(x.numel(), dtype=gt, device="cuda") for x in X],
                        M=[torch.zeros_like(x) for x in X],
                        V=[torch.zeros_like(x) for x in X] if algo != "lars" else None,
                        ratio=torch.zeros(len(X), dtype=torch.float64, device="cuda"),
                        norms=torch.zeros(2 * len(X), dtype=torch.float64, device="cuda"),
                        flag=torch.full((1,), -1, dtype=torch.int32, device="cuda"))
            side["rows"] = [(x.data_ptr(), g.data_ptr(), m.data_ptr(),
                             side["V"][i].data_ptr() if side["V"] is not None else 0, x.numel(),
                             int(w)) for i, (x, g, m, w) in
                            enumerate(zip(X, side["G"], side["M"], ps.wd_mask()))]
            self.sides.append(side)
        algo_id = _lib.LAMB_ALGO_LARS if algo == "lars" else _lib.LAMB_ALGO_LAMB
        self.plan = _lib.lamb_plan_create(self.sides[0]["rows"], self.g_kind, algo_id, chunk)
        _lib.lamb_plan_set_path(self.plan, "two-pass")

    def step(self, hp, t, nan_at=None):
        torch = self.torch
        grads = paramsets.draw_grads(self.ps, t, device="cuda")
        if nan_at is not None:
            grads[nan_at].view(-1)[0] = math.nan
        for side in self.sides:
            for G, g in zip(side["G"], grads):
                G.copy_(g.reshape(-1))
        stream = torch.cuda.current_stream().cuda_stream
        a, b = self.sides
        skip = bool(hp.skip_nonfinite)
        _lib.lamb_step_ex(self.plan, hp, stream, a["ratio"].data_ptr(), a["norms"].data_ptr(),
                          a["flag"].data_ptr() if skip else 0)
        _lib.lamb_step_static(b["rows"], self.g_kind, hp, self.chunk, stream,
                              b["ratio"].data_ptr(), b["norms"].data_ptr(),
                              b["flag"].data_ptr() if skip else 0)
        torch.cuda.synchronize()
        for key in ("X", "M", "V"):
            if a[key] is None:
                continue
            for i, (u, w) in enumerate(zip(a[key], b[key])):
                assert torch.equal(u, w), (key, i, t)
        # bit patterns (a skipped step reports NaN where its gradient was)
        for key in ("ratio", "norms"):
            assert torch.equal(a[key].view(torch.int64), b[key].view(torch.int64)), (key, t)
        if skip:
            assert int(a["flag"]) == int(b["flag"]) == (1 if nan_at is not None else 0)

    def close(self):
        self.plan.close()


def _hp(algo, ps, t, **extra):
    if algo == "lars":
        return _lib.lamb_hparams_init("lars", lr=ps.lars_lr, beta1=ps.lars_momentum,
                                      trust_coef=ps.lars_trust_coef, **extra)
    if algo == "lamb":
        return _lib.lamb_hparams_init("lamb", step=t, lr=ps.lr, beta1=ps.beta1, beta2=ps.beta2,
                                      eps=ps.eps, **extra)
    return _lib.lamb_hparams_init(algo, step=t, lr=ps.lr, **extra)


def test_static_step_equals_the_two_pass_plan_on_calls_in_a_row():
    # first call: BERT-Base (199 tensors, 5 table batches, 427,665 chunks),
    # two steps; then the smaller tiny set with other algorithms and modes
    big = Twin(1, "lamb")
    try:
        for t in (1, 2):
            big.step(_hp("lamb", big.ps, t), t)
    finally:
        big.close()
    for algo, g_dtype, chunk in (("n-lamb", "bf16", 0), ("lars", "f32", 520),
                                 ("lamb", "bf16", 64)):
        small = Twin(0, algo, g_dtype, chunk)
        try:
            for t in (1, 2, 3):
                small.step(_hp(algo, small.ps, t), t)
        finally:
            small.close()


def test_static_step_in_skip_mode():
    twin = Twin(3, "lamb")
    try:
        twin.step(_hp("lamb", twin.ps, 1, skip_nonfinite=1), 1)
        twin.step(_hp("lamb", twin.ps, 2, skip_nonfinite=1), 2, nan_at=17)
        twin.step(_hp("lamb", twin.ps, 2, skip_nonfinite=1), 3)
    finally:
        twin.close()


def test_static_step_refuses_tables_beyond_its_limits():
    torch = H.torch_cuda()
    ps = paramsets.get(0)
    twin = Twin(0, "lamb")
    n = 4_200_000  # 525,000 chunks of 8 elements: more than 2^19
    x = torch.randn(n, device="cuda")
    g = torch.zeros(n, device="cuda")
    m = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    try:
        rows = twin.sides[1]["rows"]
        hp = _hp("lamb", ps, 1)
        with pytest.raises(_lib.LambError) as e:
            _lib.lamb_step_static(rows * 513, twin.g_kind, hp, 0)  # 4104 tensors
        assert e.value.status == _lib.LAMB_EINVAL and "n_tensors" in _lib.last_error()
        big = [(x.data_ptr(), g.data_ptr(), m.data_ptr(), v.data_ptr(), n, 1)]
        before = x.clone()
        with pytest.raises(_lib.LambError) as e:
            _lib.lamb_step_static(big, _lib.LAMB_GRAD_F32, hp, 8)
        assert e.value.status == _lib.LAMB_EINVAL and "chunks" in _lib.last_error()
        torch.cuda.synchronize()
        assert torch.equal(before, x) and int(torch.count_nonzero(m)) == 0
    finally:
        twin.close()
