"""The split step (lamb_step_partials / lamb_step_finish) for optimizer state
sharded over N workers, shown on one GPU: N plans, each over one 1/N slice of
every tensor, run the first half; their totals are combined on the device
(a sum for L2 and L1, a NaN-keeping maximum for L-infinity) in the global
tensor order, as an all-reduce would; every plan then finishes from the
combined totals. The result must match the oracle's unsharded step with the
parity tolerances and the unsharded GPU step to rounding; with one shard it
must equal the two-pass path bit for bit. A non-finite gradient in any one
shard must stop every shard."""

import math

import numpy as np
import pytest

import gpu_harness as H
from paper_1904_00962_amd import _lib, paramsets

pytestmark = pytest.mark.gpu


def slices(n, shards):
    """Per-tensor split into `shards` slices of ceil(n / N) elements rounded
    up to a multiple of 8 (so that every slice of fp32 and bf16 buffers
    starts 16-byte aligned); empty slices are dropped."""
    share = -(-n // shards)
    share = (share + 7) // 8 * 8
    out = []
    for r in range(shards):
        a, b = r * share, min(n, (r + 1) * share)
        out.append((a, b) if a < b else None)
    return out


class Sharded:
    """N shard plans over slices of one set of device tensors."""

    def __init__(self, pair: H.Pair, shards: int, g_dtype: str, algo: str, chunk: int = 0):
        torch = pair.torch
        self.torch = torch
        self.pair = pair
        self.n = pair.n
        self.plans, self.index = [], []
        kind = _lib.LAMB_GRAD_BF16 if g_dtype == "bf16" else _lib.LAMB_GRAD_F32
        algo_id = _lib.LAMB_ALGO_LARS if algo == "lars" else _lib.LAMB_ALGO_LAMB
        per_tensor = [slices(x.numel(), shards) for x in pair.X]
        for r in range(shards):
            rows, idx = [], []
            for i in range(self.n):
                sl = per_tensor[i][r]
                if sl is None:
                    continue
                a, b = sl
                v = pair.V[i][a:b].data_ptr() if pair.V is not None else 0
                rows.append((pair.X[i][a:b].data_ptr(), pair.G[i][a:b].data_ptr(),
                             pair.M[i][a:b].data_ptr(), v, b - a, int(pair.wd[i])))
                idx.append(i)
            if rows:
                self.plans.append(_lib.lamb_plan_create(rows, kind, algo_id, chunk))
                self.index.append(torch.tensor(idx, dtype=torch.int64, device="cuda"))
        self.ratio = torch.zeros(self.n, dtype=torch.float64, device="cuda")
        self.norms = torch.zeros(2 * self.n, dtype=torch.float64, device="cuda")

    def step(self, hp, nonfinite=None):
        """One split step; returns the combined totals (device)."""
        torch = self.torch
        stream = torch.cuda.current_stream().cuda_stream
        n = self.n
        totals = [torch.full((2 * len(ix) + 1,), math.nan, dtype=torch.float64, device="cuda")
                  for ix in self.index]
        for plan, t in zip(self.plans, totals):
            _lib.lamb_step_partials(plan, hp, stream, t.data_ptr())
        # the exchange: every shard's totals in the global tensor order, then
        # an element-wise sum (L2, L1) or maximum (L-infinity) over shards
        grid = torch.zeros((len(self.plans), 2 * n + 1), dtype=torch.float64, device="cuda")
        for r, (ix, t) in enumerate(zip(self.index, totals)):
            k = ix.numel()
            grid[r, 2 * ix] = t[0:2 * k:2]
            grid[r, 2 * ix + 1] = t[1:2 * k:2]
            grid[r, 2 * n] = t[2 * k]
        combined = grid.amax(0) if hp.norm == _lib.LAMB_NORM_LINF else grid.sum(0)
        for r, (plan, ix) in enumerate(zip(self.plans, self.index)):
            k = ix.numel()
            back = torch.empty(2 * k + 1, dtype=torch.float64, device="cuda")
            back[0:2 * k:2] = combined[2 * ix]
            back[1:2 * k:2] = combined[2 * ix + 1]
            back[2 * k] = combined[2 * n]
            ratio = torch.zeros(k, dtype=torch.float64, device="cuda")
            norms = torch.zeros(2 * k, dtype=torch.float64, device="cuda")
            flag = nonfinite[r] if nonfinite is not None else None
            _lib.lamb_step_finish(plan, hp, stream, back.data_ptr(), ratio.data_ptr(),
                                  norms.data_ptr(), flag.data_ptr() if flag is not None else 0)
            self.ratio[ix] = ratio
            self.norms[2 * ix] = norms[0::2]
            self.norms[2 * ix + 1] = norms[1::2]
        return combined

    def close(self):
        for p in self.plans:
            p.close()


def _hparams(algo, ps, t, **extra):
    if algo == "lars":
        return _lib.lamb_hparams_init("lars", lr=ps.lars_lr, beta1=ps.lars_momentum,
                                      weight_decay=ps.weight_decay, gamma_l=ps.gamma_l,
                                      gamma_u=ps.gamma_u, trust_coef=ps.lars_trust_coef, **extra)
    variant = {"lamb": "lamb", "nlamb": "n-lamb", "nnlamb": "nn-lamb"}[algo]
    fields = dict(lr=ps.lr, beta1=ps.beta1, beta2=ps.beta2, eps=ps.eps)
    if algo != "lamb":
        fields.update(beta1=0.975, eps=1e-8)
    return _lib.lamb_hparams_init(variant, step=t, weight_decay=ps.weight_decay,
                                  gamma_l=ps.gamma_l, gamma_u=ps.gamma_u, **fields, **extra)


def _pair(cfg, algo, path="two-pass", subset=None):
    ps = paramsets.get(cfg)
    return ps, H.Pair(paramsets.draw_params(ps, device="cuda"), ps.wd_mask(), ps.g_dtype,
                      "lars" if algo == "lars" else "lamb", oracle_subset=subset, path=path)


@pytest.mark.parametrize("algo", ["lamb", "nlamb", "nnlamb", "lars"])
@pytest.mark.parametrize("cfg", [0, 3])
def test_one_shard_equals_the_two_pass_step(cfg, algo):
    """With one shard the split step is the two-pass step, bit for bit: the
    same moment pass, the same per-tensor combination order, the same apply."""
    torch = H.torch_cuda()
    ps, ref = _pair(cfg, algo, subset=[])
    _, split = _pair(cfg, algo, subset=[])
    sh = Sharded(split, 1, ps.g_dtype, algo)
    try:
        for t in (1, 2, 3):
            grads = paramsets.draw_grads(ps, t, device="cuda")
            ref.set_grads(grads)
            split.set_grads(grads)
            hp = _hparams(algo, ps, t)
            _lib.lamb_step_ex(ref.plan, hp, torch.cuda.current_stream().cuda_stream,
                              ref.ratio.data_ptr(), ref.norms.data_ptr(), 0)
            sh.step(hp)
            torch.cuda.synchronize()
            for a, b in zip(ref.X + ref.M + (ref.V or []), split.X + split.M + (split.V or [])):
                assert torch.equal(a, b)
            assert torch.equal(ref.ratio, sh.ratio) and torch.equal(ref.norms, sh.norms)
    finally:
        sh.close()
        ref.close()
        split.close()


CASES = [
    # cfg, algo, shards, norm, steps
    (0, "lamb", 2, "l2", 3), (0, "lamb", 4, "l2", 3), (0, "lamb", 8, "l2", 3),
    (0, "nlamb", 4, "l2", 2), (0, "nnlamb", 8, "l2", 2), (0, "lars", 4, "l2", 3),
    (0, "lamb", 4, "l1", 2), (0, "lamb", 8, "linf", 2), (0, "lars", 8, "linf", 2),
    (3, "lamb", 8, "l2", 2), (3, "lars", 8, "l2", 2),
    (2, "lamb", 8, "l2", 2),
]


@pytest.mark.parametrize("cfg,algo,shards,norm,steps", CASES)
def test_sharded_step_matches_oracle_and_unsharded_step(cfg, algo, shards, norm, steps):
    torch = H.torch_cuda()
    ps, pair = _pair(cfg, algo)
    _, whole = _pair(cfg, algo, path="two-pass", subset=[])
    H.log("split step cfg=%d %s shards=%d norm=%s" % (cfg, algo, shards, norm))
    sh = Sharded(pair, shards, ps.g_dtype, algo)
    try:
        assert len(sh.plans) == shards
        for t in range(1, steps + 1):
            grads = paramsets.draw_grads(ps, t, device="cuda")
            hg = pair.set_grads(grads)
            whole.set_grads(grads)
            # the unsharded step starts from the sharded step's state, so the
            # two differ only in how the norms were summed
            for a, b in zip(whole.X + whole.M + (whole.V or []), pair.X + pair.M + (pair.V or [])):
                a.copy_(b)
            hp = _hparams(algo, ps, t, norm=_lib.NORMS[norm])
            sh.step(hp)
            _lib.lamb_step_ex(whole.plan, hp, torch.cuda.current_stream().cuda_stream,
                              whole.ratio.data_ptr(), whole.norms.data_ptr(), 0)
            pair.ratio.copy_(sh.ratio)
            pair.norms.copy_(sh.norms)
            ref = H.step_ex_both_oracle(pair, hp, hg)
            rep = pair.compare(ref, "cfg%d %s x%d %s step %d" % (cfg, algo, shards, norm, t))
            H.log("  step %d: max err %.3e vs the oracle" % (t, rep.max_err))
            # the unsharded GPU step: the same norms to rounding, x to one ulp
            H.compare_ratios(sh.ratio.cpu().numpy(), whole.ratio.cpu().numpy(),
                             "ratio vs unsharded", 1e-12)
            for i in range(pair.n):
                assert torch.equal(pair.M[i], whole.M[i])
                if pair.V is not None:
                    assert torch.equal(pair.V[i], whole.V[i])
                d = (pair.X[i].view(torch.int32) - whole.X[i].view(torch.int32)).abs()
                assert int(d.max()) <= 1, i
    finally:
        sh.close()
        pair.close()
        whole.close()


@pytest.mark.parametrize("algo", ["lamb", "lars"])
def test_a_nonfinite_gradient_in_one_shard_stops_every_shard(algo):
    """skip_nonfinite: the first half only reads; a NaN in one shard's slice
    reaches every shard through the combined totals, and no shard moves."""
    torch = H.torch_cuda()
    ps, pair = _pair(0, algo)
    sh = Sharded(pair, 4, ps.g_dtype, algo)
    flags = [torch.full((1,), -1, dtype=torch.int32, device="cuda") for _ in sh.plans]
    ran = 0  # steps that ran: a skipped step does not count
    try:
        for t in (1, 2, 3):
            grads = paramsets.draw_grads(ps, t, device="cuda")
            if t == 2:
                grads[2].view(-1)[-5] = math.nan  # in the last shard's slice
            hg = pair.set_grads(grads)
            before = [a.clone() for a in pair.X + pair.M + (pair.V or [])]
            hp = _hparams(algo, ps, ran + 1, skip_nonfinite=1)
            combined = sh.step(hp, flags)
            ran += t != 2
            pair.ratio.copy_(sh.ratio)
            pair.norms.copy_(sh.norms)
            ref = H.step_ex_both_oracle(pair, hp, hg)
            torch.cuda.synchronize()
            assert [int(f) for f in flags] == [1 if t == 2 else 0] * len(flags), t
            if t == 2:
                assert float(combined[-1]) >= 1.0
                after = pair.X + pair.M + (pair.V or [])
                assert all(torch.equal(a, b) for a, b in zip(before, after))
                assert bool(np.all(np.isnan(ref)))
            else:
                pair.compare(ref, "skip %s step %d" % (algo, t))
    finally:
        sh.close()
        pair.close()
