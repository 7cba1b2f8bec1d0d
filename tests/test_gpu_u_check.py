"""The two-pass path's recomputation: the apply pass rebuilds u from the
stored moments instead of storing it, and Algorithm 2's last line uses one u
for ||u_i|| and for the update. With the plan's check on, the apply pass sums
the norms of the x it reads and of the u it recomputes per chunk, in the
moment pass's order; those sums must equal the moment pass's partials bit
for bit, for every algorithm, gradient dtype and layer norm, on the two-pass
path, on the layers the single pass leaves to the two-pass kernels, and in
the split step."""

import numpy as np
import pytest

import gpu_harness as H
from paper_1904_00962_amd import _lib, paramsets

pytestmark = pytest.mark.gpu

VARIANT = {"lamb": "lamb", "nlamb": "n-lamb", "nnlamb": "nn-lamb", "lars": "lars"}


def _hp(algo, ps, t, norm):
    if algo == "lars":
        return _lib.lamb_hparams_init("lars", lr=ps.lars_lr, beta1=ps.lars_momentum,
                                      trust_coef=ps.lars_trust_coef, norm=norm)
    extra = dict(beta1=0.975, eps=1e-8) if algo != "lamb" else {}
    return _lib.lamb_hparams_init(VARIANT[algo], step=t, lr=ps.lr, norm=norm, **extra)


def _assert_same(plan, label, expect_chunks):
    moment, apply = _lib.lamb_plan_u_partials(plan)
    assert moment.shape[0] == expect_chunks, (label, moment.shape)
    # not a vacuous check: real, positive sums
    assert np.all(np.isfinite(moment)) and np.any(moment[:, 1] > 0), label
    same = moment.view(np.uint64) == apply.view(np.uint64)
    if not np.all(same):
        k = int(np.argmin(np.all(same, axis=1)))
        raise AssertionError("%s: chunk %d moment %r apply %r" % (label, k, moment[k], apply[k]))


@pytest.mark.parametrize("algo", ["lamb", "nlamb", "nnlamb", "lars"])
@pytest.mark.parametrize("g_dtype", ["f32", "bf16"])
@pytest.mark.parametrize("norm", ["l2", "l1", "linf"])
def test_apply_pass_recomputes_the_same_u(algo, g_dtype, norm):
    torch = H.torch_cuda()
    ps = paramsets.get(0)
    pair = H.Pair(paramsets.draw_params(ps, device="cuda"), ps.wd_mask(), g_dtype,
                  "lars" if algo == "lars" else "lamb", chunk_elems=520, oracle_subset=[],
                  path="two-pass")
    try:
        _lib.lamb_plan_set_u_check(pair.plan, True)
        n_chunks = _lib.lamb_plan_info(pair.plan)[1]
        for t in (1, 2, 3):
            grads = paramsets.draw_grads(ps, t, device="cuda")
            if g_dtype == "bf16":
                grads = [g.to(torch.bfloat16) for g in grads]
            pair.set_grads(grads)
            _lib.lamb_step_ex(pair.plan, _hp(algo, ps, t, norm),
                              torch.cuda.current_stream().cuda_stream, 0, 0, 0)
            _assert_same(pair.plan, "%s %s %s step %d" % (algo, g_dtype, norm, t), n_chunks)
    finally:
        pair.close()


def test_check_on_the_layers_outside_the_single_pass():
    """BERT-Large on the default path: the head of the token embedding (all
    but its last round of tiles) takes the two-pass kernels, and the u its
    apply pass recomputes is checked."""
    torch = H.torch_cuda()
    ps = paramsets.get(2)
    pair = H.Pair(paramsets.draw_params(ps, device="cuda"), ps.wd_mask(), ps.g_dtype, "lamb",
                  oracle_subset=[])
    try:
        _, _, _, elems = _lib.lamb_plan_tiles(pair.plan, True)
        heads = [i for i, e in enumerate(elems) if e < pair.X[i].numel()]
        assert heads == [0]
        _lib.lamb_plan_set_u_check(pair.plan, True)
        head = pair.X[0].numel() - elems[0]
        expect = -(-head // _lib.lamb_plan_info(pair.plan)[2])
        for t in (1, 2):
            pair.set_grads(paramsets.draw_grads(ps, t, device="cuda"))
            _lib.lamb_step_ex(pair.plan, _hp("lamb", ps, t, "l2"),
                              torch.cuda.current_stream().cuda_stream, 0, 0, 0)
            _assert_same(pair.plan, "BERT-Large embedding step %d" % t, expect)
        # switched off, the plan reports nothing
        _lib.lamb_plan_set_u_check(pair.plan, False)
        moment, _ = _lib.lamb_plan_u_partials(pair.plan)
        assert moment.shape[0] == 0
    finally:
        pair.close()


def test_check_in_the_split_step_and_not_in_skip_mode():
    torch = H.torch_cuda()
    ps = paramsets.get(3)
    pair = H.Pair(paramsets.draw_params(ps, device="cuda"), ps.wd_mask(), ps.g_dtype, "lamb",
                  oracle_subset=[])
    totals = torch.zeros(2 * pair.n + 1, dtype=torch.float64, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    try:
        _lib.lamb_plan_set_u_check(pair.plan, True)
        n_chunks = _lib.lamb_plan_info(pair.plan)[1]
        pair.set_grads(paramsets.draw_grads(ps, 1, device="cuda"))
        hp = _hp("lamb", ps, 1, "l2")
        _lib.lamb_step_partials(pair.plan, hp, stream, totals.data_ptr())
        _lib.lamb_step_finish(pair.plan, hp, stream, totals.data_ptr())
        _assert_same(pair.plan, "ResNet-50 split step", n_chunks)
        # a skip_nonfinite step recomputes the moments in the apply pass over
        # other chunks than the moment pass's: no check, and none reported
        hp.skip_nonfinite = 1
        hp.step = 2
        flag = torch.zeros(1, dtype=torch.int32, device="cuda")
        _lib.lamb_step_ex(pair.plan, hp, stream, 0, 0, flag.data_ptr())
        moment, _ = _lib.lamb_plan_u_partials(pair.plan)
        assert moment.shape[0] == 0
    finally:
        pair.close()
