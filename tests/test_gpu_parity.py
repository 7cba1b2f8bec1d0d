"""HIP step vs the CPU oracle on the paper-shaped parameter sets.

Every step of every run is compared element by element (x, m, v) and per
tensor (trust ratio, ||x||, ||u||) under the rule in ``gpu_harness``. The
BERT-Large run uses the default chunk size, i.e. the launch configuration
the benchmark times. The 1.5B set compares a sample of whole tensors with
the oracle and checks a size-independent property on every tensor.
"""

import numpy as np
import pytest

import gpu_harness as H
from paper_1904_00962_amd import _lib, paramsets

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("chunk", [0, 1024, 8])
def test_tiny_lamb_ten_steps(chunk):
    r = H.run_config(0, 10, "lamb", chunk_elems=chunk)
    assert r.max_err <= H.STATE_TOL


def test_tiny_lars_ten_steps():
    H.run_config(0, 10, "lars", chunk_elems=512)


@pytest.mark.parametrize("path", ["auto", "wide"])
def test_tiny_lamb_hundred_steps(path):
    """100 steps compared with the oracle after every one: no drift between
    the two trajectories, and 100 alternations of the single pass's slot
    buffers on layers of up to 32 tiles."""
    r = H.run_config(0, 100, "lamb", path=path)
    assert r.max_err <= H.STATE_TOL


@pytest.mark.parametrize("algo", ["lamb", "lars", "nlamb", "nnlamb"])
def test_tiny_wide_tiles(algo):
    """The single pass with 10240-element tiles (forced on the tiny set)."""
    H.run_config(0, 6, algo, path="wide")


def test_bert_base_lamb():
    H.run_config(1, 3, "lamb")


def test_bert_large_lamb_bf16_grad():
    H.run_config(2, 3, "lamb")


def test_resnet50_lamb():
    H.run_config(3, 3, "lamb")


def test_resnet50_lars():
    H.run_config(3, 3, "lars")


@pytest.mark.parametrize("algo", ["nlamb", "nnlamb"])
def test_tiny_nesterov_variants(algo):
    H.run_config(0, 10, algo)
    H.run_config(0, 4, algo, chunk_elems=64)


@pytest.mark.parametrize("algo", ["nlamb", "nnlamb"])
def test_bert_large_nesterov_variants_bf16_grad(algo):
    H.run_config(2, 2, algo)


@pytest.mark.parametrize("algo", ["nlamb", "nnlamb"])
def test_resnet50_nesterov_variants(algo):
    H.run_config(3, 3, algo)


def test_bert_large_lars_bf16_grad():
    ps = paramsets.get(2)
    H.run_config(2, 2, "lars", oracle_subset=[0, 3, 4, 5, 6, ps.n_tensors - 1])


def test_gpt_1p5b_lamb_sampled():
    """1.56e9 parameters: one step; whole-tensor parity on a sample (the 80M
    token embedding, the first layer, the final norm), and on every tensor
    the Section 3 identity ||x_{t+1} - x_t|| = eta * phi(||x_t||). The plan
    takes 10240-element tiles, which put the 10.24M-element FFN layers on
    the single pass."""
    torch = H.torch_cuda()
    ps = paramsets.get(4)
    sample = [0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, ps.n_tensors - 2, ps.n_tensors - 1]
    H.log("parity cfg=4 sampled tensors %s" % sample)
    pair = H.Pair(paramsets.draw_params(ps, device="cuda"), ps.wd_mask(), ps.g_dtype, "lamb",
                  oracle_subset=sample)
    try:
        per, _, groups = _lib.lamb_plan_tiles(pair.plan)
        assert groups == 10
        assert [i for i, k in enumerate(per) if k == 0] == [0]  # the token embedding only
        hp = H.lamb_hp(ps)
        x_old = [x.clone() for x in pair.X]
        hg = pair.set_grads(paramsets.draw_grads(ps, 1, device="cuda"))
        pair.gpu_lamb(hp, 1)
        ref = pair.oracle_lamb(hg, hp, 1)
        pair.compare(ref, "cfg4 step 1")
        torch.cuda.synchronize()
        lr = float(np.float32(hp["lr"]))
        worst = 0.0
        for i in range(ps.n_tensors):
            xo = x_old[i].double()
            length = float(torch.linalg.vector_norm(pair.X[i].double() - xo))
            phi = min(max(float(torch.linalg.vector_norm(xo)), hp["gamma_l"]), hp["gamma_u"])
            rel = abs(length - lr * phi) / (lr * phi)
            worst = max(worst, rel)
            assert rel < 1e-4, "tensor %d: step length %.9e vs eta*phi %.9e" % (i, length, lr * phi)
        H.log("  step-length identity over all %d tensors: worst rel %.2e" % (ps.n_tensors, worst))
    finally:
        pair.close()
