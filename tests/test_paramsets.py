"""Shapes, counts, masks and seeding of the synthetic parameter sets."""

import numpy as np
import pytest

from paper_1904_00962_amd import paramsets

# (tensors, parameters, 1-D tensors without weight decay, largest tensor)
EXPECTED = {
    0: (8, 608_000, 4, 262_144),
    1: (199, 109_482_240, 123, 23_440_896),
    2: (391, 335_141_888, 243, 31_254_528),
    3: (161, 25_557_032, 107, 2_359_296),
    4: (580, 1_557_611_200, 386, 80_411_200),
}


@pytest.mark.parametrize("cfg", sorted(EXPECTED))
def test_counts(cfg):
    ps = paramsets.get(cfg)
    n, p, masked, largest = EXPECTED[cfg]
    assert ps.n_tensors == n
    assert ps.numel == p
    assert sum(1 for t in ps.tensors if not t.wd) == masked
    assert all((len(t.shape) == 1) == (not t.wd) for t in ps.tensors)
    assert max(t.numel for t in ps.tensors) == largest


def test_gradient_dtypes():
    assert [paramsets.get(c).g_dtype for c in range(5)] == ["f32", "f32", "bf16", "f32", "bf16"]


def test_seeded_draws_are_reproducible_and_subset_stable():
    ps = paramsets.get(0)
    a = [paramsets.host_array(t) for t in paramsets.draw_params(ps)]
    b = [paramsets.host_array(t) for t in paramsets.draw_params(ps, indices=[2, 5])]
    assert np.array_equal(a[2], b[0]) and np.array_equal(a[5], b[1])
    g1 = [paramsets.host_array(t) for t in paramsets.draw_grads(ps, 1)]
    g1b = [paramsets.host_array(t) for t in paramsets.draw_grads(ps, 1)]
    g2 = [paramsets.host_array(t) for t in paramsets.draw_grads(ps, 2)]
    assert all(np.array_equal(p, q) for p, q in zip(g1, g1b))
    assert not np.array_equal(g1[0], g2[0])
    assert abs(float(np.std(a[2])) - ps.sigma_x) < 1e-3
    assert abs(float(np.std(g1[2])) - ps.sigma_g) < 1e-4
    assert all(x.dtype == np.float32 for x in a + g1)


def test_bf16_gradients_round_to_nearest_even():
    ps = paramsets.get(2)
    bits = paramsets.host_array(paramsets.draw_grads(ps, 1, indices=[3])[0])
    assert bits.dtype == np.uint16 and bits.size == 1024
    import torch
    gen = torch.Generator().manual_seed(1000 * 2 + 1)
    for spec in ps.tensors[:3]:
        torch.randn(spec.numel, generator=gen)
    ref = (torch.randn(1024, generator=gen) * ps.sigma_g).numpy()
    widened = (bits.astype(np.uint32) << 16).view(np.float32)  # exact widening
    # nearest bf16: error at most half a bf16 ulp (2^-8 relative), never more
    assert np.all(np.abs(widened - ref) <= np.abs(ref) * 2.0 ** -8)
    rounded = torch.from_numpy(ref).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(rounded, bits)
