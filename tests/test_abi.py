"""The C ABI on the CPU: the library loads, exports every declared entry
point, builds the documented chunk table, and rejects bad arguments before
any HIP call (no compute is launched here)."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_1904_00962_amd import _lib, build

HEADER = os.path.join(build.INCLUDE, "lamb_mi355x.h")


@pytest.fixture(scope="module")
def lib():
    if build.is_stale():
        build.build()
    return _lib.load()


def declared_functions():
    text = open(HEADER).read()
    return re.findall(r"LAMB_API\s+[\w\s\*]+?\b(\w+)\s*\(", text)


def test_header_declares_the_bound_functions():
    assert sorted(declared_functions()) == sorted(_lib.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code in range(-8, 1):
        assert _lib.status_str(code) != "unknown status"
    assert _lib.status_str(-99) == "unknown status"


def _model_chunks(numel, chunk):
    ct, cs, cl = [], [], []
    for i, n in enumerate(numel):
        for k in range(-(-n // chunk)):
            ct.append(i)
            cs.append(k * chunk)
            cl.append(min(chunk, n - k * chunk))
    return np.array(ct), np.array(cs), np.array(cl)


@pytest.mark.parametrize("chunk", [8, 16, 1024, 32768, 65536])
def test_chunk_table_is_the_documented_split(lib, chunk):
    rng = np.random.default_rng(chunk)
    numel = [1, 7, 8, 9, chunk - 1 if chunk > 1 else 1, chunk, chunk + 1, 3 * chunk + 5]
    numel += [int(v) for v in rng.integers(1, 5 * chunk, size=20)]
    ct, cs, cl = _lib.lamb_chunk_table(numel, chunk)
    mt, ms, ml = _model_chunks(numel, chunk)
    assert np.array_equal(ct, mt) and np.array_equal(cs, ms) and np.array_equal(cl, ml)
    assert int(cl.sum()) == sum(numel)


def test_chunk_table_default_and_large_tensor(lib):
    big = (1 << 31) + 1000
    ct, cs, cl = _lib.lamb_chunk_table([big], 0)
    default = int(cl[0])
    assert default % 8 == 0 and cs[1] == default
    assert cs[-1] + cl[-1] == big and cl[-1] == big % default
    assert cs.dtype == np.int64 and cs[-1] > 2 ** 31


def test_chunk_table_errors(lib):
    for numel, chunk in (([5, 0], 8), ([5], 12), ([5], 4), ([5], -8), ([5], (1 << 30) + 8)):
        with pytest.raises(_lib.LambError) as e:
            _lib.lamb_chunk_table(numel, chunk)
        assert e.value.status == _lib.LAMB_EINVAL
    with pytest.raises(_lib.LambError) as e:
        _lib.lamb_chunk_table([1 << 40] * 3, 8)  # more than 2^31 - 1 chunks
    assert e.value.status == _lib.LAMB_EINVAL
    for numel in ([(1 << 40) + 1], [5, (1 << 63) - 1]):  # beyond 2^40 elements
        for call in (lambda: _lib.lamb_chunk_table(numel, 8),
                     lambda: _lib.lamb_tile_schedule(numel, 1024)):
            with pytest.raises(_lib.LambError) as e:
                call()
            assert e.value.status == _lib.LAMB_EINVAL and "2^40" in str(e.value)
    n = ctypes.c_int32()
    sizes = (ctypes.c_int64 * 2)(100, 100)
    arr32 = (ctypes.c_int32 * 1)()
    arr64 = (ctypes.c_int64 * 1)()
    st = lib.lamb_chunk_table(sizes, 2, 64, 1, arr32, arr64, arr32, ctypes.byref(n))
    assert st == _lib.LAMB_EINVAL and n.value == 4
    assert "capacity" in _lib.last_error()


# Fake device addresses: validation must reject these tables before any HIP
# call, so nothing ever dereferences them.
A = 1 << 40


def _row(base, numel=100, wd=1, stride=4096):
    return (base, base + stride, base + 2 * stride, base + 3 * stride, numel, wd)


@pytest.mark.parametrize("rows,algo,g,chunk,status", [
    ([], 0, 0, 0, _lib.LAMB_EINVAL),
    ([_row(A)], 0, 2, 0, _lib.LAMB_EINVAL),                    # unknown gradient dtype
    ([_row(A)], 3, 0, 0, _lib.LAMB_EINVAL),                    # unknown algorithm
    ([_row(A)], 0, 0, 12, _lib.LAMB_EINVAL),                   # chunk not a multiple of 8
    ([(0, A, A + 4096, A + 8192, 10, 1)], 0, 0, 0, _lib.LAMB_ENULL),
    ([(A, A + 4096, A + 8192, 0, 10, 1)], 0, 0, 0, _lib.LAMB_ENULL),   # LAMB needs v
    ([_row(A, numel=0)], 0, 0, 0, _lib.LAMB_EINVAL),
    ([_row(A, wd=2)], 0, 0, 0, _lib.LAMB_EINVAL),
    ([_row(A + 4)], 0, 0, 0, _lib.LAMB_EALIGN),
    ([_row(A, numel=2000)], 0, 0, 0, _lib.LAMB_EOVERLAP),       # x runs into g
    ([_row(A), _row(A + 64)], 0, 0, 0, _lib.LAMB_EOVERLAP),     # two tensors share memory
    ([(A, A, A + 8192, A + 12288, 10, 1)], 0, 0, 0, _lib.LAMB_EOVERLAP),
])
def test_plan_create_rejects_before_any_hip_call(lib, rows, algo, g, chunk, status):
    with pytest.raises(_lib.LambError) as e:
        _lib.lamb_plan_create(rows, g, algo, chunk)
    assert e.value.status == status
    assert _lib.last_error()


def test_bf16_overlap_uses_two_byte_elements(lib):
    # 100 bf16 gradients occupy 200 bytes: a neighbour 256 bytes on is fine,
    # so this table fails only later (alignment of the deliberately odd x).
    rows = [(A + 4, A + 4096, A + 8192, A + 12288, 100, 1)]
    with pytest.raises(_lib.LambError) as e:
        _lib.lamb_plan_create(rows, _lib.LAMB_GRAD_BF16, _lib.LAMB_ALGO_LAMB, 0)
    assert e.value.status == _lib.LAMB_EALIGN


def test_hparams_defaults(lib):
    hp = _lib.lamb_hparams_init("lamb")
    assert (hp.beta1, hp.beta2, hp.weight_decay, hp.step, hp.norm) == (
        pytest.approx(0.9), pytest.approx(0.999), pytest.approx(0.01), 1, _lib.LAMB_NORM_L2)
    assert hp.eps == pytest.approx(1e-6) and hp.grad_scale == 1.0 and hp.bias_correction == 1
    hp = _lib.lamb_hparams_init("n-lamb", norm="linf", lr=0.5)
    assert hp.beta1 == pytest.approx(0.975) and hp.eps == pytest.approx(1e-8)
    assert hp.norm == _lib.LAMB_NORM_LINF and hp.lr == 0.5
    hp = _lib.lamb_hparams_init("lars")
    assert hp.variant == _lib.LAMB_VARIANT_LARS and hp.trust_coef == 1.0
    with pytest.raises(_lib.LambError):
        _lib.lamb_hparams_init(9)
    assert lib.lamb_hparams_init(None, 0) == _lib.LAMB_ENULL
    assert lib.lamb_step_ex(None, ctypes.byref(hp), None, None, None, None) == _lib.LAMB_ENULL


def test_null_plan_and_outputs(lib):
    assert lib.lamb_step(None, 1e-3, 0.9, 0.999, 1e-6, 0.01, 0.0, 10.0, 1, 1, None, None,
                         None) == _lib.LAMB_ENULL
    assert lib.lars_step(None, 1e-3, 0.9, 0.01, 0.0, 10.0, 1e-3, None, None, None) == _lib.LAMB_ENULL
    assert lib.nlamb_step(None, 1e-3, 0.975, 0.999, 1e-8, 0.01, 0.0, 10.0, 1, 0, None, None,
                          None) == _lib.LAMB_ENULL
    assert lib.lamb_plan_destroy(None) == _lib.LAMB_OK
    assert lib.lamb_plan_info(None, None, None, None) == _lib.LAMB_ENULL
    assert lib.lamb_plan_set_timing(None, 4, 1) == _lib.LAMB_ENULL
    assert lib.lamb_plan_set_bf16_copies(None, None) == _lib.LAMB_ENULL
    assert lib.lamb_plan_create(None, 1, 0, 0, 0, None) == _lib.LAMB_ENULL
    assert lib.lamb_plan_set_path(None, 0) == _lib.LAMB_ENULL
    assert lib.lamb_plan_tiles(None, None, None, None, None) == _lib.LAMB_ENULL
    assert lib.lamb_plan_check(None, None) == _lib.LAMB_ENULL
    per = (ctypes.c_double * 5)()
    steps = ctypes.c_int64()
    assert lib.lamb_plan_timing(None, per, ctypes.byref(steps)) == _lib.LAMB_ENULL


def test_stream_probe_library_validates_on_the_host():
    """The measurement-only stream library (include/stream_probe.h) exports
    its entry point and rejects bad arguments before any launch."""
    if not os.path.exists(build.PROBE_LIBRARY):
        build.build_probe()
    probe = ctypes.CDLL(build.PROBE_LIBRARY)
    probe.stream_probe.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                   ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_void_p]
    fake = 1 << 20  # aligned, never dereferenced: every case fails validation
    bad = [
        (9, fake, fake, fake, fake, 1, 100, 512, 0),     # unknown pattern
        (0, fake, fake, fake, fake, 1, 0, 512, 0),       # n < 1
        (0, fake, fake, fake, fake, 1, 100, 12, 0),      # tile not a multiple of 8
        (0, fake, fake, fake, fake, 2, 100, 512, 0),     # g_bf16 not 0/1
        (0, fake, fake, fake, None, 1, 100, 512, 0),     # single pass reads g
        (0, fake + 4, fake, fake, fake, 1, 100, 512, 0), # misaligned
        (0, fake, fake, fake, fake, 1, 100, 512, 4),     # dealt tiles need 1024 | tile
        (0, fake, fake, fake, fake, 1, 100, 8192, -1),   # negative layer_tiles
    ]
    for args in bad:
        assert probe.stream_probe(*args, None) == -1, args


def test_static_step_validation_before_any_hip_call(lib):
    """lamb_step_static rejects bad tables and hyperparameters on the host
    (these fail before it looks up its device array)."""
    hp = _lib.lamb_hparams_init("lamb")
    ok = (4096, 8192, 12288, 16384, 256, 1)  # fake, aligned, disjoint addresses
    cases = [
        ([], _lib.LAMB_GRAD_F32, 0, _lib.LAMB_EINVAL),                    # no tensors
        ([ok] * 4097, _lib.LAMB_GRAD_F32, 0, _lib.LAMB_EINVAL),           # over 4096
        ([ok], 5, 0, _lib.LAMB_EINVAL),                                   # gradient dtype
        ([ok], _lib.LAMB_GRAD_F32, 12, _lib.LAMB_EINVAL),                 # chunk size
        ([(0, 8192, 12288, 16384, 256, 1)], _lib.LAMB_GRAD_F32, 0, _lib.LAMB_ENULL),
        ([(4100, 8192, 12288, 16384, 256, 1)], _lib.LAMB_GRAD_F32, 0, _lib.LAMB_EALIGN),
        ([(4096, 4608, 12288, 16384, 256, 1)], _lib.LAMB_GRAD_F32, 0, _lib.LAMB_EOVERLAP),
        # 2^22 elements in chunks of 8: 524,288 chunks fit, one element more does not
        ([(1 << 30, 1 << 31, 3 << 30, 1 << 32, (1 << 22) + 1, 1)], _lib.LAMB_GRAD_F32, 8,
         _lib.LAMB_EINVAL),
    ]
    for rows, g_dtype, chunk, status in cases:
        with pytest.raises(_lib.LambError) as e:
            _lib.lamb_step_static(rows, g_dtype, hp, chunk)
        assert e.value.status == status, (rows[:1], g_dtype, chunk, _lib.last_error())
    bad = _lib.lamb_hparams_init("lamb", beta1=1.5)
    with pytest.raises(_lib.LambError) as e:
        _lib.lamb_step_static([ok], _lib.LAMB_GRAD_F32, bad, 0)
    assert e.value.status == _lib.LAMB_EINVAL
