"""Bit identity of the library's device primitives with the host (U2): Philox4x32-10 against the
oracle's on 8.4 million random counters and three keys; the deterministic fp64 log, exp and
cos against the oracle's on the input ranges the simulator uses and far beyond; fp64 square root
and division against numpy (both correctly rounded by IEEE 754), on a few million inputs each."""
import ctypes as C

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

PHILOX, LOG, EXP, COS, SQRT, DIV = range(6)


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_05272_amd import _lib
    return _lib.load()


def run(lib, kind, x, key=0, out_dtype=np.float64, out_shape=None):
    xd = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    n = x.shape[0]
    shape = out_shape if out_shape is not None else (n,)
    od = torch.empty(shape, dtype=torch.float64 if out_dtype == np.float64 else torch.int32,
                     device="cuda")
    rc = lib.sim_device_primitive(kind, n, C.c_uint64(key), C.c_void_p(xd.data_ptr()),
                                  C.c_void_p(od.data_ptr()), None)
    assert rc == 0, lib.sim_last_error()
    torch.cuda.synchronize()
    return od.cpu().numpy().view(out_dtype)


def test_philox_bit_identical(lib, orc):
    rng = np.random.default_rng(1)
    n = 1 << 23
    ctr = rng.integers(0, 2 ** 32, size=(n, 4), dtype=np.uint64).astype(np.uint32)
    ctr[:16] = 0
    ctr[16:32] = 0xFFFFFFFF
    for key in (0, 0x5EED0005, 0xFFFFFFFFFFFFFFFF):
        got = run(lib, PHILOX, ctr, key, np.uint32, (n, 4)).reshape(n, 4)
        ref = orc.philox4x32_batch(ctr[: n // 8], key)
        assert np.array_equal(got[: n // 8], ref), hex(key)
        # and the rest spot-checked every 97th counter
        idx = np.arange(n // 8, n, 97)
        assert np.array_equal(got[idx], orc.philox4x32_batch(ctr[idx], key)), hex(key)


def fp64_inputs(rng, n, lo_exp, hi_exp):
    """Positive doubles spread uniformly in log2 space over [2^lo, 2^hi], plus random mantissas."""
    e = rng.uniform(lo_exp, hi_exp, n)
    return np.ldexp(rng.uniform(1.0, 2.0, n), np.floor(e).astype(np.int64))


def test_det_log_bit_identical(lib, orc):
    rng = np.random.default_rng(2)
    x = np.concatenate([
        (rng.integers(0, 2 ** 53, 2_000_000) + 0.5) * 2.0 ** -53,   # the uniforms it is applied to
        fp64_inputs(rng, 2_000_000, -1020, 1020),
        np.array([1.0, 2.0, 0.5, 1.0 - 2.0 ** -53, 1.0 + 2.0 ** -52, 2.2250738585072014e-308,
                  1.7976931348623157e308]),
    ])
    assert np.array_equal(run(lib, LOG, x).view(np.uint64), orc.det_log(x).view(np.uint64))


def test_det_exp_bit_identical(lib, orc):
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.uniform(-40.0, 40.0, 2_000_000), rng.uniform(-700.0, 700.0, 1_000_000),
                        rng.normal(0.0, 1e-3, 500_000),
                        np.array([0.0, -0.0, 1.0, -1.0, 709.0, -708.0, 1e-300])])
    assert np.array_equal(run(lib, EXP, x).view(np.uint64), orc.det_exp(x).view(np.uint64))


def test_det_cos_bit_identical(lib, orc):
    rng = np.random.default_rng(4)
    u = (rng.integers(0, 2 ** 53, 2_000_000) + 0.5) * 2.0 ** -53
    x = np.concatenate([2.0 * np.pi * u, rng.uniform(-20.0, 20.0, 1_000_000),
                        np.array([0.0, np.pi / 2, np.pi, 1.5 * np.pi, 2 * np.pi])])
    assert np.array_equal(run(lib, COS, x).view(np.uint64), orc.det_cos(x).view(np.uint64))


def test_sqrt_and_division_correctly_rounded(lib):
    rng = np.random.default_rng(5)
    x = np.concatenate([fp64_inputs(rng, 3_000_000, -1000, 1000),
                        np.array([0.0, 1.0, 2.0, 4.0, 2.2250738585072014e-308])])
    assert np.array_equal(run(lib, SQRT, x).view(np.uint64), np.sqrt(x).view(np.uint64))
    a = fp64_inputs(rng, 3_000_000, -500, 500) * rng.choice([-1.0, 1.0], 3_000_000)
    b = fp64_inputs(rng, 3_000_000, -500, 500)
    pairs = np.stack([a, b], axis=1).reshape(-1)
    got = run(lib, DIV, pairs.reshape(-1, 2), out_shape=(3_000_000,))
    assert np.array_equal(got.view(np.uint64), (a / b).view(np.uint64))


def test_primitive_argument_errors(lib):
    assert lib.sim_device_primitive(9, 1, C.c_uint64(0), None, None, None) == -1
    assert lib.sim_device_primitive(LOG, -1, C.c_uint64(0), None, None, None) == -1
    assert lib.sim_device_primitive(LOG, 4, C.c_uint64(0), None, None, None) == -1
    assert lib.sim_device_primitive(LOG, 0, C.c_uint64(0), None, None, None) == 0
