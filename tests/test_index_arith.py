"""The band and pass kernels split an index x into x = q d + r with
q = trunc(RN((x + 1/2) RN(1/d))) in fp32 and no correction step. The
arithmetic fact this rests on: (x + 1/2)/d lies at least 1/(2d) from an
integer, and fp32 rounding of the reciprocal and the product moves it by
less than that while x < 2^22. Checked here in numpy's IEEE fp32 (the same
round-to-nearest-even adds and multiplies the GPU executes) for every
divisor up to 2^14 and every index below 2^14, the ranges the kernels use,
and on sampled indices up to 2^22."""
import numpy as np


def _quotient(x, d):
    r = np.float32(1.0 / d)                     # the plan's RN(1/d) from fp64
    assert r == np.float32(1.0) / np.float32(d)  # the device's fp32 division agrees
    p = (x.astype(np.float32) + np.float32(0.5)) * r
    return p.astype(np.int64)                   # truncation, as v_cvt_i32_f32


def test_quotient_exact_for_kernel_ranges():
    x = np.arange(1 << 14, dtype=np.int64)
    for d in range(1, (1 << 14) + 1):
        q = _quotient(x, d)
        assert np.array_equal(q, x // d), d


def test_quotient_exact_up_to_2_22_sampled():
    rng = np.random.default_rng(7)
    for d in list(range(1, 4097)) + list(rng.integers(4097, 1 << 22, 512)):
        x = np.concatenate([rng.integers(0, 1 << 22, 2048), (1 << 22) - 1 - np.arange(16)])
        assert np.array_equal(_quotient(x, int(d)), x // int(d)), d
