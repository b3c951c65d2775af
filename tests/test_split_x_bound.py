"""The arithmetic behind fp16 weights on the fp16 matrix cores (CPU only).

Several-vector launches with only fp16 weights scale each chunk of each x
vector by 2^k (k = 14 - e, e the binary exponent of the chunk's largest |x|,
clamped to +-126) and split x 2^k into two fp16 parts, both rounded to
nearest.  include/tvl.h states: the largest |x| 2^k lies in [2^13, 2^14), and
x 2^k = hi + lo + r with |r| <= 2^-22 |x 2^k| + 2^-25.  This checks those two
statements with numpy's IEEE binary16 rounding, on random values over the
whole fp32 range and on values at the fp16 rounding and subnormal
boundaries; the GPU tests check the kernels' results against the oracle.
"""
from __future__ import annotations

import numpy as np


def split(chunk):
    chunk = np.asarray(chunk, np.float32)
    m = float(np.max(np.abs(chunk)))
    e = int(np.frexp(np.float32(m))[1]) if 0.0 < m < np.inf else 0
    k = min(max(14 - e, -126), 126)
    v = (chunk * np.float32(2.0 ** k)).astype(np.float32)  # exact: a power of two
    hi = v.astype(np.float16)
    lo = (v - hi.astype(np.float32)).astype(np.float16)
    return k, v, hi, lo


def check(chunk):
    k, v, hi, lo = split(chunk)
    m = np.max(np.abs(v))
    if np.max(np.abs(chunk)) >= 2.0 ** -112:  # the scale is not clamped
        assert 2.0 ** 13 <= m < 2.0 ** 14 or m == 0.0
    assert np.all(np.isfinite(hi)) and np.all(np.isfinite(lo))
    # v - hi is exact in fp32; the residual in double
    r = v.astype(np.float64) - hi.astype(np.float64) - lo.astype(np.float64)
    assert np.all(np.abs(r) <= 2.0 ** -22 * np.abs(v.astype(np.float64)) + 2.0 ** -25), (
        chunk[np.argmax(np.abs(r))])


def test_random_chunks_over_the_fp32_range():
    rng = np.random.default_rng(11)
    for _ in range(2000):
        lo_e, hi_e = sorted(rng.uniform(-140, 127, size=2))
        mag = 2.0 ** rng.uniform(lo_e, hi_e, size=128)
        chunk = (rng.choice([-1.0, 1.0], size=128) * mag).astype(np.float32)
        chunk[rng.random(128) < 0.05] = 0.0
        check(chunk)


def test_boundary_values():
    big = np.float32(2.0 ** 13)
    # halfway and near-halfway cases of the fp16 rounding at the top of the
    # range, values whose low part is subnormal or zero, fp32 subnormals
    ulp = 2.0 ** (13 - 10)
    vals = [big, big + ulp / 2, big + ulp / 2 + 2.0 ** -11, -(big - ulp / 4), 2.0 ** -14,
            2.0 ** -15 + 2.0 ** -30, 2.0 ** -24, 3 * 2.0 ** -26, 1.0, 1.0 + 2.0 ** -23, 0.0]
    check(np.array(vals, np.float32))
    check(np.array([2.0 ** 127 * 1.999, 1e-40, -1e-38, 3.0], np.float32))
    check(np.array([1e-45, -1e-45, 0.0], np.float32))  # only fp32 subnormals: k clamped
    check(np.zeros(8, np.float32))


def test_largest_value_maps_below_the_fp16_maximum():
    for e in range(-125, 128):
        x = np.float32(np.nextafter(np.float32(2.0 ** e), np.float32(0)))  # just below 2^e
        _, v, hi, _ = split([x])
        assert abs(float(hi[0])) <= 2.0 ** 14 < 65504.0
