"""The arithmetic behind fp16 weights on the fp16 matrix cores (CPU only).

Several-vector launches with only fp16 weights scale each chunk of each x
vector by 2^k (k = 14 - e, e the binary exponent of the chunk's largest |x|,
clamped to +-126) and split x 2^k into two fp16 parts, both rounded to
nearest.  include/tvl.h states: the largest |x| 2^k lies in [2^13, 2^14), and
x 2^k = hi + lo + r with |r| <= 2^-22 |x 2^k| + 2^-25.  This checks those two
statements with numpy's IEEE binary16 rounding, on random values over the
whole fp32 range and on values at the fp16 rounding and subnormal
boundaries.

The absolute 2^-25 is what limits the split: a chunk whose range is wider
than the two parts hold (a huge entry next to small ones) loses the small
ones, and if the weight under the huge entry is zero, S = sum_j |W_ij x_j|
does not see the huge entry, so the lost part is all of the result.  The
kernels therefore send a chunk in which any nonzero |x 2^k| is below 2^-7 to
the fp32 matrix cores (the weights converted exactly, x as it is), and the
threshold 2^-7 gives every element on the split path
|r| <= max(2^-22 |v|, 2^-25) <= 2^-18 |v|, so the split adds at most
2^-18 S to the error of the fp32 forms, for every finite x.  The model of one chunk's dot product below checks that bound,
shows the hole it closes, and measures how often the fp32 path is taken for
x ~ N(0, 1).  The GPU tests check the kernels' results against the oracle.
"""
from __future__ import annotations

import math

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


# --------------------------------------------- one chunk's dot product (model)
SPLIT_MIN = 2.0 ** -7  # a nonzero |x 2^k| below this sends the chunk to fp32


def needs_fp32(chunk) -> bool:
    """The kernels' test, for one vector's chunk (the kernels take the fp32
    path for the whole wavefront when any of its vectors needs it)."""
    _, v, _, _ = split(chunk)
    a = np.abs(v)
    return bool(np.any((a != 0) & (a < SPLIT_MIN)))


def chunk_dot(w16, chunk, guard=True):
    """sum_j w_j x_j for fp16 weights w16 and an fp32 chunk as the kernel
    forms it, in exact arithmetic apart from the split (the fp32
    accumulation, shared by every form, is left out): the split path sums
    w_j (hi_j + lo_j) 2^-k (fp16 products are exact), the fp32 path w_j x_j.
    guard=False models the form without the fp32 path."""
    w = np.asarray(w16, np.float16).astype(np.float64)
    x = np.asarray(chunk, np.float32)
    if guard and needs_fp32(x):
        return math.fsum(w * x.astype(np.float64)), "f32"
    k, _, hi, lo = split(x)
    parts = w * hi.astype(np.float64) + w * lo.astype(np.float64)  # exact in double
    return math.ldexp(math.fsum(parts), -k), "split"


def chunk_err(w16, chunk, guard=True):
    """(|model - exact| / S, path), S = sum_j |w_j x_j| (0/0 = 0)."""
    w = np.asarray(w16, np.float16).astype(np.float64)
    x = np.asarray(chunk, np.float32).astype(np.float64)
    exact = math.fsum(w * x)
    S = math.fsum(np.abs(w * x))
    got, path = chunk_dot(w16, chunk, guard)
    if S == 0.0:
        return (0.0 if got == 0.0 else math.inf), path
    return abs(got - exact) / S, path


def test_wide_chunk_family():
    """x = (2^p, 1, ..., 1) with the weight under 2^p zero and positive
    weights elsewhere: without the fp32 path the ones vanish once 2^-k puts
    them at or below half the smallest fp16 subnormal (p >= 38: error 1, the
    whole result); with it, exact."""
    rng = np.random.default_rng(5)
    w = np.abs(rng.standard_normal(128)).astype(np.float16)
    w[0] = 0.0
    for p in range(26, 61):
        x = np.ones(128, np.float32)
        x[0] = 2.0 ** p
        old, path_old = chunk_err(w, x, guard=False)
        new, path = chunk_err(w, x)
        assert path_old == "split" and path == "f32" and new == 0.0
        if p >= 38:
            assert old == 1.0, (p, old)  # the ones are gone entirely
    # the same with the huge value negative, in the middle, and tiny ones
    x = np.full(128, 3e-30, np.float32)
    x[77] = -1e10
    w = -np.abs(rng.standard_normal(128)).astype(np.float16)
    w[77] = 0.0
    assert chunk_err(w, x, guard=False)[0] == 1.0
    assert chunk_err(w, x) == (0.0, "f32")


def test_split_path_elementwise_bound():
    """Every chunk that passes the test keeps |r_j| <= 2^-18 |x_j 2^k|."""
    rng = np.random.default_rng(6)
    n_split = 0
    for _ in range(3000):
        lo_e, hi_e = sorted(rng.uniform(-130, 127, size=2))
        hi_e = min(hi_e, lo_e + rng.uniform(0, 30))  # ranges around the threshold
        x = (rng.choice([-1.0, 1.0], 128) * 2.0 ** rng.uniform(lo_e, hi_e, 128)).astype(np.float32)
        x[rng.random(128) < 0.1] = 0.0
        if needs_fp32(x):
            continue
        n_split += 1
        _, v, hi, lo = split(x)
        r = v.astype(np.float64) - hi.astype(np.float64) - lo.astype(np.float64)
        assert np.all(np.abs(r) <= 2.0 ** -18 * np.abs(v.astype(np.float64)))
    assert n_split > 500


def test_chunk_bound_over_random_data():
    """|model - exact| <= 2^-18 S for random weights (some zero under the
    largest entries) and x over every range, on both paths."""
    rng = np.random.default_rng(7)
    worst = 0.0
    for _ in range(3000):
        lo_e, hi_e = sorted(rng.uniform(-120, 120, size=2))
        x = (rng.choice([-1.0, 1.0], 128) * 2.0 ** rng.uniform(lo_e, hi_e, 128)).astype(np.float32)
        x[rng.random(128) < 0.05] = 0.0
        w = (rng.standard_normal(128) * 2.0 ** rng.integers(-20, 10)).astype(np.float16)
        w[np.argsort(-np.abs(x))[:rng.integers(0, 4)]] = 0.0
        err, _ = chunk_err(w, x)
        worst = max(worst, err)
    assert worst <= 2.0 ** -18, worst


def test_fp32_path_is_rare_for_normal_x():
    """How often a 128-column chunk of 16 x ~ N(0, 1) vectors takes the fp32
    path: an entry below about 2^-20..2^-21 of its vector's largest, ~0.3 %
    of chunks (each costs four times the matrix-core steps of a split
    chunk)."""
    rng = np.random.default_rng(8)
    n, hits = 4000, 0
    for _ in range(n):
        X = rng.standard_normal((16, 128)).astype(np.float32)
        hits += any(needs_fp32(X[b]) for b in range(16))
    assert 0.0005 < hits / n < 0.01, hits / n
