"""Pins of the CPU oracle against what the mathematics fixes (CPU only).

The oracle computes the GEMV of Kilictas & Alpay, arXiv 2601.03324, Sec. 6.1
(y = W x, row-major, every column summed) in double.  The paper prints no
numeric GEMV example, so the oracle is pinned by:

  * hand-worked cases (tests/golden/gemv_small.json),
  * exact rational arithmetic (fractions.Fraction) on tiny inputs, within the
    bound the oracle's only rounding (a sequential double sum) allows,
  * closed forms: identity W, all-ones rows (against math.fsum), one-hot x,
    zero rows, integer-valued W and x (exact), linearity,
  * the binary16 definition over all 65,536 bit patterns (against numpy),
  * the parity norm's rules (S = 0, non-finite outputs, the tolerance edge).

Each pin is a plain function so that ``test_mutants_are_caught`` can run the
whole suite against deliberately broken copies of the oracle and show that
every plausible mistake is caught by at least one pin.
"""
from __future__ import annotations

import json
import math
import os
import shutil
import subprocess
from fractions import Fraction

import numpy as np
import pytest

import oracle

U = 2.0 ** -53  # unit roundoff of double
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "gemv_small.json")


def _fr(v) -> Fraction:
    return Fraction(float(v))


def _mixed_f32(rng, n, lo=-40, hi=40):
    """fp32 values with random signs and exponents spread over 2^lo .. 2^hi."""
    v = rng.standard_normal(n) * np.exp2(rng.integers(lo, hi, n).astype(np.float64))
    return v.astype(np.float32)


# --------------------------------------------------------------------- pins
def pin_golden():
    cases = json.load(open(GOLDEN))["cases"]
    for c in cases:
        M, K, ldw = c["M"], c["K"], c["ldw"]
        x = np.array(c["x"], np.float32)
        if c["dtype"] == "f32":
            W = np.array([float(v) for v in c["W"]], np.float32).reshape(M, ldw)
            y, S = oracle.gemv_f32(W, x, K)
        else:
            W = np.array(c["W_bits"], np.uint16).reshape(M, ldw)
            y, S = oracle.gemv_f16(W, x, K)
        assert list(y) == c["y"], (c["name"], y)
        assert list(S) == c["S"], (c["name"], S)


def pin_products_exact():
    """Each product is exact in double: K = 1 GEMVs against Fraction products."""
    rng = np.random.default_rng(11)
    w = _mixed_f32(rng, 2000, -60, 60)
    for xv in _mixed_f32(rng, 12, -60, 60):
        y, S = oracle.gemv_f32(w.reshape(-1, 1), np.array([xv], np.float32))
        for i in range(len(w)):
            p = _fr(w[i]) * _fr(xv)
            assert Fraction(y[i]) == p
            assert Fraction(S[i]) == abs(p)
    # binary16 weights: every finite pattern times a few x
    bits = np.arange(0, 65536, dtype=np.uint16)
    fin = np.isfinite(bits.view(np.float16))
    bits = bits[fin]
    for xv in (np.float32(1.0), np.float32(-3.0517578e-05), np.float32(1234.5677)):
        y, _ = oracle.gemv_f16(bits.reshape(-1, 1), np.array([xv], np.float32))
        ref = bits.view(np.float16).astype(np.float64) * np.float64(xv)
        # exact: 11 x 24 significand bits fit in 53
        assert np.array_equal(y, ref)


def pin_brute_force_exact():
    """Tiny random GEMVs against exact rational sums:
    |y - exact| <= (K-1) u S and |S - S_exact| <= (K-1) u S_exact."""
    rng = np.random.default_rng(12)
    for trial in range(40):
        M = int(rng.integers(1, 9))
        K = int(rng.integers(1, 33))
        ldw = K + int(rng.integers(0, 5))
        W = np.full((M, ldw), np.nan, np.float32)
        W[:, :K] = _mixed_f32(rng, M * K, -20, 20).reshape(M, K)
        x = _mixed_f32(rng, K, -20, 20)
        y, S = oracle.gemv_f32(W, x, K)
        for i in range(M):
            prods = [_fr(W[i, j]) * _fr(x[j]) for j in range(K)]
            ex = sum(prods, Fraction(0))
            sx = sum((abs(p) for p in prods), Fraction(0))
            bound = (K - 1) * U * float(sx)
            assert abs(float(Fraction(y[i]) - ex)) <= bound, (trial, i)
            assert abs(float(Fraction(S[i]) - sx)) <= bound, (trial, i)


def pin_brute_force_exact_f16():
    rng = np.random.default_rng(13)
    for trial in range(30):
        M = int(rng.integers(1, 7))
        K = int(rng.integers(1, 40))
        ldw = K + int(rng.integers(0, 3))
        bits = rng.integers(0, 65536, (M, ldw)).astype(np.uint16)
        # keep finite weights only (replace Inf/NaN exponent patterns by zero)
        bits[(bits & 0x7C00) == 0x7C00] = 0
        x = _mixed_f32(rng, K, -10, 10)
        y, S = oracle.gemv_f16(bits, x, K)
        wf = bits.view(np.float16)
        for i in range(M):
            prods = [_fr(wf[i, j]) * _fr(x[j]) for j in range(K)]
            ex = sum(prods, Fraction(0))
            sx = sum((abs(p) for p in prods), Fraction(0))
            bound = (K - 1) * U * float(sx)
            assert abs(float(Fraction(y[i]) - ex)) <= bound
            assert abs(float(Fraction(S[i]) - sx)) <= bound


def pin_index_and_stride():
    """Non-square integer W in a padded row stride against Python integers."""
    rng = np.random.default_rng(14)
    for M, K, ldw in ((5, 7, 9), (7, 5, 32), (1, 13, 13), (9, 1, 4)):
        Wi = rng.integers(-9, 10, (M, K))
        xi = rng.integers(-9, 10, K)
        W = np.full((M, ldw), np.nan, np.float32)
        W[:, :K] = Wi
        y, S = oracle.gemv_f32(W, xi.astype(np.float32), K)
        for i in range(M):
            assert y[i] == sum(int(Wi[i, j]) * int(xi[j]) for j in range(K))
            assert S[i] == sum(abs(int(Wi[i, j]) * int(xi[j])) for j in range(K))
        Wb = np.full((M, ldw), 0x7E00, np.uint16)  # NaN padding
        Wb[:, :K] = Wi.astype(np.float16).view(np.uint16)
        y16, _ = oracle.gemv_f16(Wb, xi.astype(np.float32), K)
        assert np.array_equal(y16, y)


def pin_identity():
    rng = np.random.default_rng(15)
    for K in (1, 17, 256):
        x = _mixed_f32(rng, K)
        y, _ = oracle.gemv_f32(np.eye(K, dtype=np.float32), x)
        assert np.array_equal(y, x.astype(np.float64))
        y16, _ = oracle.gemv_f16(np.eye(K, dtype=np.float16).view(np.uint16), x)
        assert np.array_equal(y16, x.astype(np.float64))


def pin_all_ones_rows():
    """y_i = sum_j x_j: against math.fsum (correctly rounded)."""
    rng = np.random.default_rng(16)
    for K in (1, 3, 768, 4099):
        x = _mixed_f32(rng, K, -30, 30)
        y, S = oracle.gemv_f32(np.ones((2, K), np.float32), x)
        ref = math.fsum(float(v) for v in x)
        tol = max(K - 1, 0) * U * math.fsum(abs(float(v)) for v in x) + abs(ref) * U
        assert abs(y[0] - ref) <= tol and abs(y[1] - ref) <= tol


def pin_integer_exact():
    """Integer W in [-3, 3], x in [-8, 8], K <= 4096: every partial sum is an
    integer below 2^53, so the result is exact; compare with numpy int64."""
    rng = np.random.default_rng(17)
    for M, K in ((32, 4096), (3, 1000)):
        Wi = rng.integers(-3, 4, (M, K))
        xi = rng.integers(-8, 9, K)
        ref = Wi.astype(np.int64) @ xi.astype(np.int64)
        y, S = oracle.gemv_f32(Wi.astype(np.float32), xi.astype(np.float32))
        assert np.array_equal(y, ref.astype(np.float64))
        assert np.array_equal(S, (np.abs(Wi) @ np.abs(xi)).astype(np.float64))
        y16, _ = oracle.gemv_f16(Wi.astype(np.float16).view(np.uint16), xi.astype(np.float32))
        assert np.array_equal(y16, ref.astype(np.float64))


def pin_linearity():
    """W(a x + b z) = a W x + b W z, exactly, with integer data."""
    rng = np.random.default_rng(18)
    M, K = 16, 300
    W = rng.integers(-5, 6, (M, K)).astype(np.float32)
    x = rng.integers(-7, 8, K)
    z = rng.integers(-7, 8, K)
    a, b = 3, -2
    lhs, _ = oracle.gemv_f32(W, (a * x + b * z).astype(np.float32))
    yx, _ = oracle.gemv_f32(W, x.astype(np.float32))
    yz, _ = oracle.gemv_f32(W, z.astype(np.float32))
    assert np.array_equal(lhs, a * yx + b * yz)


def pin_one_hot():
    """x = e_j picks column j of W exactly."""
    rng = np.random.default_rng(19)
    M, K = 37, 29
    W = _mixed_f32(rng, M * K).reshape(M, K)
    Wb = rng.integers(0, 0x7C00, (M, K)).astype(np.uint16)  # finite, nonnegative
    for j in (0, 5, K - 1):
        e = np.zeros(K, np.float32)
        e[j] = 1.0
        y, S = oracle.gemv_f32(W, e)
        assert np.array_equal(y, W[:, j].astype(np.float64))
        assert np.array_equal(S, np.abs(W[:, j]).astype(np.float64))
        y16, _ = oracle.gemv_f16(Wb, e)
        assert np.array_equal(y16, Wb[:, j].view(np.float16).astype(np.float64))


def pin_zero_row():
    W = np.zeros((3, 10), np.float32)
    W[1] = 1.0
    x = np.arange(10, dtype=np.float32) - 4.5
    y, S = oracle.gemv_f32(W, x)
    assert y[0] == 0.0 and S[0] == 0.0 and y[2] == 0.0 and S[2] == 0.0
    assert y[1] == float(x.astype(np.float64).sum())


def pin_f16_decode_all_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([oracle.f16_to_f64(int(b)) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signs of zero and of every finite value match (bitwise on non-NaN)
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def pin_f16_subnormal_gemv():
    """W = 2^-24 (smallest binary16 subnormal) everywhere: y = 2^-24 sum x."""
    rng = np.random.default_rng(20)
    K = 777
    xi = rng.integers(-50, 51, K).astype(np.float32)
    y, _ = oracle.gemv_f16(np.full((4, K), 1, np.uint16), xi)
    assert np.all(y == math.ldexp(float(xi.astype(np.int64).sum()), -24))


def pin_check_rules():
    y_ref = np.array([1.0, 0.0, 0.0, 2.0, -3.0])
    S = np.array([2.0, 0.0, 0.0, 4.0, 6.0])
    y = np.array([1.0, 0.0, -0.0, 2.0, -3.0], np.float32)
    r = oracle.check(y, y_ref, S, 1e-5)
    assert r["bad"] == 0 and r["max_err"] == 0.0
    # S = 0 requires an exact zero
    r = oracle.check(np.array([1.0, 1e-30, 0, 2.0, -3.0], np.float32), y_ref, S, 1e-5)
    assert r["bad"] == 1 and r["argmax"] == 1 and math.isinf(r["max_err"])
    # non-finite outputs always fail
    for bad in (np.nan, np.inf, -np.inf):
        r = oracle.check(np.array([bad, 0, 0, 2.0, -3.0], np.float32), y_ref, S, 1e-5)
        assert r["bad"] == 1 and r["argmax"] == 0 and math.isinf(r["max_err"])
    # normalised error and the tolerance edge (err == tol passes)
    y = np.array([1.0, 0, 0, 2.0 + 0.5, -3.0], np.float32)  # err = 0.5/4
    r = oracle.check(y, y_ref, S, 0.125)
    assert r["bad"] == 0 and r["max_err"] == 0.125 and r["argmax"] == 3
    r = oracle.check(y, y_ref, S, 0.124)
    assert r["bad"] == 1
    assert r["mean_err"] == pytest.approx(0.125 / 5)


# ------------------------------------------------------------ RMSNorm pins
def pin_rmsnorm_closed_forms():
    """Sec. 11.2 listing: o_j = x_j g_j / sqrt(mean(x^2) + eps)."""
    # constant x = 2^-1, g = 1, eps = 0: mean square 1/4, inverse root 2, o = 1
    o = oracle.rmsnorm(np.full(8, 0.5, np.float32), np.ones(8, np.float32), 0.0)
    assert np.array_equal(o, np.ones(8))
    # a single nonzero entry: mean square x0^2 / K
    x = np.zeros(4, np.float32)
    x[0] = 2.0
    o = oracle.rmsnorm(x, np.full(4, 3.0, np.float32), 0.0)
    assert np.array_equal(o, np.array([6.0, 0, 0, 0]))
    # (3, 4): mean square 12.5 (eps inside the root)
    o = oracle.rmsnorm(np.array([3, 4], np.float32), np.array([1, -2], np.float32), 0.5)
    r = 1.0 / math.sqrt(13.0)
    assert abs(o[0] - 3 * r) <= 4 * U and abs(o[1] + 8 * r) <= 8 * U
    # zero x stays zero for any eps > 0
    assert np.array_equal(oracle.rmsnorm(np.zeros(5, np.float32), np.ones(5, np.float32), 1e-5),
                          np.zeros(5))


def pin_rmsnorm_invariances():
    rng = np.random.default_rng(21)
    for K in (1, 7, 768, 4096):
        x = rng.standard_normal(K).astype(np.float32)
        g = rng.standard_normal(K).astype(np.float32)
        base = oracle.rmsnorm(x, g, 0.0)
        # scale invariance (eps = 0): exact for powers of two
        for k in (-3, 5):
            xs = (x * np.float32(2.0 ** k)).astype(np.float32)
            assert np.array_equal(oracle.rmsnorm(xs, g, 0.0), base)
        # linear in g, exactly for a factor of 2
        assert np.array_equal(oracle.rmsnorm(x, (2 * g).astype(np.float32), 0.0), 2 * base)
        # against numpy's float64 formula (fsum of squares)
        ms = math.fsum(float(v) * float(v) for v in x) / K
        for eps in (0.0, 1e-5, 0.25):
            ref = x.astype(np.float64) * g.astype(np.float64) / math.sqrt(ms + eps)
            got = oracle.rmsnorm(x, g, eps)
            assert np.allclose(got, ref, rtol=(K + 8) * U, atol=0)


def pin_rmsnorm_gemv():
    """y = W rmsnorm(x): exact rational check on a dyadic case and the
    column-sum identity for an all-ones W."""
    x = np.array([1.0, -1.0, 1.0, -1.0], np.float32)  # mean square 1
    g = np.array([1.0, 2.0, 3.0, 4.0], np.float32)
    W = np.array([[1, 1, 1, 1], [0.5, 0, -2, 0], [0, 0, 0, 0]], np.float32)
    y, S = oracle.rmsnorm_gemv(W, x, g, 0.0)
    assert list(y) == [1 - 2 + 3 - 4, 0.5 - 6, 0.0]
    assert list(S) == [10.0, 6.5, 0.0]
    rng = np.random.default_rng(22)
    xr = rng.standard_normal(300).astype(np.float32)
    gr = rng.standard_normal(300).astype(np.float32)
    y, S = oracle.rmsnorm_gemv(np.ones((2, 300), np.float32), xr, gr, 1e-5)
    xn = oracle.rmsnorm(xr, gr, 1e-5)
    assert abs(y[0] - math.fsum(xn)) <= 300 * U * float(np.abs(xn).sum())
    # fp16 weights give the same as their fp32 values
    Wb = rng.integers(-3, 4, (5, 300)).astype(np.float16)
    y16, _ = oracle.rmsnorm_gemv(Wb.view(np.uint16), xr, gr, 1e-5)
    y32, _ = oracle.rmsnorm_gemv(Wb.astype(np.float32), xr, gr, 1e-5)
    assert np.array_equal(y16, y32)
    # padded rows: the stride is honoured
    Wp = np.full((5, 320), np.nan, np.float32)
    Wp[:, :300] = Wb.astype(np.float32)
    yp, _ = oracle.rmsnorm_gemv(Wp, xr, gr, 1e-5, K=300)
    assert np.array_equal(yp, y32)


# ------------------------------------------------------------- SwiGLU pins
def pin_swiglu():
    """h = silu(a) b with silu(z) = z / (1 + e^-z)."""
    from scipy.special import expit
    a = np.array([0.0, 1.0, -1.0, 2.5, -3.0, 40.0, -800.0, 1e-300])
    b = np.array([2.0, 3.0, -0.5, 1.0, 7.0, 0.5, 5.0, 1.0])
    h = oracle.swiglu(a, b)
    ref = a * expit(a) * b
    assert h[0] == 0.0 and h[5] == 20.0 and h[6] == 0.0 and np.all(np.isfinite(h))
    assert np.allclose(h, ref, rtol=4 * U, atol=0)
    assert abs(h[1] - 3.0 / (1.0 + math.exp(-1.0))) <= 4 * U * 3
    # zero gate input or zero b gives zero
    assert np.all(oracle.swiglu(np.zeros(3), np.array([1.0, -2.0, 3.0])) == 0.0)
    assert np.all(oracle.swiglu(np.array([1.0, -2.0, 3.0]), np.zeros(3)) == 0.0)


def _h_exact(a: float, b: float) -> float:
    """h = silu(a) b written out with math.exp (independent of the oracle)."""
    return a * b / (1.0 + math.exp(-a))


def pin_swiglu_bound(o=oracle):
    """The gate's normaliser N = |silu'(a)| |b| Sa + |silu(a)| Sb (Sec. 2.1
    FFN; the GEMV parity norm carried through h = silu(a) b).

    * hand-worked: at a = 0, silu = 0 and silu' = 1/2, so N = |b| Sa / 2; at
      a = 40 (saturated), silu' = 1 and silu = 40 to double precision; at
      a = -40, s = e^-40 / (1 + e^-40), silu = -40 s, silu' = s (1 - 40 (1 - s));
    * tightness: the largest change of h over the four corners
      (a +- t Sa, b +- t Sb), computed with math.exp, is t N to first order
      (within 1e-3 at t = 1e-7) for random a, b, Sa, Sb on both sides of
      silu's minimum (a = -1.278...) and on both signs of b;
    * the corner bound holds for a GPU-like error too: h moves by at most
      t N (1 + 1e-3) for every perturbation inside the box."""
    a = np.array([0.0, 0.0, 40.0, -40.0])
    b = np.array([3.0, -2.0, -0.5, 2.0])
    Sa = np.array([5.0, 1.0, 7.0, 3.0])
    Sb = np.array([4.0, 6.0, 1.5, 9.0])
    N = o.swiglu_bound(a, b, Sa, Sb)
    assert N[0] == 3.0 * 5.0 / 2 and N[1] == 2.0 * 1.0 / 2
    assert abs(N[2] - (0.5 * 7.0 + 40.0 * 1.5)) <= 1e-14 * N[2]
    s = math.exp(-40.0) / (1.0 + math.exp(-40.0))
    ref = abs(s * (1.0 - 40.0 * (1.0 - s))) * 2.0 * 3.0 + abs(-40.0 * s) * 9.0
    assert abs(N[3] - ref) <= 1e-12 * ref
    rng = np.random.default_rng(31)
    n = 400
    a = rng.uniform(-8.0, 8.0, n)
    a[:40] = rng.uniform(-1.6, -1.0, 40)  # around silu's minimum (silu' = 0)
    b = rng.uniform(-3.0, 3.0, n)
    Sa = np.abs(a) * rng.uniform(1.0, 4.0, n) + rng.uniform(0.0, 1.0, n)
    Sb = np.abs(b) * rng.uniform(1.0, 4.0, n) + rng.uniform(0.0, 1.0, n)
    N = o.swiglu_bound(a, b, Sa, Sb)
    t = 1e-7
    for i in range(n):
        h0 = _h_exact(a[i], b[i])
        dmax = max(abs(_h_exact(a[i] + sa * t * Sa[i], b[i] + sb * t * Sb[i]) - h0)
                   for sa in (-1.0, 1.0) for sb in (-1.0, 1.0))
        assert abs(dmax - t * N[i]) <= 1e-3 * t * N[i], (i, a[i], b[i], dmax, t * N[i])
        for da, db in rng.uniform(-1.0, 1.0, (4, 2)):
            d = abs(_h_exact(a[i] + da * t * Sa[i], b[i] + db * t * Sb[i]) - h0)
            assert d <= t * N[i] * (1 + 1e-3)


def pin_swiglu_ffn_in(o=oracle):
    """swiglu_ffn_in composes RMSNorm, both GEMVs and the gate: W1 and W3 see
    the same normalised x.  With x = c (a constant) the normalised x is
    g c / sqrt(c^2 + eps) (closed form); with W1 = 2 I and W3 = I,
    a = 2 xn and b = xn exactly, and h = silu(a) b."""
    K = 8
    c, eps = 3.0, 0.25
    x = np.full(K, c, np.float32)
    g = np.array([0.5, 1.0, 1.5, 2.0, -1.0, 0.25, 4.0, 3.0], np.float32)
    xn = [float(gj) * c / math.sqrt(c * c + eps) for gj in g]
    I = np.eye(K, dtype=np.float32)
    h, a, b, Sa, Sb = o.swiglu_ffn_in(2 * I, I, x, g, eps)
    for j in range(K):
        assert abs(a[j] - 2 * xn[j]) <= 4 * U * abs(xn[j])
        assert abs(b[j] - xn[j]) <= 4 * U * abs(xn[j])
        assert Sa[j] == abs(a[j]) and Sb[j] == abs(b[j])
        assert abs(h[j] - _h_exact(2 * xn[j], xn[j])) <= 16 * U * abs(h[j])
    # without g the raw x goes to both GEMVs
    h, a, b, _, _ = o.swiglu_ffn_in(2 * I, I, x)
    assert np.all(a == 2 * c) and np.all(b == c)
    assert np.allclose(h, _h_exact(2 * c, c), rtol=16 * U, atol=0)
    # a fp16 W1 (bit patterns) and a fp32 W3 of the same values agree
    rng = np.random.default_rng(32)
    Wi = rng.integers(-3, 4, (5, 40)).astype(np.float16)
    xr = rng.standard_normal(40).astype(np.float32)
    gr = rng.uniform(0.5, 1.5, 40).astype(np.float32)
    h16, a16, b16, _, _ = o.swiglu_ffn_in(Wi.view(np.uint16), Wi.astype(np.float32), xr, gr)
    assert np.array_equal(a16, b16)
    assert np.allclose(h16, [_h_exact(v, v) for v in a16], rtol=16 * U, atol=0)


# --------------------------------------------------- quantised-weight pins
def _q_rows(codes: np.ndarray, scales: np.ndarray, bits: int, extra: int = 0):
    """Build a quantised matrix by hand (not with the generator's quantiser):
    codes [M, K] in the signed range, scales [M, ceil(K/64)] fp32, stored
    in blocks of 4 rows with M padded to 4 (pad entries NaN: never read).  Returns
    (buffer, ldw); code rows padded to 128 bytes (+ extra) with junk."""
    M, K = codes.shape
    ldw = ((K * bits + 7) // 8 + 127) // 128 * 128 + extra
    Mp = (M + 3) // 4 * 4
    out = np.full(M * ldw + 4 * Mp * scales.shape[1], 0xAB, np.uint8)
    rows = out[:M * ldw].reshape(M, ldw)
    if bits == 8:
        rows[:, :K] = codes.astype(np.int8).view(np.uint8)
    else:
        u = (codes & 0x0F).astype(np.uint8)  # two's complement nibbles
        for j in range(K):
            if j % 2 == 0:
                rows[:, j // 2] = (rows[:, j // 2] & 0xF0) | u[:, j]
            else:
                rows[:, j // 2] = (rows[:, j // 2] & 0x0F) | (u[:, j] << 4)
    ng = scales.shape[1]
    full = np.full((Mp, ng), np.nan, np.float32)  # pad rows NaN (never read)
    full[:M] = scales
    # blocks of 4 rows: [block][group][row in block]
    plane = full.reshape(Mp // 4, 4, ng).transpose(0, 2, 1)
    out[M * ldw:] = np.ascontiguousarray(plane).reshape(-1).view(np.uint8)
    return out, ldw


def pin_quant_golden():
    """Hand-worked 4-bit row: codes (1, -2, 7), scale 1/2, x = (2, 1, -1):
    w = (0.5, -1, 3.5), y = 1 - 1 - 3.5 = -3.5, S = 5.5."""
    Wq, ldw = _q_rows(np.array([[1, -2, 7]]), np.array([[0.5]], np.float32), 4)
    assert Wq[0] == 0xE1 and Wq[1] & 0x0F == 0x07 and ldw == 128
    y, S = oracle.gemv_q(Wq, 4, ldw, 1, 3, np.array([2, 1, -1], np.float32))
    assert y[0] == -3.5 and S[0] == 5.5
    # the extreme 4-bit codes, low nibble first: byte 0x78 holds column 0 =
    # nibble 0x8 = -8 and column 1 = nibble 0x7 = 7
    Wq = np.zeros(128 + 16, np.uint8)  # one code row, scale plane of 1 group x 4 rows
    Wq[0] = 0x78
    Wq[128:] = np.array([0.25, np.nan, np.nan, np.nan], np.float32).view(np.uint8)
    y, S = oracle.gemv_q(Wq, 4, 128, 1, 2, np.array([1, 2], np.float32))
    assert y[0] == 0.25 * (-8 + 14) and S[0] == 0.25 * (8 + 14)
    # 8-bit, two rows: codes (-128, 127, 3) with scale 2^-3, (1, 1, 1) with scale 2
    Wq, ldw = _q_rows(np.array([[-128, 127, 3], [1, 1, 1]]),
                      np.array([[0.125], [2.0]], np.float32), 8)
    y, S = oracle.gemv_q(Wq, 8, ldw, 2, 3, np.array([1, 1, -4], np.float32))
    assert y[0] == (-128 + 127 - 12) * 0.125 and S[0] == (128 + 127 + 12) * 0.125
    assert y[1] == 2.0 * (1 + 1 - 4) and S[1] == 2.0 * 6


def pin_quant_matches_dequantized():
    """Power-of-two scales make every dequantised weight exact in fp32: the
    quantised oracle must then equal the fp32 oracle on numpy's dequantised
    matrix bit for bit, across group boundaries, ragged K and wide rows."""
    rng = np.random.default_rng(23)
    for bits, lo, hi in ((8, -128, 127), (4, -8, 7)):
        for M, K, extra in ((5, 1, 0), (7, 63, 128), (3, 64, 0), (9, 130, 0), (4, 1000, 256)):
            codes = rng.integers(lo, hi + 1, (M, K))
            scales = np.exp2(rng.integers(-12, 3, (M, (K + 63) // 64))).astype(np.float32)
            Wq, ldw = _q_rows(codes, scales, bits, extra)
            deq = (codes * np.repeat(scales, 64, axis=1)[:, :K]).astype(np.float32)
            x = rng.standard_normal(K).astype(np.float32)
            yq, Sq = oracle.gemv_q(Wq, bits, ldw, M, K, x)
            yf, Sf = oracle.gemv_f32(deq, x)
            assert np.array_equal(yq, yf) and np.array_equal(Sq, Sf), (bits, M, K)
            # single weights at the group edges of every row
            for i in range(M):
                for j in {0, min(63, K - 1), min(64, K - 1), K - 1}:
                    assert oracle.q_weight(Wq, bits, ldw, M, K, i, j) == float(deq[i, j])


def pin_quant_exact_rational():
    """Arbitrary fp32 scales (not powers of two): against exact rational sums of
    s * q * x.  A product s q x can need 24 + 8 + 24 significand bits, more
    than double holds, so the bound is K * 2^-52 * S (product and sum
    roundings), not equality."""
    from fractions import Fraction
    rng = np.random.default_rng(24)
    for bits, lo, hi in ((8, -127, 127), (4, -7, 7)):
        for M, K in ((1, 1), (3, 65), (4, 130), (2, 200)):
            codes = rng.integers(lo, hi + 1, (M, K))
            scales = rng.uniform(1e-3, 1.0, (M, (K + 63) // 64)).astype(np.float32)
            Wq, ldw = _q_rows(codes, scales, bits)
            x = rng.standard_normal(K).astype(np.float32)
            y, S = oracle.gemv_q(Wq, bits, ldw, M, K, x)
            for i in range(M):
                exact = sum(Fraction(float(scales[i, j // 64])) * int(codes[i, j])
                            * Fraction(float(x[j])) for j in range(K))
                s_abs = sum(abs(Fraction(float(scales[i, j // 64])) * int(codes[i, j])
                                * Fraction(float(x[j]))) for j in range(K))
                assert abs(Fraction(y[i]) - exact) <= K * Fraction(2) ** -52 * s_abs, (bits, M, K, i)
                assert abs(Fraction(S[i]) - s_abs) <= K * Fraction(2) ** -52 * s_abs


PINS = [pin_golden, pin_products_exact, pin_brute_force_exact, pin_brute_force_exact_f16,
        pin_index_and_stride, pin_identity, pin_all_ones_rows, pin_integer_exact,
        pin_linearity, pin_one_hot, pin_zero_row, pin_f16_decode_all_patterns,
        pin_f16_subnormal_gemv, pin_check_rules, pin_rmsnorm_closed_forms,
        pin_rmsnorm_invariances, pin_rmsnorm_gemv, pin_swiglu, pin_swiglu_bound,
        pin_swiglu_ffn_in, pin_quant_golden,
        pin_quant_matches_dequantized, pin_quant_exact_rational]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_oracle_pin(pin):
    pin()


# ------------------------------------------------------------------ mutants
# Plausible mistakes, each applied to a private copy of oracle.c.  None of
# them may survive the pins above.  (Mutants that could read out of bounds
# are not used: they would crash the test process rather than fail a pin.)
MUTANTS = {
    "dropped_last_term_f32": ("for (int64_t j = 0; j < K; ++j) {\n            const double p = (double)row[j]",
                              "for (int64_t j = 0; j < K - 1; ++j) {\n            const double p = (double)row[j]"),
    "dropped_last_term_f16": ("for (int64_t j = 0; j < K; ++j) {\n            const double p = oracle_f16",
                              "for (int64_t j = 1; j < K; ++j) {\n            const double p = oracle_f16"),
    "stride_K_not_ldw_f32": ("const float *row = W + i * ldw;", "const float *row = W + i * K;"),
    "stride_K_not_ldw_f16": ("const uint16_t *row = W + i * ldw;", "const uint16_t *row = W + i * K;"),
    "product_rounded_to_f32": ("(double)row[j] * (double)x[j]", "(double)(row[j] * x[j])"),
    "float_accumulator": ("double acc = 0.0, s = 0.0;", "float acc = 0.0f; double s = 0.0;"),
    "sign_flip": ("            acc += p;", "            acc -= p;"),
    "S_not_absolute": ("            s += fabs(p);", "            s += p;"),
    "f16_subnormal_scale": ("ldexp((double)m, -24)", "ldexp((double)m, -25)"),
    "f16_exponent_bias": ("e - 25);", "e - 24);"),
    "f16_sign_dropped": ("return sign ? -v : v;", "return v;"),
    "f16_mantissa_width": ("ldexp((double)(1024 + m)", "ldexp((double)(512 + m)"),
    "check_S0_rule": ("e = (yi == 0.0) ? 0.0 : INFINITY;", "e = 0.0;"),
    "check_nonfinite": ("if (!isfinite(yi)) {", "if (0) {"),
    "check_tol_strict": ("if (e > tol) ++bad;", "if (e >= tol) ++bad;"),
    "rms_eps_outside_root": ("1.0 / sqrt(ms + eps)", "1.0 / sqrt(ms) + eps"),
    "rms_sum_not_mean": ("const double ms = ss / (double)K;", "const double ms = ss;"),
    "rms_g_dropped": ("(double)x[j] * (double)g[j] * inv", "(double)x[j] * inv"),
    "rms_no_root": ("1.0 / sqrt(ms + eps)", "1.0 / (ms + eps)"),
    "rms_abs_not_square": ("ss += (double)x[j] * (double)x[j];", "ss += fabs((double)x[j]);"),
    "gemvdx_stride": ("((const float *)W)[i * ldw + j]", "((const float *)W)[i * K + j]"),
    "gemvdx_f16_bits_as_int": ("is_f16 ? oracle_f16_to_f64(((const uint16_t *)W)[i * ldw + j])",
                               "is_f16 ? (double)(((const uint16_t *)W)[i * ldw + j])"),
    "swiglu_sign": ("a[i] / (1.0 + exp(-a[i])) * b[i]", "a[i] / (1.0 + exp(a[i])) * b[i]"),
    "swiglu_sigmoid_only": ("a[i] / (1.0 + exp(-a[i])) * b[i]", "1.0 / (1.0 + exp(-a[i])) * b[i]"),
    "swiglu_no_b": ("a[i] / (1.0 + exp(-a[i])) * b[i]", "a[i] / (1.0 + exp(-a[i]))"),
    "q_group_32": ("scales[(i / 4) * 4 * ng + 4 * (j / 64) + i % 4]",
                   "scales[(i / 4) * 4 * ng + 4 * (j / 32) + i % 4]"),
    "q_scale_row_major": ("scales[(i / 4) * 4 * ng + 4 * (j / 64) + i % 4]",
                          "scales[i * ng + j / 64]"),
    "q_scale_group_major": ("scales[(i / 4) * 4 * ng + 4 * (j / 64) + i % 4]",
                            "scales[(j / 64) * ((M + 3) / 4 * 4) + i]"),
    "q4_nibble_order": ("(j % 2 == 0) ? (byte & 0x0f) : (byte >> 4)", "(j % 2 == 0) ? (byte >> 4) : (byte & 0x0f)"),
    "q4_offset_not_twos_complement": ("q = (double)(u >= 8 ? u - 16 : u);", "q = (double)(u - 8);"),
    "q4_sign_threshold": ("q = (double)(u >= 8 ? u - 16 : u);", "q = (double)(u > 8 ? u - 16 : u);"),
    "q8_unsigned": ("q = (double)(int8_t)row[j];", "q = (double)row[j];"),
    "q_code_row_stride": ("const uint8_t *row = W + i * ldw;\n    double q;",
                          "const uint8_t *row = W + i * K * bits / 8;\n    double q;"),
}


def test_mutants_are_caught(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = open(oracle._SRC).read()
    survivors = []
    for name, (old, new) in MUTANTS.items():
        assert old in src, name
        msrc = src.replace(old, new, 1)
        cpath = tmp_path / f"{name}.c"
        cpath.write_text(msrc)
        so = tmp_path / f"lib{name}.so"
        subprocess.check_call(["gcc", *oracle.CFLAGS, "-o", str(so), str(cpath), "-lm"])
        caught = []
        with oracle.using(str(so)):
            for pin in PINS:
                try:
                    pin()
                except (AssertionError, ValueError, OverflowError):
                    # a pin that cannot even evaluate the mutant's output
                    # (NaN or Inf where an exact value belongs) catches it too
                    caught.append(pin.__name__)
        if not caught:
            survivors.append(name)
    assert not survivors, f"mutants not caught by any pin: {survivors}"


# Plausible mistakes in the Python part of the oracle (the SwiGLU gate's
# normaliser and the FFN-input composition), each applied to a private copy of
# oracle/__init__.py that still calls the real C library.
PY_MUTANTS = {
    "bound_dsilu_abs_dropped": ("np.abs(dsilu) * np.abs(b) * Sa", "dsilu * np.abs(b) * Sa"),
    "bound_silu_abs_dropped": ("np.abs(a * sig) * Sb", "a * sig * Sb"),
    "bound_Sa_Sb_swapped": ("np.abs(dsilu) * np.abs(b) * Sa + np.abs(a * sig) * Sb",
                            "np.abs(dsilu) * np.abs(b) * Sb + np.abs(a * sig) * Sa"),
    "bound_b_dropped": ("np.abs(dsilu) * np.abs(b) * Sa", "np.abs(dsilu) * Sa"),
    "bound_dsilu_is_sigmoid": ("dsilu = sig * (1.0 + a * (1.0 - sig))", "dsilu = sig"),
    "bound_dsilu_sign": ("dsilu = sig * (1.0 + a * (1.0 - sig))",
                         "dsilu = sig * (1.0 - a * (1.0 - sig))"),
    "bound_sigmoid_sign": ("sig = 1.0 / (1.0 + np.exp(-a))", "sig = 1.0 / (1.0 + np.exp(a))"),
    "bound_second_term_dropped": ("np.abs(dsilu) * np.abs(b) * Sa + np.abs(a * sig) * Sb",
                                  "np.abs(dsilu) * np.abs(b) * Sa"),
    "ffn_W3_sees_raw_x": ("b, Sb = gemv_dx(W3, xd, K)",
                          "b, Sb = gemv_dx(W3, np.asarray(x, np.float32).astype(np.float64), K)"),
    "ffn_W1_sees_raw_x": ("a, Sa = gemv_dx(W1, xd, K)",
                          "a, Sa = gemv_dx(W1, np.asarray(x, np.float32).astype(np.float64), K)"),
    "ffn_W1_W3_swapped": ("a, Sa = gemv_dx(W1, xd, K)\n    b, Sb = gemv_dx(W3, xd, K)",
                          "a, Sa = gemv_dx(W3, xd, K)\n    b, Sb = gemv_dx(W1, xd, K)"),
    "ffn_gate_on_b": ("return swiglu(a, b), a, b, Sa, Sb", "return swiglu(b, a), a, b, Sa, Sb"),
}
PY_PINS = [pin_swiglu_bound, pin_swiglu_ffn_in]


def test_python_mutants_are_caught():
    import types
    src = open(oracle.__file__).read()
    survivors = []
    for name, (old, new) in PY_MUTANTS.items():
        assert src.count(old) == 1, name
        mod = types.ModuleType("oracle_mutant_" + name)
        mod.__file__ = oracle.__file__  # same liboracle.so
        exec(compile(src.replace(old, new, 1), oracle.__file__, "exec"), mod.__dict__)
        caught = []
        for pin in PY_PINS:
            try:
                pin(mod)
            except (AssertionError, ValueError, OverflowError):
                caught.append(pin.__name__)
        if not caught:
            survivors.append(name)
    assert not survivors, f"mutants not caught by any pin: {survivors}"
