"""The seeded input generator (CPU only).

Checks it against an independent Python rendering of SplitMix64 (Steele, Lea &
Flood, OOPSLA 2014), numpy's float32 -> float16 cast (round to nearest even),
and the properties the tests and the benchmark rely on: any slice can be
regenerated on its own, the output does not depend on the thread count, and
the distributions have the requested moments.
"""
from __future__ import annotations

import os
import subprocess
import sys

import numpy as np

import synth

M64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15


def _py_splitmix64(seed: int, n: int):
    """Sequential SplitMix64: state += gamma; output mix(state)."""
    out, s = [], seed & M64
    for _ in range(n):
        s = (s + GAMMA) & M64
        z = s
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
        out.append(z ^ (z >> 31))
    return out


def test_splitmix64_matches_sequential_definition():
    for seed in (0, 1, 0xDEADBEEF, M64):
        ref = _py_splitmix64(seed, 50)
        got = [synth.u64(seed, k) for k in range(50)]
        assert got == ref
    # the widely quoted first output for seed 0
    assert synth.u64(0, 0) == 0xE220A8397B1DCDAF


def test_f16_rne_matches_numpy():
    rng = np.random.default_rng(3)
    v = np.concatenate([
        (rng.standard_normal(200000) * np.exp2(rng.integers(-30, 18, 200000))).astype(np.float32),
        np.array([0.0, -0.0, 65504.0, 65519.99, 65520.0, -65520.0, 1e9, np.inf, -np.inf,
                  2.0 ** -24, 2.0 ** -25, 2.0 ** -25 * 1.0000001, 3 * 2.0 ** -26,
                  2.0 ** -14, 2.0 ** -14 * (1 - 2 ** -11), 5.9604645e-08, 6.1035156e-05],
                 np.float32),
        # every fp32 with a tie in the dropped bits near 1.0 and in the subnormal range
        (np.float32(1.0) + np.arange(-300, 300, dtype=np.float32) * np.float32(2 ** -12)),
        (np.arange(1, 3000, dtype=np.float32) * np.float32(2 ** -25)),
    ])
    got = synth.f32_to_f16_bits(v)
    with np.errstate(over="ignore"):
        ref = v.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, ref)
    nan = synth.f32_to_f16_bits(np.array([np.nan], np.float32))
    assert np.isnan(nan.view(np.float16)[0])


def test_slices_regenerate():
    k = synth.key(9, 1, 2, 3)
    full = synth.normal_f32(10001, k, 0.02)
    part = synth.normal_f32(77, k, 0.02, offset=5001)
    assert np.array_equal(full[5001:5078], part)
    odd = synth.normal_f32(1, k, 0.02, offset=4)
    assert odd[0] == full[4]
    fu = synth.uniform_f32(1000, k, -0.05, 0.05)
    assert np.array_equal(fu[333:400], synth.uniform_f32(67, k, -0.05, 0.05, offset=333))
    h = synth.normal_f16(5000, k, 0.02)
    assert np.array_equal(h, synth.f32_to_f16_bits(synth.normal_f32(5000, k, 0.02)))


def test_thread_count_independent(tmp_path):
    code = ("import sys, numpy as np; sys.path.insert(0, %r); import synth;"
            "np.save(sys.argv[1], synth.normal_f32(300001, synth.key(2, 5, 4, 0, 0), 0.02))"
            % os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    outs = []
    for t in ("1", "5"):
        f = tmp_path / f"o{t}.npy"
        env = dict(os.environ, OMP_NUM_THREADS=t)
        subprocess.check_call([sys.executable, "-c", code, str(f)], env=env)
        outs.append(np.load(f))
    assert np.array_equal(outs[0], outs[1])


def test_moments():
    n = 1 << 20
    z = synth.normal_f32(n, synth.key(1), 1.0).astype(np.float64)
    assert abs(z.mean()) < 5 / np.sqrt(n)
    assert abs(z.var() - 1.0) < 5 * np.sqrt(2.0 / n)
    assert abs((z ** 3).mean()) < 5 * np.sqrt(15.0 / n)
    assert abs((z ** 4).mean() - 3.0) < 5 * np.sqrt(96.0 / n)
    u = synth.uniform_f32(n, synth.key(2), -0.05, 0.05).astype(np.float64)
    assert u.min() >= -0.05 and u.max() <= 0.05
    assert abs(u.mean()) < 5 * 0.1 / np.sqrt(12 * n)
    i = synth.int_f32(n, synth.key(3), -3, 3)
    assert set(np.unique(i)) == {-3, -2, -1, 0, 1, 2, 3}


def test_workload_tables():
    W = synth.WORKLOADS
    assert W["sweep110m"].algo_bytes() == 438_874_112
    assert W["sweep110m"].weight_bytes() == 438_042_624
    assert len(W["sweep110m"].mats) == 85
    assert W["sweep7b"].algo_bytes() == 26_438_448_128
    assert len(W["sweep7b"].mats) == 225
    assert W["stack70b8"].algo_bytes() == 13_695_385_600
    assert len(W["stack70b8"].mats) == 56
    assert W["gemv768"].algo_bytes() == 2_365_440
    assert W["cls32000"].algo_bytes() == 98_435_072
    plain = [wl for wl in W.values() if not wl.mats[0].quantised]
    keys = {m.w_key for wl in plain for m in wl.mats}
    assert len(keys) == sum(len(wl.mats) for wl in plain)
    # the quantised workloads quantise the fp32 draws of their source token:
    # 110M: 109,510,656 code bytes + 6,844,416 scale bytes (8-bit)
    for src, q in (("sweep110m", "sweep110m_q8"), ("sweep110m", "sweep110m_q4"),
                   ("sweep7b", "sweep7b_q8"), ("sweep7b", "sweep7b_q4")):
        assert [m.w_key for m in W[q].mats] == [m.w_key for m in W[src].mats]
        assert [(m.M, m.K) for m in W[q].mats] == [(m.M, m.K) for m in W[src].mats]
    assert W["sweep110m_q8"].weight_bytes() == 109_510_656 + 6_844_416
    assert W["sweep110m_q4"].weight_bytes() == 109_510_656 // 2 + 6_844_416
    assert W["sweep110m_q8"].algo_bytes() == 117_186_560
    # row regeneration equals the full draw
    m = W["sweep110m"].mats[4]
    full = m.weights()
    assert np.array_equal(full[100:103], m.weights(100, 3))


def test_quantize_rows_format_and_error():
    """The generator's block quantiser writes the format the oracle decodes:
    scale = max|w| / qmax per 64 columns, every weight within half a step of
    its fp32 value, zero groups exactly zero."""
    import oracle
    rng = np.random.default_rng(5)
    for bits, qmax in ((8, 127), (4, 7)):
        for M, K in ((3, 1), (4, 63), (5, 130), (2, 1000)):
            w = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
            w[0, :min(K, 64)] = 0.0  # an all-zero group
            ldw = synth.q_row_bytes(K, bits)
            Wq = synth.quantize_rows(w, bits, pad=0xCD)
            assert Wq.size == synth.q_matrix_bytes(M, K, bits)
            for i in range(M):
                for j in range(K):
                    g = j // 64
                    s = float(np.abs(w[i, g * 64:min(K, g * 64 + 64)]).max()) / qmax
                    d = oracle.q_weight(Wq, bits, ldw, M, K, i, j)
                    assert abs(d - float(w[i, j])) <= 0.5 * s * (1 + 1e-6) + 1e-12
                    if s == 0.0:
                        assert d == 0.0
