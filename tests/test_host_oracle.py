"""The thread-pool form of the oracle used by the full-size GPU checks gives
the oracle's own results bit for bit (CPU only)."""
from __future__ import annotations

import numpy as np

import host_oracle
import oracle
import synth


def test_blocks_cover_rows_once():
    for M in (1, 3, 4, 5, 63, 64, 65, 1000, 32000):
        for align in (1, 4):
            bl = host_oracle._blocks(M, align)
            assert bl[0][0] == 0 and bl[-1][1] == M
            assert all(b[1] == c[0] for b, c in zip(bl, bl[1:]))
            assert all(a % align == 0 for a, _ in bl)


def test_gemv_blocks_equal_whole():
    rng = np.random.default_rng(3)
    for M, K in ((1, 7), (130, 300), (1001, 64)):
        W = (rng.standard_normal((M, K + 5)) * 0.02).astype(np.float32)
        x = rng.standard_normal(K).astype(np.float32)
        y, S = host_oracle.gemv(W, x, 0)
        y0, S0 = oracle.gemv_f32(W, x, K)
        assert np.array_equal(y, y0) and np.array_equal(S, S0)
        Wh = synth.f32_to_f16_bits(W)
        y, S = host_oracle.gemv(Wh, x, 1)
        y0, S0 = oracle.gemv_f16(Wh, x, K)
        assert np.array_equal(y, y0) and np.array_equal(S, S0)
        xd = rng.standard_normal(K + 5)
        y, S = host_oracle.gemv_dx(Wh, xd)
        y0, S0 = oracle.gemv_dx(Wh, xd)
        assert np.array_equal(y, y0) and np.array_equal(S, S0)


def test_gemv_q_blocks_equal_whole():
    rng = np.random.default_rng(4)
    for bits in (8, 4):
        for M, K in ((1, 64), (6, 100), (257, 700), (1001, 130)):
            W = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
            buf = synth.quantize_rows(W, bits)
            ldw = synth.q_row_bytes(K, bits)
            x = rng.standard_normal(K).astype(np.float32)
            y, S = host_oracle.gemv_q(buf, bits, ldw, M, K, x)
            y0, S0 = oracle.gemv_q(buf, bits, ldw, M, K, x)
            assert np.array_equal(y, y0) and np.array_equal(S, S0), (bits, M, K)


def test_swiglu_blocks_equal_whole():
    rng = np.random.default_rng(5)
    M, K = 300, 257
    W1 = synth.f32_to_f16_bits((rng.standard_normal((M, K)) * 0.02).astype(np.float32))
    W3 = synth.f32_to_f16_bits((rng.standard_normal((M, K)) * 0.02).astype(np.float32))
    x = rng.standard_normal(K).astype(np.float32)
    g = rng.uniform(0.5, 1.5, K).astype(np.float32)
    for gg in (g, None):
        got = host_oracle.swiglu_ffn_in(W1, W3, x, gg, 1e-5)
        ref = oracle.swiglu_ffn_in(W1, W3, x, gg, 1e-5)
        for a, b in zip(got, ref):
            assert np.array_equal(a, b)
