"""tvl_gemv_noalloc through the C ABI (MI355X): the allocation-free variant of
tvl_gemv_ex for callers that cannot allocate device memory.

Every case makes two calls in a row, the second with a smaller input, through
both entry points with the same tuning.  The two entry points launch the same
kernels, so their outputs must be bitwise equal, and both must match the CPU
oracle within the GEMV tolerance (1e-5 of sum_j |W_ij x_j| for fp32 weights,
2e-3 for fp16).  K splits too large for the static scratch are rejected
before anything is enqueued.
"""
from __future__ import annotations

import ctypes
import sys

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2601_03324_amd import tvl  # noqa: E402  (raises if libtvl.so is missing)

DEV = "cuda"
TOL = {0: 1e-5, 1: 2e-3}
SHAPE_ERR = -2
PARTIALS, COUNTERS = 1 << 20, 1 << 16  # the static scratch's capacity


def log(msg):
    print(msg, flush=True, file=sys.stderr)


def matrix(M, K, dt, seed):
    rng = np.random.default_rng(seed)
    Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    host = Wf if dt == 0 else Wf.astype(np.float16).view(np.uint16)
    ldw = tvl.tvl_row_stride(K, dt)
    if dt == 0:
        buf = torch.zeros((M, ldw), dtype=torch.float32, device=DEV)
        buf[:, :K] = torch.from_numpy(host).to(DEV)
    else:
        buf = torch.zeros((M, ldw), dtype=torch.int16, device=DEV)
        buf[:, :K] = torch.from_numpy(host.view(np.int16)).to(DEV)
    x = rng.standard_normal(K).astype(np.float32)
    return host, buf, ldw, x


def run(fn, buf, ldw, dt, x, M, K, tuning):
    xd = torch.from_numpy(x).to(DEV)
    y = torch.full((M,), float("nan"), dtype=torch.float32, device=DEV)
    fn(buf, ldw, dt, xd, y, M, K, tuning)
    torch.cuda.synchronize()
    return y.cpu().numpy()


# (first call, second smaller call): (M, K, dtype, tuning)
CASES = [
    # default choice: a K split for few long rows (S = 2, then S = 4)
    ((96, 16384, 0, None), (40, 9000, 0, None)),
    ((128, 20000, 1, None), (17, 17000, 1, None)),
    # forced splits in both x modes, ragged K
    ((1000, 5000, 1, dict(ksplit=7)), (300, 4100, 1, dict(ksplit=3))),
    ((4096, 3000, 0, dict(rows_per_wave=8, waves_per_block=4, unroll=1, ksplit=16, flags=2)),
     (100, 2999, 0, dict(rows_per_wave=8, waves_per_block=4, unroll=1, ksplit=16, flags=2))),
    ((2000, 6000, 0, dict(rows_per_wave=1, waves_per_block=4, unroll=8, ksplit=4, flags=1)),
     (129, 700, 0, dict(rows_per_wave=1, waves_per_block=4, unroll=8, ksplit=4, flags=1))),
    # a split that fills the scratch exactly: S * M = 2^20 partials
    ((PARTIALS // 256, 4096, 0, dict(ksplit=256)), (1000, 4096, 0, dict(ksplit=256))),
    # row splits (no scratch at all)
    ((2048, 768, 0, None), (500, 300, 0, None)),
]


@pytest.mark.parametrize("first,second", CASES, ids=[f"case{i}" for i in range(len(CASES))])
def test_noalloc_matches_gemv_ex(first, second):
    for n, (M, K, dt, tuning) in enumerate((first, second)):
        log(f"noalloc: call {n + 1}: M={M} K={K} dtype={dt} tuning={tuning}")
        host, buf, ldw, x = matrix(M, K, dt, seed=M * 7919 + K + dt)
        y_ex = run(tvl.tvl_gemv_ex, buf, ldw, dt, x, M, K, tuning)
        y_na = run(tvl.tvl_gemv_noalloc, buf, ldw, dt, x, M, K, tuning)
        assert np.array_equal(y_ex.view(np.uint32), y_na.view(np.uint32)), (M, K, dt, tuning)
        yref, S = oracle.gemv_f32(host, x) if dt == 0 else oracle.gemv_f16(host, x)
        r = oracle.check(y_na, yref, S, TOL[dt])
        assert r["bad"] == 0, r
        # a rerun reuses the scratch: the counters were left at zero
        y_again = run(tvl.tvl_gemv_noalloc, buf, ldw, dt, x, M, K, tuning)
        assert np.array_equal(y_again.view(np.uint32), y_na.view(np.uint32))


@pytest.mark.parametrize("M,tuning", [
    (PARTIALS // 2 + 1, dict(ksplit=2)),  # 2^20 + 2 partials
    (COUNTERS + 1, dict(rows_per_wave=1, waves_per_block=1, unroll=4, ksplit=2, flags=2)),
], ids=["partials", "counters"])
def test_noalloc_rejects_splits_beyond_the_scratch(M, tuning):
    K = 64
    log(f"noalloc: rejection M={M} tuning={tuning}")
    W = torch.zeros((M, K), dtype=torch.float32, device=DEV)
    x = torch.zeros(K, dtype=torch.float32, device=DEV)
    y = torch.full((M,), float("nan"), dtype=torch.float32, device=DEV)
    t = tvl.tvl_tuning(**tuning)
    st = tvl.lib.tvl_gemv_noalloc(W.data_ptr(), K, 0, x.data_ptr(), y.data_ptr(), M, K,
                                  ctypes.byref(t), None)
    assert st == SHAPE_ERR
    assert b"static scratch" in tvl.lib.tvl_last_error()
    torch.cuda.synchronize()
    assert torch.isnan(y).all()  # nothing was enqueued


@pytest.mark.parametrize("dt,tuning", [(3, dict(flags=1)), (3, None), (2, None)],
                         ids=["q4-x-in-lds", "q4", "q8"])
def test_noalloc_quantised(dt, tuning):
    """Quantised weights need no scratch: tvl_gemv_noalloc gives the same
    bits as tvl_gemv_ex (x staged in LDS: dynamic LDS, not an allocation),
    two calls, the second smaller, both within the oracle's bar."""
    import synth
    bits = 4 if dt == 3 else 8
    for n, (M, K) in enumerate(((640, 4096), (70, 1000))):
        log(f"noalloc quantised: call {n + 1}: M={M} K={K} dtype={dt} tuning={tuning}")
        rng = np.random.default_rng(M + K + dt)
        w = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
        ldw = tvl.tvl_row_stride(K, dt)
        Wq = synth.quantize_rows(w, bits, ldw=ldw)
        Wd = tvl.upload_quant(Wq, M, K, dt, ldw, DEV)
        x = rng.standard_normal(K).astype(np.float32)
        y_ex = run(tvl.tvl_gemv_ex, Wd.buf, ldw, dt, x, M, K, tuning)
        y_na = run(tvl.tvl_gemv_noalloc, Wd.buf, ldw, dt, x, M, K, tuning)
        assert np.array_equal(y_ex.view(np.uint32), y_na.view(np.uint32)), (M, K, dt)
        yref, S = oracle.gemv_q(Wq, bits, ldw, M, K, x)
        assert oracle.check(y_na, yref, S, 1e-5)["bad"] == 0, (M, K, dt)
