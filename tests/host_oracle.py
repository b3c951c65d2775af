"""The CPU oracle over whole large matrices on every host thread (test helper).

The oracle is single-threaded C; ctypes releases the GIL for each call, so
row blocks of one matrix run side by side in a thread pool.  Each block is
the plain definition applied to those rows (the oracle's own calls, nothing
reordered inside a row), so the result is the oracle's, bit for bit, for any
number of threads.  This is what lets the full-size workloads (the 7B token,
the 70B-shaped stacks, 7 GB of 8-bit codes) be checked on every output
instead of sampled rows.
"""
from __future__ import annotations

import concurrent.futures as cf
import os

import numpy as np

import oracle

_POOL = None


def host_threads() -> int:
    """Threads this process may use (its CPU affinity), at most 16."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def pool() -> cf.ThreadPoolExecutor:
    global _POOL
    if _POOL is None:
        _POOL = cf.ThreadPoolExecutor(host_threads())
    return _POOL


def _blocks(M: int, align: int = 1):
    """About four row blocks per thread, each a multiple of `align` rows
    (the last one excepted)."""
    per = -(-M // (host_threads() * 4))
    step = -(-per // align) * align
    return [(r, min(M, r + step)) for r in range(0, M, step)]


def _join(parts):
    return (np.concatenate([p[0] for p in parts]), np.concatenate([p[1] for p in parts]))


def gemv(W: np.ndarray, x: np.ndarray, dt: int):
    """(y, S) of fp32 (dt 0) or binary16-bits (dt 1) W [M, ldw] and fp32 x."""
    fn = oracle.gemv_f32 if dt == 0 else oracle.gemv_f16
    K = x.shape[0]
    futs = [pool().submit(fn, W[a:b], x, K) for a, b in _blocks(W.shape[0])]
    return _join([f.result() for f in futs])


def gemv_dx(W: np.ndarray, xd: np.ndarray):
    """(y, S) of fp32 or binary16-bits W and a double x."""
    futs = [pool().submit(oracle.gemv_dx, W[a:b], xd) for a, b in _blocks(W.shape[0])]
    return _join([f.result() for f in futs])


def gemv_q(buf: np.ndarray, bits: int, ldw: int, M: int, K: int, x: np.ndarray):
    """(y, S) of a block-quantised matrix (code plane of M rows of ldw bytes,
    then fp32 scales in blocks of 4 rows, ceil(K/64) per row).  A block of
    rows [a, b) with a % 4 == 0 is itself such a matrix: its code rows, then
    its own scale blocks, which are contiguous in the plane."""
    ng = (K + 63) // 64
    Mp = (M + 3) // 4 * 4
    buf = np.ascontiguousarray(buf, np.uint8).reshape(-1)
    codes = buf[:M * ldw]
    scales = buf[M * ldw:M * ldw + 4 * Mp * ng]

    def block(a, b):
        bp = (b + 3) // 4 * 4  # scale blocks of rows [a, b), the last one padded
        sub = np.concatenate([codes[a * ldw:b * ldw], scales[4 * a * ng:4 * bp * ng]])
        return oracle.gemv_q(sub, bits, ldw, b - a, K, x)

    futs = [pool().submit(block, a, b) for a, b in _blocks(M, align=4)]
    return _join([f.result() for f in futs])


def swiglu_ffn_in(W1: np.ndarray, W3: np.ndarray, x: np.ndarray, g, eps: float):
    """oracle.swiglu_ffn_in on row blocks: (h, a, b, Sa, Sb)."""
    futs = [pool().submit(oracle.swiglu_ffn_in, W1[a:b], W3[a:b], x, g, eps)
            for a, b in _blocks(W1.shape[0])]
    parts = [f.result() for f in futs]
    return tuple(np.concatenate([p[i] for p in parts]) for i in range(5))
