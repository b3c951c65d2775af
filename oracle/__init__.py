"""Plain CPU oracle for the TVL GEMV path (ctypes over ``oracle.c``).

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this package.  It shares no code
with the HIP library and never imports it.

Every function here marshals numpy arrays into the C oracle, where the
arithmetic is, except ``swiglu_bound`` (the tolerance normaliser of the SwiGLU
gate, a few numpy lines).  The definitions cited there are from Kilictas & Alpay,
arXiv 2601.03324: the GEMV of Sec. 6.1 (naive loop and the GEMV listing,
row-major ``w + i*n + j``), its traffic/FLOP model in Sec. 3.1, and the
accepted summation-order drift of Sec. 5.2.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

CFLAGS = ["-std=c99", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` with gcc into ``liboracle.so`` next to it."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def load(path: str) -> ctypes.CDLL:
    """Open an oracle shared library at ``path`` and declare its signatures."""
    L = ctypes.CDLL(path)
    P, I64, D = ctypes.c_void_p, ctypes.c_int64, ctypes.c_double
    L.oracle_f16_to_f64.argtypes = [ctypes.c_uint16]
    L.oracle_f16_to_f64.restype = D
    for name in ("oracle_gemv_f32", "oracle_gemv_f16"):
        fn = getattr(L, name)
        fn.argtypes = [P, I64, P, I64, I64, P, P]
        fn.restype = None
    L.oracle_check.argtypes = [P, P, P, I64, D, P, P, P]
    L.oracle_check.restype = I64
    L.oracle_rmsnorm.argtypes = [P, P, I64, D, P]
    L.oracle_rmsnorm.restype = None
    L.oracle_gemv_dx.argtypes = [P, ctypes.c_int32, I64, P, I64, I64, P, P]
    L.oracle_gemv_dx.restype = None
    L.oracle_swiglu.argtypes = [P, P, I64, P]
    L.oracle_swiglu.restype = None
    L.oracle_gemv_q.argtypes = [P, ctypes.c_int32, I64, P, I64, I64, P, P]
    L.oracle_gemv_q.restype = None
    L.oracle_q_weight.argtypes = [P, ctypes.c_int32, I64, I64, I64, I64, I64]
    L.oracle_q_weight.restype = D
    return L


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        _lib = load(_LIB)
    return _lib


@contextlib.contextmanager
def using(path: str):
    """Temporarily route every call of this module to the library at ``path``
    (the pin suite uses it to show that a deliberately broken oracle fails)."""
    global _lib
    saved = _lib
    _lib = load(path)
    try:
        yield _lib
    finally:
        _lib = saved


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _rows(W: np.ndarray, K: int | None):
    if W.ndim != 2 or not W.flags.c_contiguous:
        raise ValueError("W must be a C-contiguous 2-D array [M, ldw]")
    M, ldw = W.shape
    K = ldw if K is None else int(K)
    if not (0 <= K <= ldw):
        raise ValueError("need 0 <= K <= ldw")
    return M, ldw, K


def gemv_f32(W: np.ndarray, x: np.ndarray, K: int | None = None):
    """Return (y, S) in float64 for fp32 W [M, ldw] (first K columns used)."""
    W = np.ascontiguousarray(W, dtype=np.float32)
    M, ldw, K = _rows(W, K)
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.shape[0] < K:
        raise ValueError("x shorter than K")
    y = np.empty(M, dtype=np.float64)
    S = np.empty(M, dtype=np.float64)
    lib().oracle_gemv_f32(_ptr(W), ldw, _ptr(x), M, K, _ptr(y), _ptr(S))
    return y, S


def gemv_f16(W_bits: np.ndarray, x: np.ndarray, K: int | None = None):
    """Return (y, S) in float64 for binary16 W given as uint16 bit patterns."""
    W_bits = np.ascontiguousarray(W_bits)
    if W_bits.dtype == np.float16:
        W_bits = W_bits.view(np.uint16)
    if W_bits.dtype != np.uint16:
        raise ValueError("W_bits must be uint16 (binary16 bit patterns)")
    M, ldw, K = _rows(W_bits, K)
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.shape[0] < K:
        raise ValueError("x shorter than K")
    y = np.empty(M, dtype=np.float64)
    S = np.empty(M, dtype=np.float64)
    lib().oracle_gemv_f16(_ptr(W_bits), ldw, _ptr(x), M, K, _ptr(y), _ptr(S))
    return y, S


def f16_to_f64(bits: int) -> float:
    return lib().oracle_f16_to_f64(int(bits) & 0xFFFF)


def check(y_gpu: np.ndarray, y_ref: np.ndarray, S: np.ndarray, tol: float):
    """Normalised parity check.  Returns dict(bad, max_err, argmax, mean_err)."""
    y_gpu = np.ascontiguousarray(y_gpu, dtype=np.float32)
    y_ref = np.ascontiguousarray(y_ref, dtype=np.float64)
    S = np.ascontiguousarray(S, dtype=np.float64)
    M = y_gpu.shape[0]
    if y_ref.shape[0] != M or S.shape[0] != M:
        raise ValueError("length mismatch")
    mx = ctypes.c_double()
    am = ctypes.c_int64()
    mean = ctypes.c_double()
    bad = lib().oracle_check(_ptr(y_gpu), _ptr(y_ref), _ptr(S), M, float(tol),
                             ctypes.addressof(mx), ctypes.addressof(am),
                             ctypes.addressof(mean))
    return {"bad": int(bad), "max_err": mx.value, "argmax": am.value,
            "mean_err": mean.value}


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm of fp32 x with fp32 weight g, in double (Sec. 11.2 listing order)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    g = np.ascontiguousarray(g, dtype=np.float32)
    K = x.shape[0]
    if g.shape[0] != K:
        raise ValueError("g and x lengths differ")
    out = np.empty(K, dtype=np.float64)
    lib().oracle_rmsnorm(_ptr(x), _ptr(g), K, float(eps), _ptr(out))
    return out


def gemv_dx(W: np.ndarray, xd: np.ndarray, K: int | None = None):
    """(y, S) for fp32 W or binary16 bits W and a double x."""
    W = np.ascontiguousarray(W)
    if W.dtype == np.float16:
        W = W.view(np.uint16)
    if W.dtype not in (np.float32, np.uint16):
        raise ValueError("W must be float32 or uint16 (binary16 bits)")
    M, ldw, K = _rows(W, K)
    xd = np.ascontiguousarray(xd, dtype=np.float64)
    if xd.shape[0] < K:
        raise ValueError("x shorter than K")
    y = np.empty(M, dtype=np.float64)
    S = np.empty(M, dtype=np.float64)
    lib().oracle_gemv_dx(_ptr(W), 1 if W.dtype == np.uint16 else 0, ldw, _ptr(xd), M, K,
                         _ptr(y), _ptr(S))
    return y, S


def rmsnorm_gemv(W: np.ndarray, x: np.ndarray, g: np.ndarray, eps: float,
                 K: int | None = None):
    """y = W rmsnorm(x; g, eps): (y, S) with S_i = sum_j |W_ij xn_j|."""
    return gemv_dx(W, rmsnorm(x, g, eps), K)


def swiglu(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """h = silu(a) * b elementwise, in double."""
    a = np.ascontiguousarray(a, dtype=np.float64)
    b = np.ascontiguousarray(b, dtype=np.float64)
    if a.shape != b.shape:
        raise ValueError("a and b shapes differ")
    h = np.empty_like(a)
    lib().oracle_swiglu(_ptr(a), _ptr(b), a.shape[0], _ptr(h))
    return h


def swiglu_ffn_in(W1: np.ndarray, W3: np.ndarray, x: np.ndarray, g: np.ndarray | None = None,
                  eps: float = 1e-5, K: int | None = None):
    """The FFN input half of a Llama-2 layer: h = silu(W1 xn) * (W3 xn), with
    xn = rmsnorm(x; g, eps) when g is given, else x.  Returns
    (h, a, b, Sa, Sb): the gate, both GEMVs and their normalisers."""
    xd = rmsnorm(x, g, eps) if g is not None else np.asarray(x, np.float32).astype(np.float64)
    a, Sa = gemv_dx(W1, xd, K)
    b, Sb = gemv_dx(W3, xd, K)
    return swiglu(a, b), a, b, Sa, Sb


def swiglu_bound(a: np.ndarray, b: np.ndarray, Sa: np.ndarray, Sb: np.ndarray) -> np.ndarray:
    """Normaliser of the SwiGLU gate's error (Sec. 2.1 FFN, h = silu(a) * b with
    a = W1 x and b = W3 x): the GEMV parity norm carried through the gate to
    first order.  If a and b are within tau*Sa and tau*Sb of their exact
    values, h moves by at most tau * N + O(tau^2) with

        N = |silu'(a)| |b| Sa + |silu(a)| Sb,
        silu'(z) = s(z) (1 + z (1 - s(z))),  s(z) = 1 / (1 + e^-z),

    which the four corners (a +- tau Sa, b +- tau Sb) attain.  The fp32
    evaluation of silu and of the product adds a few units of 2^-24 of
    |h| <= |silu(a)| |b| <= |silu(a)| Sb, i.e. under 3 % of tau * N at
    tau = 1e-5, so N needs no term of its own for it (while e^-a stays finite
    in fp32, a > -88).  N = 0 only where h = 0 (b = 0, or a = 0 with Sb > 0).
    err_i = |h_gpu - h_ref| / N_i."""
    a = np.asarray(a, np.float64)
    sig = 1.0 / (1.0 + np.exp(-a))
    dsilu = sig * (1.0 + a * (1.0 - sig))
    return np.abs(dsilu) * np.abs(b) * Sa + np.abs(a * sig) * Sb


def gemv_q(Wq: np.ndarray, bits: int, ldw: int, M: int, K: int, x: np.ndarray):
    """(y, S) for a block-quantised matrix given as one uint8 buffer: the code
    plane (M rows of ldw bytes) followed by the fp32 scale plane in blocks of
    4 rows (M rounded up to 4, ceil(K/64) groups); 8- or 4-bit codes (format
    in oracle.c)."""
    Wq = np.ascontiguousarray(Wq, dtype=np.uint8).reshape(-1)
    if bits not in (4, 8):
        raise ValueError("bits must be 4 or 8")
    need = M * ldw + 4 * ((M + 3) // 4 * 4) * ((K + 63) // 64)
    if Wq.size < need:
        raise ValueError(f"buffer of {Wq.size} bytes, need {need}")
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.empty(M, dtype=np.float64)
    S = np.empty(M, dtype=np.float64)
    lib().oracle_gemv_q(_ptr(Wq), bits, ldw, _ptr(x), M, K, _ptr(y), _ptr(S))
    return y, S


def q_weight(Wq: np.ndarray, bits: int, ldw: int, M: int, K: int, i: int, j: int) -> float:
    Wq = np.ascontiguousarray(Wq, dtype=np.uint8).reshape(-1)
    return lib().oracle_q_weight(_ptr(Wq), bits, ldw, M, K, i, j)
