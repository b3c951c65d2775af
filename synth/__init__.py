"""Seeded synthetic inputs for the TVL GEMV path (ctypes over ``synth.c``).

This module is shared by the oracle side and the HIP side.  It draws numbers
and rounds them to storage types; it holds none of the GEMV arithmetic.

The workloads stand in for the paper's Llama-2 checkpoints (Kilictas & Alpay,
arXiv 2601.03324, Sec. 7.1 runs the 110M "stories" model; Sec. 1 motivates the
70B case): the decode-step weight shapes of Llama-2 110M, 7B and an 8-layer
70B-shaped stack, with N(0, 0.02^2) weights (uniform for the single 768x768
case) and N(0, 1) activations, every matrix with its own seeded x.  GEMV time
does not depend on the values, so nothing about speed hinges on them.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB = os.path.join(_HERE, "libsynth.so")


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-std=c99", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(_LIB)
        P, I64, U64, D = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_double
        L.synth_u64.argtypes = [U64, U64]
        L.synth_u64.restype = U64
        L.synth_key.argtypes = [U64, P, ctypes.c_int]
        L.synth_key.restype = U64
        L.synth_f32_to_f16_bits.argtypes = [ctypes.c_float]
        L.synth_f32_to_f16_bits.restype = ctypes.c_uint16
        L.synth_f32_to_f16.argtypes = [P, P, I64]
        L.synth_uniform_f32.argtypes = [P, I64, U64, U64, D, D]
        L.synth_normal_f32.argtypes = [P, I64, U64, U64, D]
        L.synth_normal_f16.argtypes = [P, I64, U64, U64, D]
        L.synth_int_f32.argtypes = [P, I64, U64, U64, I64, I64]
        L.synth_int_f16.argtypes = [P, I64, U64, U64, I64, I64]
        L.synth_q_row_bytes.argtypes = [I64, ctypes.c_int]
        L.synth_q_row_bytes.restype = I64
        L.synth_quantize_rows.argtypes = [P, I64, I64, ctypes.c_int, P, I64]
        for n in ("synth_f32_to_f16", "synth_uniform_f32", "synth_normal_f32",
                  "synth_normal_f16", "synth_int_f32", "synth_int_f16", "synth_quantize_rows"):
            getattr(L, n).restype = None
        _lib = L
    return _lib


# ----------------------------------------------------------------- primitives
def u64(key: int, k: int) -> int:
    return int(lib().synth_u64(key, k))


def key(*fields: int, root: int = 0) -> int:
    arr = (ctypes.c_uint64 * len(fields))(*[int(f) for f in fields])
    return int(lib().synth_key(root, arr, len(fields)))


def uniform_f32(n: int, k: int, a: float, b: float, offset: int = 0, out=None):
    out = np.empty(n, np.float32) if out is None else out
    lib().synth_uniform_f32(out.ctypes.data, n, k, offset, a, b)
    return out


def normal_f32(n: int, k: int, sigma: float = 1.0, offset: int = 0, out=None):
    out = np.empty(n, np.float32) if out is None else out
    lib().synth_normal_f32(out.ctypes.data, n, k, offset, sigma)
    return out


def normal_f16(n: int, k: int, sigma: float, offset: int = 0, out=None):
    """binary16 bit patterns (uint16) of the RNE-rounded N(0, sigma^2) fp32 values."""
    out = np.empty(n, np.uint16) if out is None else out
    lib().synth_normal_f16(out.ctypes.data, n, k, offset, sigma)
    return out


def int_f32(n: int, k: int, lo: int, hi: int, offset: int = 0):
    out = np.empty(n, np.float32)
    lib().synth_int_f32(out.ctypes.data, n, k, offset, lo, hi)
    return out


def int_f16(n: int, k: int, lo: int, hi: int, offset: int = 0):
    out = np.empty(n, np.uint16)
    lib().synth_int_f16(out.ctypes.data, n, k, offset, lo, hi)
    return out


def f32_to_f16_bits(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    out = np.empty(a.shape, np.uint16)
    lib().synth_f32_to_f16(a.ctypes.data, out.ctypes.data, a.size)
    return out


def q_row_bytes(K: int, bits: int) -> int:
    """Bytes of one code row: ceil(K * bits / 8) rounded up to 128."""
    return int(lib().synth_q_row_bytes(K, bits))


def q_matrix_bytes(M: int, K: int, bits: int, ldw: int | None = None) -> int:
    """Code plane (M rows of ldw bytes) + scale plane (M rounded up to 4
    rows x ceil(K/64) groups, fp32, in blocks of 4 rows)."""
    ldw = q_row_bytes(K, bits) if ldw is None else ldw
    return M * ldw + 4 * ((M + 3) // 4 * 4) * ((K + 63) // 64)


def quantize_rows(w: np.ndarray, bits: int, ldw: int | None = None, pad: int = 0) -> np.ndarray:
    """fp32 [M, K] -> one uint8 buffer: the code plane (M rows of ldw bytes)
    then the fp32 scale plane; code padding = `pad`."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    M, K = w.shape
    ldw = q_row_bytes(K, bits) if ldw is None else ldw
    out = np.full(q_matrix_bytes(M, K, bits, ldw), pad, np.uint8)
    lib().synth_quantize_rows(w.ctypes.data, M, K, bits, out.ctypes.data, ldw)
    return out


# ----------------------------------------------------------------- workloads
MATRIX_IDS = {"wq": 0, "wk": 1, "wv": 2, "wo": 3, "w1": 4, "w3": 5, "w2": 6, "cls": 7}
KIND_W, KIND_X = 0, 1


@dataclass(frozen=True)
class MatSpec:
    """One weight matrix of a workload and the recipe of its inputs."""
    name: str
    M: int
    K: int
    dtype: str  # "f32", "f16", or block-quantised "q8" / "q4" (weights); x and y are fp32
    dist: tuple  # ("normal", sigma) or ("uniform", a, b)
    cfg: int
    layer: int
    mat: int

    @property
    def w_key(self) -> int:
        return key(self.cfg, self.layer, self.mat, KIND_W, 0)

    def x_key(self, rep: int = 0) -> int:
        return key(self.cfg, self.layer, self.mat, KIND_X, rep)

    @property
    def bits(self) -> int:
        return {"f32": 32, "f16": 16, "q8": 8, "q4": 4}[self.dtype]

    @property
    def quantised(self) -> bool:
        return self.dtype in ("q8", "q4")

    @property
    def wbytes(self) -> int:
        """Weight bytes a GEMV must read: the values, and for block-quantised
        weights the codes plus one fp32 scale per 64 columns (no padding)."""
        if self.quantised:
            return self.M * ((self.K * self.bits + 7) // 8) + 4 * self.M * ((self.K + 63) // 64)
        return self.M * self.K * self.bits // 8

    def algo_bytes(self) -> int:
        """Algorithmic bytes of one GEMV: |W| + |x| + |y| (paper Sec. 3.1)."""
        return self.wbytes + 4 * self.K + 4 * self.M

    def weights(self, row0: int = 0, nrows: int | None = None) -> np.ndarray:
        """Rows [row0, row0+nrows) as a dense [nrows, K] array (fp32, or uint16
        bits); for "q8" / "q4" the fp32 draw quantised row by row into one
        uint8 buffer (code plane of nrows rows, then their scale plane)."""
        nrows = self.M - row0 if nrows is None else nrows
        n, off = nrows * self.K, row0 * self.K
        if self.quantised:
            w = normal_f32(n, self.w_key, self.dist[1], off).reshape(nrows, self.K)
            return quantize_rows(w, self.bits)
        if self.dist[0] == "uniform":
            w = uniform_f32(n, self.w_key, self.dist[1], self.dist[2], off)
            if self.dtype == "f16":
                w = f32_to_f16_bits(w)
        elif self.dtype == "f32":
            w = normal_f32(n, self.w_key, self.dist[1], off)
        else:
            w = normal_f16(n, self.w_key, self.dist[1], off)
        return w.reshape(nrows, self.K)

    def x(self, rep: int = 0) -> np.ndarray:
        return normal_f32(self.K, self.x_key(rep), 1.0)


@dataclass(frozen=True)
class Workload:
    name: str
    cfg: int
    mats: tuple = field(default_factory=tuple)
    reps: int = 1  # x vectors per matrix (the classifier case draws 100)

    def algo_bytes(self) -> int:
        return sum(m.algo_bytes() for m in self.mats)

    def weight_bytes(self) -> int:
        return sum(m.wbytes for m in self.mats)

    def flops(self) -> int:
        return sum(2 * m.M * m.K for m in self.mats)


def _llama(cfg: int, layers: int, dim: int, hidden: int, vocab: int | None,
           dtype: str, kv: int | None = None, sigma: float = 0.02) -> tuple:
    kv = dim if kv is None else kv
    shapes = [("wq", dim, dim), ("wk", kv, dim), ("wv", kv, dim), ("wo", dim, dim),
              ("w1", hidden, dim), ("w3", hidden, dim), ("w2", dim, hidden)]
    mats = []
    for l in range(layers):
        for nm, M, K in shapes:
            mats.append(MatSpec(f"L{l}.{nm}", M, K, dtype, ("normal", sigma), cfg, l,
                                MATRIX_IDS[nm]))
    if vocab:
        mats.append(MatSpec("cls", vocab, dim, dtype, ("normal", sigma), cfg, 0,
                            MATRIX_IDS["cls"]))
    return tuple(mats)


WORKLOADS = {
    # a single fp32 GEMV, W U(-0.05, 0.05), x N(0, 1), seed 0
    "gemv768": Workload("gemv768", 1, (MatSpec("w", 768, 768, "f32", ("uniform", -0.05, 0.05),
                                               1, 0, 0),)),
    # one decode token of Llama-2 110M ("stories"), fp32: 12 layers + tied classifier
    "sweep110m": Workload("sweep110m", 2, _llama(2, 12, 768, 2048, 32000, "f32")),
    # the 110M classifier alone, 100 fresh x
    "cls32000": Workload("cls32000", 3, (MatSpec("cls", 32000, 768, "f32", ("normal", 0.02),
                                                 3, 0, MATRIX_IDS["cls"]),), reps=100),
    # one decode token of Llama-2 7B, fp32: 32 layers + classifier
    "sweep7b": Workload("sweep7b", 4, _llama(4, 32, 4096, 11008, 32000, "f32")),
    # 8 layers of a Llama-2 70B-shaped stack, fp16 weights (GQA: wk, wv are 1024 x 8192)
    "stack70b8": Workload("stack70b8", 5, _llama(5, 8, 8192, 28672, None, "f16", kv=1024)),
    # the same 110M and 7B tokens with block-quantised weights: the fp32 draws
    # above, quantised per 64 columns to 8-bit or 4-bit codes
    "sweep110m_q8": Workload("sweep110m_q8", 2, _llama(2, 12, 768, 2048, 32000, "q8")),
    "sweep110m_q4": Workload("sweep110m_q4", 2, _llama(2, 12, 768, 2048, 32000, "q4")),
    "sweep7b_q8": Workload("sweep7b_q8", 4, _llama(4, 32, 4096, 11008, 32000, "q8")),
    "sweep7b_q4": Workload("sweep7b_q4", 4, _llama(4, 32, 4096, 11008, 32000, "q4")),
}


# ------------------------------------------------------- fused decode items
KIND_G = 2  # RMSNorm weight vectors


@dataclass(frozen=True)
class VecSpec:
    """A seeded fp32 vector (an activation x or an RMSNorm weight g)."""
    K: int
    cfg: int
    layer: int
    group: int
    kind: int  # KIND_X or KIND_G

    def values(self) -> np.ndarray:
        k = key(self.cfg, self.layer, 100 + self.group, self.kind, 0)
        if self.kind == KIND_G:  # RMSNorm weights: positive, around 1
            return uniform_f32(self.K, k, 0.5, 1.5)
        return normal_f32(self.K, k, 1.0)


@dataclass(frozen=True)
class FusedSpec:
    """One item of a fused decode sweep: a GEMV or a SwiGLU pair (W = w1,
    W3 = w3), with x optionally RMS-normalised by g first (eps 1e-5)."""
    name: str
    W: MatSpec
    x: VecSpec
    W3: MatSpec | None = None
    g: VecSpec | None = None
    eps: float = 1e-5

    @property
    def M(self) -> int:
        return self.W.M

    @property
    def K(self) -> int:
        return self.W.K

    def algo_bytes(self) -> int:
        """|W| (+|W3|) + |x| (+|g|) + |y|: every input read once, y written once."""
        b = self.W.wbytes + 4 * self.K + 4 * self.M
        if self.W3 is not None:
            b += self.W3.wbytes
        if self.g is not None:
            b += 4 * self.K
        return b


@dataclass(frozen=True)
class FusedWorkload:
    name: str
    cfg: int
    items: tuple

    def algo_bytes(self) -> int:
        return sum(i.algo_bytes() for i in self.items)

    def weight_bytes(self) -> int:
        return sum(i.W.wbytes + (i.W3.wbytes if i.W3 is not None else 0) for i in self.items)


# groups of activation / norm vectors within a layer
G_ATT, G_WO, G_FFN, G_W2, G_FINAL = 0, 1, 2, 3, 4


def _llama_fused(cfg: int, layers: int, dim: int, hidden: int, vocab: int | None,
                 dtype: str, kv: int | None = None, sigma: float = 0.02) -> tuple:
    """A Llama-2 decode token as fused items: RMSNorm -> wq, wk, wv (one shared
    normalised input); wo; RMSNorm -> SwiGLU(w1, w3); w2; final RMSNorm -> cls."""
    kv = dim if kv is None else kv
    items = []
    for l in range(layers):
        def mat(nm, M, K):
            return MatSpec(f"L{l}.{nm}", M, K, dtype, ("normal", sigma), cfg, l, MATRIX_IDS[nm])
        xa, ga = VecSpec(dim, cfg, l, G_ATT, KIND_X), VecSpec(dim, cfg, l, G_ATT, KIND_G)
        for nm, M in (("wq", dim), ("wk", kv), ("wv", kv)):
            items.append(FusedSpec(f"L{l}.{nm}", mat(nm, M, dim), xa, g=ga))
        items.append(FusedSpec(f"L{l}.wo", mat("wo", dim, dim), VecSpec(dim, cfg, l, G_WO, KIND_X)))
        xf, gf = VecSpec(dim, cfg, l, G_FFN, KIND_X), VecSpec(dim, cfg, l, G_FFN, KIND_G)
        items.append(FusedSpec(f"L{l}.w1w3", mat("w1", hidden, dim), xf, W3=mat("w3", hidden, dim),
                               g=gf))
        items.append(FusedSpec(f"L{l}.w2", mat("w2", dim, hidden),
                               VecSpec(hidden, cfg, l, G_W2, KIND_X)))
    if vocab:
        items.append(FusedSpec("cls", MatSpec("cls", vocab, dim, dtype, ("normal", sigma), cfg, 0,
                                              MATRIX_IDS["cls"]),
                               VecSpec(dim, cfg, 0, G_FINAL, KIND_X),
                               g=VecSpec(dim, cfg, 0, G_FINAL, KIND_G)))
    return tuple(items)


FUSED_WORKLOADS = {
    # the 110M decode token with its RMSNorms and SwiGLU gates fused (73 items)
    "fused110m": FusedWorkload("fused110m", 2, _llama_fused(2, 12, 768, 2048, 32000, "f32")),
    # 8 fused layers of the 70B-shaped stack, fp16 weights (40 items)
    "fused70b8": FusedWorkload("fused70b8", 5, _llama_fused(5, 8, 8192, 28672, None, "f16",
                                                            kv=1024)),
}
