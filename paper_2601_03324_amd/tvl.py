"""Thin Python binding of the TVL GEMV C ABI (``include/tvl.h``, ``libtvl.so``).

Argument marshalling only: every function forwards to the C entry point of
the same name, which enqueues HIP kernels.  Pointers may be given as ints or
as torch tensors (their ``data_ptr()``); ``stream=None`` means torch's current
stream on the current device.  Nothing here computes a GEMV: when the library
is missing, importing this module raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtvl.so")

TVL_F32, TVL_F16, TVL_Q8, TVL_Q4 = 0, 1, 2, 3
TVL_FLAG_X_LDS = 1
TVL_FLAG_X_DIRECT = 2
STATUS = {0: "TVL_OK", -1: "TVL_ERR_NULL", -2: "TVL_ERR_SHAPE", -3: "TVL_ERR_ALIGN",
          -4: "TVL_ERR_DTYPE", -5: "TVL_ERR_ALIAS", -6: "TVL_ERR_HIP", -7: "TVL_ERR_NOMEM",
          -8: "TVL_ERR_ARG"}

# (rows per wave, waves per block, unroll) triples the library instantiates
LDS_SHAPES = ((1, 4, 4), (1, 4, 8), (2, 4, 2), (2, 4, 3), (2, 4, 4), (2, 4, 8), (4, 4, 1),
              (4, 4, 2), (4, 4, 3), (4, 4, 4), (8, 4, 1), (8, 4, 2), (2, 8, 4), (2, 8, 8),
              (4, 8, 2), (1, 2, 8), (2, 2, 8), (4, 2, 4), (8, 2, 2))
DIRECT_SHAPES = tuple((r, w, u) for w in (1, 4)
                      for (r, u) in ((1, 4), (1, 8), (2, 2), (2, 3), (2, 4), (2, 8), (4, 1),
                                     (4, 2), (4, 3), (4, 4), (8, 1), (8, 2))) + (
    (1, 8, 8), (2, 8, 3), (2, 8, 4), (4, 8, 2))

# every symbol include/tvl.h declares
EXPORTS = ("tvl_version", "tvl_row_stride", "tvl_pack_rows", "tvl_gemv", "tvl_gemv_ex",
           "tvl_gemv_noalloc", "tvl_gemv_item",
           "tvl_gemv_batch_sweep", "tvl_sweep_plan_create", "tvl_sweep_plan_run",
           "tvl_sweep_plan_info", "tvl_sweep_plan_destroy", "tvl_release_workspaces",
           "tvl_util_read_stream", "tvl_util_copy", "tvl_status_str", "tvl_last_error")


class TvlError(RuntimeError):
    def __init__(self, status: int, fn: str, detail: str):
        self.status = status
        super().__init__(f"{fn}: {STATUS.get(status, status)}: {detail}")


TVL_OP_GEMV, TVL_OP_SWIGLU = 0, 1


class tvl_item(ctypes.Structure):
    _fields_ = [("W", ctypes.c_void_p), ("ldw", ctypes.c_int64), ("x", ctypes.c_void_p),
                ("y", ctypes.c_void_p), ("M", ctypes.c_int64), ("K", ctypes.c_int64),
                ("dtype", ctypes.c_int32), ("op", ctypes.c_int32), ("W3", ctypes.c_void_p),
                ("g", ctypes.c_void_p), ("eps", ctypes.c_float), ("nrhs", ctypes.c_int32),
                ("ldx", ctypes.c_int64), ("ldy", ctypes.c_int64)]


class tvl_tuning(ctypes.Structure):
    _fields_ = [("rows_per_wave", ctypes.c_int32), ("waves_per_block", ctypes.c_int32),
                ("unroll", ctypes.c_int32), ("ksplit", ctypes.c_int32),
                ("grid", ctypes.c_int32), ("flags", ctypes.c_int32)]


assert ctypes.sizeof(tvl_item) == 96


def _bind_hip_runtime() -> None:
    """One HIP runtime per process.  torch ships its own libamdhip64 (same
    soname as the system one); device pointers and stream handles from torch
    are only valid in that runtime instance.  Loading it globally before
    libtvl.so makes the library's libamdhip64.so.7 dependency resolve to the
    already-loaded copy instead of a second runtime from /opt/rocm."""
    try:
        import torch
    except ImportError:
        return
    hip = os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so")
    if os.path.exists(hip):
        ctypes.CDLL(hip, mode=ctypes.RTLD_GLOBAL)


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2601_03324_amd.build.build() "
                          f"(hipcc --offload-arch=gfx950)")
    _bind_hip_runtime()
    L = ctypes.CDLL(LIB_PATH)
    P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    sig = {
        "tvl_version": ([], I32),
        "tvl_row_stride": ([I64, I32], I64),
        "tvl_pack_rows": ([P, I64, P, I64, I64, I32, P], I32),
        "tvl_gemv": ([P, I64, I32, P, P, I64, I64, P], I32),
        "tvl_gemv_ex": ([P, I64, I32, P, P, I64, I64, P, P], I32),
        "tvl_gemv_noalloc": ([P, I64, I32, P, P, I64, I64, P, P], I32),
        "tvl_gemv_item": ([P, P, P], I32),
        "tvl_gemv_batch_sweep": ([P, I32, P], I32),
        "tvl_sweep_plan_create": ([P, I32, P, P], I32),
        "tvl_sweep_plan_run": ([P, P], I32),
        "tvl_sweep_plan_info": ([P, P, P, P], I32),
        "tvl_sweep_plan_destroy": ([P], I32),
        "tvl_release_workspaces": ([], I32),
        "tvl_util_read_stream": ([P, I64, P, I64, P, P], I32),
        "tvl_util_copy": ([P, P, I64, P], I32),
        "tvl_status_str": ([I32], ctypes.c_char_p),
        "tvl_last_error": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    return L


lib = _load()


def _p(v) -> int:
    if v is None:
        return 0
    if isinstance(v, int):
        return v
    if hasattr(v, "data_ptr"):
        return int(v.data_ptr())
    raise TypeError(f"expected an int pointer or a tensor, got {type(v)}")


def _stream(stream) -> int:
    if stream is None:
        import torch
        if torch.cuda.is_available():
            return int(torch.cuda.current_stream().cuda_stream)
        return 0
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


def _chk(st: int, fn: str) -> None:
    if st != 0:
        raise TvlError(st, fn, (lib.tvl_last_error() or b"").decode())


def _tuning(t) -> tvl_tuning | None:
    if t is None or isinstance(t, tvl_tuning):
        return t
    return tvl_tuning(**t)


# ------------------------------------------------------------------ entry points
def tvl_version() -> int:
    return lib.tvl_version()


def tvl_row_stride(K: int, dtype: int) -> int:
    return lib.tvl_row_stride(K, dtype)


def tvl_pack_rows(dst, ldw: int, src, M: int, K: int, dtype: int, stream=None) -> None:
    _chk(lib.tvl_pack_rows(_p(dst), ldw, _p(src), M, K, dtype, _stream(stream)), "tvl_pack_rows")


def tvl_gemv(W, ldw: int, dtype: int, x, y, M: int, K: int, stream=None) -> None:
    _chk(lib.tvl_gemv(_p(W), ldw, dtype, _p(x), _p(y), M, K, _stream(stream)), "tvl_gemv")


def tvl_gemv_ex(W, ldw: int, dtype: int, x, y, M: int, K: int, tuning=None, stream=None) -> None:
    t = _tuning(tuning)
    _chk(lib.tvl_gemv_ex(_p(W), ldw, dtype, _p(x), _p(y), M, K,
                         ctypes.byref(t) if t is not None else None, _stream(stream)),
         "tvl_gemv_ex")


def tvl_gemv_noalloc(W, ldw: int, dtype: int, x, y, M: int, K: int, tuning=None,
                     stream=None) -> None:
    t = _tuning(tuning)
    _chk(lib.tvl_gemv_noalloc(_p(W), ldw, dtype, _p(x), _p(y), M, K,
                              ctypes.byref(t) if t is not None else None, _stream(stream)),
         "tvl_gemv_noalloc")


def item(W, ldw: int, x, y, M: int, K: int, dtype: int, op: int = TVL_OP_GEMV, W3=None,
         g=None, eps: float = 0.0, nrhs: int = 1, ldx: int = 0, ldy: int = 0) -> tvl_item:
    """One tvl_item; pointers as ints or tensors."""
    return tvl_item(_p(W), ldw, _p(x), _p(y), M, K, dtype, op, _p(W3) or None, _p(g) or None,
                    eps, nrhs, ldx, ldy)


def make_items(items) -> ctypes.Array:
    """items: iterable of tvl_item, (W, ldw, x, y, M, K, dtype) tuples, or
    dicts of item() keywords."""
    lst = list(items)
    arr = (tvl_item * max(len(lst), 1))()
    for i, it in enumerate(lst):
        if isinstance(it, tvl_item):
            arr[i] = it
        elif isinstance(it, dict):
            arr[i] = item(**it)
        else:
            arr[i] = item(*it)
    return arr, len(lst)


def tvl_gemv_item(it, tuning=None, stream=None) -> None:
    """Run one item (GEMV or SwiGLU, with or without RMSNorm) in one launch."""
    if isinstance(it, dict):
        it = item(**it)
    elif not isinstance(it, tvl_item):
        it = item(*it)
    t = _tuning(tuning)
    _chk(lib.tvl_gemv_item(ctypes.byref(it), ctypes.byref(t) if t is not None else None,
                           _stream(stream)), "tvl_gemv_item")


def tvl_gemv_batch_sweep(items, stream=None) -> None:
    arr, n = items if isinstance(items, tuple) else make_items(items)
    _chk(lib.tvl_gemv_batch_sweep(arr, n, _stream(stream)), "tvl_gemv_batch_sweep")


class Plan:
    """Owner of a tvl_plan*; ``run()`` is exactly one kernel launch."""

    def __init__(self, handle: int):
        self.handle = ctypes.c_void_p(handle)

    def run(self, stream=None) -> None:
        _chk(lib.tvl_sweep_plan_run(self.handle, _stream(stream)), "tvl_sweep_plan_run")

    def info(self) -> dict:
        nt, g, r = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int32()
        _chk(lib.tvl_sweep_plan_info(self.handle, ctypes.byref(nt), ctypes.byref(g),
                                     ctypes.byref(r)), "tvl_sweep_plan_info")
        return {"ntiles": nt.value, "grid": g.value, "rows_per_tile": r.value}

    def destroy(self) -> None:
        if self.handle:
            _chk(lib.tvl_sweep_plan_destroy(self.handle), "tvl_sweep_plan_destroy")
            self.handle = ctypes.c_void_p(0)

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def tvl_sweep_plan_create(items, tuning=None) -> Plan:
    arr, n = items if isinstance(items, tuple) else make_items(items)
    t = _tuning(tuning)
    h = ctypes.c_void_p()
    _chk(lib.tvl_sweep_plan_create(arr, n, ctypes.byref(t) if t is not None else None,
                                   ctypes.byref(h)), "tvl_sweep_plan_create")
    return Plan(h.value or 0)


def tvl_release_workspaces() -> None:
    _chk(lib.tvl_release_workspaces(), "tvl_release_workspaces")


def tvl_util_read_stream(src, nbytes: int, sink, sink_len: int, stream=None) -> int:
    g = ctypes.c_int64()
    _chk(lib.tvl_util_read_stream(_p(src), nbytes, _p(sink), sink_len, ctypes.byref(g),
                                  _stream(stream)), "tvl_util_read_stream")
    return g.value


def tvl_util_copy(dst, src, nbytes: int, stream=None) -> None:
    _chk(lib.tvl_util_copy(_p(dst), _p(src), nbytes, _stream(stream)), "tvl_util_copy")


def tvl_status_str(status: int) -> str:
    return lib.tvl_status_str(status).decode()


def tvl_last_error() -> str:
    return (lib.tvl_last_error() or b"").decode()


# ------------------------------------------------------------- device buffers
@dataclass
class TvlMatrix:
    """A weight matrix resident on the GPU in the TVL layout (rows of ldw)."""
    buf: object  # torch tensor owning the memory
    M: int
    K: int
    ldw: int
    dtype: int

    @property
    def ptr(self) -> int:
        return int(self.buf.data_ptr())


def upload_matrix(host, dtype: int, device="cuda", stream=None) -> TvlMatrix:
    """Copy a dense host matrix (numpy fp32, or uint16 binary16 bits) to the GPU
    and lay it out in TVL rows with tvl_pack_rows (pad zeroed)."""
    import numpy as np
    import torch
    host = np.ascontiguousarray(host)
    M, K = host.shape
    ldw = tvl_row_stride(K, dtype)
    tdt = torch.float32 if dtype == TVL_F32 else torch.int16
    src = torch.from_numpy(host.view(np.float32 if dtype == TVL_F32 else np.int16))
    if ldw == K:
        buf = src.to(device, non_blocking=False)
    else:
        dense = src.to(device)
        buf = torch.empty((M, ldw), dtype=tdt, device=device)
        tvl_pack_rows(buf, ldw, dense, M, K, dtype, stream)
        torch.cuda.current_stream().synchronize()
        del dense
    if buf.data_ptr() % 128:
        raise RuntimeError("device allocation is not 128-byte aligned")
    return TvlMatrix(buf, M, K, ldw, dtype)


def quant_matrix_bytes(M: int, K: int, dtype: int, ldw: int | None = None) -> int:
    """Bytes of a block-quantised matrix: M code rows of ldw bytes, then the
    fp32 scale plane in blocks of 4 rows (M rounded up to 4 rows, each with
    ceil(K/64) scales; a block holds its 4 rows' scales group by group)."""
    ldw = tvl_row_stride(K, dtype) if ldw is None else ldw
    return M * ldw + 4 * ((M + 3) // 4 * 4) * ((K + 63) // 64)


def upload_quant(host, M: int, K: int, dtype: int, ldw: int | None = None,
                 device="cuda") -> TvlMatrix:
    """Copy an already-quantised matrix (one uint8 buffer: code plane, then
    scale plane) to the GPU as is."""
    import numpy as np
    import torch
    if dtype not in (TVL_Q8, TVL_Q4):
        raise ValueError("upload_quant: dtype must be TVL_Q8 or TVL_Q4")
    ldw = tvl_row_stride(K, dtype) if ldw is None else ldw
    host = np.ascontiguousarray(host, dtype=np.uint8).reshape(-1)
    if host.size != quant_matrix_bytes(M, K, dtype, ldw):
        raise ValueError(f"upload_quant: {host.size} bytes, expected "
                         f"{quant_matrix_bytes(M, K, dtype, ldw)}")
    buf = torch.from_numpy(host).to(device)
    if buf.data_ptr() % 128:
        raise RuntimeError("device allocation is not 128-byte aligned")
    return TvlMatrix(buf, M, K, ldw, dtype)
