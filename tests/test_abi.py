"""The C-ABI library on a host without a GPU (CPU only).

The library must load, export every entry point ``include/tvl.h`` declares,
and reject every bad argument with the documented status before it makes any
HIP call (fake pointers are passed; none is ever dereferenced).
"""
from __future__ import annotations

import ctypes
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tvl.h")

tvl = pytest.importorskip("paper_2601_03324_amd.tvl",
                          reason="libtvl.so not built (run __graft_entry__.build())")
L = tvl.lib

OK, NULL, SHAPE, ALIGN, DTYPE, ALIAS, HIP, NOMEM, ARG = 0, -1, -2, -3, -4, -5, -6, -7, -8
A = 1 << 40  # fake, 128-byte aligned device addresses far apart
B = 2 << 40
C = 3 << 40


def declared_symbols():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"TVL_API\s+[\w\s\*]+?\b(tvl_\w+)\s*\(", txt)))


def test_exports_every_declared_symbol():
    syms = declared_symbols()
    assert len(syms) >= 15
    for s in syms:
        assert hasattr(L, s), s
    assert set(syms) == set(tvl.EXPORTS)
    assert tvl.tvl_version() == 100


def test_missing_library_fails_loudly(tmp_path, monkeypatch):
    monkeypatch.setattr(tvl, "LIB_PATH", str(tmp_path / "libtvl.so"))
    with pytest.raises(ImportError):
        tvl._load()


def test_item_layout_matches_header():
    assert ctypes.sizeof(tvl.tvl_item) == 96
    assert tvl.tvl_item.nrhs.offset == 76
    assert tvl.tvl_item.ldx.offset == 80
    assert tvl.tvl_item.ldy.offset == 88
    assert tvl.tvl_item.dtype.offset == 48
    assert tvl.tvl_item.op.offset == 52
    assert tvl.tvl_item.W3.offset == 56
    assert tvl.tvl_item.g.offset == 64
    assert tvl.tvl_item.eps.offset == 72
    assert ctypes.sizeof(tvl.tvl_tuning) == 24


D = 4 << 40  # another fake, far-away device address (g, W3)
E = 5 << 40


@pytest.mark.parametrize("kw,st", [
    (dict(op=2), ARG), (dict(op=1), NULL), (dict(op=1, W3=D + 64), ALIGN),
    (dict(W3=D), ARG), (dict(g=D + 4), ALIGN), (dict(g=D, eps=-1.0), ARG),
    (dict(g=D, eps=float("nan")), ARG), (dict(g=D, eps=float("inf")), ARG),
    (dict(op=1, W3=D, y=D + 128), ALIAS), (dict(g=D, eps=1e-5, y=D + 1024), ALIAS),
    (dict(nrhs=17, ldx=768, ldy=768), ARG), (dict(nrhs=-1), ARG),
    (dict(nrhs=2, ldx=767, ldy=768), SHAPE), (dict(nrhs=2, ldx=768, ldy=700), SHAPE),
    (dict(nrhs=2, ldx=770, ldy=768), ALIGN), (dict(nrhs=2, ldx=768, ldy=768, g=D), ARG),
    (dict(nrhs=2, ldx=768, ldy=768, op=1, W3=D), ARG),
    # the second y row runs into the second x row's neighbour: y rows span (n-1)*ldy + M
    (dict(nrhs=4, ldx=1024, ldy=1024, y=B + 4 * 3 * 1024), ALIAS),
])
def test_fused_item_rejects(kw, st):
    base = dict(W=A, ldw=768, x=B, y=C, M=768, K=768, dtype=0)
    it = tvl.item(**{**base, **kw})
    assert L.tvl_gemv_item(ctypes.byref(it), None, None) == st
    arr, n = tvl.make_items([it])
    assert L.tvl_gemv_batch_sweep(arr, n, None) == st


@pytest.mark.parametrize("nrhs", list(range(2, 17)))
def test_multi_item_default_shape_exists(nrhs):
    """Every vector count has a default several-vector kernel, for fp32,
    fp16 and mixed launches: validation passes and the call only fails at the
    device query of a GPU-less host."""
    for dt in (0, 1):
        it = tvl.item(A, 768, B, C, 768, 768, dt, nrhs=nrhs, ldx=768, ldy=768)
        assert L.tvl_gemv_item(ctypes.byref(it), None, None) == HIP
        arr, n = tvl.make_items([it])
        assert L.tvl_gemv_batch_sweep(arr, n, None) == HIP
    mixed = [tvl.item(A, 768, B, C, 768, 768, 0, nrhs=nrhs, ldx=768, ldy=768),
             tvl.item(D, 768, B, E, 768, 768, 1, nrhs=nrhs, ldx=768, ldy=768)]
    arr, n = tvl.make_items(mixed)
    assert L.tvl_gemv_batch_sweep(arr, n, None) == HIP


def test_fused_item_needs_direct_shape():
    it = tvl.item(A, 768, B, C, 768, 768, 0, g=D, eps=1e-5)
    t = tvl.tvl_tuning(flags=1)  # LDS-x
    assert L.tvl_gemv_item(ctypes.byref(it), ctypes.byref(t), None) == ARG
    t = tvl.tvl_tuning(ksplit=2)
    assert L.tvl_gemv_item(ctypes.byref(it), ctypes.byref(t), None) == ARG
    t = tvl.tvl_tuning(rows_per_wave=1, waves_per_block=4, unroll=8, flags=2)  # no fused form
    assert L.tvl_gemv_item(ctypes.byref(it), ctypes.byref(t), None) == ARG
    assert L.tvl_gemv_item(None, None, None) == NULL


@pytest.mark.parametrize("K,dt,ldw", [(1, 0, 32), (32, 0, 32), (33, 0, 64), (768, 0, 768),
                                      (11008, 0, 11008), (1, 1, 64), (64, 1, 64), (65, 1, 128),
                                      (28672, 1, 28672), (100, 0, 128), (100, 1, 128)])
def test_row_stride(K, dt, ldw):
    assert tvl.tvl_row_stride(K, dt) == ldw


@pytest.mark.parametrize("K,dt,ldw", [(1, 2, 128), (128, 2, 128), (129, 2, 256), (768, 2, 768),
                                      (100, 3, 128), (256, 3, 128), (257, 3, 256), (768, 3, 384),
                                      (4096, 3, 2048), (11008, 2, 11008), (11008, 3, 5504)])
def test_row_stride_quantised(K, dt, ldw):
    # code bytes ceil(K * bits / 8) rounded up to 128; the scales live apart
    assert tvl.tvl_row_stride(K, dt) == ldw
    assert synth.q_row_bytes(K, 8 if dt == 2 else 4) == ldw


def test_quantised_item_rejects():
    base = dict(W=A, ldw=768, x=B, y=C, M=768, K=768, dtype=2)
    for kw in (dict(g=D, eps=1e-5), dict(op=1, W3=D), dict(nrhs=2, ldx=768, ldy=768)):
        it = tvl.item(**{**base, **kw})
        assert L.tvl_gemv_item(ctypes.byref(it), None, None) == ARG
    assert L.tvl_pack_rows(A, 896, B, 4, 768, 2, None) == DTYPE
    # quantised and fused items may not share one launch
    arr, n = tvl.make_items([base, dict(W=A + (1 << 30), ldw=768, x=B, y=C + (1 << 20), M=768,
                                        K=768, dtype=0, g=D, eps=1e-5)])
    assert L.tvl_gemv_batch_sweep(arr, n, None) == ARG


def test_quantised_alias_covers_scale_plane():
    # 768 x 768 8-bit: code plane 768*768 bytes, then 768*12 fp32 scales
    end_codes = A + 768 * 768
    for y in (end_codes, end_codes + 4 * 768 * 12 - 4):
        it = tvl.item(W=A, ldw=768, x=B, y=y, M=768, K=768, dtype=2)
        assert L.tvl_gemv_item(ctypes.byref(it), None, None) == ALIAS


def test_row_stride_rejects():
    assert tvl.tvl_row_stride(0, 0) == -1
    assert tvl.tvl_row_stride(5, 7) == -1
    assert tvl.tvl_row_stride(-3, 1) == -1


def gemv(W=A, ldw=768, dt=0, x=B, y=C, M=768, K=768, tuning=None, fn="tvl_gemv_ex"):
    t = None if tuning is None else ctypes.byref(tvl.tvl_tuning(**tuning))
    return getattr(L, fn)(W, ldw, dt, x, y, M, K, t, None)


REJECTS = [
    (dict(W=0), NULL), (dict(x=0), NULL), (dict(y=0), NULL),
    (dict(dt=4), DTYPE), (dict(dt=-1), DTYPE),
    (dict(dt=2, ldw=640), SHAPE), (dict(dt=3, ldw=256), SHAPE), (dict(dt=2, ldw=896, tuning=dict(ksplit=2)), ARG),
    # quantised weights with x in LDS: only (4,4,1) (8,4,1) (8,2,1) (4,4,2), and x of
    # K columns in whole KiB within 160 KB (K <= 40,960)
    (dict(dt=3, ldw=512, tuning=dict(rows_per_wave=2, waves_per_block=4, unroll=2, flags=1)),
     ARG),
    (dict(dt=3, K=40961, ldw=20608, tuning=dict(flags=1)), SHAPE),
    (dict(dt=2, K=(1 << 24) + 128, ldw=(1 << 24) + 128), SHAPE),
    (dict(dt=3, ldw=(1 << 24) + 128), SHAPE),
    (dict(M=0), SHAPE), (dict(K=0), SHAPE), (dict(M=-5), SHAPE), (dict(M=1 << 31), SHAPE),
    (dict(K=(1 << 30) + 1, ldw=(1 << 30) + 32), SHAPE), (dict(ldw=767), SHAPE),
    (dict(W=A + 64), ALIGN), (dict(ldw=770), ALIGN), (dict(dt=1, ldw=800), ALIGN),
    (dict(x=B + 8), ALIGN), (dict(y=C + 2), ALIGN),
    (dict(y=A + 4096), ALIAS), (dict(y=B - 4), ALIAS), (dict(x=C + 1024), ALIAS),
    (dict(tuning=dict(rows_per_wave=3)), ARG), (dict(tuning=dict(unroll=-1)), ARG),
    (dict(tuning=dict(rows_per_wave=8, unroll=16)), ARG), (dict(tuning=dict(flags=4)), ARG),
    (dict(tuning=dict(flags=3)), ARG),
    (dict(tuning=dict(ksplit=5000)), ARG),
]


@pytest.mark.parametrize("fn", ["tvl_gemv_ex", "tvl_gemv_noalloc"])
@pytest.mark.parametrize("kw,st", REJECTS)
def test_gemv_rejects(kw, st, fn):
    """tvl_gemv_noalloc validates exactly like tvl_gemv_ex."""
    assert gemv(fn=fn, **kw) == st
    assert tvl.tvl_last_error() != ""
    assert tvl.tvl_status_str(st).startswith(tvl.STATUS[st])


def test_quantised_x_in_lds_accepted():
    """Quantised weights with x in LDS pass validation up to the LDS limit and
    reach the device query (no GPU here); a flag-only tuning keeps the default
    rows and waves, which have an LDS-x form."""
    for K, ldw in ((768, 384), (11008, 5504), (40960, 20480)):
        for tuning in (dict(flags=1), dict(rows_per_wave=8, waves_per_block=2, unroll=1,
                                           flags=1)):
            assert gemv(dt=3, K=K, ldw=ldw, tuning=tuning) in (OK, HIP), (K, tuning)
    arr, n = tvl.make_items([dict(W=A, ldw=5504, x=B, y=C, M=768, K=11008, dtype=3)])
    h = ctypes.c_void_p()
    t = tvl.tvl_tuning(flags=1)
    assert L.tvl_sweep_plan_create(arr, n, ctypes.byref(t), ctypes.byref(h)) in (OK, HIP)
    arr, n = tvl.make_items([dict(W=A, ldw=20608, x=B, y=C, M=8, K=40961, dtype=3)])
    assert L.tvl_sweep_plan_create(arr, n, ctypes.byref(t), ctypes.byref(h)) == SHAPE
    assert "LDS" in tvl.tvl_last_error()


def test_alias_boundaries_are_exact():
    # y ends exactly where W starts: no overlap, so validation passes and the
    # call gets as far as the device query (which fails without a GPU)
    M = 768
    st = gemv(W=A, y=A - 4 * M)
    assert st in (OK, HIP)
    assert gemv(W=A, y=A - 4 * M + 4) == ALIAS
    # the matrix spans M whole rows of ldw = 1024 > K elements
    end = A + M * 1024 * 4
    assert gemv(W=A, ldw=1024, y=end) in (OK, HIP)
    assert gemv(W=A, ldw=1024, y=end - 4) == ALIAS


def items(*specs):
    arr, n = tvl.make_items(specs)
    return arr, n


def test_sweep_rejects_and_enqueues_nothing():
    good = (A, 768, B, C, 768, 768, 0)
    bad_align = (A + 8, 768, B, C + (1 << 20), 768, 768, 0)
    arr, n = items(good, bad_align)
    assert L.tvl_gemv_batch_sweep(arr, n, None) == ALIGN
    assert "item 1" in tvl.tvl_last_error()
    # two outputs overlapping
    arr, n = items(good, (A + (1 << 30), 768, B, C + 100 * 4, 768, 768, 0))
    assert L.tvl_gemv_batch_sweep(arr, n, None) == ALIAS
    # output of one item over the x of another
    arr, n = items(good, (A + (1 << 30), 768, C + 16, C + (1 << 24), 768, 768, 0))
    assert L.tvl_gemv_batch_sweep(arr, n, None) == ALIAS
    # several-vector items cannot share a plan with fused items
    arr, n = tvl.make_items([dict(W=A, ldw=768, x=B, y=C, M=768, K=768, dtype=0, nrhs=2,
                                  ldx=768, ldy=768),
                             dict(W=A, ldw=768, x=B, y=C + (1 << 20), M=768, K=768, dtype=0,
                                  g=D, eps=1e-5)])
    h = ctypes.c_void_p()
    assert L.tvl_sweep_plan_create(arr, n, None, ctypes.byref(h)) == ARG
    assert L.tvl_gemv_batch_sweep(arr, n, None) == ARG
    assert L.tvl_gemv_batch_sweep(None, 3, None) == NULL
    assert L.tvl_gemv_batch_sweep(None, -1, None) == SHAPE
    # an empty sweep is a no-op that needs no device
    assert L.tvl_gemv_batch_sweep(None, 0, None) == OK


def test_shared_inputs_are_not_aliases():
    # tied weights and a shared x are legal: only outputs may not overlap
    arr, n = items((A, 768, B, C, 768, 768, 0), (A, 768, B, C + 4096, 768, 768, 0))
    st = L.tvl_gemv_batch_sweep(arr, n, None)
    assert st in (OK, HIP)


def test_plan_api_rejects():
    h = ctypes.c_void_p()
    arr, n = items((A, 768, B, C, 768, 768, 0))
    assert L.tvl_sweep_plan_create(arr, n, None, None) == NULL
    t = tvl.tvl_tuning(ksplit=2)
    assert L.tvl_sweep_plan_create(arr, n, ctypes.byref(t), ctypes.byref(h)) == ARG
    assert h.value is None
    assert L.tvl_sweep_plan_run(None, None) == NULL
    assert L.tvl_sweep_plan_info(None, None, None, None) == NULL
    assert L.tvl_sweep_plan_destroy(None) == OK  # idempotent on NULL
    assert L.tvl_sweep_plan_destroy(None) == OK


def test_pack_and_utils_reject():
    assert L.tvl_pack_rows(0, 32, B, 4, 4, 0, None) == NULL
    assert L.tvl_pack_rows(A, 4, B, 4, 4, 0, None) == ALIGN
    assert L.tvl_pack_rows(A, 32, B, 4, 40, 0, None) == SHAPE
    assert L.tvl_pack_rows(A, 32, A + 64, 4, 4, 0, None) == ALIAS
    assert L.tvl_pack_rows(A, 32, B + 2, 4, 4, 0, None) == ALIGN
    assert L.tvl_pack_rows(A, 32, B, 4, 4, 9, None) == DTYPE
    assert L.tvl_util_copy(A, A + 16, 64, None) == ALIAS
    assert L.tvl_util_copy(A, B, 60, None) == SHAPE
    assert L.tvl_util_read_stream(A, 64, B, 0, None, None) == SHAPE
    assert L.tvl_util_read_stream(A + 8, 64, B, 4, None, None) == ALIGN


@pytest.mark.parametrize("flag,shapes", [(1, "LDS_SHAPES"), (2, "DIRECT_SHAPES")])
def test_instantiated_shapes_match_binding(flag, shapes):
    """Probe every (R, W, U) in each x mode: the instantiated ones pass
    validation (and then fail at the device query on a host without a GPU),
    the rest are rejected."""
    seen = set()
    for R in (1, 2, 3, 4, 8, 16):
        for W in (1, 2, 4, 8, 16):
            for U in range(1, 17):
                st = gemv(tuning=dict(rows_per_wave=R, waves_per_block=W, unroll=U, flags=flag))
                if st != ARG:
                    seen.add((R, W, U))
    assert seen == set(getattr(tvl, shapes))


def test_status_strings():
    for code, name in tvl.STATUS.items():
        assert tvl.tvl_status_str(code).startswith(name)
    assert tvl.tvl_status_str(42) == "unknown tvl_status"
