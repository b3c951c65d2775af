"""The launch shapes (CPU only): include/tvl.h lists exactly the shapes the
GPU tests run, and the library accepts every listed shape and rejects
others, for the several-vector forms (fp32 and fp16 items, single items and
plans), the fused forms, the quantised forms (8- and 4-bit, direct x and x in
LDS) and the plain single-vector forms (each x mode).  No GPU here: an
accepted call fails only at the device query (TVL_ERR_HIP).
"""
from __future__ import annotations

import ctypes
import os
import re

import pytest

from multi_shapes import (FUSED_SHAPES, MFMA, MFMA16, MFMA_DMA, MFMA_HX, MFMA_LDS, MFMA_XS, MULTI,
                          QUANT_LDS_SHAPES, QUANT_SHAPES)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
tvl = pytest.importorskip("paper_2601_03324_amd.tvl",
                          reason="libtvl.so not built (run __graft_entry__.build())")
L = tvl.lib
HIP, ARG = -6, -8
A, B, C = 1 << 40, 2 << 40, 3 << 40  # fake device addresses, never dereferenced

MATRIX = MFMA + MFMA16 + MFMA_LDS + MFMA_DMA + MFMA_HX + MFMA_XS


def header_section(start, end):
    text = open(os.path.join(ROOT, "include", "tvl.h")).read()
    return text[text.index(start):text.index(end)]


def test_header_lists_the_tested_matrix_core_shapes():
    sec = header_section("on the matrix cores:", "Launches holding block-quantised")
    listed = {tuple(map(int, m)) for m in re.findall(r"\((\d+),(\d+),(\d+)\)", sec)}
    assert listed == set(MATRIX)
    assert len(MATRIX) == len(set(MATRIX))


def test_header_lists_the_tested_valu_shapes():
    sec = header_section("on the vector ALUs:", "on the matrix cores:")
    listed = set()
    for cls, body in re.findall(r"(\d+): ((?:\(\d+,\d+,\d+\)\s*)+)", sec):
        listed |= {(*map(int, m), int(cls)) for m in re.findall(r"\((\d+),(\d+),(\d+)\)", body)}
    assert listed == set(MULTI)


def call(shape, nrhs, dt):
    r, w, u = shape
    it = tvl.item(A, 768, B, C, 768, 768, dt, nrhs=nrhs, ldx=768, ldy=768)
    t = tvl.tvl_tuning(rows_per_wave=r, waves_per_block=w, unroll=u, flags=2)
    single = L.tvl_gemv_item(ctypes.byref(it), ctypes.byref(t), None)
    arr, n = tvl.make_items([it])
    h = ctypes.c_void_p()
    plan = L.tvl_sweep_plan_create(arr, n, ctypes.byref(t), ctypes.byref(h))
    assert not h.value
    return single, plan


@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
@pytest.mark.parametrize("shape", MATRIX, ids=[f"{r}-{w}-{u}" for r, w, u in MATRIX])
def test_library_accepts_every_matrix_core_shape(shape, dt):
    for nrhs in (2, 9, 16):
        assert call(shape, nrhs, dt) == (HIP, HIP), (shape, nrhs)


@pytest.mark.parametrize("shape", MULTI, ids=[f"{r}-{w}-{u}-{b}" for r, w, u, b in MULTI])
def test_library_accepts_every_valu_shape(shape):
    r, w, u, b = shape
    assert call((r, w, u), b, 0) == (HIP, HIP)


@pytest.mark.parametrize("shape", [(16, 4, 99), (16, 3, 202), (64, 2, 202), (16, 8, 203),
                                   (64, 4, 303), (32, 1, 62), (16, 2, 8), (128, 1, 2)])
def test_unlisted_shapes_are_rejected(shape):
    assert call(shape, 8, 0) == (ARG, ARG)


def test_header_lists_the_tested_fused_shapes():
    sec = header_section("Launches holding RMSNorm or SwiGLU items", "Launches holding several")
    listed = {tuple(map(int, m)) for m in re.findall(r"\((\d+),(\d+),(\d+)\)", sec)}
    assert listed == set(FUSED_SHAPES)


@pytest.mark.parametrize("shape", FUSED_SHAPES, ids=[f"{r}-{w}-{u}" for r, w, u in FUSED_SHAPES])
def test_library_accepts_every_fused_shape(shape):
    r, w, u = shape
    D = 4 << 40
    for dt in (0, 1):
        it = tvl.item(A, 768, B, C, 768, 768, dt, g=D, eps=1e-5)
        t = tvl.tvl_tuning(rows_per_wave=r, waves_per_block=w, unroll=u, flags=2)
        assert L.tvl_gemv_item(ctypes.byref(it), ctypes.byref(t), None) == HIP
        arr, n = tvl.make_items([it])
        h = ctypes.c_void_p()
        assert L.tvl_sweep_plan_create(arr, n, ctypes.byref(t), ctypes.byref(h)) == HIP


def triples(text):
    return [tuple(map(int, m)) for m in re.findall(r"\((\d+),(\d+),(\d+)\)", text)]


def test_header_lists_the_tested_quantised_shapes():
    sec = header_section("Launches holding block-quantised items", "typedef struct tvl_tuning")
    direct, lds = sec.split("x in LDS")
    assert triples(direct) == QUANT_SHAPES
    assert triples(lds) == QUANT_LDS_SHAPES


def quant_call(shape, flags, dt):
    r, w, u = shape
    ldw = 768 if dt == 2 else 384  # K = 768 codes, 128-byte rows
    t = tvl.tvl_tuning(rows_per_wave=r, waves_per_block=w, unroll=u, flags=flags)
    single = L.tvl_gemv_ex(A, ldw, dt, B, C, 768, 768, ctypes.byref(t), None)
    arr, n = tvl.make_items([dict(W=A, ldw=ldw, x=B, y=C, M=768, K=768, dtype=dt)])
    h = ctypes.c_void_p()
    plan = L.tvl_sweep_plan_create(arr, n, ctypes.byref(t), ctypes.byref(h))
    assert not h.value
    return single, plan


@pytest.mark.parametrize("dt", [2, 3], ids=["q8", "q4"])
@pytest.mark.parametrize("flags,listed", [(2, QUANT_SHAPES), (1, QUANT_LDS_SHAPES)],
                         ids=["direct-x", "x-in-lds"])
def test_library_accepts_exactly_the_listed_quantised_shapes(flags, listed, dt):
    """Every (R, W, U) probed: the listed ones pass validation as a single
    GEMV and as a plan, the rest are rejected by both."""
    seen = set()
    for R in (1, 2, 3, 4, 8, 16):
        for W in (1, 2, 4, 8):
            for U in range(1, 10):
                single, plan = quant_call((R, W, U), flags, dt)
                assert (single == ARG) == (plan == ARG), (R, W, U)
                if single != ARG:
                    assert single == HIP and plan == HIP, (R, W, U)
                    seen.add((R, W, U))
    assert seen == set(listed)


def plain_lists(sec):
    """{(R, W, U)} from 'W=a [and W=b]: (R,U) ...' groups."""
    out = set()
    parts = re.split(r"W=(\d+)(?: and W=(\d+))?:", sec)
    for k in range(1, len(parts), 3):
        ws = [int(parts[k])] + ([int(parts[k + 1])] if parts[k + 1] else [])
        for r, u in re.findall(r"\((\d+),(\d+)\)", parts[k + 2]):
            out |= {(int(r), w, int(u)) for w in ws}
    return out


def test_header_lists_the_plain_shapes_of_each_x_mode():
    sec = header_section("*   LDS-x:", "Launches holding RMSNorm")
    lds, direct = sec.split("direct-x:")
    assert plain_lists(lds) == set(tvl.LDS_SHAPES)
    assert plain_lists(direct) == set(tvl.DIRECT_SHAPES)
    assert len(tvl.LDS_SHAPES) == len(set(tvl.LDS_SHAPES))
    assert len(tvl.DIRECT_SHAPES) == len(set(tvl.DIRECT_SHAPES))
