"""Property-based checks of the C ABI's argument validation (CPU only).

Random items, valid and invalid in every field, go through
``tvl_gemv_batch_sweep`` and ``tvl_gemv_item`` on a host without a GPU.  The
library must return a documented status and never crash or touch memory (all
pointers are fake, far-apart addresses).  For single items the status must be
one that the rules in ``include/tvl.h`` allow: a rule the item breaks, or --
when it breaks none -- the device query's failure (no GPU here).  The rules
are restated below from the header, independently of the C code.
"""
from __future__ import annotations

import ctypes
import math

import pytest

hypothesis = pytest.importorskip("hypothesis")
from hypothesis import given, settings, strategies as st  # noqa: E402

tvl = pytest.importorskip("paper_2601_03324_amd.tvl",
                          reason="libtvl.so not built (run __graft_entry__.build())")
L = tvl.lib

OK, NULL, SHAPE, ALIGN, DTYPE, ALIAS, HIP, NOMEM, ARG = 0, -1, -2, -3, -4, -5, -6, -7, -8
DOCUMENTED = {OK, NULL, SHAPE, ALIGN, DTYPE, ALIAS, HIP, NOMEM, ARG}

# each pointer kind in its own 2^44-byte region (so only huge spans overlap)
REGION = {"W": 1 << 44, "x": 2 << 44, "y": 3 << 44, "g": 4 << 44, "W3": 5 << 44}


def ptr(kind):
    base = REGION[kind]
    return st.sampled_from([0, base, base + 4, base + 16, base + 64, base + 128, base + 4096])


def size_of(dt):
    return {0: 4, 1: 2}.get(dt, 1)


def q_row_bytes(K, dt):
    bits = 4 if dt == 3 else 8
    return ((K * bits + 7) // 8 + 127) // 128 * 128


ITEM = st.fixed_dictionaries({
    "W": ptr("W"), "x": ptr("x"), "y": ptr("y"), "W3": ptr("W3"), "g": ptr("g"),
    "M": st.sampled_from([-1, 0, 1, 7, 768, 32000, (1 << 31) - 1, 1 << 31]),
    "K": st.sampled_from([-5, 0, 1, 63, 768, 4096, 1 << 30, (1 << 30) + 1]),
    "ldw_extra": st.sampled_from([-1, 0, 1, 32, 64, 1 << 20]),
    "dtype": st.sampled_from([-1, 0, 1, 2, 3, 4]),
    "op": st.sampled_from([-1, 0, 1, 2]),
    "eps": st.sampled_from([0.0, 1e-5, -1.0, float("nan"), float("inf")]),
    "nrhs": st.sampled_from([-1, 0, 1, 2, 5, 16, 17]),
    "ldx_extra": st.sampled_from([-4, 0, 1, 4]),
    "ldy_extra": st.sampled_from([-1, 0, 3]),
})


def make(d):
    K, M, dt = d["K"], d["M"], d["dtype"]
    if dt in (2, 3) and K > 0:
        ldw = q_row_bytes(K, dt) + d["ldw_extra"]
    else:
        ldw = max(K, 0) + d["ldw_extra"]
    ldx = max(K, 0) + d["ldx_extra"]
    ldy = max(M, 0) + d["ldy_extra"]
    it = tvl.item(d["W"], ldw, d["x"], d["y"], M, K, dt, op=d["op"], W3=d["W3"] or None,
                  g=d["g"] or None, eps=d["eps"], nrhs=d["nrhs"], ldx=ldx, ldy=ldy)
    return it, ldw, ldx, ldy


def allowed(d, ldw, ldx, ldy):
    """Statuses the header's rules allow for this single item."""
    W, x, y, W3, g = d["W"], d["x"], d["y"], d["W3"], d["g"]
    M, K, dt, op, nrhs, eps = d["M"], d["K"], d["dtype"], d["op"], d["nrhs"], d["eps"]
    quant = dt in (2, 3)
    v = set()
    if not W or not x or not y or (op == 1 and not W3):
        v.add(NULL)
    if dt not in (0, 1, 2, 3):
        v.add(DTYPE)
    if M < 1 or M > (1 << 31) - 1 or K < 1 or K > (1 << 30):
        v.add(SHAPE)
    if K >= 1:
        if (not quant and ldw < K) or (quant and ldw < q_row_bytes(K, dt)):
            v.add(SHAPE)
        if quant and (K > (1 << 24) or ldw > (1 << 24)):
            v.add(SHAPE)
    if M >= 1 and ldw > 0 and ldw > (1 << 61) // M // size_of(dt):
        v.add(SHAPE)
    if quant and M >= 1 and K >= 1 and 4 * ((M + 3) // 4 * 4) * ((K + 63) // 64) > 0x7FFFFFFF:
        v.add(SHAPE)
    if W % 128 or (ldw * size_of(dt)) % 128 or x % 16 or y % 4:
        v.add(ALIGN)
    if nrhs < 0 or nrhs > 16 or op not in (0, 1):
        v.add(ARG)
    if nrhs > 1:
        if op != 0 or g:
            v.add(ARG)
        if ldx < K or ldy < M or ldx > (1 << 40) or ldy > (1 << 40):
            v.add(SHAPE)
        if ldx % 4:
            v.add(ALIGN)
    if quant and (op != 0 or g or nrhs > 1):
        v.add(ARG)
    if op == 1 and W3 and W3 % 128:
        v.add(ALIGN)
    if op != 1 and W3:
        v.add(ARG)
    if g and g % 16:
        v.add(ALIGN)
    if g and (not math.isfinite(eps) or eps < 0):
        v.add(ARG)
    # the output against every input (the restrict contract)
    nv = nrhs if nrhs > 1 else 1
    if M >= 1 and K >= 1 and ldw > 0:
        def over(a0, a1, b0, b1):
            return a0 < b1 and b0 < a1
        qplane = 4 * ((M + 3) // 4 * 4) * ((K + 63) // 64) if quant else 0
        yr = (y, y + 4 * ((nv - 1) * max(ldy, 0) + M))
        ins = [(W, W + M * ldw * size_of(dt) + qplane),
               (x, x + 4 * ((nv - 1) * max(ldx, 0) + K))]
        if op == 1 and W3:
            ins.append((W3, W3 + M * ldw * size_of(dt)))
        if g:
            ins.append((g, g + 4 * K))
        if any(over(*yr, *r) for r in ins):
            v.add(ALIAS)
    return v or {HIP}


@st.composite
def near_valid_item(draw):
    """A valid item, then 0-2 corrupted fields (so most cases break exactly one
    rule, or none)."""
    dt = draw(st.sampled_from([0, 1, 2, 3]))
    quant = dt in (2, 3)
    multi = not quant and draw(st.booleans())
    nrhs = draw(st.sampled_from([2, 5, 16])) if multi else draw(st.sampled_from([0, 1]))
    fused = not quant and not multi and draw(st.booleans())
    op = draw(st.sampled_from([0, 1])) if fused else 0
    d = {"W": REGION["W"] + draw(st.sampled_from([0, 128])),
         "x": REGION["x"] + draw(st.sampled_from([0, 16])),
         "y": REGION["y"] + draw(st.sampled_from([0, 4])),
         "W3": REGION["W3"] if op == 1 else 0,
         "g": REGION["g"] if fused and draw(st.booleans()) else 0,
         "M": draw(st.sampled_from([1, 7, 768, 32000])),
         "K": draw(st.sampled_from([1, 63, 768, 4096])),
         "ldw_extra": 0, "dtype": dt, "op": op, "eps": draw(st.sampled_from([0.0, 1e-5])),
         "nrhs": nrhs, "ldx_extra": 4 if multi else 0, "ldy_extra": draw(st.sampled_from([0, 3]))}
    if dt == 1 and d["K"] % 64:  # fp16 rows: a 128-byte multiple
        d["ldw_extra"] = -d["K"] % 64
    if dt == 0 and d["K"] % 32:
        d["ldw_extra"] = -d["K"] % 32
    if multi and d["K"] % 4:
        d["ldx_extra"] = 4 - d["K"] % 4
    corrupt = draw(st.lists(st.sampled_from([
        ("W", 0), ("x", 0), ("y", 0), ("W", REGION["W"] + 64), ("x", REGION["x"] + 4),
        ("y", REGION["y"] + 2), ("dtype", 7), ("M", 0), ("K", 0), ("K", (1 << 30) + 1),
        ("ldw_extra", -1), ("nrhs", 17), ("nrhs", -1), ("op", 2), ("eps", float("nan")),
        ("g", REGION["g"] + 4), ("W3", REGION["W3"]), ("ldx_extra", -1), ("ldy_extra", -1),
        ("y", REGION["W"]), ("y", REGION["x"] + 8), ("g", REGION["g"]), ("op", 1)]),
        max_size=2))
    for k, val in corrupt:
        d[k] = val
    return d


@settings(max_examples=1500, deadline=None)
@given(near_valid_item())
def test_near_valid_item_status_follows_the_rules(d):
    _check_single(d)


@settings(max_examples=600, deadline=None)
@given(ITEM)
def test_single_item_status_follows_the_rules(d):
    _check_single(d)


def _check_single(d):
    it, ldw, ldx, ldy = make(d)
    arr, n = tvl.make_items([it])
    st1 = L.tvl_gemv_batch_sweep(arr, n, None)
    assert st1 in allowed(d, ldw, ldx, ldy), (d, st1, tvl.tvl_last_error())
    if st1 != OK:
        assert tvl.tvl_last_error() != ""
    # the same item through the single-item entry point and a second call
    st2 = L.tvl_gemv_item(ctypes.byref(it), None, None)
    assert st2 in allowed(d, ldw, ldx, ldy) | ({ARG} if st1 == HIP else set()), (d, st1, st2)
    assert L.tvl_gemv_batch_sweep(arr, n, None) == st1


@settings(max_examples=300, deadline=None)
@given(st.lists(ITEM, min_size=0, max_size=5))
def test_batches_get_a_documented_status(ds):
    items = [make(d)[0] for d in ds]
    arr, n = tvl.make_items(items) if items else (None, 0)
    s = L.tvl_gemv_batch_sweep(arr, n, None)
    assert s in DOCUMENTED
    if n == 0:
        assert s == OK  # nothing to do, nothing enqueued
    else:
        assert s != OK  # no GPU: a batch that validates fails at the device query
        h = ctypes.c_void_p()
        assert L.tvl_sweep_plan_create(arr, n, None, ctypes.byref(h)) == s
        assert not h.value
