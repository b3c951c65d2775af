"""GPU parity of block-quantised weights (8-bit and 4-bit codes, one fp32
scale per 64 columns; Sec. 8.2 proposes 4-bit weights unpacked on the fly,
Sec. 2.2 names 4/8-bit quantisation) against the CPU oracle, which decodes
every weight exactly and sums in double.

Parity norm: |y - ref| / sum_j |w_ij x_j| with the decoded weights, 1e-5
(the kernel converts codes exactly and accumulates in fp32, as for fp32
weights).  With integer x and power-of-two scales every partial sum is
exact, so those cases must match bit for bit.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import synth
from multi_shapes import QUANT_LDS_SHAPES, QUANT_SHAPES  # direct x; x staged in LDS

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2601_03324_amd import tvl  # noqa: E402

TOL = 1e-5
DEV = "cuda"
BITS = {tvl.TVL_Q8: 8, tvl.TVL_Q4: 4}
RAGGED = [(1, 1), (3, 17), (17, 3), (64, 63), (65, 65), (257, 255), (1000, 1000), (33, 4095),
          (130, 11008), (5, 28672), (2048, 768), (768, 2048), (9, 2049), (31, 1023)]


def log(msg):
    print(msg, flush=True, file=sys.stderr)


def quant_case(seed, M, K, dt, extra=0, pad=0xCD):
    """Seeded fp32 weights quantised by the generator, x ~ N(0, 1); code rows
    of ldw = stride + extra bytes whose padding holds `pad`."""
    rng = np.random.default_rng(seed)
    w = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    x = rng.standard_normal(K).astype(np.float32)
    ldw = tvl.tvl_row_stride(K, dt) + extra
    Wq = synth.quantize_rows(w, BITS[dt], ldw=ldw, pad=pad)
    return Wq, ldw, x


def run_item(Wq, ldw, dt, x, M, K, tuning=None):
    Wd = tvl.upload_quant(Wq, M, K, dt, ldw, DEV)
    xd = torch.from_numpy(x).to(DEV)
    y = torch.full((M,), float("nan"), dtype=torch.float32, device=DEV)
    if tuning is None:
        tvl.tvl_gemv(Wd.buf, ldw, dt, xd, y, M, K)
    else:
        tvl.tvl_gemv_ex(Wd.buf, ldw, dt, xd, y, M, K, tuning)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def check(y, yref, S, what):
    r = oracle.check(y, yref, S, TOL)
    assert r["bad"] == 0, f"{what}: {r}"
    return r["max_err"]


@pytest.mark.parametrize("dt", [tvl.TVL_Q8, tvl.TVL_Q4], ids=["q8", "q4"])
@pytest.mark.parametrize("M,K", RAGGED, ids=[f"{m}x{k}" for m, k in RAGGED])
def test_quant_gemv(M, K, dt):
    log(f"quant gemv {M}x{K} dtype={dt}")
    Wq, ldw, x = quant_case(M * 7919 + K * 13 + dt, M, K, dt)
    yref, S = oracle.gemv_q(Wq, BITS[dt], ldw, M, K, x)
    check(run_item(Wq, ldw, dt, x, M, K), yref, S, f"{M}x{K} dt={dt}")


@pytest.mark.parametrize("shape", QUANT_SHAPES, ids=[f"R{r}W{w}U{u}" for r, w, u in QUANT_SHAPES])
@pytest.mark.parametrize("dt", [tvl.TVL_Q8, tvl.TVL_Q4], ids=["q8", "q4"])
def test_quant_shapes(shape, dt):
    r, w, u = shape
    log(f"quant shape {shape} dtype={dt}")
    for M, K in ((37, 5000), (130, 768), (7, 4097), (70, 1536), (300, 640), (9, 11008)):
        Wq, ldw, x = quant_case(M + K + r * 100 + u, M, K, dt)
        yref, S = oracle.gemv_q(Wq, BITS[dt], ldw, M, K, x)
        t = dict(rows_per_wave=r, waves_per_block=w, unroll=u, flags=2)
        check(run_item(Wq, ldw, dt, x, M, K, t), yref, S, f"{shape} {M}x{K}")


@pytest.mark.parametrize("shape", QUANT_LDS_SHAPES,
                         ids=[f"R{r}W{w}U{u}" for r, w, u in QUANT_LDS_SHAPES])
@pytest.mark.parametrize("dt", [tvl.TVL_Q8, tvl.TVL_Q4], ids=["q8", "q4"])
def test_quant_x_in_lds(shape, dt):
    """x staged in LDS per row tile: ragged K (not a multiple of 4, 32 or a
    chunk), every lane-group size (K = 255 .. 11008 gives G = 8 .. 64), rows
    past M, and NaN in the floats right after x (the staging's last 16-byte
    load brings them into LDS; the ragged last chunk must mask them)."""
    r, w, u = shape
    t = dict(rows_per_wave=r, waves_per_block=w, unroll=u, flags=1)
    for M, K in ((37, 5000), (130, 768), (7, 4097), (70, 1536), (300, 640), (9, 11008),
                 (1, 1), (3, 17), (65, 65), (257, 255), (33, 4095), (5, 2049), (31, 1023)):
        Wq, ldw, x = quant_case(M * 31 + K + r * 100 + w, M, K, dt)
        yref, S = oracle.gemv_q(Wq, BITS[dt], ldw, M, K, x)
        Wd = tvl.upload_quant(Wq, M, K, dt, ldw, DEV)
        xbuf = torch.full((64 + K + 64,), float("nan"), dtype=torch.float32, device=DEV)
        xd = xbuf[64:64 + K]  # NaN right after x: staged, never used
        xd.copy_(torch.from_numpy(x))
        y = torch.full((M,), float("nan"), dtype=torch.float32, device=DEV)
        tvl.tvl_gemv_ex(Wd.buf, ldw, dt, xd, y, M, K, t)
        torch.cuda.synchronize()
        check(y.cpu().numpy(), yref, S, f"LDS-x {shape} {M}x{K}")


@pytest.mark.parametrize("K", [16385, 28672, 40960])
def test_quant_x_in_lds_large_k(K):
    """x in LDS beyond 64 KB of dynamic LDS (K > 16,384) up to the 160 KB
    limit (K = 40,960), 4-bit and 8-bit, single GEMV and plan."""
    for dt in (tvl.TVL_Q4, tvl.TVL_Q8):
        M = 67
        Wq, ldw, x = quant_case(K + dt, M, K, dt)
        yref, S = oracle.gemv_q(Wq, BITS[dt], ldw, M, K, x)
        y = run_item(Wq, ldw, dt, x, M, K, dict(flags=1))
        check(y, yref, S, f"LDS-x K={K} dt={dt}")
        Wd = tvl.upload_quant(Wq, M, K, dt, ldw, DEV)
        xd = torch.from_numpy(x).to(DEV)
        yd = torch.full((M,), float("nan"), dtype=torch.float32, device=DEV)
        plan = tvl.tvl_sweep_plan_create([(Wd.ptr, Wd.ldw, xd, yd, M, K, dt)], dict(flags=1))
        try:
            plan.run()
            torch.cuda.synchronize()
        finally:
            plan.destroy()
        check(yd.cpu().numpy(), yref, S, f"LDS-x plan K={K} dt={dt}")


def test_quant_x_in_lds_plan_mixed():
    """A plan of 8-bit, 4-bit, fp32 and fp16 items with only the LDS-x flag
    set (default rows and waves): the quantised items read x from LDS, the
    plain ones directly; every output, two runs, bit-identical."""
    rng = np.random.default_rng(4242)
    cases, items, keep = [], [], []
    for i, (M, K, dt) in enumerate([(768, 768, tvl.TVL_Q8), (2048, 768, tvl.TVL_Q4),
                                    (768, 2048, tvl.TVL_Q4), (33, 4095, tvl.TVL_Q8),
                                    (500, 300, tvl.TVL_F32), (257, 255, tvl.TVL_F16),
                                    (1, 1, tvl.TVL_Q4), (300, 11008, tvl.TVL_Q4)]):
        x = rng.standard_normal(K).astype(np.float32)
        if dt in BITS:
            Wq, ldw, _ = quant_case(2000 + i, M, K, dt)
            Wd = tvl.upload_quant(Wq, M, K, dt, ldw, DEV)
            yref, S = oracle.gemv_q(Wq, BITS[dt], ldw, M, K, x)
        else:
            Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
            if dt == tvl.TVL_F32:
                Wd = tvl.upload_matrix(Wf, dt, DEV)
                yref, S = oracle.gemv_f32(Wf, x)
            else:
                Wh = synth.f32_to_f16_bits(Wf)
                Wd = tvl.upload_matrix(Wh, dt, DEV)
                yref, S = oracle.gemv_f16(Wh, x)
        xd = torch.from_numpy(x).to(DEV)
        y = torch.full((M,), float("nan"), dtype=torch.float32, device=DEV)
        keep.append((Wd, xd))
        items.append((Wd.ptr, Wd.ldw, xd, y, M, K, dt))
        cases.append((y, yref, S, f"item {i} {M}x{K} dt={dt}"))
    plan = tvl.tvl_sweep_plan_create(items, dict(flags=1))
    outs = []
    try:
        for rep in range(2):
            for y, *_ in cases:
                y.fill_(float("nan"))
            plan.run()
            torch.cuda.synchronize()
            outs.append([y.cpu().numpy().copy() for y, *_ in cases])
            for y, yref, S, what in cases:
                check(y.cpu().numpy(), yref, S, f"LDS-x rep {rep} {what}")
    finally:
        plan.destroy()
    for a, b, (_, _, _, what) in zip(outs[0], outs[1], cases):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), what


@pytest.mark.parametrize("dt", [tvl.TVL_Q8, tvl.TVL_Q4], ids=["q8", "q4"])
def test_quant_two_million_rows(dt):
    """2^21 + 5 rows of 100 columns (two scale groups, the last one ragged;
    a scale plane of 2,097,152 + 8 rows in 4-row blocks): the default, x in
    LDS, another shape and a plan, every output against the oracle."""
    M, K = (1 << 21) + 5, 100
    log(f"quant {M} rows dtype={dt}")
    Wq, ldw, x = quant_case((1 << 21) + dt, M, K, dt)
    yref, S = oracle.gemv_q(Wq, BITS[dt], ldw, M, K, x)
    for t in (None, dict(flags=1), dict(rows_per_wave=4, waves_per_block=4, unroll=1, flags=2)):
        check(run_item(Wq, ldw, dt, x, M, K, t), yref, S, f"{M}x{K} {t}")
    Wd = tvl.upload_quant(Wq, M, K, dt, ldw, DEV)
    xd = torch.from_numpy(x).to(DEV)
    yd = torch.full((M,), float("nan"), dtype=torch.float32, device=DEV)
    plan = tvl.tvl_sweep_plan_create([(Wd.ptr, Wd.ldw, xd, yd, M, K, dt)])
    try:
        plan.run()
        torch.cuda.synchronize()
    finally:
        plan.destroy()
    check(yd.cpu().numpy(), yref, S, f"{M}x{K} plan")


@pytest.mark.parametrize("dt", [tvl.TVL_Q8, tvl.TVL_Q4], ids=["q8", "q4"])
def test_quant_inf_in_x_gives_ieee_results(dt):
    """+inf in x: rows whose code in that column is positive, negative or 0
    give +inf, -inf or NaN (0 * inf), as IEEE arithmetic on the decoded
    weights does; every shape, direct x and x in LDS."""
    rng = np.random.default_rng(5 + dt)
    M, K = 301, 1001
    tunings = [None] + [dict(rows_per_wave=r, waves_per_block=w_, unroll=u, flags=2)
                        for r, w_, u in QUANT_SHAPES] + \
        [dict(rows_per_wave=r, waves_per_block=w_, unroll=u, flags=1)
         for r, w_, u in QUANT_LDS_SHAPES]
    for col in (0, 517, K - 1):
        w = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
        w[:, col] = np.tile(np.float32([0.05, -0.05, 0.0]), M // 3 + 1)[:M]
        x = rng.standard_normal(K).astype(np.float32)
        x[col] = np.inf
        ldw = tvl.tvl_row_stride(K, dt)
        Wq = synth.quantize_rows(w, BITS[dt], ldw=ldw)
        want = np.tile(np.int8([1, -1, 0]), M // 3 + 1)[:M]
        for t in tunings:
            y = run_item(Wq, ldw, dt, x, M, K, t)
            cls = np.where(np.isnan(y), 0, np.where(np.isinf(y), np.sign(y), 2)).astype(np.int8)
            assert np.array_equal(cls, want), (col, t)


@pytest.mark.parametrize("dt", [tvl.TVL_Q8, tvl.TVL_Q4], ids=["q8", "q4"])
def test_quant_wide_rows_and_junk_padding(dt):
    """ldw beyond the minimum, padding full of junk codes: never read into y."""
    for M, K, extra in ((65, 1000, 128), (3, 130, 1024), (100, 4095, 384)):
        for pad in (0x00, 0x77, 0xFF):
            Wq, ldw, x = quant_case(K + extra + pad, M, K, dt, extra, pad)
            yref, S = oracle.gemv_q(Wq, BITS[dt], ldw, M, K, x)
            check(run_item(Wq, ldw, dt, x, M, K), yref, S, f"{M}x{K}+{extra} pad={pad:#x}")


@pytest.mark.parametrize("dt", [tvl.TVL_Q8, tvl.TVL_Q4], ids=["q8", "q4"])
def test_quant_exact_on_integers(dt):
    """Codes over the full range, power-of-two scales, integer x (and the
    same x scaled into the fp32 subnormals): the result is exact, so it must
    equal the oracle bit for bit."""
    bits = BITS[dt]
    for M, K in ((77, 4096), (5, 3000), (300, 129)):
        rng = np.random.default_rng(M * K + bits)
        ldw = tvl.tvl_row_stride(K, dt)
        ng = (K + 63) // 64
        codes = rng.integers(0, 256 if bits == 8 else 16, (M, ldw * 8 // bits)).astype(np.uint8)
        if bits == 8:
            plane = codes
        else:
            plane = codes[:, 0::2] | (codes[:, 1::2] << 4)
        scales = np.exp2(rng.integers(-2, 1, (M, ng))).astype(np.float32)
        Mp = (M + 3) // 4 * 4
        full = np.full((Mp, ng), np.float32(1e30))  # junk in the padding rows
        full[:M] = scales
        sp = np.ascontiguousarray(full.reshape(Mp // 4, 4, ng).transpose(0, 2, 1))  # 4-row blocks
        Wq = np.concatenate([plane.reshape(-1), sp.reshape(-1).view(np.uint8)])
        x = rng.integers(-4, 5, K).astype(np.float32)
        yref, _ = oracle.gemv_q(Wq, bits, ldw, M, K, x)
        y = run_item(Wq, ldw, dt, x, M, K)
        assert np.array_equal(y.astype(np.float64), yref), f"{M}x{K}"
        # the same with subnormal x (k 2^-140): exact only if subnormal x,
        # products and partial sums are kept, direct x and x in LDS
        xs = (x * 2.0 ** -140).astype(np.float32)
        yref, _ = oracle.gemv_q(Wq, bits, ldw, M, K, xs)
        assert np.array_equal(yref.astype(np.float32).astype(np.float64), yref)
        for t in (None, dict(flags=1), dict(flags=2)):
            y = run_item(Wq, ldw, dt, xs, M, K, t)
            assert np.array_equal(y.astype(np.float64), yref), f"{M}x{K} subnormal x {t}"


@pytest.mark.parametrize("dt", [tvl.TVL_Q8, tvl.TVL_Q4], ids=["q8", "q4"])
def test_quant_extreme_scales(dt):
    """Huge weights (scales up to 1e37 / 7: the 4-bit kernels fold the codes'
    1/16 into the scale, so a scale must stay below 2^124) with tiny x, and
    tiny weights (subnormal scales) with huge x: every product and sum stays
    finite and normal, so the results must meet the bar; default and every
    shape (direct x and x in LDS)."""
    rng = np.random.default_rng(9 + dt)
    M, K = 64, 1000
    tunings = [None] + [dict(rows_per_wave=r, waves_per_block=w_, unroll=u, flags=2)
                        for r, w_, u in QUANT_SHAPES] + \
        [dict(rows_per_wave=r, waves_per_block=w_, unroll=u, flags=1)
         for r, w_, u in QUANT_LDS_SHAPES]
    huge = np.clip(rng.standard_normal((M, K)) * 3e36, -1e37, 1e37).astype(np.float32)
    tiny = (rng.standard_normal((M, K)) * 2e-38).astype(np.float32)
    for w, xs in ((huge, 1e-8), (tiny, 1e30)):
        x = (rng.standard_normal(K) * xs).astype(np.float32)
        ldw = tvl.tvl_row_stride(K, dt)
        Wq = synth.quantize_rows(w, BITS[dt], ldw=ldw)
        yref, S = oracle.gemv_q(Wq, BITS[dt], ldw, M, K, x)
        assert np.all(np.isfinite(yref))
        for t in tunings:
            check(run_item(Wq, ldw, dt, x, M, K, t), yref, S, f"extreme scales x~{xs} {t}")


def test_quant_plan_mixed_with_float_items():
    """One plan over 8-bit, 4-bit, fp32 and fp16 items, run twice."""
    rng = np.random.default_rng(99)
    cases, items, keep = [], [], []
    for i, (M, K, dt) in enumerate([(768, 768, tvl.TVL_Q8), (2048, 768, tvl.TVL_Q4),
                                    (768, 2048, tvl.TVL_Q4), (33, 4095, tvl.TVL_Q8),
                                    (500, 300, tvl.TVL_F32), (257, 255, tvl.TVL_F16),
                                    (1, 1, tvl.TVL_Q4)]):
        x = rng.standard_normal(K).astype(np.float32)
        if dt in BITS:
            Wq, ldw, _ = quant_case(1000 + i, M, K, dt)
            Wd = tvl.upload_quant(Wq, M, K, dt, ldw, DEV)
            yref, S = oracle.gemv_q(Wq, BITS[dt], ldw, M, K, x)
        else:
            Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
            if dt == tvl.TVL_F32:
                Wd = tvl.upload_matrix(Wf, dt, DEV)
                yref, S = oracle.gemv_f32(Wf, x)
            else:
                Wh = synth.f32_to_f16_bits(Wf)
                Wd = tvl.upload_matrix(Wh, dt, DEV)
                yref, S = oracle.gemv_f16(Wh, x)
        xd = torch.from_numpy(x).to(DEV)
        y = torch.full((M,), float("nan"), dtype=torch.float32, device=DEV)
        keep.append((Wd, xd))
        items.append((Wd.ptr, Wd.ldw, xd, y, M, K, dt))
        cases.append((y, yref, S, f"item {i} {M}x{K} dt={dt}"))
    plan = tvl.tvl_sweep_plan_create(items)
    try:
        for rep in range(2):
            for y, *_ in cases:
                y.fill_(float("nan"))
            plan.run()
            torch.cuda.synchronize()
            for y, yref, S, what in cases:
                check(y.cpu().numpy(), yref, S, f"rep {rep} {what}")
    finally:
        plan.destroy()
    for y, *_ in cases:
        y.fill_(float("nan"))
    tvl.tvl_gemv_batch_sweep(items)
    torch.cuda.synchronize()
    for y, yref, S, what in cases:
        check(y.cpu().numpy(), yref, S, f"batch sweep {what}")


@pytest.mark.parametrize("dt", [tvl.TVL_Q8, tvl.TVL_Q4], ids=["q8", "q4"])
def test_quant_7b_layer_shapes(dt):
    """Full-size Llama-2-7B projections (4096 x 4096, 11008 x 4096,
    4096 x 11008) and the 32000-row classifier, every row checked."""
    for M, K in ((4096, 4096), (11008, 4096), (4096, 11008), (32000, 4096)):
        log(f"quant 7B shape {M}x{K} dtype={dt}")
        Wq, ldw, x = quant_case(M ^ K ^ dt, M, K, dt)
        yref, S = oracle.gemv_q(Wq, BITS[dt], ldw, M, K, x)
        check(run_item(Wq, ldw, dt, x, M, K), yref, S, f"{M}x{K}")


@pytest.mark.parametrize("name", ["sweep110m_q8", "sweep110m_q4", "sweep7b_q8", "sweep7b_q4"])
def test_quant_sweeps_in_one_launch(name):
    """Whole decode tokens with block-quantised weights in the launch the
    bench times (one plan, the library's default shape): every output of
    every matrix against the oracle, on the very bytes uploaded."""
    import host_oracle
    import synth.device as sdev
    wl = synth.WORKLOADS[name]
    log(f"{name}: generating and uploading {wl.weight_bytes() / 1e9:.2f} GB")
    cases = []
    for i, m in enumerate(wl.mats):
        Wq = m.weights()
        x = m.x(0)
        g = sdev.DevGemv(m, sdev.upload(m, Wq, DEV), torch.from_numpy(x).to(DEV),
                         torch.full((m.M,), float("nan"), dtype=torch.float32, device=DEV))
        yref, S = host_oracle.gemv_q(Wq, m.bits, synth.q_row_bytes(m.K, m.bits), m.M, m.K, x)
        cases.append((g, yref, S))
        del Wq
    plan = tvl.tvl_sweep_plan_create([g.item() for g, _, _ in cases])
    plan.run()
    torch.cuda.synchronize()
    worst = 0.0
    for g, yref, S in cases:
        worst = max(worst, check(g.y.cpu().numpy(), yref, S, f"{name} {g.spec.name}"))
    log(f"{name}: every output, max normalised error {worst:.3e}")
    plan.destroy()
    del cases
    torch.cuda.empty_cache()
