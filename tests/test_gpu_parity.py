"""GPU parity: the HIP path through the C ABI against the CPU oracle (MI355X).

Tolerance (normalised per output by S_i = sum_j |W_ij x_j|): 1e-5 for fp32
weights, 2e-3 for fp16 weights.  Where the arithmetic is exact (identity,
integer-valued data, one-hot x, subnormal fp16 weights, zero rows) the GPU
must match bit for bit.  Every launch shape the library instantiates is run.
"""
from __future__ import annotations

import sys
import zlib

import numpy as np
import pytest

import host_oracle
import oracle
import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2601_03324_amd import tvl  # noqa: E402  (raises if libtvl.so is missing)
import synth.device as sdev  # noqa: E402

TOL = {0: 1e-5, 1: 2e-3}
DEV = "cuda"

# every (R, waves, U) the library instantiates, plus K-split and cached loads
# every (R, waves, U) the library instantiates in both x modes, plus K splits
SHAPES = ([(r, w, u, 1) for r, w, u in tvl.LDS_SHAPES]
          + [(r, w, u, 2) for r, w, u in tvl.DIRECT_SHAPES])
VARIANTS = ([None, dict(flags=1), dict(flags=2)]
            + [dict(rows_per_wave=r, waves_per_block=w, unroll=u, flags=f) for r, w, u, f in SHAPES]
            + [dict(ksplit=2), dict(ksplit=3), dict(ksplit=7),
               dict(rows_per_wave=1, waves_per_block=4, unroll=8, ksplit=4, flags=1),
               dict(rows_per_wave=8, waves_per_block=2, unroll=2, ksplit=5, flags=1),
               dict(rows_per_wave=2, waves_per_block=4, unroll=4, ksplit=3, flags=1),
               dict(rows_per_wave=1, waves_per_block=1, unroll=4, ksplit=4, flags=2),
               dict(rows_per_wave=4, waves_per_block=1, unroll=4, ksplit=2, flags=2),
               dict(rows_per_wave=2, waves_per_block=4, unroll=3, ksplit=6, flags=2),
               dict(rows_per_wave=8, waves_per_block=4, unroll=1, ksplit=16, flags=2)])


def vname(v):
    return "auto" if v is None else "-".join(f"{k[0]}{val}" for k, val in v.items())


def log(msg):
    print(msg, flush=True, file=sys.stderr)


def dev_matrix(host, dt, ldw=None, pad=None):
    """Device TVL buffer; pad (elements K..ldw-1) = 0 or a poison value."""
    M, K = host.shape
    ldw = tvl.tvl_row_stride(K, dt) if ldw is None else ldw
    if dt == 0:
        buf = torch.full((M, ldw), float("nan") if pad is None else pad, dtype=torch.float32,
                         device=DEV) if ldw != K else None
        src = torch.from_numpy(np.ascontiguousarray(host, np.float32))
    else:
        fill = 0x7E00 if pad is None else pad  # binary16 NaN
        fill = fill - 65536 if fill >= 32768 else fill
        buf = torch.full((M, ldw), fill, dtype=torch.int16, device=DEV) if ldw != K else None
        src = torch.from_numpy(np.ascontiguousarray(host, np.uint16).view(np.int16))
    if buf is None:
        buf = src.to(DEV)
    else:
        buf[:, :K] = src.to(DEV)
    assert buf.data_ptr() % 128 == 0
    return buf, ldw


def run_gemv(buf, ldw, dt, x_host, M, K, tuning=None, y_fill=float("nan")):
    x = torch.from_numpy(np.ascontiguousarray(x_host, np.float32)).to(DEV)
    y = torch.full((M,), y_fill, dtype=torch.float32, device=DEV)
    if tuning is None:
        tvl.tvl_gemv(buf, ldw, dt, x, y, M, K)
    else:
        tvl.tvl_gemv_ex(buf, ldw, dt, x, y, M, K, tuning)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def ref(host, x, dt):
    return oracle.gemv_f32(host, x) if dt == 0 else oracle.gemv_f16(host, x)


def assert_parity(y, yref, S, dt, what):
    r = oracle.check(y, yref, S, TOL[dt])
    assert r["bad"] == 0, f"{what}: {r}"
    return r


# ------------------------------------------------------------ single GEMV
def test_config_gemv768_all_variants():
    """768x768 fp32, W ~ U(-0.05, 0.05), x ~ N(0, 1), seed 0."""
    m = synth.WORKLOADS["gemv768"].mats[0]
    W, x = m.weights(), m.x()
    yref, S = oracle.gemv_f32(W, x)
    buf, ldw = dev_matrix(W, 0)
    worst = 0.0
    for v in VARIANTS:
        y = run_gemv(buf, ldw, 0, x, m.M, m.K, v)
        worst = max(worst, assert_parity(y, yref, S, 0, vname(v))["max_err"])
    log(f"gemv768: max normalised error over {len(VARIANTS)} variants = {worst:.3e}")


RAGGED = [(1, 1), (3, 17), (17, 3), (63, 64), (64, 63), (65, 65), (255, 257), (256, 256),
          (257, 255), (1000, 1000), (4095, 33), (33, 4095), (130, 11008), (5, 28672),
          (2048, 768), (768, 2048)]


@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
@pytest.mark.parametrize("M,K", RAGGED, ids=[f"{m}x{k}" for m, k in RAGGED])
def test_ragged_shapes_all_variants(M, K, dt):
    rng = np.random.default_rng(M * 100003 + K * 7 + dt)
    Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    W = Wf if dt == 0 else synth.f32_to_f16_bits(Wf)
    x = rng.standard_normal(K).astype(np.float32)
    yref, S = ref(W, x, dt)
    buf, ldw = dev_matrix(W, dt)
    for v in VARIANTS:
        y = run_gemv(buf, ldw, dt, x, M, K, v)
        assert_parity(y, yref, S, dt, f"{M}x{K} {vname(v)}")


@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
def test_padding_poison_is_never_read(dt):
    """Rows padded to a 128-byte stride with NaN in the pad: results are
    bitwise those of the same data in a zero-padded buffer."""
    rng = np.random.default_rng(5)
    for M, K, extra in ((37, 13, 1), (70, 101, 2), (9, 777, 3), (300, 1029, 1)):
        Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
        W = Wf if dt == 0 else synth.f32_to_f16_bits(Wf)
        x = rng.standard_normal(K).astype(np.float32)
        ldw = tvl.tvl_row_stride(K, dt) + extra * (32 if dt == 0 else 64)
        poison, ldw1 = dev_matrix(W, dt, ldw=ldw)       # NaN pad
        clean, _ = dev_matrix(W, dt, ldw=ldw, pad=0)      # zero pad
        yref, S = ref(W, x, dt)
        for v in VARIANTS:
            a = run_gemv(poison, ldw1, dt, x, M, K, v)
            b = run_gemv(clean, ldw1, dt, x, M, K, v)
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), vname(v)
            assert_parity(a, yref, S, dt, f"poison {M}x{K} {vname(v)}")


def test_pack_rows_layout():
    rng = np.random.default_rng(6)
    for dt, (M, K) in ((0, (19, 45)), (1, (23, 70)), (0, (5, 32))):
        Wf = (rng.standard_normal((M, K))).astype(np.float32)
        W = Wf if dt == 0 else synth.f32_to_f16_bits(Wf)
        mat = tvl.upload_matrix(W, dt, DEV)
        assert mat.ldw == tvl.tvl_row_stride(K, dt)
        got = mat.buf.cpu().numpy()
        view = got.view(np.float32 if dt == 0 else np.uint16)
        assert np.array_equal(view[:, :K], W.view(view.dtype))
        assert np.all(view[:, K:] == 0)


# ------------------------------------------------------------ closed forms
@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
def test_identity_bitwise(dt):
    rng = np.random.default_rng(7)
    for K in (1, 100, 256, 1000):
        x = (rng.standard_normal(K) * np.exp2(rng.integers(-20, 20, K))).astype(np.float32)
        I = np.eye(K, dtype=np.float32)
        W = I if dt == 0 else I.astype(np.float16).view(np.uint16)
        buf, ldw = dev_matrix(W, dt)
        for v in VARIANTS:
            y = run_gemv(buf, ldw, dt, x, K, K, v)
            assert np.array_equal(y.view(np.uint32), x.view(np.uint32)), (K, vname(v))


@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
def test_integer_data_bitwise(dt):
    """W in [-3, 3], x in [-8, 8], K <= 4096: every fp32 partial sum is an
    integer below 2^24, so any summation order is exact."""
    for M, K, seed in ((64, 4096, 1), (257, 1000, 2), (3, 77, 3)):
        kw, kx = synth.key(99, seed, 0), synth.key(99, seed, 1)
        W = (synth.int_f32(M * K, kw, -3, 3) if dt == 0 else synth.int_f16(M * K, kw, -3, 3))
        W = W.reshape(M, K)
        x = synth.int_f32(K, kx, -8, 8)
        yref, _ = ref(W, x, dt)
        buf, ldw = dev_matrix(W, dt)
        for v in VARIANTS:
            y = run_gemv(buf, ldw, dt, x, M, K, v)
            assert np.array_equal(y.astype(np.float64), yref), (M, K, vname(v))


def test_one_hot_and_zero_rows():
    rng = np.random.default_rng(8)
    M, K = 300, 515
    W = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    W[7] = 0.0
    W[299] = 0.0
    buf, ldw = dev_matrix(W, 0)
    for j in (0, 1, 256, 514):
        e = np.zeros(K, np.float32)
        e[j] = 1.0
        for v in VARIANTS:
            y = run_gemv(buf, ldw, 0, e, M, K, v)
            assert np.array_equal(y, W[:, j]), (j, vname(v))
    x = rng.standard_normal(K).astype(np.float32)
    for v in VARIANTS:
        y = run_gemv(buf, ldw, 0, x, M, K, v)
        assert y[7] == 0.0 and y[299] == 0.0


def test_f16_subnormal_weights_not_flushed():
    """W = 2^-24 (smallest binary16 subnormal) everywhere, integer x:
    y = 2^-24 * sum(x) exactly (a flush to zero would give 0)."""
    for M, K in ((64, 777), (5, 8192)):
        x = synth.int_f32(K, synth.key(98, K), -50, 50)
        W = np.full((M, K), 1, np.uint16)
        buf, ldw = dev_matrix(W, 1)
        want = np.float32(np.ldexp(float(x.astype(np.int64).sum()), -24))
        for v in VARIANTS:
            y = run_gemv(buf, ldw, 1, x, M, K, v)
            assert np.all(y == want), (M, K, vname(v), y[:4], want)


def test_nan_in_x_propagates():
    rng = np.random.default_rng(9)
    M, K = 200, 1000
    W = (rng.standard_normal((M, K)) * 0.02 + 0.5).astype(np.float32)
    buf, ldw = dev_matrix(W, 0)
    x = rng.standard_normal(K).astype(np.float32)
    x[123] = np.nan
    for v in VARIANTS:
        y = run_gemv(buf, ldw, 0, x, M, K, v)
        assert np.all(np.isnan(y)), vname(v)


def ieee_class(y):
    """-1 / +1 for -inf / +inf, 0 for NaN, 2 for finite."""
    return np.where(np.isnan(y), 0, np.where(np.isinf(y), np.sign(y), 2)).astype(np.int8)


def inf_case(rng, M, K, col):
    """Weights whose column `col` is positive, negative or zero by row, x with
    +inf there: y_i is +inf, -inf or NaN (0 * inf) by IEEE whatever the
    order of the sum (the other terms are finite)."""
    W = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    W[:, col] = np.tile(np.float32([0.5, -0.25, 0.0]), M // 3 + 1)[:M]
    x = rng.standard_normal(K).astype(np.float32)
    x[col] = np.inf
    want = np.tile(np.int8([1, -1, 0]), M // 3 + 1)[:M]
    return W, x, want


@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
def test_inf_in_x_gives_ieee_results(dt):
    """+inf in x: every plain variant gives +inf, -inf or NaN exactly where
    IEEE arithmetic does (the sign of the weight in that column; NaN where
    it is 0), with the inf in the first, a middle and the ragged last chunk."""
    rng = np.random.default_rng(77 + dt)
    M, K = 301, 1001
    for col in (0, 517, K - 1):
        W, x, want = inf_case(rng, M, K, col)
        Wd = W if dt == 0 else synth.f32_to_f16_bits(W)
        buf, ldw = dev_matrix(Wd, dt)
        for v in VARIANTS:
            y = run_gemv(buf, ldw, dt, x, M, K, v)
            assert np.array_equal(ieee_class(y), want), (col, vname(v))


@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
def test_subnormal_x_not_flushed(dt):
    """x_j = k_j 2^-140 (fp32 subnormals) and integer weights: every product
    and every partial sum is a multiple of 2^-149 below 2^-116, so the sums
    are exact in fp32 only if subnormal x, products and partial sums are
    kept (not flushed to zero); each plain variant must equal the oracle
    bit for bit."""
    rng = np.random.default_rng(140 + dt)
    M, K = 257, 1001
    Wi = rng.integers(-4, 5, (M, K)).astype(np.float32)
    W = Wi if dt == 0 else synth.f32_to_f16_bits(Wi)
    x = (rng.integers(-100, 101, K) * 2.0 ** -140).astype(np.float32)
    assert np.all(np.abs(x[x != 0]) < np.finfo(np.float32).tiny)
    yref, _ = ref(W, x, dt)
    assert np.any(yref != 0)
    buf, ldw = dev_matrix(W, dt)
    for v in VARIANTS:
        y = run_gemv(buf, ldw, dt, x, M, K, v)
        assert np.array_equal(y.astype(np.float64), yref), vname(v)


def test_output_overwritten_and_rerun_bitwise():
    """y is overwritten whatever it held; 10 reruns of each variant are
    bitwise identical (the K-split combine has a fixed order)."""
    rng = np.random.default_rng(10)
    M, K = 1024, 8192
    W = synth.f32_to_f16_bits((rng.standard_normal((M, K)) * 0.02).astype(np.float32))
    x = rng.standard_normal(K).astype(np.float32)
    buf, ldw = dev_matrix(W, 1)
    for v in VARIANTS:
        first = run_gemv(buf, ldw, 1, x, M, K, v, y_fill=float("nan"))
        for i in range(10):
            again = run_gemv(buf, ldw, 1, x, M, K, v, y_fill=1e30 if i % 2 else -7.0)
            assert np.array_equal(first.view(np.uint32), again.view(np.uint32)), vname(v)


# ------------------------------------------------------------------ sweeps
def _check_gemvs(gemvs, what, rows=None):
    worst = {0: 0.0, 1: 0.0}
    for g in gemvs:
        m = g.spec
        y = g.y.cpu().numpy()
        if rows is None:
            W = m.weights()
            yref, S = ref(W, g.x.cpu().numpy(), sdev.dtype_code(m))
            r = assert_parity(y, yref, S, sdev.dtype_code(m), f"{what} {m.name}")
        else:
            idx = sdev.sample_rows(m.M, rows, zlib.crc32(m.name.encode()))
            W = np.stack([m.weights(int(i), 1)[0] for i in idx])
            yref, S = ref(W, g.x.cpu().numpy(), sdev.dtype_code(m))
            r = assert_parity(y[idx], yref, S, sdev.dtype_code(m), f"{what} {m.name}")
        dt = sdev.dtype_code(m)
        worst[dt] = max(worst[dt], r["max_err"])
    return worst


def test_sweep110m_plan_batch_and_grid():
    """One decode token of Llama-2 110M (85 GEMVs, fp32) in one launch: every
    output against the oracle; batch-sweep and a persistent grid are bitwise
    equal to the plan."""
    wl = synth.WORKLOADS["sweep110m"]
    gemvs = sdev.load(wl, DEV)
    items = [g.item() for g in gemvs]
    plan = tvl.tvl_sweep_plan_create(items)
    info = plan.info()
    rpt = info["rows_per_tile"]
    assert info["ntiles"] == sum((m.M + rpt - 1) // rpt for m in wl.mats)
    plan.run()
    torch.cuda.synchronize()
    worst = _check_gemvs(gemvs, "sweep110m")
    log(f"sweep110m: max normalised error {worst[0]:.3e}, tiles {info['ntiles']}")
    base = [g.y.clone() for g in gemvs]
    for g in gemvs:
        g.y.fill_(float("nan"))
    tvl.tvl_gemv_batch_sweep(items)
    torch.cuda.synchronize()
    for g, b in zip(gemvs, base):
        assert torch.equal(g.y, b), g.spec.name
    for grid in (256, 1000):
        p2 = tvl.tvl_sweep_plan_create(items, dict(grid=grid))
        for g in gemvs:
            g.y.fill_(float("nan"))
        p2.run()
        torch.cuda.synchronize()
        for g, b in zip(gemvs, base):
            assert torch.equal(g.y, b), (grid, g.spec.name)
        p2.destroy()
    # every sweep launch shape
    for r, w, u, f in SHAPES:
        p3 = tvl.tvl_sweep_plan_create(items, dict(rows_per_wave=r, waves_per_block=w, unroll=u,
                                                   flags=f))
        for g in gemvs:
            g.y.fill_(float("nan"))
        p3.run()
        torch.cuda.synchronize()
        _check_gemvs(gemvs[:8] + gemvs[-1:], f"sweep110m R{r}W{w}U{u}F{f}")
        p3.destroy()
    plan.destroy()


@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
def test_two_million_rows_every_output(dt):
    """2^21 + 17 rows of 40 columns (ragged, NaN in each row's padding): the
    largest grids and tile tables of the tests (131,073 tiles of 16 rows in a
    plan; single GEMVs in both x modes, 8 rows per wavefront and a K split
    over all rows), every output against the oracle."""
    M, K = (1 << 21) + 17, 40
    rng = np.random.default_rng((1 << 21) + dt)
    Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    W = Wf if dt == 0 else synth.f32_to_f16_bits(Wf)
    del Wf
    x = rng.standard_normal(K).astype(np.float32)
    yref, S = host_oracle.gemv(W, x, dt)
    buf, ldw = dev_matrix(W, dt)
    del W
    for v in (None, dict(flags=1), dict(flags=2), dict(ksplit=2),
              dict(rows_per_wave=8, waves_per_block=4, unroll=1, flags=2)):
        log(f"{M} rows dt={dt} {vname(v)}")
        y = run_gemv(buf, ldw, dt, x, M, K, v)
        assert_parity(y, yref, S, dt, f"{M}x{K} {vname(v)}")
    xd = torch.from_numpy(x).to(DEV)
    yd = torch.full((M,), float("nan"), device=DEV)
    plan = tvl.tvl_sweep_plan_create([(buf, ldw, xd, yd, M, K, dt)])
    try:
        plan.run()
        torch.cuda.synchronize()
        assert_parity(yd.cpu().numpy(), yref, S, dt, f"{M}x{K} plan {plan.info()}")
    finally:
        plan.destroy()


def test_empty_sweeps_are_no_ops():
    """A plan of no items has no tiles and runs as a no-op (no launch), also
    under each kind of tuning; an empty batch sweep returns at once; the
    stream stays usable and a following GEMV is exact."""
    for tuning in (None, dict(flags=1), dict(flags=2),
                   dict(rows_per_wave=4, waves_per_block=4, unroll=1, flags=2)):
        plan = tvl.tvl_sweep_plan_create([], tuning)
        try:
            assert plan.info()["ntiles"] == 0
            plan.run()
            plan.run()
        finally:
            plan.destroy()
    tvl.tvl_gemv_batch_sweep([])
    torch.cuda.synchronize()
    W = np.eye(64, dtype=np.float32)
    x = np.arange(64, dtype=np.float32)
    buf, ldw = dev_matrix(W, 0)
    assert np.array_equal(run_gemv(buf, ldw, 0, x, 64, 64), x)


def test_sweep_mixed_dtypes_and_ragged():
    rng = np.random.default_rng(11)
    specs = [(1, 1, 0), (3, 17, 1), (257, 255, 0), (65, 1000, 1), (1000, 65, 0),
             (17, 11008, 0), (9, 28672, 1), (2048, 768, 0), (130, 4095, 1)]
    hosts, mats, xs, ys = [], [], [], []
    for M, K, dt in specs:
        Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
        W = Wf if dt == 0 else synth.f32_to_f16_bits(Wf)
        buf, ldw = dev_matrix(W, dt)  # NaN-poisoned pad where ldw > K
        hosts.append(W)
        mats.append((buf, ldw))
        xs.append(rng.standard_normal(K).astype(np.float32))
        ys.append(torch.full((M,), float("nan"), device=DEV))
    xd = [torch.from_numpy(x).to(DEV) for x in xs]
    items = [(mats[i][0], mats[i][1], xd[i], ys[i], M, K, dt)
             for i, (M, K, dt) in enumerate(specs)]
    for tuning in (None, dict(flags=1), dict(flags=2),
                   dict(rows_per_wave=4, waves_per_block=8, unroll=2, flags=1),
                   dict(rows_per_wave=1, waves_per_block=2, unroll=8, grid=7, flags=1),
                   dict(rows_per_wave=8, waves_per_block=1, unroll=2, flags=2),
                   dict(rows_per_wave=2, waves_per_block=4, unroll=3, grid=5, flags=2)):
        plan = tvl.tvl_sweep_plan_create(items, tuning)
        plan.run()
        torch.cuda.synchronize()
        for i, (M, K, dt) in enumerate(specs):
            yref, S = ref(hosts[i], xs[i], dt)
            assert_parity(ys[i].cpu().numpy(), yref, S, dt, f"mixed {M}x{K} {tuning}")
        plan.destroy()


def test_tied_weights_shared_by_items():
    """Two items share one W (the tied classifier) and one x."""
    m = synth.WORKLOADS["sweep110m"].mats[4]
    W, x = m.weights(), m.x()
    buf, ldw = dev_matrix(W, 0)
    xd = torch.from_numpy(x).to(DEV)
    y1 = torch.full((m.M,), float("nan"), device=DEV)
    y2 = torch.full((m.M,), float("nan"), device=DEV)
    tvl.tvl_gemv_batch_sweep([(buf, ldw, xd, y1, m.M, m.K, 0), (buf, ldw, xd, y2, m.M, m.K, 0)])
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    yref, S = oracle.gemv_f32(W, x)
    assert_parity(y1.cpu().numpy(), yref, S, 0, "tied")


def test_cls32000_100_reps():
    """The 110M classifier (32000x768 fp32) with 100 fresh x, every output."""
    wl = synth.WORKLOADS["cls32000"]
    m = wl.mats[0]
    W = m.weights()
    buf, ldw = dev_matrix(W, 0)
    worst = 0.0
    for rep in range(wl.reps):
        x = m.x(rep)
        y = run_gemv(buf, ldw, 0, x, m.M, m.K)
        yref, S = oracle.gemv_f32(W, x)
        worst = max(worst, assert_parity(y, yref, S, 0, f"cls rep {rep}")["max_err"])
    log(f"cls32000 x100: max normalised error {worst:.3e}")


def load_with_refs(wl):
    """Upload every matrix of ``wl`` and take the oracle's (y, S) of every row
    from the same host array, generated once (row blocks on every host
    thread)."""
    out = []
    for i, m in enumerate(wl.mats):
        W = m.weights()
        x = m.x(0)
        g = sdev.DevGemv(m, sdev.upload(m, W, DEV), torch.from_numpy(x).to(DEV),
                         torch.full((m.M,), float("nan"), dtype=torch.float32, device=DEV))
        dt = sdev.dtype_code(m)
        if m.quantised:
            yref, S = host_oracle.gemv_q(W, m.bits, synth.q_row_bytes(m.K, m.bits), m.M, m.K, x)
        else:
            yref, S = host_oracle.gemv(W, x, dt)
        out.append((g, yref, S))
        del W
        if i % 16 == 0 or i == len(wl.mats) - 1:
            log(f"  {wl.name}: {i + 1}/{len(wl.mats)} matrices uploaded and referenced")
    return out


@pytest.mark.parametrize("name", ["sweep7b", "stack70b8"])
def test_large_sweeps_every_output(name):
    """Llama-2 7B (fp32, 225 GEMVs, 26.4 GB) and an 8-layer 70B-shaped stack
    (fp16 weights, 56 GEMVs, 13.7 GB) in one launch each, in the launch the
    bench times: every output of every matrix against the oracle."""
    wl = synth.WORKLOADS[name]
    log(f"{name}: generating and uploading {wl.weight_bytes() / 1e9:.1f} GB")
    cases = load_with_refs(wl)
    plan = tvl.tvl_sweep_plan_create([g.item() for g, _, _ in cases])
    plan.run()
    torch.cuda.synchronize()
    worst, n = 0.0, 0
    for g, yref, S in cases:
        r = assert_parity(g.y.cpu().numpy(), yref, S, sdev.dtype_code(g.spec),
                          f"{name} {g.spec.name}")
        worst = max(worst, r["max_err"])
        n += g.spec.M
    log(f"{name}: {n} outputs, max normalised error {worst:.3e}")
    plan.destroy()
    del cases
    torch.cuda.empty_cache()


def test_batch_sweep_cache_under_threads():
    """Four host threads, each on its own stream, call tvl_gemv_batch_sweep
    over 80 distinct one-item lists: more lists than the library's plan cache
    holds, so cached plans are evicted while other threads look them up and
    launch them.  Every output of every call is checked against the oracle."""
    import threading
    rng = np.random.default_rng(99)
    M, K, nlist, nthr = 64, 256, 80, 4
    W = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    buf, ldw = dev_matrix(W, 0)
    xs = rng.standard_normal((nlist, K)).astype(np.float32)
    X = torch.from_numpy(xs).to(DEV)
    Y = torch.full((nthr, nlist, M), float("nan"), device=DEV)
    torch.cuda.synchronize()
    errors = []

    def worker(t):
        try:
            s = torch.cuda.Stream()
            for rep in range(3):
                for i in range(nlist):
                    j = (7 * i + 13 * t + rep) % nlist
                    tvl.tvl_gemv_batch_sweep([(buf, ldw, X[j], Y[t, j], M, K, 0)], s)
            s.synchronize()
        except Exception as exc:  # reported below
            errors.append((t, exc))

    ths = [threading.Thread(target=worker, args=(t,)) for t in range(nthr)]
    for th in ths:
        th.start()
    for th in ths:
        th.join()
    torch.cuda.synchronize()
    assert not errors, errors
    Yh = Y.cpu().numpy()
    for j in range(nlist):
        ref, S = oracle.gemv_f32(W, xs[j])
        for t in range(nthr):
            r = oracle.check(Yh[t, j], ref, S, 1e-5)
            assert r["bad"] == 0, (t, j, r)
    tvl.tvl_release_workspaces()


def test_ksplit_workspaces_under_threads():
    """K-split GEMVs (few long rows) from four host threads, each on its own
    stream, while a fifth thread frees the K-split workspaces again and
    again: a call must never launch with a workspace another thread has just
    freed or replaced.  Every result is checked against the oracle."""
    import threading
    import time
    rng = np.random.default_rng(123)
    M, K, nthr, reps = 64, 12288, 4, 25  # 48 KB rows, M <= 128: the library's K split
    W = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    buf, ldw = dev_matrix(W, 0)
    xs = rng.standard_normal((reps, K)).astype(np.float32)
    X = torch.from_numpy(xs).to(DEV)
    Y = torch.full((nthr, reps, M), float("nan"), device=DEV)
    torch.cuda.synchronize()
    errors, done = [], threading.Event()

    def worker(t):
        try:
            s = torch.cuda.Stream()
            for r in range(reps):
                tvl.tvl_gemv(buf, ldw, 0, X[r], Y[t, r], M, K, stream=s)
            s.synchronize()
        except Exception as exc:  # reported below
            errors.append((t, exc))

    def releaser():
        try:
            while not done.is_set():
                tvl.tvl_release_workspaces()
                time.sleep(0.001)
        except Exception as exc:
            errors.append(("release", exc))

    rel = threading.Thread(target=releaser)
    rel.start()
    ths = [threading.Thread(target=worker, args=(t,)) for t in range(nthr)]
    for th in ths:
        th.start()
    for th in ths:
        th.join()
    done.set()
    rel.join()
    torch.cuda.synchronize()
    assert not errors, errors
    Yh = Y.cpu().numpy()
    for r in range(reps):
        ref, S = oracle.gemv_f32(W, xs[r])
        for t in range(nthr):
            res = oracle.check(Yh[t, r], ref, S, 1e-5)
            assert res["bad"] == 0, (t, r, res)
    tvl.tvl_release_workspaces()
