"""GPU parity of the several-vector GEMV (beam search with B hypotheses,
Sec. 9.1: one pass over the weights serves every hypothesis).  Each output
vector is checked against the oracle's GEMV of its own x (the plain
definition, applied per vector), with the GEMV parity norm.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import host_oracle
import oracle
import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2601_03324_amd import tvl  # noqa: E402
import synth.device as sdev  # noqa: E402

TOL = {0: 1e-5, 1: 2e-3}
DEV = "cuda"
from multi_shapes import MFMA, MFMA16, MFMA_DMA, MFMA_HX, MFMA_LDS, MFMA_XS, MULTI  # noqa: E402


def tunings(nrhs):
    out = [None]
    for r, w, u, b in MULTI:
        if b >= nrhs and (b == 2 or b // 2 < nrhs):  # the kernels the library would pick from
            out.append(dict(rows_per_wave=r, waves_per_block=w, unroll=u, flags=2))
    for r, w, u in MFMA + MFMA16 + MFMA_LDS + MFMA_DMA + MFMA_HX + MFMA_XS:
        out.append(dict(rows_per_wave=r, waves_per_block=w, unroll=u, flags=2))
    return out


def dev_matrix(host, dt):
    M, K = host.shape
    ldw = tvl.tvl_row_stride(K, dt)
    if dt == 0:
        buf = torch.full((M, ldw), float("nan"), dtype=torch.float32, device=DEV)
        buf[:, :K] = torch.from_numpy(np.ascontiguousarray(host, np.float32)).to(DEV)
    else:
        buf = torch.full((M, ldw), 0x7E00, dtype=torch.int16, device=DEV)
        buf[:, :K] = torch.from_numpy(np.ascontiguousarray(host, np.uint16).view(np.int16)).to(DEV)
    return buf, ldw


def run(buf, ldw, dt, X, M, K, nrhs, ldy, t):
    """X: host [nrhs, K]; x rows padded to ldx with NaN (never read); y rows
    of ldy floats, the gap after each row holds a sentinel that must stay."""
    ldx = (K + 3) // 4 * 4 + 4
    Xd = torch.full((nrhs, ldx), float("nan"), device=DEV)
    Xd[:, :K] = torch.from_numpy(X).to(DEV)
    Yd = torch.full((nrhs, ldy), -12345.0, device=DEV)
    tvl.tvl_gemv_item(dict(W=buf, ldw=ldw, x=Xd, y=Yd, M=M, K=K, dtype=dt, nrhs=nrhs, ldx=ldx,
                           ldy=ldy), t)
    torch.cuda.synchronize()
    Y = Yd.cpu().numpy()
    assert np.all(Y[:, M:] == -12345.0), "wrote past M in a y row"
    return Y[:, :M]


SHAPES = [(1, 1), (3, 17), (64, 63), (65, 65), (257, 255), (1000, 1000), (33, 4095),
          (130, 11008), (5, 28672), (2048, 768)]


@pytest.mark.parametrize("nrhs", [2, 3, 4, 5, 8, 11, 16])
@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
@pytest.mark.parametrize("M,K", SHAPES, ids=[f"{m}x{k}" for m, k in SHAPES])
def test_multi_vectors(M, K, dt, nrhs):
    rng = np.random.default_rng(M * 31 + K * 7 + dt * 3 + nrhs)
    Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    W = Wf if dt == 0 else synth.f32_to_f16_bits(Wf)
    X = rng.standard_normal((nrhs, K)).astype(np.float32)
    refs = [(oracle.gemv_f32 if dt == 0 else oracle.gemv_f16)(W, X[b]) for b in range(nrhs)]
    buf, ldw = dev_matrix(W, dt)
    for t in tunings(nrhs):
        Y = run(buf, ldw, dt, X, M, K, nrhs, M + 3, t)
        for b in range(nrhs):
            r = oracle.check(Y[b], refs[b][0], refs[b][1], TOL[dt])
            assert r["bad"] == 0, (M, K, nrhs, b, t, r)


@pytest.mark.parametrize("dt,nrhs", [(0, 16), (0, 3), (1, 8)], ids=["f32-16", "f32-3", "f16-8"])
def test_multi_million_rows(dt, nrhs):
    """2^20 + 3 rows of 72 columns (ragged) with several vectors, through the
    library's default form (shared x on the matrix cores, the VALU form, and
    split x on the fp16 matrix cores), every output of every vector against
    the oracle."""
    M, K = (1 << 20) + 3, 72
    rng = np.random.default_rng((1 << 20) + 10 * dt + nrhs)
    Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    W = Wf if dt == 0 else synth.f32_to_f16_bits(Wf)
    del Wf
    X = rng.standard_normal((nrhs, K)).astype(np.float32)
    refs = [host_oracle.gemv(W, X[b], dt) for b in range(nrhs)]
    buf, ldw = dev_matrix(W, dt)
    del W
    Y = run(buf, ldw, dt, X, M, K, nrhs, M + 5, None)
    for b in range(nrhs):
        r = oracle.check(Y[b], refs[b][0], refs[b][1], TOL[dt])
        assert r["bad"] == 0, (M, K, nrhs, b, r)


@pytest.mark.parametrize("dt,nrhs", [(0, 3), (0, 8), (0, 16), (1, 3)],
                         ids=["f32-3", "f32-8", "f32-16", "f16-3"])
def test_multi_inf_in_x_gives_ieee_results(dt, nrhs):
    """+inf in one column of one vector: that vector's outputs are +inf,
    -inf or NaN exactly as IEEE arithmetic gives them (the sign of the
    weight in that column, NaN where it is 0), the other vectors' stay
    finite; every form with fp32 products (the vector ALUs, the fp32
    matrix cores; fp16 weights on the vector ALUs).  The fp16 matrix-core
    form with split x holds for finite x only."""
    rng = np.random.default_rng(41 + 10 * dt + nrhs)
    M, K = 301, 1001
    ts = tunings(nrhs) if dt == 0 else [t for t in tunings(nrhs)
                                        if t is None or t["unroll"] < 10]
    for col in (0, 517, K - 1):
        Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
        Wf[:, col] = np.tile(np.float32([0.5, -0.25, 0.0]), M // 3 + 1)[:M]
        W = Wf if dt == 0 else synth.f32_to_f16_bits(Wf)
        X = rng.standard_normal((nrhs, K)).astype(np.float32)
        X[1, col] = np.inf
        want = np.tile(np.int8([1, -1, 0]), M // 3 + 1)[:M]
        buf, ldw = dev_matrix(W, dt)
        for t in ts:
            Y = run(buf, ldw, dt, X, M, K, nrhs, M + 3, t)
            cls = np.where(np.isnan(Y), 0, np.where(np.isinf(Y), np.sign(Y), 2)).astype(np.int8)
            assert np.array_equal(cls[1], want), (col, t)
            others = np.delete(cls, 1, axis=0)
            assert np.all(others == 2), (col, t)


@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
@pytest.mark.parametrize("nrhs", [3, 8, 16])
def test_multi_subnormal_x(nrhs, dt):
    """Weights of small integers and subnormal x (k 2^-140): every product
    and partial sum is exact only if subnormals are kept; every form must
    equal the oracle bit for bit (with fp16 weights on the fp16 matrix
    cores each chunk's range is too wide for the split: the chunk runs on
    the fp32 matrix cores)."""
    rng = np.random.default_rng(1400 + nrhs + 7 * dt)
    M, K = 301, 1001
    Wi = rng.integers(-4, 5, (M, K)).astype(np.float32)
    W = Wi if dt == 0 else synth.f32_to_f16_bits(Wi)
    X = (rng.integers(-100, 101, (nrhs, K)) * 2.0 ** -140).astype(np.float32)
    refs = [oracle.gemv_f32(Wi, X[b])[0] for b in range(nrhs)]
    buf, ldw = dev_matrix(W, dt)
    for t in tunings(nrhs):
        Y = run(buf, ldw, dt, X, M, K, nrhs, M + 3, t)
        for b in range(nrhs):
            assert np.array_equal(Y[b].astype(np.float64), refs[b]), (nrhs, b, t)


def test_multi_matches_single_bitwise_on_integers():
    """Integer data: every vector's result is exact, so it equals the
    single-vector result bit for bit."""
    M, K = 300, 2000
    W = synth.int_f32(M * K, synth.key(77, 1), -3, 3).reshape(M, K)
    X = synth.int_f32(8 * K, synth.key(77, 2), -8, 8).reshape(8, K)
    buf, ldw = dev_matrix(W, 0)
    for t in tunings(8):
        Y = run(buf, ldw, 0, X, M, K, 8, M, t)
        for b in range(8):
            ref, _ = oracle.gemv_f32(W, X[b])
            assert np.array_equal(Y[b].astype(np.float64), ref), (b, t)


def test_beam4_sweep110m():
    """The 110M decode token for 4 hypotheses (85 items x 4 vectors), one
    launch; every output of every vector against the oracle."""
    wl = synth.WORKLOADS["sweep110m"]
    ms = sdev.load_multi(wl, 4, DEV)
    hosts = [m.weights() for m in wl.mats]
    for t in (None, dict(rows_per_wave=2, waves_per_block=4, unroll=2, flags=2),
              dict(rows_per_wave=4, waves_per_block=4, unroll=1, flags=2, grid=500),
              dict(rows_per_wave=8, waves_per_block=4, unroll=1, flags=2),
              dict(rows_per_wave=16, waves_per_block=2, unroll=1, flags=2, grid=700),
              dict(rows_per_wave=32, waves_per_block=2, unroll=4, flags=2),
              dict(rows_per_wave=64, waves_per_block=1, unroll=4, flags=2, grid=300),
              dict(rows_per_wave=16, waves_per_block=4, unroll=2, flags=2),
              dict(rows_per_wave=32, waves_per_block=1, unroll=2, flags=2, grid=900),
              dict(rows_per_wave=16, waves_per_block=2, unroll=33, flags=2),
              dict(rows_per_wave=32, waves_per_block=1, unroll=32, flags=2, grid=600),
              dict(rows_per_wave=16, waves_per_block=1, unroll=33, flags=2),
              dict(rows_per_wave=16, waves_per_block=4, unroll=202, flags=2),
              dict(rows_per_wave=32, waves_per_block=2, unroll=202, flags=2, grid=400),
              dict(rows_per_wave=32, waves_per_block=1, unroll=52, flags=2, grid=500)):
        for d in ms:
            d.Y.fill_(float("nan"))
        plan = tvl.tvl_sweep_plan_create([d.item() for d in ms], t)
        plan.run()
        torch.cuda.synchronize()
        for d, Wh in zip(ms, hosts):
            m = d.spec
            Y = d.Y.cpu().numpy()
            for b in range(4):
                ref, S = host_oracle.gemv(Wh, m.x(b), 0)
                r = oracle.check(Y[b], ref, S, 1e-5)
                assert r["bad"] == 0, (m.name, b, t, r)
        plan.destroy()


def test_multi_plan_mixed_dtypes():
    """One plan holding fp32 and fp16 several-vector items with different
    vector counts (the mixed-dtype kernels), every output against the oracle,
    also with grids of 1 and 3 workgroups looping over all tiles."""
    rng = np.random.default_rng(4242)
    # (M, K, dtype, vectors); one-vector items share several-vector launches too
    specs = [(300, 1000, 0, 5), (130, 2050, 1, 11), (77, 768, 0, 16), (1, 33, 1, 2),
             (50, 300, 0, 1), (40, 640, 1, 1)]
    host, items, keep = [], [], []
    for M, K, dt, nb in specs:
        Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
        W = Wf if dt == 0 else synth.f32_to_f16_bits(Wf)
        X = rng.standard_normal((nb, K)).astype(np.float32)
        buf, ldw = dev_matrix(W, dt)
        ldx = (K + 3) // 4 * 4
        Xd = torch.full((nb, ldx), float("nan"), device=DEV)
        Xd[:, :K] = torch.from_numpy(X).to(DEV)
        Yd = torch.full((nb, M + 1), -12345.0, device=DEV)
        items.append(tvl.item(buf.data_ptr(), ldw, Xd.data_ptr(), Yd.data_ptr(), M, K, dt,
                              nrhs=nb, ldx=ldx, ldy=M + 1))
        host.append((W, X, dt, nb, Yd))
        keep += [buf, Xd, Yd]
    # small grids: each workgroup loops over tiles of both dtypes, and its
    # wavefronts drift apart (one may run an fp32 tile next to an fp16 one)
    for t in [None] + [dict(rows_per_wave=r, waves_per_block=w, unroll=u, flags=2)
                       for r, w, u in MFMA + MFMA16 + MFMA_LDS + MFMA_DMA + MFMA_HX + MFMA_XS] + [
            dict(rows_per_wave=r, waves_per_block=w, unroll=u, flags=2, grid=g)
            for r, w, u in MFMA_LDS + MFMA_DMA + MFMA_HX + MFMA_XS if w > 1
            for g in (1, 3)]:
        for *_, Yd in host:
            Yd[:, :-1].fill_(float("nan"))
        plan = tvl.tvl_sweep_plan_create(items, t)
        plan.run()
        torch.cuda.synchronize()
        for W, X, dt, nb, Yd in host:
            Y = Yd.cpu().numpy()
            assert np.all(Y[:, -1] == -12345.0), ("wrote past M", t)
            for b in range(nb):
                ref, S = (oracle.gemv_f32 if dt == 0 else oracle.gemv_f16)(W, X[b])
                r = oracle.check(Y[b, :-1], ref, S, TOL[dt])
                assert r["bad"] == 0, (W.shape, dt, nb, b, t, r)
        plan.destroy()


@pytest.mark.parametrize("nb", [8, 16])
def test_beam_sweep110m_default(nb):
    """The 110M decode token for 8 and 16 hypotheses in the launch the bench
    times (the library's default several-vector kernel, tiles in XCD-aware
    order): every output of every matrix and every vector."""
    wl = synth.WORKLOADS["sweep110m"]
    ms = sdev.load_multi(wl, nb, DEV)
    for d in ms:
        d.Y.fill_(float("nan"))
    plan = tvl.tvl_sweep_plan_create([d.item() for d in ms])
    plan.run()
    torch.cuda.synchronize()
    worst = 0.0
    for d in ms:
        m = d.spec
        Y = d.Y.cpu().numpy()
        Wh = m.weights()
        for b in range(nb):
            ref, S = host_oracle.gemv(Wh, m.x(b), 0)
            r = oracle.check(Y[b], ref, S, 1e-5)
            assert r["bad"] == 0, (m.name, nb, b, r)
            worst = max(worst, r["max_err"])
    print(f"beam{nb}_110m: every output, max normalised error {worst:.3e}", file=sys.stderr,
          flush=True)
    plan.destroy()


@pytest.mark.parametrize("nb", [8, 16])
def test_beam_70b_layer_default(nb):
    """One 70B-shaped fp16 layer (7 GEMVs, 1.71 GB) for 8 and 16 hypotheses in
    the launch the bench times (the library's default: split x on the fp16
    matrix cores, x shared by the block): every output of every matrix and
    every vector, within the fp32 parity bar (1e-5 of the norm)."""
    src = synth.WORKLOADS["stack70b8"]
    wl = synth.Workload("stack70b8[:7]", src.cfg, tuple(src.mats[:7]))
    ms = sdev.load_multi(wl, nb, DEV)
    for d in ms:
        d.Y.fill_(float("nan"))
    plan = tvl.tvl_sweep_plan_create([d.item() for d in ms])
    plan.run()
    torch.cuda.synchronize()
    worst = 0.0
    for d in ms:
        m = d.spec
        Wh = m.weights()
        Y = d.Y.cpu().numpy()
        for b in range(nb):
            ref, S = host_oracle.gemv(Wh, m.x(b), 1)
            r = oracle.check(Y[b], ref, S, 1e-5)
            assert r["bad"] == 0, (m.name, nb, b, r)
            worst = max(worst, r["max_err"])
        del Wh
    print(f"beam{nb}_70b: every output, max normalised error {worst:.3e}", file=sys.stderr,
          flush=True)
    plan.destroy()
    del ms
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dt,ldw,M", [(0, (1 << 27) - 64, 5), (0, (1 << 28) - 64, 3),
                                       (0, 1 << 28, 3), (1, (1 << 27) - 64, 9),
                                       (1, (1 << 28) - 64, 5), (1, 1 << 28, 5)],
                         ids=["f32-4rows-limit", "f32-2rows-limit", "f32-direct",
                              "f16-8rows-limit", "f16-4rows-limit", "f16-direct"])
def test_multi_huge_row_stride(dt, ldw, M):
    """Row strides at the limits of the matrix-core forms that address a
    load's rows through one buffer descriptor (31-bit size): 2 fp32 or 4 fp16
    rows (LDS-staged form, 128-column streamed chunks), 4 fp32 or 8 fp16 rows
    (64-column streamed chunks), and one past (those launches fall back to the
    direct-load form).  3, 5 or 9 rows (a partial group) of 0.25-1 GiB, 8
    vectors, every launch shape."""
    K, nb = 300, 8
    rng = np.random.default_rng(ldw % 1000 + dt)
    Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    W = Wf if dt == 0 else synth.f32_to_f16_bits(Wf)
    X = rng.standard_normal((nb, K)).astype(np.float32)
    if dt == 0:
        buf = torch.empty((M, ldw), dtype=torch.float32, device=DEV)
        buf[:, K:K + 64].fill_(float("nan"))  # padding next to the row: never used
        buf[:, :K] = torch.from_numpy(W).to(DEV)
    else:
        buf = torch.empty((M, ldw), dtype=torch.int16, device=DEV)
        buf[:, K:K + 64].fill_(0x7E00)
        buf[:, :K] = torch.from_numpy(W.view(np.int16)).to(DEV)
    refs = [(oracle.gemv_f32 if dt == 0 else oracle.gemv_f16)(W, X[b]) for b in range(nb)]
    for t in [None] + [dict(rows_per_wave=r, waves_per_block=w, unroll=u, flags=2)
                       for r, w, u in MFMA_LDS + MFMA16 + MFMA_DMA + MFMA_HX + MFMA_XS]:
        Y = run(buf, ldw, dt, X, M, K, nb, M, t)
        for b in range(nb):
            r = oracle.check(Y[b], refs[b][0], refs[b][1], TOL[dt])
            assert r["bad"] == 0, (dt, ldw, t, b, r)
    del buf
    torch.cuda.empty_cache()


@pytest.mark.parametrize("M,K", [(100, 1000), (37, 4099), (300, 768)])
def test_split_x_keeps_fp32_accuracy(M, K):
    """fp16 weights on the fp16 matrix cores with x split into two scaled fp16
    parts: the result stays within the fp32 parity bar (1e-5 of the norm), for
    x spanning 10^-20 .. 10^20 (each 128-column chunk with its own scale;
    chunks of zeros and of tiny values included)."""
    rng = np.random.default_rng(M + K)
    W = synth.f32_to_f16_bits((rng.standard_normal((M, K)) * 0.02).astype(np.float32))
    nb = 16
    mag = 10.0 ** rng.uniform(-20, 20, size=(nb, K))
    X = (rng.standard_normal((nb, K)) * mag).astype(np.float32)
    X[0, :256] = 0.0                 # two zero chunks
    X[1, 128:256] *= 1e-18           # a chunk of tiny values
    X[2] = rng.standard_normal(K).astype(np.float32)  # plain N(0, 1)
    refs = [oracle.gemv_f16(W, X[b]) for b in range(nb)]
    buf, ldw = dev_matrix(W, 1)
    for r, w, u in MFMA_HX + [t for t in MFMA_XS if t[2] > 300]:
        Y = run(buf, ldw, 1, X, M, K, nb, M, dict(rows_per_wave=r, waves_per_block=w,
                                                  unroll=u, flags=2))
        for b in range(nb):
            res = oracle.check(Y[b], refs[b][0], refs[b][1], 1e-5)
            assert res["bad"] == 0, (M, K, (r, w, u), b, res)


def test_split_x_wide_chunks():
    """Chunks whose range two fp16 parts cannot hold: a huge entry beside
    small ones, the weight under the huge entry zero and every other weight
    positive (so S is the small entries' sum).  Split as is, the small
    entries would round to zero (normalised error 1); such chunks take the
    fp32 matrix cores, so every output stays within the fp32 bar (1e-5 of the
    norm).  Full chunks and the ragged last chunk (K = 1000: 896 + 104 at 128
    columns, 960 + 40 at 64), every split-x launch shape, 16 vectors."""
    M, K, nb = 300, 1000, 16
    rng = np.random.default_rng(1000)
    X = rng.standard_normal((nb, K)).astype(np.float32)
    huge = {0: (0, 2.0 ** 40, 1.0), 1: (200, -1e10, 3e-30), 5: (700, 2.0 ** 60, 1.0),
            9: (990, 1e30, 1e-3), 12: (64, 2.0 ** 37, 1.0)}
    Wf = np.abs(rng.standard_normal((M, K)) * 0.02).astype(np.float32) + 1e-3
    for b, (col, big, small) in huge.items():
        c0 = col // 128 * 128
        X[b, c0:c0 + 128] = small
        X[b, col] = big
        Wf[:, col] = 0.0
    W = synth.f32_to_f16_bits(Wf)
    refs = [oracle.gemv_f16(W, X[b]) for b in range(nb)]
    buf, ldw = dev_matrix(W, 1)
    for r, w, u in MFMA_HX + [t for t in MFMA_XS if t[2] > 300]:
        Y = run(buf, ldw, 1, X, M, K, nb, M, dict(rows_per_wave=r, waves_per_block=w,
                                                  unroll=u, flags=2))
        for b in range(nb):
            res = oracle.check(Y[b], refs[b][0], refs[b][1], 1e-5)
            assert res["bad"] == 0, ((r, w, u), b, res)
    # the library's default for only fp16 weights and 16 vectors is a split-x form
    Y = run(buf, ldw, 1, X, M, K, nb, M, None)
    for b in range(nb):
        assert oracle.check(Y[b], refs[b][0], refs[b][1], 1e-5)["bad"] == 0, b


def test_split_x_wide_chunks_every_column_position():
    """The range test must look at every column: chunks whose only small
    nonzero entries sit at one position modulo 4 (1, 2, 3 or 0), beside one
    huge entry under a zero weight and zeros elsewhere.  Split as is, the
    small entries would round to zero (normalised error 1).  Every split-x
    shape and the default, 16 vectors, fp32 bar."""
    M, K, nb = 200, 1024, 16
    rng = np.random.default_rng(4)
    Wf = np.abs(rng.standard_normal((M, K)) * 0.02).astype(np.float32) + 1e-3
    X = np.zeros((nb, K), np.float32)
    for b in range(nb):
        pos, c0 = b % 4, (b % 8) * 128  # one chunk of 128 (two of 64) per vector
        big = c0 + (pos + 2) % 4  # the huge entry, never at the small ones' position
        X[b, c0 + pos:c0 + 128:4] = 1.0 if b < 8 else 3e-3
        X[b, big] = 2.0 ** 40 if b < 8 else 1e30
        Wf[:, big] = 0.0
        X[b, (c0 + 512) % K:(c0 + 512) % K + 128] = rng.standard_normal(128)  # a normal chunk
    W = synth.f32_to_f16_bits(Wf)
    refs = [oracle.gemv_f16(W, X[b]) for b in range(nb)]
    buf, ldw = dev_matrix(W, 1)
    for t in [dict(rows_per_wave=r, waves_per_block=w, unroll=u, flags=2)
              for r, w, u in MFMA_HX + [t for t in MFMA_XS if t[2] > 300]] + [None]:
        Y = run(buf, ldw, 1, X, M, K, nb, M, t)
        for b in range(nb):
            res = oracle.check(Y[b], refs[b][0], refs[b][1], 1e-5)
            assert res["bad"] == 0, (t, b, b % 4, res)


def test_split_x_extreme_finite_x():
    """Every finite x: chunks near the fp32 maximum (3e38), of subnormals
    (1e-39, 1e-44), of both beside ordinary values, and of zeros; small
    weights keep every product and sum finite.  fp32 bar through every
    split-x shape and the default, 16 vectors."""
    M, K, nb = 100, 768, 16
    rng = np.random.default_rng(5)
    W = synth.f32_to_f16_bits((rng.standard_normal((M, K)) * 0.02).astype(np.float32))
    X = rng.standard_normal((nb, K)).astype(np.float32)
    X[0, :128] = 3e38 * np.sign(rng.standard_normal(128)).astype(np.float32)
    X[1, :128] = np.float32(1e-39) * rng.standard_normal(128).astype(np.float32)
    X[2, :128] = np.float32(1e-44)  # subnormals down to a few ulps of the smallest
    X[3, 128:256] = 0.0
    X[3, 130] = 3e38                 # the maximum beside zeros
    X[4, 256:384] *= np.float32(1e-39)
    X[4, 300] = 2.5e38               # subnormals beside the maximum: the fp32 path
    X[5, 384:512] = np.float32(1.4e-45)  # the smallest subnormal
    X[6] = 0.0
    refs = [oracle.gemv_f16(W, X[b]) for b in range(nb)]
    assert all(np.all(np.isfinite(r[0])) for r in refs)
    buf, ldw = dev_matrix(W, 1)
    for t in [dict(rows_per_wave=r, waves_per_block=w, unroll=u, flags=2)
              for r, w, u in MFMA_HX + [t for t in MFMA_XS if t[2] > 300]] + [None]:
        Y = run(buf, ldw, 1, X, M, K, nb, M, t)
        for b in range(nb):
            res = oracle.check(Y[b], refs[b][0], refs[b][1], 1e-5)
            assert res["bad"] == 0, (t, b, res)


@pytest.mark.parametrize("nb", [5, 8, 16])
def test_split_x_forms_agree_bitwise(nb):
    """The split-x forms compute the same per-vector scale, split and
    matrix-core steps per chunk whether each wavefront splits x itself (U =
    13x) or each splits a share once per block (U = 30x): for the same chunk
    width every shape gives the same bits, including chunks that take the
    fp32 path and the ragged last chunk."""
    M, K = 300, 1000
    rng = np.random.default_rng(77 + nb)
    W = synth.f32_to_f16_bits((rng.standard_normal((M, K)) * 0.02).astype(np.float32))
    X = rng.standard_normal((nb, K)).astype(np.float32)
    X[0, 130] = 2.0 ** 50  # a wide chunk (128 columns: chunk 1; 64 columns: chunk 2)
    X[nb - 1, 900:] *= 1e-30
    buf, ldw = dev_matrix(W, 1)
    for cc in (128, 64):
        shapes = ([t for t in MFMA_HX if t[2] % 10 == (3 if cc == 128 else 2)]
                  + [t for t in MFMA_XS if t[2] > 300 and t[2] % 10 == (3 if cc == 128 else 2)])
        outs = []
        for r, w, u in shapes:
            Y = run(buf, ldw, 1, X, M, K, nb, M, dict(rows_per_wave=r, waves_per_block=w,
                                                       unroll=u, flags=2))
            outs.append(((r, w, u), Y.view(np.uint32).copy()))
        for shape, Y in outs[1:]:
            assert np.array_equal(Y, outs[0][1]), (cc, outs[0][0], shape)
        refs = [oracle.gemv_f16(W, X[b]) for b in range(nb)]
        Y = outs[0][1].view(np.float32)
        for b in range(nb):
            assert oracle.check(Y[b], refs[b][0], refs[b][1], 1e-5)["bad"] == 0, (cc, b)


@pytest.mark.parametrize("ldx", [(1 << 27) - 64, 1 << 27], ids=["xs-limit", "fallback"])
def test_multi_huge_x_stride(ldx):
    """x strides at the shared-x forms' limit (4 x vectors of one 64-column
    chunk row in a buffer descriptor's 31-bit size) and one past it (those
    launches fall back to the direct-load form; the split-x shared form reads
    x through plain pointers and runs as is): 5 vectors of 0.5 GiB each (a
    partial group of 4), fp32 and fp16 weights, every launch shape."""
    M, K, nb = 100, 300, 5
    rng = np.random.default_rng(ldx % 1000)
    Xh = rng.standard_normal((nb, K)).astype(np.float32)
    Xd = torch.empty((nb, ldx), dtype=torch.float32, device=DEV)
    Xd[:, K:K + 64].fill_(float("nan"))  # next to each vector: never used
    Xd[:, :K] = torch.from_numpy(Xh).to(DEV)
    for dt in (0, 1):
        Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
        W = Wf if dt == 0 else synth.f32_to_f16_bits(Wf)
        buf, ldw = dev_matrix(W, dt)
        refs = [(oracle.gemv_f32 if dt == 0 else oracle.gemv_f16)(W, Xh[b]) for b in range(nb)]
        for t in [None] + [dict(rows_per_wave=r, waves_per_block=w, unroll=u, flags=2)
                           for r, w, u in MFMA_XS + MFMA_DMA + MFMA_HX + MFMA_LDS]:
            Yd = torch.full((nb, M), float("nan"), device=DEV)
            tvl.tvl_gemv_item(dict(W=buf, ldw=ldw, x=Xd, y=Yd, M=M, K=K, dtype=dt, nrhs=nb,
                                   ldx=ldx, ldy=M), t)
            torch.cuda.synchronize()
            Y = Yd.cpu().numpy()
            for b in range(nb):
                r = oracle.check(Y[b], refs[b][0], refs[b][1], TOL[dt])
                assert r["bad"] == 0, (ldx, dt, t, b, r)
    del Xd
    torch.cuda.empty_cache()
