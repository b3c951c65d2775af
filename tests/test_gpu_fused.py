"""GPU parity of the fused items: RMSNorm before the GEMV (Sec. 2.1, the
Sec. 11.2 listing) and the SwiGLU gate of the FFN (Sec. 2.1), against the
CPU oracle (which normalises first, then multiplies, in double).

GEMV outputs use the GEMV parity norm (|y - ref| / sum_j |W_ij xn_j|, 1e-5
for fp32 weights, 2e-3 for fp16).  SwiGLU outputs h = silu(a) b use the
first-order propagation of that norm through the gate
(oracle.swiglu_bound), with the same tolerances.
"""
from __future__ import annotations

import sys
import zlib

import numpy as np
import pytest

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
from multi_shapes import FUSED_SHAPES  # noqa: E402
TUNINGS = [None] + [dict(rows_per_wave=r, waves_per_block=w, unroll=u, flags=2)
                    for r, w, u in FUSED_SHAPES]


def log(msg):
    print(msg, flush=True, file=sys.stderr)


def dev_matrix(host, dt, ldw=None):
    """TVL buffer with NaN in the padding (never read)."""
    M, K = host.shape
    ldw = tvl.tvl_row_stride(K, dt) if ldw is None else ldw
    if dt == 0:
        buf = torch.full((M, ldw), float("nan"), dtype=torch.float32, device=DEV)
        buf[:, :K] = torch.from_numpy(np.ascontiguousarray(host, np.float32)).to(DEV)
    else:
        buf = torch.full((M, ldw), 0x7E00, dtype=torch.int16, device=DEV)
        buf[:, :K] = torch.from_numpy(np.ascontiguousarray(host, np.uint16).view(np.int16)).to(DEV)
    return buf, ldw


def rand_w(rng, M, K, dt):
    Wf = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    return Wf if dt == 0 else synth.f32_to_f16_bits(Wf)


def check_gemv(y, yref, S, dt, what):
    r = oracle.check(y, yref, S, TOL[dt])
    assert r["bad"] == 0, f"{what}: {r}"
    return r["max_err"]


def check_swiglu(h, href, bound, dt, what):
    r = oracle.check(h, href, bound, TOL[dt])
    assert r["bad"] == 0, f"{what}: {r}"
    return r["max_err"]


RAGGED = [(1, 1), (3, 17), (17, 3), (64, 63), (65, 65), (257, 255), (1000, 1000), (33, 4095),
          (130, 11008), (5, 28672), (2048, 768), (768, 2048)]


@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
@pytest.mark.parametrize("M,K", RAGGED, ids=[f"{m}x{k}" for m, k in RAGGED])
def test_rmsnorm_gemv_item(M, K, dt):
    rng = np.random.default_rng(M * 7919 + K * 13 + dt)
    W = rand_w(rng, M, K, dt)
    x = rng.standard_normal(K).astype(np.float32)
    g = rng.uniform(0.5, 1.5, K).astype(np.float32)
    yref, S = oracle.rmsnorm_gemv(W, x, g, 1e-5)
    buf, ldw = dev_matrix(W, dt)
    xd, gd = torch.from_numpy(x).to(DEV), torch.from_numpy(g).to(DEV)
    for t in TUNINGS:
        y = torch.full((M,), float("nan"), device=DEV)
        tvl.tvl_gemv_item(dict(W=buf, ldw=ldw, x=xd, y=y, M=M, K=K, dtype=dt, g=gd, eps=1e-5), t)
        torch.cuda.synchronize()
        check_gemv(y.cpu().numpy(), yref, S, dt, f"rmsnorm {M}x{K} {t}")


@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
@pytest.mark.parametrize("norm", [False, True], ids=["plain", "norm"])
@pytest.mark.parametrize("M,K", RAGGED, ids=[f"{m}x{k}" for m, k in RAGGED])
def test_swiglu_item(M, K, norm, dt):
    rng = np.random.default_rng(M * 104729 + K * 31 + dt * 2 + norm)
    W1, W3 = rand_w(rng, M, K, dt), rand_w(rng, M, K, dt)
    # a larger scale makes the gate nonlinear over the whole silu range
    x = (rng.standard_normal(K) * 4).astype(np.float32)
    g = rng.uniform(0.5, 1.5, K).astype(np.float32) if norm else None
    href, a, b, Sa, Sb = oracle.swiglu_ffn_in(W1, W3, x, g, 1e-5)
    bound = oracle.swiglu_bound(a, b, Sa, Sb)
    b1, ldw = dev_matrix(W1, dt)
    b3, _ = dev_matrix(W3, dt)
    xd = torch.from_numpy(x).to(DEV)
    gd = torch.from_numpy(g).to(DEV) if norm else None
    for t in TUNINGS:
        y = torch.full((M,), float("nan"), device=DEV)
        tvl.tvl_gemv_item(dict(W=b1, ldw=ldw, x=xd, y=y, M=M, K=K, dtype=dt,
                               op=tvl.TVL_OP_SWIGLU, W3=b3, g=gd, eps=1e-5), t)
        torch.cuda.synchronize()
        check_swiglu(y.cpu().numpy(), href, bound, dt, f"swiglu {M}x{K} norm={norm} {t}")


def ieee_class(y):
    """-1 / +1 for -inf / +inf, 0 for NaN, 2 for finite."""
    y = np.asarray(y, np.float64)
    return np.where(np.isnan(y), 0, np.where(np.isinf(y), np.sign(y), 2)).astype(np.int8)


@pytest.mark.parametrize("dt", [0, 1], ids=["f32", "f16"])
def test_fused_inf_in_x_matches_the_oracle(dt):
    """+inf in x, fused items: with RMSNorm the normalised x is NaN at that
    column and 0 elsewhere, so every output is NaN; a SwiGLU pair without
    RMSNorm gives silu(a) * b with a, b = +-inf or NaN by the weights' signs
    (silu(-inf) is NaN, silu(+inf) = +inf).  The GPU's +inf / -inf / NaN /
    finite pattern must equal the oracle's, every fused shape."""
    rng = np.random.default_rng(606 + dt)
    M, K, col = 301, 1001, 517
    W1 = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    W3 = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    W1[:, col] = np.tile(np.float32([0.5, -0.25, 0.0]), M // 3 + 1)[:M]
    W3[:, col] = np.tile(np.float32([0.5, 0.5, -0.5, 0.0]), M // 4 + 1)[:M]
    if dt == 1:
        W1, W3 = synth.f32_to_f16_bits(W1), synth.f32_to_f16_bits(W3)
    x = rng.standard_normal(K).astype(np.float32)
    x[col] = np.inf
    g = rng.uniform(0.5, 1.5, K).astype(np.float32)
    yref, _ = oracle.rmsnorm_gemv(W1, x, g, 1e-5)
    href = oracle.swiglu_ffn_in(W1, W3, x, None, 1e-5)[0]
    assert np.all(np.isnan(yref))
    want = ieee_class(href)
    assert set(np.unique(want)) == {-1, 0, 1}
    b1, ldw = dev_matrix(W1, dt)
    b3, _ = dev_matrix(W3, dt)
    xd, gd = torch.from_numpy(x).to(DEV), torch.from_numpy(g).to(DEV)
    for t in TUNINGS:
        y = torch.full((M,), 0.0, device=DEV)
        tvl.tvl_gemv_item(dict(W=b1, ldw=ldw, x=xd, y=y, M=M, K=K, dtype=dt, g=gd, eps=1e-5), t)
        h = torch.full((M,), 0.0, device=DEV)
        tvl.tvl_gemv_item(dict(W=b1, ldw=ldw, x=xd, y=h, M=M, K=K, dtype=dt,
                               op=tvl.TVL_OP_SWIGLU, W3=b3), t)
        torch.cuda.synchronize()
        assert np.all(np.isnan(y.cpu().numpy())), t
        assert np.array_equal(ieee_class(h.cpu().numpy()), want), t


def test_fused_closed_forms():
    """Exact cases: identity W after RMSNorm of a +-1 vector (mean square 1,
    eps 0) gives g * x bitwise; a zero W3 row gives h = 0; a saturated gate
    gives h = b (large positive a) or 0 (large negative a); NaN in x
    propagates through the normalisation to every output."""
    K = 256
    x = np.where(np.arange(K) % 3 == 0, -1.0, 1.0).astype(np.float32)
    g = (np.arange(K) % 7 + 1).astype(np.float32)
    I = np.eye(K, dtype=np.float32)
    buf, ldw = dev_matrix(I, 0)
    xd, gd = torch.from_numpy(x).to(DEV), torch.from_numpy(g).to(DEV)
    for t in TUNINGS:
        y = torch.full((K,), float("nan"), device=DEV)
        tvl.tvl_gemv_item(dict(W=buf, ldw=ldw, x=xd, y=y, M=K, K=K, dtype=0, g=gd, eps=0.0), t)
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy(), x * g), t
    # SwiGLU: W1 = 100 I (gate saturates at silu(100 x)), W3 = I with zero rows
    W1 = (100 * np.eye(K)).astype(np.float32)
    W3 = np.eye(K, dtype=np.float32)
    W3[5] = 0.0
    b1, _ = dev_matrix(W1, 0)
    b3, _ = dev_matrix(W3, 0)
    for t in TUNINGS:
        y = torch.full((K,), float("nan"), device=DEV)
        tvl.tvl_gemv_item(dict(W=b1, ldw=ldw, x=xd, y=y, M=K, K=K, dtype=0,
                               op=tvl.TVL_OP_SWIGLU, W3=b3), t)
        torch.cuda.synchronize()
        h = y.cpu().numpy()
        assert h[5] == 0.0
        pos, neg = x > 0, x < 0
        pos[5] = neg[5] = False
        assert np.all(h[pos] == 100.0)   # silu(100) * 1 = 100 (sigmoid rounds to 1)
        assert np.all(h[neg] == 0.0)     # expf(100) overflows fp32: silu(-100) = -0
    xn = x.copy()
    xn[9] = np.nan
    xnd = torch.from_numpy(xn).to(DEV)
    y = torch.zeros(K, device=DEV)
    tvl.tvl_gemv_item(dict(W=buf, ldw=ldw, x=xnd, y=y, M=K, K=K, dtype=0, g=gd, eps=1e-5))
    torch.cuda.synchronize()
    assert np.all(np.isnan(y.cpu().numpy()))


def test_fused_rerun_bitwise():
    rng = np.random.default_rng(3)
    M, K = 1000, 4096
    W1, W3 = rand_w(rng, M, K, 1), rand_w(rng, M, K, 1)
    b1, ldw = dev_matrix(W1, 1)
    b3, _ = dev_matrix(W3, 1)
    xd = torch.from_numpy(rng.standard_normal(K).astype(np.float32)).to(DEV)
    gd = torch.from_numpy(rng.uniform(0.5, 1.5, K).astype(np.float32)).to(DEV)
    for t in TUNINGS:
        outs = []
        for i in range(5):
            y = torch.full((M,), float("nan") if i % 2 else 7.0, device=DEV)
            tvl.tvl_gemv_item(dict(W=b1, ldw=ldw, x=xd, y=y, M=M, K=K, dtype=1,
                                   op=tvl.TVL_OP_SWIGLU, W3=b3, g=gd, eps=1e-5), t)
            torch.cuda.synchronize()
            outs.append(y.cpu().numpy().view(np.uint32))
        for o in outs[1:]:
            assert np.array_equal(o, outs[0]), t


def _check_fused_gemvs(gemvs, what, rows=None):
    worst = 0.0
    for d in gemvs:
        it = d.spec
        dt = sdev.dtype_code(it.W)
        idx = (np.arange(it.M) if rows is None
               else sdev.sample_rows(it.M, rows, zlib.crc32(it.name.encode())))
        W = it.W.weights() if rows is None else np.stack([it.W.weights(int(i), 1)[0] for i in idx])
        x = it.x.values()
        g = it.g.values() if it.g is not None else None
        y = d.y.cpu().numpy()[idx]
        if it.W3 is None:
            xd = oracle.rmsnorm(x, g, it.eps) if g is not None else x.astype(np.float64)
            yref, S = oracle.gemv_dx(W, xd)
            worst = max(worst, check_gemv(y, yref, S, dt, f"{what} {it.name}"))
        else:
            W3 = (it.W3.weights() if rows is None
                  else np.stack([it.W3.weights(int(i), 1)[0] for i in idx]))
            href, a, b, Sa, Sb = oracle.swiglu_ffn_in(W, W3, x, g, it.eps)
            bound = oracle.swiglu_bound(a, b, Sa, Sb)
            worst = max(worst, check_swiglu(y, href, bound, dt, f"{what} {it.name}"))
    return worst


def test_fused110m_sweep():
    """The 110M decode token as 73 fused items (RMSNorm -> wq/wk/wv, wo,
    RMSNorm -> SwiGLU(w1, w3), w2, final RMSNorm -> classifier) in one
    launch; every output against the oracle, in every fused launch shape."""
    wl = synth.FUSED_WORKLOADS["fused110m"]
    gemvs = sdev.load_fused(wl, DEV)
    items = [d.item() for d in gemvs]
    for t in TUNINGS + [dict(grid=300)]:
        for d in gemvs:
            d.y.fill_(float("nan"))
        plan = tvl.tvl_sweep_plan_create(items, t)
        plan.run()
        torch.cuda.synchronize()
        worst = _check_fused_gemvs(gemvs, f"fused110m {t}")
        plan.destroy()
    log(f"fused110m: max normalised error {worst:.3e}")


def test_fused70b8_every_output():
    """8 layers of the 70B-shaped stack as 48 fused items (fp16 weights, 13.7
    GB) in the launch the bench times: every output of every item against
    the oracle (each matrix generated once; row blocks of the oracle on every
    host thread)."""
    import host_oracle
    wl = synth.FUSED_WORKLOADS["fused70b8"]
    log(f"fused70b8: uploading {wl.weight_bytes() / 1e9:.1f} GB")
    vecs, cases = {}, []

    def vec(v):
        if v is not None and v not in vecs:
            vecs[v] = torch.from_numpy(v.values()).to(DEV)
        return None if v is None else vecs[v]

    for i, it in enumerate(wl.items):
        W = it.W.weights()
        W3 = it.W3.weights() if it.W3 is not None else None
        d = sdev.DevFused(it, tvl.upload_matrix(W, sdev.dtype_code(it.W), DEV),
                          tvl.upload_matrix(W3, sdev.dtype_code(it.W3), DEV) if W3 is not None
                          else None, vec(it.x), vec(it.g),
                          torch.full((it.M,), float("nan"), device=DEV))
        x = it.x.values()
        g = it.g.values() if it.g is not None else None
        if W3 is None:
            xd = oracle.rmsnorm(x, g, it.eps) if g is not None else x.astype(np.float64)
            yref, S = host_oracle.gemv_dx(W, xd)
            cases.append((d, yref, S, None))
        else:
            href, a, b, Sa, Sb = host_oracle.swiglu_ffn_in(W, W3, x, g, it.eps)
            cases.append((d, href, None, oracle.swiglu_bound(a, b, Sa, Sb)))
        del W, W3
        if i % 8 == 0 or i == len(wl.items) - 1:
            log(f"  fused70b8: {i + 1}/{len(wl.items)} items uploaded and referenced")
    plan = tvl.tvl_sweep_plan_create([d.item() for d, *_ in cases])
    plan.run()
    torch.cuda.synchronize()
    worst = 0.0
    for d, yref, S, bound in cases:
        dt = sdev.dtype_code(d.spec.W)
        y = d.y.cpu().numpy()
        what = f"fused70b8 {d.spec.name}"
        worst = max(worst, check_gemv(y, yref, S, dt, what) if bound is None
                    else check_swiglu(y, yref, bound, dt, what))
    log(f"fused70b8: every output, max normalised error {worst:.3e}")
    plan.destroy()
    del cases
    torch.cuda.empty_cache()


def test_mixed_plain_and_fused_plan():
    """Plain and fused items, fp32 and fp16, in one plan."""
    rng = np.random.default_rng(17)
    specs = [(257, 255, 0, "gemv", False), (65, 1000, 1, "gemv", True),
             (1000, 65, 0, "swiglu", True), (9, 28672, 1, "swiglu", False),
             (130, 4095, 1, "gemv", False), (2048, 768, 0, "swiglu", True)]
    keep, items, refs = [], [], []
    for M, K, dt, op, norm in specs:
        W1 = rand_w(rng, M, K, dt)
        W3 = rand_w(rng, M, K, dt) if op == "swiglu" else None
        x = rng.standard_normal(K).astype(np.float32)
        g = rng.uniform(0.5, 1.5, K).astype(np.float32) if norm else None
        b1, ldw = dev_matrix(W1, dt)
        b3 = dev_matrix(W3, dt)[0] if W3 is not None else None
        xd = torch.from_numpy(x).to(DEV)
        gd = torch.from_numpy(g).to(DEV) if norm else None
        y = torch.full((M,), float("nan"), device=DEV)
        keep += [b1, b3, xd, gd, y]
        items.append(dict(W=b1, ldw=ldw, x=xd, y=y, M=M, K=K, dtype=dt,
                          op=tvl.TVL_OP_SWIGLU if W3 is not None else tvl.TVL_OP_GEMV,
                          W3=b3, g=gd, eps=1e-5 if norm else 0.0))
        refs.append((W1, W3, x, g, dt, y))
    for t in TUNINGS:
        plan = tvl.tvl_sweep_plan_create(items, t)
        plan.run()
        torch.cuda.synchronize()
        for W1, W3, x, g, dt, y in refs:
            if W3 is None:
                yref, S = (oracle.rmsnorm_gemv(W1, x, g, 1e-5) if g is not None
                           else oracle.gemv_dx(W1, x.astype(np.float64)))
                check_gemv(y.cpu().numpy(), yref, S, dt, f"mixed gemv {t}")
            else:
                href, a, b, Sa, Sb = oracle.swiglu_ffn_in(W1, W3, x, g, 1e-5)
                check_swiglu(y.cpu().numpy(), href, oracle.swiglu_bound(a, b, Sa, Sb), dt,
                             f"mixed swiglu {t}")
        plan.destroy()
