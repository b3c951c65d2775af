"""HIP graph capture of library calls (MI355X).

A graph captured from tvl_gemv_batch_sweep (cached plan) and a K-split
tvl_gemv keeps using the library's plan tables and K-split workspace.  Those
must stay valid when the plan cache is later emptied (more item lists than
it holds) and when the stream's workspace is replaced by a larger one: the
library keeps such buffers until tvl_release_workspaces.  Each replay, with
eager work and synchronisations between replays, must equal the eager
result bit for bit, and the eager result must match the oracle.  Building a
plan while the stream is capturing is refused and enqueues nothing.
"""
from __future__ import annotations

import ctypes
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

DEV = "cuda"
ARG = -8


def matrix(rng, M, K):
    W = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    return W, torch.from_numpy(W).to(DEV)


def test_capture_survives_eviction_and_workspace_growth():
    rng = np.random.default_rng(2024)
    s = torch.cuda.Stream()
    sid = int(s.cuda_stream)
    # a two-item batch sweep and a K split (64 rows of 48 KB: split by default)
    specs = [(300, 704), (129, 2048)]  # K * 4 bytes a multiple of 128: ldw = K
    hosts, items, ys, xs = [], [], [], []
    for M, K in specs:
        W, Wd = matrix(rng, M, K)
        x = rng.standard_normal(K).astype(np.float32)
        xd = torch.from_numpy(x).to(DEV)
        y = torch.full((M,), float("nan"), device=DEV)
        hosts.append((W, x, Wd, xd))
        ys.append(y)
        items.append((Wd, K, xd, y, M, K, 0))
    Mk, Kk = 64, 12288
    Wk, Wkd = matrix(rng, Mk, Kk)
    xk = rng.standard_normal(Kk).astype(np.float32)
    xkd = torch.from_numpy(xk).to(DEV)
    yk = torch.full((Mk,), float("nan"), device=DEV)
    outs = ys + [yk]

    def calls():
        tvl.tvl_gemv_batch_sweep(items, sid)
        tvl.tvl_gemv(Wkd, Kk, 0, xkd, yk, Mk, Kk, stream=sid)

    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        calls()  # eager: builds the plan and the stream's workspace
    s.synchronize()
    eager = [y.clone() for y in outs]
    for (W, x, _, _), y in zip(hosts + [(Wk, xk, None, None)], eager):
        yref, S = oracle.gemv_f32(W, x)
        r = oracle.check(y.cpu().numpy(), yref, S, 1e-5)
        assert r["bad"] == 0, r

    # an item list without a plan cannot be captured: refused, nothing enqueued
    other, n_other = tvl.make_items([(hosts[0][2], 704, hosts[0][3], ys[0], 300, 699, 0)])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        calls()
        st = tvl.lib.tvl_gemv_batch_sweep(ctypes.cast(other, ctypes.c_void_p), n_other, sid)
    assert st == ARG
    assert b"captured" in tvl.lib.tvl_last_error()

    # empty the plan cache (more lists than it holds) and grow the stream's
    # K-split workspace (8192 rows x 16 slices: twice its first size)
    big_y = torch.empty(8192, device=DEV)
    with torch.cuda.stream(s):
        for i in range(70):
            tvl.tvl_gemv_batch_sweep([(hosts[0][2], 704, hosts[0][3], big_y, 300 - i, 704, 0)],
                                     sid)
        W2, W2d = matrix(rng, 8192, 1024)
        x2d = torch.from_numpy(rng.standard_normal(1024).astype(np.float32)).to(DEV)
        tvl.tvl_gemv_ex(W2d, 1024, 0, x2d, big_y, 8192, 1024, dict(ksplit=16), sid)
    s.synchronize()
    yref, S = oracle.gemv_f32(W2, x2d.cpu().numpy())
    assert oracle.check(big_y.cpu().numpy(), yref, S, 1e-5)["bad"] == 0

    for rep in range(3):
        for y in outs:
            y.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for y, e in zip(outs, eager):
            assert torch.equal(y, e), rep
        with torch.cuda.stream(s):  # eager work between replays
            calls()
        s.synchronize()
        for y, e in zip(outs, eager):
            assert torch.equal(y, e), rep
    del g
    torch.cuda.synchronize()
    tvl.tvl_release_workspaces()


def test_capture_quantised_x_in_lds():
    """A plan of 4-bit and 8-bit items with x staged in LDS (dynamic LDS per
    launch) captured into a HIP graph: every replay, with eager work and
    synchronisations between replays, equals the eager result bit for bit."""
    rng = np.random.default_rng(31)
    s = torch.cuda.Stream()
    sid = int(s.cuda_stream)
    items, outs, keep = [], [], []
    for M, K, dt in ((300, 4096, tvl.TVL_Q4), (129, 11008, tvl.TVL_Q4), (77, 768, tvl.TVL_Q8)):
        w = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
        bits = 4 if dt == tvl.TVL_Q4 else 8
        ldw = tvl.tvl_row_stride(K, dt)
        Wq = synth.quantize_rows(w, bits, ldw=ldw)
        Wd = tvl.upload_quant(Wq, M, K, dt, ldw, DEV)
        x = rng.standard_normal(K).astype(np.float32)
        xd = torch.from_numpy(x).to(DEV)
        y = torch.full((M,), float("nan"), device=DEV)
        keep.append((Wd, xd, Wq, x, M, K, bits, ldw))
        items.append((Wd.ptr, Wd.ldw, xd, y, M, K, dt))
        outs.append(y)
    plan = tvl.tvl_sweep_plan_create(items, dict(flags=1))
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        plan.run(sid)
    s.synchronize()
    eager = [y.clone() for y in outs]
    for (_, _, Wq, x, M, K, bits, ldw), y in zip(keep, eager):
        yref, S = oracle.gemv_q(Wq, bits, ldw, M, K, x)
        assert oracle.check(y.cpu().numpy(), yref, S, 1e-5)["bad"] == 0, (M, K, bits)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        plan.run(sid)
    for rep in range(3):
        for y in outs:
            y.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for y, e in zip(outs, eager):
            assert torch.equal(y, e), rep
        with torch.cuda.stream(s):  # eager work between replays
            plan.run(sid)
        s.synchronize()
        for y, e in zip(outs, eager):
            assert torch.equal(y, e), rep
    del g
    torch.cuda.synchronize()
    plan.destroy()


def f16_bits(w):
    return torch.from_numpy(synth.f32_to_f16_bits(w).view(np.int16)).to(DEV)


def plan_kind(kind, rng):
    """(item dicts, outputs, kept buffers, tuning) of one plan kind."""
    items, outs, keep = [], [], []

    def out(n):
        y = torch.full((n,), float("nan"), device=DEV)
        outs.append(y)
        return y

    def vec(n):
        v = torch.from_numpy(rng.standard_normal(n).astype(np.float32)).to(DEV)
        keep.append(v)
        return v

    def mat(M, K, dt):
        w = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
        d = torch.from_numpy(w).to(DEV) if dt == 0 else f16_bits(w)
        keep.append(d)
        return d

    tuning = None
    if kind in ("plain", "plain-lds"):
        for M, K, dt in ((768, 768, 0), (2048, 768, 0), (300, 1024, 1), (129, 4096, 0)):
            items.append(dict(W=mat(M, K, dt), ldw=K, x=vec(K), y=out(M), M=M, K=K, dtype=dt))
        tuning = dict(flags=1) if kind == "plain-lds" else None
    elif kind == "fused":
        K = 768
        g = vec(K)
        items.append(dict(W=mat(768, K, 0), ldw=K, x=vec(K), y=out(768), M=768, K=K, dtype=0,
                          g=g, eps=1e-5))
        items.append(dict(W=mat(2048, K, 0), ldw=K, x=vec(K), y=out(2048), M=2048, K=K, dtype=0,
                          op=tvl.TVL_OP_SWIGLU, W3=mat(2048, K, 0), g=g, eps=1e-5))
        items.append(dict(W=mat(512, 2048, 1), ldw=2048, x=vec(2048), y=out(512), M=512,
                          K=2048, dtype=1))
    else:  # several vectors: fp32 on the shared-x matrix-core form, fp16 with
        # split x, mixed weights, and the vector ALUs
        nb, dts = {"multi-f32-16": (16, (0, 0)), "multi-f16-8": (8, (1, 1)),
                   "multi-mixed-8": (8, (0, 1)), "multi-4": (4, (0, 1))}[kind]
        for (M, K), dt in zip(((768, 768), (2048, 2048)), dts):
            ldx, ldy = K + 4, M + 8
            X = vec(nb * ldx)
            Y = torch.full((nb * ldy,), float("nan"), device=DEV)
            outs.append(Y)
            items.append(dict(W=mat(M, K, dt), ldw=K, x=X, y=Y, M=M, K=K, dtype=dt, nrhs=nb,
                              ldx=ldx, ldy=ldy))
    return items, outs, keep, tuning


@pytest.mark.parametrize("kind", ["plain", "plain-lds", "fused", "multi-f32-16", "multi-f16-8",
                                  "multi-mixed-8", "multi-4"])
def test_capture_every_plan_kind(kind):
    """A plan of each kind (plain fp32/fp16 in both x modes, RMSNorm and
    SwiGLU items, several vectors through each default form: shared x with
    weights streamed into LDS, split x on the fp16 matrix cores, mixed
    weights, the vector ALUs) run twice inside one captured HIP graph: five
    replays, with eager runs and synchronisations between them, each equal
    to the eager result bit for bit."""
    rng = np.random.default_rng(zlib.crc32(kind.encode()))
    items, outs, keep, tuning = plan_kind(kind, rng)
    s = torch.cuda.Stream()
    sid = int(s.cuda_stream)
    plan = tvl.tvl_sweep_plan_create(items, tuning)
    try:
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            plan.run(sid)
        s.synchronize()
        eager = [y.clone() for y in outs]
        assert all(bool(torch.isfinite(e).any()) for e in eager)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            plan.run(sid)
            plan.run(sid)
        for rep in range(5):
            for y in outs:
                y.fill_(float("nan"))
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            for y, e in zip(outs, eager):  # bit patterns: unwritten gaps stay NaN
                assert torch.equal(y.view(torch.int32), e.view(torch.int32)), (kind, rep)
            with torch.cuda.stream(s):  # eager work between replays
                plan.run(sid)
            s.synchronize()
            for y, e in zip(outs, eager):
                assert torch.equal(y.view(torch.int32), e.view(torch.int32)), (kind, rep)
        del g
        torch.cuda.synchronize()
    finally:
        plan.destroy()
