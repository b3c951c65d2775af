"""Put a synthetic workload on the GPU (torch allocations, TVL row layout).

Input plumbing shared by the GPU tests and the benchmark: draws each matrix
with the generator of this package, uploads it, and gives every GEMV its own
x and y buffers.  No GEMV arithmetic happens here.
"""
from __future__ import annotations

import sys
from dataclasses import dataclass

import numpy as np

from . import MatSpec, Workload


@dataclass
class DevGemv:
    spec: MatSpec
    W: object  # TvlMatrix
    x: object  # torch fp32 [K]
    y: object  # torch fp32 [M]

    def item(self):
        from paper_2601_03324_amd import tvl
        return (self.W.ptr, self.W.ldw, self.x, self.y, self.spec.M, self.spec.K, self.W.dtype)


def dtype_code(spec: MatSpec) -> int:
    return {"f32": 0, "f16": 1, "q8": 2, "q4": 3}[spec.dtype]


def upload(spec: MatSpec, host, device="cuda"):
    """A TvlMatrix of ``spec``'s weights (``host`` = spec.weights())."""
    from paper_2601_03324_amd import tvl
    if spec.quantised:
        return tvl.upload_quant(host, spec.M, spec.K, dtype_code(spec), device=device)
    return tvl.upload_matrix(host, dtype_code(spec), device)


def load(wl: Workload, device="cuda", rep: int = 0, progress: bool = False,
         share_from: list | None = None) -> list:
    """Upload every matrix of ``wl``.  ``share_from`` reuses the weight buffers
    of an earlier load (fresh x and y only)."""
    import torch
    from paper_2601_03324_amd import tvl
    out = []
    for i, m in enumerate(wl.mats):
        if share_from is not None:
            Wd = share_from[i].W
        else:
            Wd = upload(m, m.weights(), device)
        x = torch.from_numpy(m.x(rep)).to(device)
        y = torch.full((m.M,), float("nan"), dtype=torch.float32, device=device)
        out.append(DevGemv(m, Wd, x, y))
        if progress and (i % 16 == 0 or i == len(wl.mats) - 1):
            print(f"  loaded {wl.name} {i + 1}/{len(wl.mats)}", flush=True, file=sys.stderr)
    return out


def clone_weights(gemvs: list, device="cuda") -> list:
    """A second copy of every weight matrix (same values, new addresses) with
    its own x and y: lets a benchmark alternate between copies so that the
    256 MB last-level cache cannot serve a sweep from the previous one."""
    import torch
    from paper_2601_03324_amd import tvl
    out = []
    for g in gemvs:
        buf = g.W.buf.clone()
        Wd = tvl.TvlMatrix(buf, g.W.M, g.W.K, g.W.ldw, g.W.dtype)
        out.append(DevGemv(g.spec, Wd, g.x.clone(), torch.empty_like(g.y)))
    return out


def sample_rows(M: int, n: int, seed: int) -> np.ndarray:
    """First, last and n-2 seeded random rows of an M-row matrix (sorted, unique)."""
    rng = np.random.default_rng(seed)
    rows = {0, M - 1}
    rows.update(int(r) for r in rng.integers(0, M, max(n - 2, 0)))
    return np.array(sorted(rows), dtype=np.int64)


@dataclass
class DevFused:
    spec: object  # FusedSpec
    W: object     # TvlMatrix
    W3: object    # TvlMatrix or None
    x: object     # torch fp32 [K]
    g: object     # torch fp32 [K] or None
    y: object     # torch fp32 [M]

    def item(self) -> dict:
        from paper_2601_03324_amd import tvl
        return dict(W=self.W.ptr, ldw=self.W.ldw, x=self.x, y=self.y, M=self.spec.M,
                    K=self.spec.K, dtype=self.W.dtype,
                    op=tvl.TVL_OP_SWIGLU if self.W3 is not None else tvl.TVL_OP_GEMV,
                    W3=self.W3.ptr if self.W3 is not None else None, g=self.g,
                    eps=self.spec.eps if self.g is not None else 0.0)


def load_fused(wl, device="cuda", progress: bool = False) -> list:
    """Upload every item of a fused workload; x and g vectors shared by a
    group (e.g. wq, wk, wv) are uploaded once and shared."""
    import torch
    from paper_2601_03324_amd import tvl
    vecs = {}

    def vec(v):
        if v is None:
            return None
        if v not in vecs:
            vecs[v] = torch.from_numpy(v.values()).to(device)
        return vecs[v]

    out = []
    for i, it in enumerate(wl.items):
        Wd = tvl.upload_matrix(it.W.weights(), dtype_code(it.W), device)
        W3 = tvl.upload_matrix(it.W3.weights(), dtype_code(it.W3), device) if it.W3 else None
        y = torch.full((it.M,), float("nan"), dtype=torch.float32, device=device)
        out.append(DevFused(it, Wd, W3, vec(it.x), vec(it.g), y))
        if progress and (i % 8 == 0 or i == len(wl.items) - 1):
            print(f"  loaded {wl.name} {i + 1}/{len(wl.items)}", flush=True, file=sys.stderr)
    return out


@dataclass
class DevMulti:
    spec: MatSpec
    W: object   # TvlMatrix
    X: object   # torch fp32 [B, ldx]
    Y: object   # torch fp32 [B, ldy]
    B: int

    def item(self) -> dict:
        return dict(W=self.W.ptr, ldw=self.W.ldw, x=self.X, y=self.Y, M=self.spec.M,
                    K=self.spec.K, dtype=self.W.dtype, nrhs=self.B, ldx=self.X.shape[1],
                    ldy=self.Y.shape[1])


def load_multi(wl: Workload, B: int, device="cuda", share_from: list | None = None) -> list:
    """Every matrix of ``wl`` with B x vectors (reps 0..B-1 of its x stream),
    stored as B rows padded to a multiple of 4 floats; y as B rows of M."""
    import torch
    from paper_2601_03324_amd import tvl
    out = []
    for i, m in enumerate(wl.mats):
        Wd = share_from[i].W if share_from is not None else tvl.upload_matrix(
            m.weights(), dtype_code(m), device)
        ldx = (m.K + 3) // 4 * 4
        X = torch.zeros((B, ldx), dtype=torch.float32)
        for b in range(B):
            X[b, :m.K] = torch.from_numpy(m.x(b))
        Y = torch.full((B, m.M), float("nan"), dtype=torch.float32, device=device)
        out.append(DevMulti(m, Wd, X.to(device), Y, B))
    return out
