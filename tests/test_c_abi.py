"""The C ABI from plain C (tests/c_driver/tvl_c_driver.c, built by
``__graft_entry__.build()``): no Python and no torch between the caller and
``libtvl.so``.

On a host without a GPU the driver must load both libraries and report that
there is no device (exit status 77); on a GPU it packs three matrices, runs a
plan, a cached batch and single GEMVs, then two several-vector items (8 fp32
and 16 fp16 beam vectors), and checks every output against the C oracle.
"""
from __future__ import annotations

import os
import subprocess

import pytest

BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_driver", "tvl_c_driver")


def run_driver():
    assert os.path.exists(BIN), "tests/c_driver/tvl_c_driver missing: run __graft_entry__.build()"
    return subprocess.run([BIN], capture_output=True, text=True, timeout=120)


def _have_gpu() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:  # torch missing: treat as no GPU
        return False


@pytest.mark.skipif(_have_gpu(), reason="a GPU is present (the gpu test runs the driver)")
def test_c_driver_links_and_reports_no_gpu():
    if not os.path.exists(BIN):  # like the other ABI tests before build()
        pytest.skip("tests/c_driver/tvl_c_driver not built (run __graft_entry__.build())")
    r = run_driver()
    assert r.returncode == 77, (r.returncode, r.stdout, r.stderr)
    assert "no GPU" in r.stdout


@pytest.mark.gpu
def test_c_driver_on_gpu():
    r = run_driver()
    print(r.stdout)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert "all checks passed" in r.stdout
    # 3 items x (plan + 2 batches + gemv), and 2 several-vector items
    assert r.stdout.count("max normalised error") == 14
