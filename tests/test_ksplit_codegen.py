"""The K split's publication of partial sums, as compiled for gfx950 (CPU only).

k_gemv_ksplit publishes each slice's partials without a release fence (one
would write back the whole L2 per workgroup); it relies on the partials being
agent-scope atomic stores (written through, sc1), on the wait for their
acknowledgement before the barrier and the counter's atomic add, and on an
acquire fence (buffer_inv sc1) in the last workgroup before its coherent
(sc1) loads of the partials.  This compiles the kernel source for gfx950 and
checks each of those instructions in every instantiation, so a change in code
generation that drops one fails here rather than silently on the GPU.
"""
from __future__ import annotations

import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2601_03324_amd", "csrc")


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    from paper_2601_03324_amd import build as b
    try:
        cc = b.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("ksplit") / "tvl_gemv.s"
    subprocess.check_call([cc, *[f for f in b.FLAGS if f not in ("-fPIC",)], "-I", b.INCLUDE,
                           "-I", CSRC, "--cuda-device-only", "-S", "-o", str(out),
                           os.path.join(CSRC, "tvl_gemv.hip")],
                          stderr=subprocess.DEVNULL)
    return out.read_text()


def bodies(asm):
    names = re.findall(r"^(_ZN3tvl12_GLOBAL__N_113k_gemv_ksplit\w+):", asm, re.M)
    assert names, "no k_gemv_ksplit instantiation found"
    for n in names:
        i = asm.index(n + ":")
        j = asm.index(".Lfunc_end", i)
        yield n, [ln.strip() for ln in asm[i:j].split("\n")
                  if ln.strip() and not ln.strip().startswith((";", "."))]


def test_ksplit_publication_codegen(asm):
    n = 0
    for name, body in bodies(asm):
        n += 1
        at = [k for k, ln in enumerate(body) if ln.startswith("global_atomic_add")]
        assert len(at) == 1, name
        a = at[0]
        stores = [k for k in range(a) if body[k].startswith("global_store")]
        assert stores, name
        # every store before the counter update is a partial: written through
        assert all(re.search(r"\bsc1\b", body[k]) for k in stores), name
        between = body[stores[-1] + 1:a]
        assert "s_waitcnt vmcnt(0)" in " ".join(between), name  # acknowledged ...
        waves = int(re.search(r"ksplitI(?:f|DF16_)Li\d+ELi(\d+)E", name).group(1))
        if waves > 1:  # ... by every wavefront (one wavefront needs no barrier)
            assert any(ln.startswith("s_barrier") for ln in between), name
        after = body[a + 1:]
        inv = [k for k, ln in enumerate(after) if re.match(r"buffer_inv\b.*\bsc1\b", ln)]
        loads = [k for k, ln in enumerate(after) if ln.startswith("global_load")]
        assert inv and loads, name
        assert inv[0] < loads[0], name  # acquire before reading the partials
        assert all(re.search(r"\bsc1\b", after[k]) for k in loads), name
    assert n >= 40  # both weight dtypes x every instantiated shape and x mode
