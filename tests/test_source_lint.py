"""Source checks of the HIP kernels (CPU only).

__builtin_bit_cast of an ext-vector element (``v[e]``, ``xb[q][e]``) is
lowered by this compiler to the bits of element 0 of the vector, whatever
the index: the split-x range test once read only every fourth column that
way.  A value's bits are taken with __float_as_uint / __uint_as_float on the
element's value instead.  This test rejects the pattern in every kernel
source: a bit_cast whose operand ends in a subscript of a vector-typed
name (f4, u4, h8, ...).
"""
from __future__ import annotations

import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2601_03324_amd", "csrc")
VECTOR_TYPES = ("f4", "u4", "h4", "h8", "f8", "f2", "u2", "V")


def vector_names(src: str) -> set:
    """Names declared with a vector type (scalars, arrays and references)."""
    names = set()
    for t in VECTOR_TYPES:
        for m in re.finditer(rf"\b(?:const\s+)?{t}\s+(?:\(&)?\s*(\w+)", src):
            names.add(m.group(1))
    return names


def test_no_bit_cast_of_vector_elements():
    bad = []
    for f in sorted(os.listdir(CSRC)):
        if not f.endswith((".hip", ".h", ".cpp")):
            continue
        src = open(os.path.join(CSRC, f)).read()
        vecs = vector_names(src)
        for m in re.finditer(r"__builtin_bit_cast\(\s*[\w:]+\s*,\s*([\w.]+)((?:\[[^\]]*\])+)\s*\)", src):
            name, subs = m.group(1), m.group(2)
            # arrays of vectors: one subscript per array dimension is a whole
            # vector; the declaration tells how many dimensions the array has
            decl = re.search(rf"\b(?:{'|'.join(VECTOR_TYPES)})\s+(?:\(&)?\s*{re.escape(name)}\)?((?:\[[^\]]*\])*)", src)
            dims = len(re.findall(r"\[", decl.group(1))) if decl else 0
            if name in vecs and len(re.findall(r"\[", subs)) > dims:
                line = src[:m.start()].count("\n") + 1
                bad.append(f"{f}:{line}: {m.group(0)}")
    assert not bad, "bit_cast of a vector element (reads element 0):\n" + "\n".join(bad)


def test_lint_catches_the_pattern():
    src = "f4 xb[4];\nuint32_t b = __builtin_bit_cast(uint32_t, xb[q][e]);\n"
    vecs = vector_names(src)
    m = re.search(r"__builtin_bit_cast\(\s*[\w:]+\s*,\s*([\w.]+)((?:\[[^\]]*\])+)\s*\)", src)
    decl = re.search(r"\bf4\s+xb((?:\[[^\]]*\])*)", src)
    assert m and "xb" in vecs and len(re.findall(r"\[", m.group(2))) > len(re.findall(r"\[", decl.group(1)))
