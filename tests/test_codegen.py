"""Guards on the code this repository builds (CPU only, no GPU).

hipcc (ROCm 7.2, clang) miscompiles __builtin_bit_cast of an element of an
ext_vector_type value: bit_cast(float, w[i]) and bit_cast(float, w.y) read
element 0 whatever the index, so a 16-byte vector load shrinks to one dword
used four times.  The kernels copy such an element to a scalar first; these
tests keep the pattern out of the sources and check the effect in the
generated assembly of the row reductions, where it first appeared.
"""

import os
import re

import pytest

from paper_2510_08726_amd import build as libbuild

CSRC = libbuild.CSRC


def test_no_bit_cast_of_a_vector_element_in_the_sources():
    pat = re.compile(r"__builtin_bit_cast\(\s*[\w:]+\s*,\s*\w+\s*(\[[^\]]*\]|\.[xyzw])\s*\)")
    bad = []
    for f in sorted(os.listdir(CSRC)):
        if f.endswith((".hip", ".h", ".cpp")):
            for n, line in enumerate(open(os.path.join(CSRC, f)), 1):
                if pat.search(line):
                    bad.append(f"{f}:{n}: {line.strip()}")
    assert not bad, "\n".join(bad)


def test_pattern_finder_catches_the_miscompiled_forms():
    pat = re.compile(r"__builtin_bit_cast\(\s*[\w:]+\s*,\s*\w+\s*(\[[^\]]*\]|\.[xyzw])\s*\)")
    assert pat.search("f[i] = __builtin_bit_cast(float, w[i]);")
    assert pat.search("x = __builtin_bit_cast(f16x2, v.y);")
    assert not pat.search("x = __builtin_bit_cast(float, u);")
    assert not pat.search("x = __builtin_bit_cast(vec8, make_uint4(a, b, c, d));")


def _kernels(asm):
    out, name = {}, None
    for line in open(asm):
        m = re.match(r"^(_ZN4attn\S*):", line)
        if m:
            name = m.group(1)
            out[name] = []
        elif name and line.startswith("\t"):
            out[name].append(line.split()[0] if line.split() else "")
        if line.startswith(".Lfunc_end"):
            name = None
    return out


# Kernels that read X: the 16-byte loads each issues at least (its unrolled
# loads plus a tail load, or the 16 vectors a lane holds), and its 4-byte
# loads (rms_apply_kernel reads the two fp32 partials of a chunk; X is never
# read 4 bytes at a time).
_X_READERS = {"norm_split_kernel": (9, 0), "rms_apply_kernel": (5, 2), "l2_row_kernel": (9, 0),
              "rms_row_kernel": (16, 0)}


def test_norm_kernels_load_whole_vectors():
    asm = os.path.join(libbuild.unit_dir("norms"), f"norms-hip-amdgcn-amd-amdhsa-{libbuild.ARCH}.s")
    if not os.path.exists(asm):
        import __graft_entry__
        __graft_entry__.build()
    kernels = _kernels(asm)
    for name, (least, dwords) in _X_READERS.items():
        ks = {k: v for k, v in kernels.items() if name in k}
        assert len(ks) == (6 if name == "norm_split_kernel" else 3), name
        for k, ops in ks.items():
            assert ops.count("global_load_dwordx4") >= least, k
            assert ops.count("global_load_dword") == dwords, k
