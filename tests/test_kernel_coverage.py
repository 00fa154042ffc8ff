"""Every compiled kernel instantiation is exercised by a GPU test (CPU check).

The kernel names come from the device assembly of this repository's own
build; the names the cases dispatch to come from the library's host-only
dispatch query, which shares its decisions with the launchers.
"""

import os
import re

import pytest

import paper_2510_08726_amd as pa
from paper_2510_08726_amd import build as libbuild
from kernel_cases import DECODE_VARIANT_CASES, NORM_CASES, PREFILL_VARIANT_CASES

_ARG = re.compile(r"Li(-?\d+)E|DF16_|DF16b|Lb([01])E|^f")


def _canonical(mangled):
    m = re.match(r"_ZN4attn12_GLOBAL__N_1\d+(\w+?)ENS_\d+\w+ParamsE$", mangled)   # not a template
    if m:
        return m.group(1)
    m = re.match(r"_ZN4attn12_GLOBAL__N_1\d+(\w+?)I(.*)EEvNS_\d+\w+ParamsE$", mangled)
    assert m, mangled
    args = []
    for t in _ARG.finditer(m.group(2)):
        if t.group(1) is not None:
            args.append(t.group(1))
        elif t.group(2) is not None:
            args.append(t.group(2))
        elif t.group(0) == "f":
            args.append("f32")
        else:
            args.append("f16" if t.group(0) == "DF16_" else "bf16")
    return f"{m.group(1)}<{','.join(args)}>"


@pytest.fixture(scope="module")
def compiled():
    files = libbuild.device_asm_files()
    if not all(os.path.exists(f) for f in files) or not os.path.exists(pa.library_path()):
        import __graft_entry__
        __graft_entry__.build()
    names = set()
    for f in files:
        names.update(re.findall(r"^\s*\.amdhsa_kernel\s+(\S+)", open(f).read(), flags=re.M))
    # every kernel but the peak probes of peaks.h (measured by the bench)
    return {_canonical(n) for n in names if "hbm_read_kernel" not in n and "mfma_loop_kernel" not in n}


def test_canonical_names():
    assert _canonical("_ZN4attn12_GLOBAL__N_114prefill_kernelILi128EDF16_Lb1ELb0ELb1ELb0EEEvNS_13PrefillParamsE") \
        == "prefill_kernel<128,f16,1,0,1,0>"
    assert _canonical("_ZN4attn12_GLOBAL__N_119decode_split_kernelILi64EDF16bLi8ELb1ELb0EEEvNS_12DecodeParamsE") \
        == "decode_split_kernel<64,bf16,8,1,0>"


def test_every_compiled_kernel_is_exercised(compiled):
    import torch
    dt = {"f16": torch.float16, "bf16": torch.bfloat16}
    used = set()
    for B, Hq, Hkv, Lq, Lk, D, d, causal, alibi, cap, win in PREFILL_VARIANT_CASES:
        used.update(pa.attn_fwd_kernels(D, dt[d], causal, alibi, cap or 0.0, win or 0))
    for B, Hq, Hkv, Lk, D, d, alibi, cap, S in DECODE_VARIANT_CASES:
        used.update(pa.attn_decode_kernels(Hq, Hkv, D, dt[d], alibi, cap or 0.0))
    ndt = {"f16": torch.float16, "bf16": torch.bfloat16, "f32": torch.float32}
    for N, M, d, C in NORM_CASES:   # tests/test_gpu_norms.py runs both operations on each
        for op in ("l2", "rms"):
            used.update(pa.norm_kernels(op, M, ndt[d], C or pa.norm_chunks(op, N, M, ndt[d])))
    assert len(compiled) == 32 + 64 + 16 + 4 + 16, sorted(compiled)
    assert used == compiled, (sorted(compiled - used), sorted(used - compiled))


def test_dispatch_query_rejects_what_the_entry_points_reject():
    import torch
    with pytest.raises(pa.AttnError):
        pa.attn_fwd_kernels(96, torch.float16, 1, 0)
    with pytest.raises(pa.AttnError):
        pa.attn_fwd_kernels(128, torch.float16, 0, 0, 0.0, 16)      # window without the causal mask
    with pytest.raises(pa.AttnError):
        pa.attn_fwd_kernels(128, torch.float16, 1, 1, 3.0, 0)       # SoftCap with ALiBi
    with pytest.raises(pa.AttnError):
        pa.attn_decode_kernels(6, 4, 128, torch.float16, 0)         # Hq % Hkv != 0
