"""The C ABI on the host: the library loads, exports every declared symbol and
rejects bad arguments before any HIP call (no GPU needed, no compute call).

Pointers passed here are never dereferenced: every call below fails host-side
validation, which runs before anything is enqueued.
"""

import ctypes
import os
import re

import pytest

import paper_2510_08726_amd as pa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = ctypes.c_void_p(0x1000)   # non-NULL, never dereferenced on these paths
NULL = None


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(pa.library_path()):
        import __graft_entry__
        __graft_entry__.build()
    return pa.load_library()


def declared_functions():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names.update(re.findall(r"\b((?:attn|peaks|norm|rmsnorm)_[a-z0-9_]+)\s*\(", src))
    return sorted(names)


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert {"attn_fwd", "attn_fwd_mod", "attn_decode", "attn_decode_mod", "attn_decode_workspace_bytes",
            "attn_decode_num_splits", "attn_status_string", "attn_last_hip_error"} <= set(names)
    assert {"peaks_hbm_read", "peaks_mfma", "attn_decode_noalloc", "norm_l2", "rmsnorm_rowmax",
            "norm_chunks", "norm_workspace_bytes"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name


def test_norm_chunk_heuristic(lib):
    """Host logic of the row reductions' split (no device here: 256 compute
    units): one chunk per row when the rows fill >= 85 % of the compute
    units' rounds (for RMSNorm, rows of <= 256 KiB), else about 512
    workgroups with chunks of >= 4096 elements."""
    F16, BF16, F32 = 0, 1, 2
    for rms in (0, 1):
        assert lib.norm_chunks(rms, 256, 1 << 17, BF16) == 1     # 256 KiB rows, one round of 256
        assert lib.norm_chunks(rms, 512, 1 << 16, F32) == 1
        assert lib.norm_chunks(rms, 480, 4096, F16) == 1         # 480 of 512 slots: 94 %
        assert lib.norm_chunks(rms, 300, 1 << 17, BF16) == 2     # 300 of 512 slots: 512 / N
        assert lib.norm_chunks(rms, 255, 1 << 17, BF16) == 3     # fewer rows than compute units
        assert lib.norm_chunks(rms, 32, 1 << 10, F16) == 1       # chunks of >= 4096 elements
        assert lib.norm_chunks(rms, 32, 1 << 17, F16) == 16      # 512 workgroups
        assert lib.norm_chunks(rms, 1, 40000, BF16) == 10        # 512 / N, capped by M / 4096
        assert lib.norm_chunks(rms, 0, 8, F16) == 0 and lib.norm_chunks(rms, 8, 8, 7) == 0
    assert lib.norm_chunks(0, 256, 1 << 17, F32) == 1            # the L2 norm: any row length
    assert lib.norm_chunks(1, 256, 1 << 17, F32) == 2            # RMSNorm: a 512 KiB row


def test_norm_kernel_query():
    """The kernels each row-reduction path launches (host only)."""
    import torch
    f16, bf16, f32 = torch.float16, torch.bfloat16, torch.float32
    assert pa.norm_kernels("l2", 1 << 17, f32, 2) == ["norm_split_kernel<f32,0>", "l2_combine_kernel"]
    assert pa.norm_kernels("rms", 1 << 17, bf16, 2) == ["norm_split_kernel<bf16,1>", "rms_apply_kernel<bf16>"]
    assert pa.norm_kernels("l2", 1 << 20, f16, 1) == ["l2_row_kernel<f16>"]          # any row length
    assert pa.norm_kernels("rms", 1 << 17, bf16, 1) == ["rms_row_kernel<bf16>"]      # 256 KiB: held in registers
    assert pa.norm_kernels("rms", 1 << 16, f32, 1) == ["rms_row_kernel<f32>"]
    assert pa.norm_kernels("rms", (1 << 17) + 8, bf16, 1) == ["norm_split_kernel<bf16,1>", "rms_apply_kernel<bf16>"]
    assert pa.norm_kernels("rms", (1 << 16) + 4, f32, 1) == ["norm_split_kernel<f32,1>", "rms_apply_kernel<f32>"]
    for bad in ((1 << 17, bf16, 0), (1001, f16, 1), (0, f16, 1)):
        with pytest.raises(pa.AttnError):
            pa.norm_kernels("rms", *bad)


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4, -5):
        s = pa.attn_status_string(code)
        assert s.startswith("ATTN_")
    assert "unknown" in pa.attn_status_string(-99)
    assert pa.attn_last_hip_error() == 0


def fwd(lib, q=FAKE, k=FAKE, v=FAKE, o=FAKE, B=1, Hq=2, Hkv=2, Lq=8, Lk=8, D=64, causal=0,
        scale=0.125, slopes=NULL, cap=0.0, window=0, dtype=0):
    rc = lib.attn_fwd_mod(q, k, v, o, B, Hq, Hkv, Lq, Lk, D, causal, scale, slopes, cap, window, dtype, NULL)
    if cap == 0.0 and window == 0:
        # the boundary's own signature answers the same way
        assert lib.attn_fwd(q, k, v, o, B, Hq, Hkv, Lq, Lk, D, causal, scale, slopes, dtype, NULL) == rc
    return rc


@pytest.mark.parametrize("kw,code", [
    (dict(q=NULL), pa.ATTN_ERR_NULL), (dict(k=NULL), pa.ATTN_ERR_NULL),
    (dict(v=NULL), pa.ATTN_ERR_NULL), (dict(o=NULL), pa.ATTN_ERR_NULL),
    (dict(B=0), pa.ATTN_ERR_SHAPE), (dict(Hq=0), pa.ATTN_ERR_SHAPE),
    (dict(Hkv=0), pa.ATTN_ERR_SHAPE), (dict(Lq=0), pa.ATTN_ERR_SHAPE),
    (dict(Lk=-3), pa.ATTN_ERR_SHAPE), (dict(Hq=6, Hkv=4), pa.ATTN_ERR_SHAPE),
    (dict(scale=float("nan")), pa.ATTN_ERR_SHAPE), (dict(scale=float("inf")), pa.ATTN_ERR_SHAPE),
    (dict(D=96), pa.ATTN_ERR_UNSUPPORTED), (dict(D=256), pa.ATTN_ERR_UNSUPPORTED),
    (dict(causal=1, cap=-2.0), pa.ATTN_ERR_SHAPE), (dict(causal=1, cap=float("nan")), pa.ATTN_ERR_SHAPE),
    (dict(cap=30.0), pa.ATTN_ERR_UNSUPPORTED),                       # SoftCap without the causal mask
    (dict(causal=1, cap=30.0, slopes=FAKE), pa.ATTN_ERR_UNSUPPORTED),  # SoftCap with ALiBi
    (dict(causal=1, window=-1), pa.ATTN_ERR_SHAPE),
    (dict(window=16), pa.ATTN_ERR_UNSUPPORTED),                      # window without the causal mask
    (dict(causal=1, window=4, D=96), pa.ATTN_ERR_UNSUPPORTED),
    (dict(causal=1, window=4, q=NULL), pa.ATTN_ERR_NULL),
    (dict(dtype=2), pa.ATTN_ERR_UNSUPPORTED),
    (dict(B=1 << 20, Hq=1 << 10, Hkv=1 << 10, Lq=1 << 20, Lk=1 << 20), pa.ATTN_ERR_SHAPE),
    # one head's K or V must stay below 2^31 bytes (32-bit offsets in the prefill copies)
    (dict(Lk=1 << 23, D=128), pa.ATTN_ERR_SHAPE), (dict(Lk=1 << 24, D=64), pa.ATTN_ERR_SHAPE),
])
def test_fwd_rejects_bad_arguments(lib, kw, code):
    assert fwd(lib, **kw) == code


def dec(lib, q=FAKE, k=FAKE, v=FAKE, o=FAKE, B=2, Hq=8, Hkv=2, Lk=100, D=128, scale=0.1,
        slopes=NULL, cap=0.0, S=4, ws=FAKE, ws_bytes=1 << 30, dtype=0):
    rc = lib.attn_decode_mod(q, k, v, o, B, Hq, Hkv, Lk, D, scale, slopes, cap, S, ws, ws_bytes, dtype, NULL)
    if cap == 0.0:
        assert lib.attn_decode(q, k, v, o, B, Hq, Hkv, Lk, D, scale, slopes, S, ws, ws_bytes, dtype, NULL) == rc
    return rc


@pytest.mark.parametrize("kw,code", [
    (dict(q=NULL), pa.ATTN_ERR_NULL), (dict(ws=NULL), pa.ATTN_ERR_NULL),
    (dict(B=0), pa.ATTN_ERR_SHAPE), (dict(Hq=6, Hkv=4), pa.ATTN_ERR_SHAPE),
    (dict(Lk=0), pa.ATTN_ERR_SHAPE), (dict(S=-1), pa.ATTN_ERR_SHAPE),
    (dict(scale=float("nan")), pa.ATTN_ERR_SHAPE),
    (dict(cap=-1.0), pa.ATTN_ERR_SHAPE), (dict(cap=float("nan")), pa.ATTN_ERR_SHAPE),
    (dict(cap=float("inf")), pa.ATTN_ERR_SHAPE),
    (dict(D=32), pa.ATTN_ERR_UNSUPPORTED), (dict(dtype=7), pa.ATTN_ERR_UNSUPPORTED),
    (dict(ws_bytes=100), pa.ATTN_ERR_WORKSPACE),
    (dict(ws=ctypes.c_void_p(0x1004)), pa.ATTN_ERR_WORKSPACE),   # not 16-byte aligned
])
def test_decode_rejects_bad_arguments(lib, kw, code):
    assert dec(lib, **kw) == code


def test_workspace_size_formula(lib):
    for B, Hq, D, S in [(1, 1, 64, 1), (8, 32, 128, 32), (16, 32, 128, 64), (3, 5, 64, 7)]:
        n = B * Hq * S * (D + 2) * 4
        got = pa.attn_decode_workspace_bytes(B, Hq, D, S)
        assert got >= n and got - n < 256 and got % 256 == 0
    assert pa.attn_decode_workspace_bytes(0, 1, 64, 1) == 0
    assert pa.attn_decode_workspace_bytes(1, 1, 96, 1) == 0
    assert pa.attn_decode_workspace_bytes(1, 1, 64, 0) == 0


def test_workspace_check_uses_resolved_split_count(lib):
    """With num_splits = 0 the size check uses the heuristic's chunk count."""
    S = pa.attn_decode_num_splits(2, 8, 2, 100, 128)
    need = pa.attn_decode_workspace_bytes(2, 8, 128, S)
    assert dec(lib, S=0, ws_bytes=need - 256) == pa.ATTN_ERR_WORKSPACE


def test_num_splits_heuristic(lib):
    # One query head per KV head: about one workgroup per compute unit (256
    # compute units without a device), chunks of >= 256 keys.
    assert pa.attn_decode_num_splits(8, 32, 32, 8192, 128) == 1
    assert pa.attn_decode_num_splits(1, 32, 32, 32768, 128) == 8
    assert pa.attn_decode_num_splits(4, 32, 32, 16384, 64) == 2
    assert pa.attn_decode_num_splits(32, 32, 32, 2048, 128) == 1
    assert pa.attn_decode_num_splits(1, 1, 1, 1, 64) == 1
    assert pa.attn_decode_num_splits(1, 1, 1, 300, 64) == 2    # chunks of >= 256 keys
    assert pa.attn_decode_num_splits(0, 1, 1, 300, 64) == 0
    # 2..32 query heads per KV head: one workgroup per (chunk, KV head, batch),
    # about one per compute unit (256 on MI355X, also the fallback without a
    # device), chunks of >= 128 keys.
    assert pa.attn_decode_num_splits(16, 32, 8, 32768, 128) == 2
    assert pa.attn_decode_num_splits(1, 4, 2, 200, 128) == 2    # chunks of >= 128 keys
    for B, Hq, Hkv, Lk in [(1, 4, 2, 777), (4, 16, 16, 5000), (2, 64, 8, 100000), (1, 64, 1, 5000)]:
        S = pa.attn_decode_num_splits(B, Hq, Hkv, Lk, 128)
        grouped = 2 <= Hq // Hkv <= 32
        assert 1 <= S <= -(-Lk // (128 if grouped else 256))


def test_binding_rejects_cpu_tensors():
    import torch
    q = torch.zeros(1, 1, 4, 64, dtype=torch.float16)
    with pytest.raises(ValueError):
        pa.attn_fwd(q, q, q)


def test_boundary_signatures_match_the_scope_table():
    """attn_fwd / attn_decode take exactly the boundary's arguments (no modifier
    inserted between them); the modifiers live in the *_mod entry points."""
    src = open(os.path.join(ROOT, "include", "attn.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)

    def params(name):
        m = re.search(r"\b%s\s*\(([^)]*)\)\s*;" % name, src)
        return [re.split(r"[\s*]+", p.strip())[-1] for p in m.group(1).split(",")]
    assert params("attn_fwd") == ["Q", "K", "V", "O", "B", "Hq", "Hkv", "Lq", "Lk", "D", "causal", "scale",
                                  "alibi_slopes", "dtype", "stream"]
    assert params("attn_decode") == ["Q", "K", "V", "O", "B", "Hq", "Hkv", "Lk", "D", "scale", "alibi_slopes",
                                     "num_splits", "workspace", "workspace_bytes", "dtype", "stream"]
    assert params("attn_fwd_mod")[-4:] == ["softcap", "window", "dtype", "stream"]
    assert params("attn_decode_mod")[10:13] == ["alibi_slopes", "softcap", "num_splits"]
