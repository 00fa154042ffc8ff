"""attn_decode_noalloc (static workspace, no allocation) through the C ABI
against attn_decode_mod with a caller workspace, on two calls in a row, the
second with a smaller input."""

import ctypes

import numpy as np
import pytest
import torch

import paper_2510_08726_amd as pa
from paper_2510_08726_amd.workloads import alibi_slopes, random_tensors
from gpu_common import assert_close, host32, oracle_fwd

pytestmark = pytest.mark.gpu

CASES = [  # B, Hq, Hkv, Lk, D, dtype, alibi, softcap, num_splits
    (8, 32, 8, 5000, 128, "f16", False, None, 0),     # grouped kernel, the library's split count
    (2, 16, 16, 1000, 64, "bf16", True, 2.0, 7),       # vector kernel, ALiBi and SoftCap
]


def _call(lib, fn, q, k, v, o, sl, cap, S, ws=None):
    B, Hq, _, D = q.shape
    Hkv, Lk = k.shape[1], k.shape[2]
    vp = ctypes.c_void_p
    dt = 0 if q.dtype == torch.float16 else 1
    stream = vp(torch.cuda.current_stream().cuda_stream)
    slp = None if sl is None else vp(sl.data_ptr())
    if fn == "noalloc":
        return lib.attn_decode_noalloc(vp(q.data_ptr()), vp(k.data_ptr()), vp(v.data_ptr()), vp(o.data_ptr()),
                                       B, Hq, Hkv, Lk, D, D ** -0.5, slp, float(cap or 0.0), S, dt, stream)
    return lib.attn_decode_mod(vp(q.data_ptr()), vp(k.data_ptr()), vp(v.data_ptr()), vp(o.data_ptr()),
                               B, Hq, Hkv, Lk, D, D ** -0.5, slp, float(cap or 0.0), S, vp(ws.data_ptr()),
                               ws.numel(), dt, stream)


def test_noalloc_matches_workspace_entry_point_twice_shrinking():
    lib = pa.load_library()
    dev = torch.device("cuda")
    for n, case in enumerate(CASES):
        B, Hq, Hkv, Lk, D, dt, alibi, cap, S = case
        print(f"no-alloc decode call {n}: {case}", flush=True)
        q, k, v = (t.to(dev) for t in random_tensors([(B, Hq, 1, D), (B, Hkv, Lk, D), (B, Hkv, Lk, D)], dt,
                                                     seed=100 + n))
        if cap:
            q = (q.float() * 4).to(q.dtype)
        sl = alibi_slopes(Hq).to(dev) if alibi else None
        Sres = S or pa.attn_decode_num_splits(B, Hq, Hkv, Lk, D)
        ws = torch.empty(pa.attn_decode_workspace_bytes(B, Hq, D, Sres), dtype=torch.uint8, device=dev)
        o_ref = torch.full_like(q, float("nan"))
        o_new = torch.full_like(q, float("nan"))
        assert _call(lib, "mod", q, k, v, o_ref, sl, cap, S, ws) == pa.ATTN_OK
        assert _call(lib, "noalloc", q, k, v, o_new, sl, cap, S) == pa.ATTN_OK
        torch.cuda.synchronize()
        # the same kernels on the same partials: bitwise equal
        assert torch.equal(o_new, o_ref)
        ref = oracle_fwd(q.cpu(), k.cpu(), v.cpu(), scale=D ** -0.5, causal=True,
                         slopes=None if sl is None else sl.cpu(), softcap=cap)
        assert_close(host32(o_new), ref, f"no-alloc decode {case}")


def test_noalloc_rejects_a_workspace_beyond_its_limit():
    lib = pa.load_library()
    dev = torch.device("cuda")
    q = torch.zeros(64, 64, 1, 128, dtype=torch.float16, device=dev)
    k = torch.zeros(64, 64, 8, 128, dtype=torch.float16, device=dev)
    o = torch.zeros_like(q)
    # 64 * 64 * 8 splits * 130 floats = 17 MB > 16 MiB: refused before any launch
    assert pa.attn_decode_workspace_bytes(64, 64, 128, 8) > pa.ATTN_DECODE_NOALLOC_BYTES
    assert _call(lib, "noalloc", q, k, k, o, None, None, 8) == pa.ATTN_ERR_WORKSPACE
