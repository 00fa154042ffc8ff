"""Every compiled kernel instantiation once on the GPU against the fp64 oracle
(the cases of tests/kernel_cases.py; the CPU test test_kernel_coverage checks
that they reach every kernel in the build)."""

import zlib

import numpy as np
import pytest
import torch

import paper_2510_08726_amd as pa
from paper_2510_08726_amd.workloads import alibi_slopes, random_tensors
from gpu_common import assert_close, host32, oracle_fwd, run_fwd
from kernel_cases import DECODE_VARIANT_CASES, PREFILL_VARIANT_CASES, case_id

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("case", PREFILL_VARIANT_CASES, ids=case_id)
def test_prefill_variant(case):
    B, Hq, Hkv, Lq, Lk, D, dt, causal, alibi, cap, win = case
    print(f"prefill variant {case} -> {pa.attn_fwd_kernels(D, {'f16': torch.float16, 'bf16': torch.bfloat16}[dt], causal, alibi, cap or 0.0, win or 0)}",
          flush=True)
    q, k, v = random_tensors([(B, Hq, Lq, D), (B, Hkv, Lk, D), (B, Hkv, Lk, D)], dt,
                             seed=zlib.crc32(repr(case).encode()) % 1000)
    if cap:
        q = (q.float() * 4).to(q.dtype)
    sl = alibi_slopes(Hq) if alibi else None
    o = run_fwd(q, k, v, scale=D ** -0.5, causal=causal, slopes=sl, softcap=cap, window=win)
    ref = oracle_fwd(q, k, v, scale=D ** -0.5, causal=causal, slopes=sl, softcap=cap, window=win)
    assert_close(host32(o), ref, f"prefill variant {case}")


@pytest.mark.parametrize("case", DECODE_VARIANT_CASES, ids=case_id)
def test_decode_variant(case):
    B, Hq, Hkv, Lk, D, dt, alibi, cap, S = case
    print(f"decode variant {case} -> {pa.attn_decode_kernels(Hq, Hkv, D, {'f16': torch.float16, 'bf16': torch.bfloat16}[dt], alibi, cap or 0.0)}",
          flush=True)
    q, k, v = random_tensors([(B, Hq, 1, D), (B, Hkv, Lk, D), (B, Hkv, Lk, D)], dt,
                             seed=zlib.crc32(repr(case).encode()) % 1000)
    if cap:
        q = (q.float() * 4).to(q.dtype)
    sl = alibi_slopes(Hq) if alibi else None
    dev = torch.device("cuda")
    o = pa.attn_decode(q.to(dev), k.to(dev), v.to(dev), scale=D ** -0.5,
                       alibi_slopes=None if sl is None else sl.to(dev), softcap=cap, num_splits=S)
    torch.cuda.synchronize()
    ref = oracle_fwd(q, k, v, scale=D ** -0.5, causal=True, slopes=sl, softcap=cap)
    assert_close(host32(o), ref, f"decode variant {case}")
    assert np.all(np.isfinite(host32(o)))
