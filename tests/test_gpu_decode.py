"""GPU parity of split-k decode (attn_decode) against the fp64 oracle.

Besides the final output, the workspace partials written by the split kernel
(the local nests) are compared element by element with the oracle's own
local nests, and the result must not depend on the number of chunks.
"""

import functools
import zlib

import numpy as np
import pytest
import torch

import paper_2510_08726_amd as pa
from oracle import splitk
from paper_2510_08726_amd.workloads import WORKLOADS, alibi_slopes, make_inputs, random_tensors
from gpu_common import assert_close, host32, host64, oracle_fwd, run_fwd

pytestmark = pytest.mark.gpu


def run_decode(q, k, v, *, scale, slopes=None, softcap=None, num_splits=0):
    dev = torch.device("cuda")
    B, Hq, _, D = q.shape
    Hkv, Lk = k.shape[1], k.shape[2]
    S = num_splits or pa.attn_decode_num_splits(B, Hq, Hkv, Lk, D)
    ws = torch.empty(pa.attn_decode_workspace_bytes(B, Hq, D, S), dtype=torch.uint8, device=dev)
    o = pa.attn_decode(q.to(dev), k.to(dev), v.to(dev), scale=scale,
                       alibi_slopes=None if slopes is None else slopes.to(dev),
                       softcap=softcap, num_splits=num_splits, workspace=ws)
    torch.cuda.synchronize()
    return o, ws, S


CASES = [  # B, Hq, Hkv, Lk, D, dtype, S, alibi
    (2, 8, 2, 1000, 128, "f16", 3, False),
    (3, 4, 4, 777, 64, "bf16", 5, False),
    (2, 16, 2, 4096, 128, "f16", 0, False),
    (1, 6, 2, 333, 128, "bf16", 4, True),      # 3 query heads per KV head
    (2, 8, 8, 1024, 64, "f16", 1, True),
    (1, 4, 1, 10, 128, "f16", 6, False),       # chunks of 2 keys, the last chunk empty
    (1, 2, 2, 1, 64, "f16", 4, False),         # one key, three empty chunks
    (1, 32, 4, 2500, 128, "bf16", 100, False),
    (2, 16, 1, 3000, 64, "bf16", 7, True),     # 16 query heads per KV head
    (1, 32, 1, 700, 128, "f16", 3, True),      # 32 query heads per KV head: every MFMA column
    (2, 4, 2, 515, 64, "bf16", 2, True),       # 2 query heads per KV head, D 64
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
def test_decode_matches_oracle(case):
    B, Hq, Hkv, Lk, D, dt, S, alibi = case
    print(f"decode case {case}", flush=True)
    q, k, v = random_tensors([(B, Hq, 1, D), (B, Hkv, Lk, D), (B, Hkv, Lk, D)], dt, seed=zlib.crc32(repr(case).encode()) % 1000)
    sl = alibi_slopes(Hq) if alibi else None
    scale = D ** -0.5
    o, ws, Sres = run_decode(q, k, v, scale=scale, slopes=sl, num_splits=S)
    ref = oracle_fwd(q, k, v, scale=scale, causal=True, slopes=sl)
    assert_close(host32(o), ref, f"decode {case}")

    # the local nests, element by element (natural-log units)
    o_l, m_l, s_l = [t.cpu().numpy().astype(np.float64) for t in pa.decode_partials(ws, B, Hq, D, Sres)]
    ro, rm, rs = splitk.split_local(host32(q), host32(k), host32(v), scale=scale, num_splits=Sres,
                                    causal=True, alibi_slopes=None if sl is None else host64(sl))
    ro, rm, rs = ro[:, :, 0], rm[:, :, 0], rs[:, :, 0]
    empty = np.isneginf(rm)
    assert np.array_equal(np.isneginf(m_l), empty)
    assert np.all(s_l[empty] == 0) and np.all(o_l[empty] == 0)
    live = ~empty
    np.testing.assert_allclose(m_l[live], rm[live], atol=1e-4, rtol=1e-5)
    np.testing.assert_allclose(s_l[live], rs[live], rtol=2e-4)
    # The chunk-normalised partial is a weighted mean of V rows.  The weights
    # that multiply V are rounded to the input type (the compute definition
    # casts exp before the second matmul), a relative error of up to 2^-11
    # (fp16) or 2^-9 (bf16) per weight, so a chunk of few keys can be off by
    # about that times max |V| (~4 for N(0,1) rows).
    tol = 2e-3 if dt == "f16" else 8e-3
    np.testing.assert_allclose((o_l / np.where(live, s_l, 1)[..., None])[live],
                               (ro / np.where(live, rs, 1)[..., None])[live], atol=tol)


def test_decode_independent_of_split_count_and_equals_prefill_row():
    B, Hq, Hkv, Lk, D = 2, 8, 2, 3000, 128
    q, k, v = random_tensors([(B, Hq, 1, D), (B, Hkv, Lk, D), (B, Hkv, Lk, D)], "f16", seed=31)
    scale = D ** -0.5
    outs = [host32(run_decode(q, k, v, scale=scale, num_splits=S)[0]) for S in (1, 2, 16, 64, 3000)]
    single = host32(run_fwd(q, k, v, scale=scale, causal=True))
    ref = oracle_fwd(q, k, v, scale=scale, causal=True)
    for o in outs + [single]:
        assert_close(o, ref, "decode vs oracle")
    for o in outs[1:] + [single]:
        assert_close(o, outs[0], "decode(S) vs decode(1)")


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (8, 2)], ids=["per-head", "grouped"])
def test_one_chunk_output_is_the_combine_of_its_partial(Hq, Hkv):
    """With one chunk the split kernel writes O itself (the combine does not
    run); it must be what the combine computes from the single partial, whose
    weight is exp(0) = 1: o_l / sum_l, rounded once to fp16."""
    B, Lk, D = 2, 777, 128
    print(f"one-chunk decode {B}x{Hq}/{Hkv} Lk {Lk}", flush=True)
    q, k, v = random_tensors([(B, Hq, 1, D), (B, Hkv, Lk, D), (B, Hkv, Lk, D)], "f16", seed=37)
    o, ws, S = run_decode(q, k, v, scale=D ** -0.5, num_splits=1)
    ol, _, sl = (t.cpu().numpy() for t in pa.decode_partials(ws, B, Hq, D, 1))
    expect = (ol[:, :, 0] / sl[:, :, 0, None]).astype(np.float16)
    got = o.cpu().numpy().reshape(B, Hq, D)
    assert np.array_equal(got.view(np.uint16), expect.view(np.uint16))
    assert_close(host32(o), oracle_fwd(q, k, v, scale=D ** -0.5, causal=True), "one-chunk decode vs oracle")


def test_decode_is_deterministic():
    q, k, v = random_tensors([(4, 8, 1, 128), (4, 2, 5000, 128), (4, 2, 5000, 128)], "bf16", seed=32)
    a = run_decode(q, k, v, scale=0.1, num_splits=13)[0]
    b = run_decode(q, k, v, scale=0.1, num_splits=13)[0]
    assert torch.equal(a, b)


@functools.lru_cache(maxsize=1)
def _workload_run(name):
    w = WORKLOADS[name]
    q, k, v, sl = make_inputs(w)
    o, ws, S = run_decode(q, k, v, scale=w.sm_scale, slopes=sl, softcap=w.softcap or None,
                          num_splits=w.num_splits)
    return w, q, k, v, sl, o.cpu()


@pytest.mark.parametrize("name", ["mha_decode", "gqa_long_decode", "alibi_decode", "softcap_decode"])
def test_decode_workload_full(name):
    """Every output row of the full-size decode workloads vs the oracle."""
    print(f"decode workload {name}", flush=True)
    w, q, k, v, sl, o = _workload_run(name)
    ref = oracle_fwd(q, k, v, scale=w.sm_scale, causal=True, slopes=sl, softcap=w.softcap or None)
    assert_close(host32(o), ref, name)


SOFTCAP_CASES = [  # B, Hq, Hkv, Lk, D, dtype, S, alibi, cap, score gain
    (2, 8, 8, 1000, 128, "f16", 3, False, 2.0, 4.0),     # one head per KV head: vector kernel
    (2, 8, 2, 777, 64, "bf16", 5, False, 1.0, 4.0),      # 4 query heads per KV head: matrix kernel
    (1, 32, 16, 2500, 128, "f16", 0, False, 5.0, 8.0),   # Gemma 2 27B head layout
    (1, 16, 1, 300, 128, "bf16", 4, True, 3.0, 4.0),     # 16 per KV head, with ALiBi after the cap
    (2, 6, 6, 333, 64, "f16", 2, True, 0.5, 1.0),        # vector kernel with ALiBi after the cap
    (1, 4, 2, 1, 128, "f16", 3, False, 1.0, 4.0),        # one key, two empty chunks
]


@pytest.mark.parametrize("case", SOFTCAP_CASES, ids=lambda c: "x".join(map(str, c)))
def test_decode_softcap_matches_oracle(case):
    """SoftCap decode vs the oracle.  The query is scaled up ("score gain") so
    that the scores reach the cap and the capped result differs from the
    uncapped one by far more than the tolerance."""
    B, Hq, Hkv, Lk, D, dt, S, alibi, cap, gain = case
    print(f"softcap decode case {case}", flush=True)
    q, k, v = random_tensors([(B, Hq, 1, D), (B, Hkv, Lk, D), (B, Hkv, Lk, D)], dt,
                             seed=zlib.crc32(repr(case).encode()) % 1000)
    q = (q.float() * gain).to(q.dtype)
    sl = alibi_slopes(Hq) if alibi else None
    scale = D ** -0.5
    o, ws, Sres = run_decode(q, k, v, scale=scale, slopes=sl, softcap=cap, num_splits=S)
    ref = oracle_fwd(q, k, v, scale=scale, causal=True, slopes=sl, softcap=cap)
    assert_close(host32(o), ref, f"softcap decode {case}")
    if Lk > 1:
        plain = oracle_fwd(q, k, v, scale=scale, causal=True, slopes=sl)
        assert np.abs(plain - ref).max() > 0.05, "the cap must matter in this case"
    # the local nests carry the capped scores
    o_l, m_l, s_l = [t.cpu().numpy().astype(np.float64) for t in pa.decode_partials(ws, B, Hq, D, Sres)]
    ro, rm, rs = splitk.split_local(host32(q), host32(k), host32(v), scale=scale, num_splits=Sres,
                                    causal=True, alibi_slopes=None if sl is None else host64(sl),
                                    softcap=cap)
    live = ~np.isneginf(rm[:, :, 0])
    assert np.array_equal(np.isneginf(m_l), ~live)
    np.testing.assert_allclose(m_l[live], rm[:, :, 0][live], atol=1e-4, rtol=1e-5)
    np.testing.assert_allclose(s_l[live], rs[:, :, 0][live], rtol=2e-4)


def test_decode_softcap_saturates_exactly():
    """Scores far beyond the cap: every capped score is +-cap, so the output is
    the closed-form mix e^cap V_j* + e^-cap (others), whatever the kernel."""
    B, Hq, Hkv, Lk, D, cap = 1, 2, 2, 64, 64, 1.5
    q = torch.zeros(B, Hq, 1, D)
    q[..., 0] = 1.0
    k = torch.zeros(B, Hkv, Lk, D)
    k[..., 0] = -1000.0
    k[:, :, 17, 0] = 1000.0
    v = random_tensors([(B, Hkv, Lk, D)], "f16", seed=77)[0]
    q, k = q.half(), k.half()
    o = host32(run_decode(q, k, v, scale=1.0, softcap=cap, num_splits=4)[0])
    w = np.full(Lk, np.exp(-cap))
    w[17] = np.exp(cap)
    ref = (w[:, None] * host64(v)[0]).sum(1) / w.sum()          # [Hq, D]
    assert np.all(np.isfinite(o))
    np.testing.assert_allclose(o[0, :, 0], ref, atol=2e-3)
