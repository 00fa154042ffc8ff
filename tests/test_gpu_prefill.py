"""GPU parity of the fused prefill kernel (attn_fwd) against the fp64 oracle.

Small shapes span several 256-row query blocks and 32-key tiles with ragged
tails and are compared element by element; the full-size workloads run in the
launch configuration the bench times and are compared on sampled rows the
oracle computes one by one.
"""

import functools
import zlib

import numpy as np
import pytest
import torch

import paper_2510_08726_amd as pa
from paper_2510_08726_amd.workloads import WORKLOADS, alibi_slopes, make_inputs, random_tensors
from gpu_common import assert_close, host32, host64, oracle_fwd, run_fwd

pytestmark = pytest.mark.gpu

CASES = [  # B, Hq, Hkv, Lq, Lk, D, dtype, causal, alibi
    (1, 2, 2, 128, 128, 64, "f16", False, False),
    (2, 4, 4, 333, 333, 64, "f16", True, False),
    (2, 4, 2, 200, 457, 128, "bf16", True, False),
    (1, 4, 4, 300, 300, 128, "f16", False, False),
    (2, 8, 2, 257, 257, 128, "bf16", True, True),
    (1, 2, 2, 190, 64, 64, "f16", True, False),     # Lq > Lk: the first rows see no key
    (1, 2, 1, 1, 300, 128, "f16", True, False),     # a single query row
    (1, 3, 1, 65, 65, 64, "bf16", False, True),     # 3 query heads per KV head
    (1, 4, 4, 700, 700, 64, "bf16", True, True),    # ALiBi: keys visited last to first, 3 query blocks
    (1, 2, 2, 300, 777, 128, "f16", True, True),    # ALiBi causal with Lk > Lq
    (1, 2, 2, 520, 300, 64, "f16", False, True),    # ALiBi without mask, Lq > Lk, ragged keys
    (1, 2, 2, 530, 200, 128, "bf16", True, True),   # ALiBi causal, Lq > Lk: rows and waves with no key
    (1, 2, 1, 600, 1000, 128, "bf16", False, False),
    (1, 4, 4, 130, 70, 128, "f16", False, False),
    (1, 2, 2, 1, 1, 64, "bf16", True, True),
    (1, 2, 2, 520, 520, 64, "f16", True, True),
    (1, 1, 1, 129, 1000, 128, "bf16", False, False),
    (1, 16, 2, 300, 300, 128, "bf16", True, False),   # 8 query heads per KV head: one head per wave
    (2, 8, 1, 70, 70, 64, "f16", True, True),         # 8 per KV head with ALiBi, a single ragged block
    (1, 12, 3, 100, 260, 128, "f16", False, False),   # 4 query heads per KV head, Lk > Lq
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
def test_prefill_matches_oracle(case):
    B, Hq, Hkv, Lq, Lk, D, dt, causal, alibi = case
    print(f"prefill case {case}", flush=True)
    q, k, v = random_tensors([(B, Hq, Lq, D), (B, Hkv, Lk, D), (B, Hkv, Lk, D)], dt, seed=zlib.crc32(repr(case).encode()) % 1000)
    sl = alibi_slopes(Hq) if alibi else None
    scale = D ** -0.5
    o = run_fwd(q, k, v, scale=scale, causal=causal, slopes=sl)
    ref = oracle_fwd(q, k, v, scale=scale, causal=causal, slopes=sl)
    assert_close(host32(o), ref, f"prefill {case}")
    if causal and Lq > Lk:
        assert torch.all(o[:, :, :Lq - Lk] == 0)


@pytest.mark.parametrize("scale,alibi", [(0.0, False), (0.0, True), (-0.2, False), (-0.2, True), (3.0, False),
                                         (3.0, True)])
def test_prefill_special_scales(scale, alibi):
    """scale 0 (uniform / geometric weights), negative scale, large scores."""
    B, H, L, D = 1, 4, 200, 64
    q, k, v = random_tensors([(B, H, L, D)] * 3, "f16", seed=21)
    sl = alibi_slopes(H) if alibi else None
    o = run_fwd(q, k, v, scale=scale, causal=True, slopes=sl)
    ref = oracle_fwd(q, k, v, scale=scale, causal=True, slopes=sl)
    assert_close(host32(o), ref, f"scale={scale} alibi={alibi}")


def test_prefill_constant_v():
    B, H, L, D = 1, 2, 300, 128
    q, k = random_tensors([(B, H, L, D)] * 2, "f16", seed=22)
    c = torch.linspace(-3, 3, D, dtype=torch.float16)
    v = c.expand(B, H, L, D).contiguous()
    o = run_fwd(q, k, v, scale=D ** -0.5, causal=True)
    err = (o.float().cpu() - c.float()).abs().max().item()
    assert err <= 2e-3, err


def test_prefill_peak_in_last_tile_selects_its_value_row():
    """The repair factor must discount every earlier tile once the max jumps."""
    B, H, L, D = 1, 1, 300, 64
    q, k, v = random_tensors([(B, H, L, D)] * 3, "f16", seed=23)
    q = q * 0.05
    k = k * 0.05
    jstar = L - 1
    q[..., 0] = 5.0
    k[0, 0, jstar, 0] = 6.0          # q.k* = 30 for every row, others < ~0.5
    q, k = q.contiguous(), k.contiguous()
    o = run_fwd(q, k, v, scale=1.0, causal=False)
    np.testing.assert_allclose(host32(o)[0, 0], np.broadcast_to(host32(v)[0, 0, jstar], (L, D)), atol=2e-3)


@pytest.mark.parametrize("direction", [1, -1])
def test_prefill_monotone_scores(direction):
    """Scores that rise (the max moves at every tile) or fall along the keys."""
    B, H, L, D = 1, 2, 400, 64
    _, _, v = random_tensors([(B, H, L, D)] * 3, "bf16", seed=24)
    u = torch.zeros(D)
    u[0] = 1.0
    q = (u * 2.0).expand(B, H, L, D).to(torch.bfloat16).contiguous()
    ramp = torch.linspace(0, 8, L) * direction
    k = (ramp[:, None] * u[None, :]).expand(B, H, L, D).to(torch.bfloat16).contiguous()
    o = run_fwd(q, k, v, scale=1.0, causal=True)
    ref = oracle_fwd(q, k, v, scale=1.0, causal=True)
    assert_close(host32(o), ref, f"monotone {direction}")


def test_prefill_is_deterministic():
    w = WORKLOADS["causal_mha_prefill"]
    q, k, v = random_tensors([(2, 8, 700, 128), (2, 8, 700, 128), (2, 8, 700, 128)], "f16", seed=25)
    a = run_fwd(q, k, v, scale=w.sm_scale, causal=True)
    b = run_fwd(q, k, v, scale=w.sm_scale, causal=True)
    assert torch.equal(a, b)


# ---------------------------------------------------------------------------
# full-size workloads (the bench's launch configuration)

@functools.lru_cache(maxsize=1)
def _workload_run(name):
    w = WORKLOADS[name]
    q, k, v, sl = make_inputs(w)
    dev = torch.device("cuda")
    # NaN-filled output: a row that no work item writes cannot pass.
    o = torch.full(q.shape, float("nan"), dtype=q.dtype, device=dev)
    pa.attn_fwd(q.to(dev), k.to(dev), v.to(dev), o, causal=w.causal, scale=w.sm_scale,
                alibi_slopes=None if sl is None else sl.to(dev), softcap=w.softcap or None,
                window=w.window or None)
    torch.cuda.synchronize()
    return w, q, k, v, sl, o.cpu()


def _wave_block_rows(L):
    """The first and the last row of every 32-row wave block (every wave of
    every work item of the persistent schedule), plus a few in between."""
    rows = set()
    for r0 in range(0, L, 32):
        rows.update((r0, min(r0 + 31, L - 1)))
    rows.update(range(L // 2 - 3, L // 2 + 3))
    return sorted(rows)


@pytest.mark.parametrize("name", ["tiny_noncausal", "causal_mha_prefill", "gqa_causal_prefill",
                                  "alibi_causal_prefill", "softcap_causal_prefill", "window_causal_prefill"])
def test_prefill_workload_full_size(name):
    """Every (batch, head).  The causal MHA workload (and the tiny one) is
    compared on every row; the others on the first and last row of every
    32-row wave block, so every wave of every work item is checked."""
    print(f"prefill workload {name}", flush=True)
    w, q, k, v, sl, o = _workload_run(name)
    got = host32(o)
    assert np.all(np.isfinite(got)), "every output row is written"
    full = name in ("tiny_noncausal", "causal_mha_prefill")
    rows = None if full else _wave_block_rows(w.Lq)
    ref = oracle_fwd(q, k, v, scale=w.sm_scale, causal=w.causal, slopes=sl, softcap=w.softcap or None,
                     window=w.window or None, rows=rows)
    assert_close(got if full else got[:, :, rows], ref, f"{name} {'all rows' if full else 'wave-block rows'}")


MULTI_ROUND_CASES = [  # B, Hq, Hkv, L_q, L_k, D, dtype, alibi, window: more work items than workgroups
    (4, 64, 64, 600, 600, 64, "f16", False, None),     # 1280 items: 2-3 rounds per workgroup
    (4, 64, 64, 600, 600, 64, "bf16", True, None),     # ALiBi: keys last to first
    (2, 64, 8, 600, 600, 128, "f16", False, None),     # 8 query heads per KV head: 608 items
    (3, 48, 48, 400, 650, 64, "f16", False, None),     # Lq < Lk
    (3, 48, 48, 650, 400, 128, "bf16", False, None),   # Lq > Lk: rows and waves with no key
    (4, 64, 32, 600, 600, 64, "f16", False, 90),       # sliding window, 2 heads per KV head
]


@pytest.mark.parametrize("case", MULTI_ROUND_CASES, ids=lambda c: "x".join(map(str, c)))
def test_prefill_multi_round_matches_oracle_everywhere(case):
    """The persistent schedule's later rounds: the next item's staging before
    the current output, the snake order, compared on every output element."""
    B, Hq, Hkv, Lq, Lk, D, dt, alibi, win = case
    print(f"multi-round prefill case {case}", flush=True)
    q, k, v = random_tensors([(B, Hq, Lq, D), (B, Hkv, Lk, D), (B, Hkv, Lk, D)], dt,
                             seed=zlib.crc32(repr(case).encode()) % 1000)
    sl = alibi_slopes(Hq) if alibi else None
    dev = torch.device("cuda")
    o = torch.full((B, Hq, Lq, D), float("nan"), dtype=q.dtype, device=dev)
    pa.attn_fwd(q.to(dev), k.to(dev), v.to(dev), o, causal=True, scale=D ** -0.5,
                alibi_slopes=None if sl is None else sl.to(dev), window=win)
    torch.cuda.synchronize()
    got = host32(o)
    ref = oracle_fwd(q, k, v, scale=D ** -0.5, causal=True, slopes=sl, window=win)
    assert_close(got, ref, f"multi-round {case}")
    if Lq > Lk:
        assert np.all(got[:, :, :Lq - Lk] == 0)


SOFTCAP_CASES = [  # B, Hq, Hkv, Lq, Lk, D, dtype, cap, score gain
    (1, 4, 4, 300, 300, 128, "f16", 2.0, 4.0),
    (2, 8, 4, 257, 257, 64, "bf16", 1.0, 4.0),      # 2 query heads per KV head, ragged tail
    (1, 16, 2, 200, 330, 128, "bf16", 5.0, 8.0),    # 8 query heads per KV head, Lq < Lk
    (1, 2, 1, 96, 40, 64, "f16", 3.0, 4.0),         # Lq > Lk: the first rows see no key
]


@pytest.mark.parametrize("case", SOFTCAP_CASES, ids=lambda c: "x".join(map(str, c)))
def test_prefill_softcap_matches_oracle(case):
    """Causal SoftCap prefill vs the oracle; the query is scaled up so that the
    cap changes the result by far more than the tolerance."""
    B, Hq, Hkv, Lq, Lk, D, dt, cap, gain = case
    print(f"softcap prefill case {case}", flush=True)
    q, k, v = random_tensors([(B, Hq, Lq, D), (B, Hkv, Lk, D), (B, Hkv, Lk, D)], dt,
                             seed=zlib.crc32(repr(case).encode()) % 1000)
    q = (q.float() * gain).to(q.dtype)
    scale = D ** -0.5
    o = run_fwd(q, k, v, scale=scale, causal=True, softcap=cap)
    ref = oracle_fwd(q, k, v, scale=scale, causal=True, softcap=cap)
    assert_close(host32(o), ref, f"softcap prefill {case}")
    plain = oracle_fwd(q, k, v, scale=scale, causal=True)
    assert np.abs(plain - ref).max() > 0.05, "the cap must matter in this case"


def test_prefill_softcap_last_row_equals_decode():
    """The last query row of causal SoftCap prefill is the SoftCap decode of that token."""
    B, Hq, Hkv, L, D, cap = 2, 8, 2, 700, 128, 2.5
    q, k, v = random_tensors([(B, Hq, L, D), (B, Hkv, L, D), (B, Hkv, L, D)], "f16", seed=61)
    q = (q.float() * 4).to(q.dtype)
    o = host32(run_fwd(q, k, v, scale=D ** -0.5, causal=True, softcap=cap))
    dev = torch.device("cuda")
    od = pa.attn_decode(q[:, :, -1:].contiguous().to(dev), k.to(dev), v.to(dev), scale=D ** -0.5,
                        softcap=cap, num_splits=3)
    torch.cuda.synchronize()
    assert_close(o[:, :, -1:], host64(od.cpu()).astype(np.float64), "prefill last row vs decode")


WINDOW_CASES = [  # B, Hq, Hkv, Lq, Lk, D, dtype, window, alibi, softcap
    (1, 2, 2, 300, 300, 128, "f16", 1, False, None),        # one key per row: O = V[i]
    (2, 4, 2, 333, 333, 64, "bf16", 45, False, None),       # band edges inside tiles, ragged tail
    (1, 4, 4, 700, 700, 128, "f16", 100, False, None),      # several 128-row blocks, edges off the grid
    (1, 2, 1, 257, 600, 128, "bf16", 64, False, None),      # Lq < Lk, band edge on the tile grid
    (1, 2, 2, 400, 150, 64, "f16", 70, False, None),        # Lq > Lk: the first rows see no key
    (1, 16, 2, 300, 300, 128, "bf16", 33, False, None),     # 8 query heads per KV head
    (1, 4, 4, 520, 520, 64, "f16", 96, True, None),         # ALiBi: keys visited last to first
    (1, 2, 2, 300, 777, 128, "bf16", 200, True, None),      # ALiBi, Lk > Lq
    (1, 4, 2, 300, 300, 128, "f16", 57, False, 3.0),        # with SoftCap (Gemma 2 local layers)
    (1, 2, 2, 129, 129, 64, "f16", 5000, False, None),      # window wider than every row: causal
]


@pytest.mark.parametrize("case", WINDOW_CASES, ids=lambda c: "x".join(map(str, c)))
def test_prefill_window_matches_oracle(case):
    B, Hq, Hkv, Lq, Lk, D, dt, W, alibi, cap = case
    print(f"window prefill case {case}", flush=True)
    q, k, v = random_tensors([(B, Hq, Lq, D), (B, Hkv, Lk, D), (B, Hkv, Lk, D)], dt,
                             seed=zlib.crc32(repr(case).encode()) % 1000)
    if cap:
        q = (q.float() * 4).to(q.dtype)
    sl = alibi_slopes(Hq) if alibi else None
    scale = D ** -0.5
    o = run_fwd(q, k, v, scale=scale, causal=True, slopes=sl, softcap=cap, window=W)
    ref = oracle_fwd(q, k, v, scale=scale, causal=True, slopes=sl, softcap=cap, window=W)
    assert_close(host32(o), ref, f"window prefill {case}")
    if W == 1:
        G = Hq // Hkv
        off = Lk - Lq
        vv = host32(v).repeat(G, axis=1)
        rows = [i for i in range(Lq) if i + off >= 0]
        np.testing.assert_array_equal(host32(o)[:, :, rows], vv[:, :, [i + off for i in rows]])


def test_prefill_window_scale_zero_is_band_mean():
    """scale = 0: every row averages V over its band (closed form)."""
    B, H, L, D, W = 1, 2, 300, 64, 37
    q, k, v = random_tensors([(B, H, L, D)] * 3, "f16", seed=66)
    o = host32(run_fwd(q, k, v, scale=0.0, causal=True, window=W))
    vv = host64(v)
    ref = np.stack([vv[:, :, max(0, i - W + 1):i + 1].mean(axis=2) for i in range(L)], axis=2)
    np.testing.assert_allclose(o, ref, atol=4e-3)
