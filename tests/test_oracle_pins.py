"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

None of these compares the oracle with a retyped copy of itself: they use
invariants of softmax attention, closed forms of special cases, brute force
over tiny exact inputs, hand-derived fixtures (tests/golden) and PyTorch's
float64 CPU ``scaled_dot_product_attention`` as a library special case.
``test_oracle_mutants.py`` shows that plausible mistakes fail these pins.
"""

import itertools
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2510_08726_amd.workloads import alibi_slopes

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape, seed):
    return np.random.Generator(np.random.PCG64(seed)).standard_normal(shape)


def _sdpa(q, k, v, *, scale, causal=False, slopes=None):
    """PyTorch float64 CPU attention; bias and causal mask built bottom-right."""
    q, k, v = (torch.from_numpy(np.ascontiguousarray(x)) for x in (q, k, v))
    B, Hq, Lq, D = q.shape
    Hkv, Lk = k.shape[1], k.shape[2]
    off = Lk - Lq
    i = torch.arange(Lq, dtype=torch.float64)[:, None] + off
    j = torch.arange(Lk, dtype=torch.float64)[None, :]
    mask = torch.zeros(Hq, Lq, Lk, dtype=torch.float64)
    if slopes is not None:
        mask = mask - torch.as_tensor(slopes, dtype=torch.float64)[:, None, None] * (i - j)
    if causal:
        mask = mask.masked_fill(j > i, float("-inf"))
    G = Hq // Hkv
    k = k.repeat_interleave(G, dim=1)
    v = v.repeat_interleave(G, dim=1)
    return F.scaled_dot_product_attention(q, k, v, attn_mask=mask[None], scale=scale).numpy()


# ---------------------------------------------------------------------------
# invariants

@pytest.mark.parametrize("causal,alibi,cap", [(False, False, None), (True, False, None), (True, True, None),
                                           (True, False, 1.5), (True, True, 0.7)])
def test_probability_rows_sum_to_one(causal, alibi, cap):
    q, k = _rand((1, 4, 37, 16), 1), _rand((1, 2, 53, 16), 2)
    sl = alibi_slopes(4).double().numpy() if alibi else None
    for hq in range(4):
        p = oracle.softmax_probs(q, k, scale=0.25, causal=causal, alibi_slopes=sl, softcap=cap, hq=hq)
        assert np.all(p >= 0)
        np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-12)
        if causal:   # masked entries carry exactly zero probability
            off = 53 - 37
            for i in range(37):
                assert np.all(p[i, i + off + 1:] == 0.0)


@pytest.mark.parametrize("causal", [False, True])
def test_constant_v_gives_constant_output(causal):
    q, k = _rand((2, 4, 19, 8), 3), _rand((2, 2, 19, 8), 4)
    c = _rand((2, 2, 1, 8), 5)
    v = np.broadcast_to(c, (2, 2, 19, 8)).copy()
    o = oracle.attention(q, k, v, scale=0.4, causal=causal)
    expect = np.repeat(c, 2, axis=1)                        # query heads of each group
    np.testing.assert_allclose(o, np.broadcast_to(expect, o.shape), atol=1e-12)


def test_one_hot_peak_selects_value_row():
    """A score that exceeds every other by >= 20 picks its V row (K != V)."""
    D, Lk = 8, 40
    rng = np.random.Generator(np.random.PCG64(7))
    k = rng.standard_normal((1, 1, Lk, D)) * 0.1
    v = rng.standard_normal((1, 1, Lk, D))
    q = np.zeros((1, 1, 3, D))
    peaks = [Lk - 1, 0, 17]                                 # last, first, middle key
    for i, j in enumerate(peaks):
        q[0, 0, i] = k[0, 0, j] * 0.0
        q[0, 0, i, i] = 1.0
        k[0, 0, j, i] = 40.0                                  # q_i . k_j = 40 >> others
    o = oracle.attention(q, k, v, scale=1.0)
    for i, j in enumerate(peaks):
        np.testing.assert_allclose(o[0, 0, i], v[0, 0, j], atol=Lk * math.exp(-20) * 10)


def test_single_key_returns_its_value():
    q, k, v = _rand((1, 2, 5, 4), 8), _rand((1, 2, 1, 4), 9), _rand((1, 2, 1, 4), 10)
    o = oracle.attention(q, k, v, scale=0.7)
    np.testing.assert_allclose(o, np.broadcast_to(v, o.shape), atol=1e-15)


def test_two_keys_logistic_closed_form():
    """Lk = 2: o = sigma(s0 - s1) v0 + sigma(s1 - s0) v1, scores summed by hand."""
    q, k, v = _rand((1, 1, 6, 5), 11), _rand((1, 1, 2, 5), 12), _rand((1, 1, 2, 5), 13)
    scale = 0.37
    o = oracle.attention(q, k, v, scale=scale)
    for i in range(6):
        s = [scale * sum(q[0, 0, i, d] * k[0, 0, j, d] for d in range(5)) for j in range(2)]
        w0 = 1.0 / (1.0 + math.exp(s[1] - s[0]))
        for d in range(5):
            assert abs(o[0, 0, i, d] - (w0 * v[0, 0, 0, d] + (1 - w0) * v[0, 0, 1, d])) < 1e-13


@pytest.mark.parametrize("Lq,Lk", [(7, 7), (5, 12), (1, 9)])
def test_causal_scale_zero_is_prefix_mean(Lq, Lk):
    """scale = 0 removes the scores: row i averages the Lk - Lq + i + 1 visible V rows."""
    q, k, v = _rand((1, 1, Lq, 3), 14), _rand((1, 1, Lk, 3), 15), _rand((1, 1, Lk, 3), 16)
    o = oracle.attention(q, k, v, scale=0.0, causal=True)
    for i in range(Lq):
        n = i + (Lk - Lq) + 1
        np.testing.assert_allclose(o[0, 0, i], v[0, 0, :n].mean(axis=0), atol=1e-14)


def test_alibi_scale_zero_geometric_closed_form():
    """scale = 0 with ALiBi: weights r^(i-j), r = e^-slope, over the visible keys."""
    H, L = 4, 11
    q, k, v = _rand((1, H, L, 2), 17), _rand((1, H, L, 2), 18), _rand((1, H, L, 2), 19)
    sl = alibi_slopes(H).double().numpy()
    o = oracle.attention(q, k, v, scale=0.0, causal=True, alibi_slopes=sl)
    for h in range(H):
        r = math.exp(-sl[h])
        for i in range(L):
            w = np.array([r ** (i - j) for j in range(i + 1)])
            expect = (w[:, None] * v[0, h, :i + 1]).sum(axis=0) / w.sum()
            np.testing.assert_allclose(o[0, h, i], expect, atol=1e-13)


def test_alibi_row_shift_invariance():
    """-slope (i - j) and +slope j differ by a per-row constant: same softmax."""
    H, L = 2, 9
    q, k, v = _rand((1, H, L, 4), 20), _rand((1, H, L, 4), 21), _rand((1, H, L, 4), 22)
    sl = np.array([0.5, 0.125])
    o = oracle.attention(q, k, v, scale=0.5, causal=True, alibi_slopes=sl)
    for h in range(H):
        s = 0.5 * q[0, h] @ k[0, h].T + sl[h] * np.arange(L)[None, :]
        s = np.where(np.tril(np.ones((L, L))) > 0, s, -np.inf)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        np.testing.assert_allclose(o[0, h], (p / p.sum(1, keepdims=True)) @ v[0, h], atol=1e-13)


def test_gqa_equals_mha_with_repeated_heads():
    q, k, v = _rand((2, 8, 13, 4), 23), _rand((2, 2, 21, 4), 24), _rand((2, 2, 21, 4), 25)
    o = oracle.attention(q, k, v, scale=0.3, causal=True)
    o_mha = oracle.attention(q, np.repeat(k, 4, axis=1), np.repeat(v, 4, axis=1),
                             scale=0.3, causal=True)
    np.testing.assert_array_equal(o, o_mha)
    # Hkv == Hq is plain multi-head attention: head h uses K/V head h
    o1 = oracle.attention(q[:, :1], k[:, :1], v[:, :1], scale=0.3, causal=True)
    np.testing.assert_array_equal(o[:, :1], o1)


def test_fully_masked_rows_are_zero():
    """Causal with Lq > Lk: the first Lq - Lk rows see no key and give 0, not NaN."""
    q, k, v = _rand((1, 1, 9, 4), 26), _rand((1, 1, 4, 4), 27), _rand((1, 1, 4, 4), 28)
    o = oracle.attention(q, k, v, scale=0.5, causal=True)
    assert np.all(o[0, 0, :5] == 0.0)
    assert np.all(np.isfinite(o))
    np.testing.assert_allclose(o[0, 0, 5], v[0, 0, 0], atol=1e-15)   # first live row sees key 0 only


def test_large_scores_stay_finite():
    """Scores near +-1e4 would overflow exp without the max subtraction."""
    q, k, v = _rand((1, 2, 16, 8), 29), _rand((1, 2, 16, 8), 30), _rand((1, 2, 16, 8), 31)
    o = oracle.attention(q, k, v, scale=2000.0, causal=True)
    assert np.all(np.isfinite(o))
    s = q[0, 0] @ k[0, 0].T
    for i in range(16):
        j = int(np.argmax(np.where(np.arange(16) <= i, s[i], -np.inf)))
        np.testing.assert_allclose(o[0, 0, i], v[0, 0, j], atol=1e-6)


def test_rows_subset_matches_full():
    q, k, v = _rand((1, 2, 40, 8), 32), _rand((1, 2, 40, 8), 33), _rand((1, 2, 40, 8), 34)
    full = oracle.attention(q, k, v, scale=0.3, causal=True)
    rows = [0, 7, 39, 21]
    sub = oracle.attention(q, k, v, scale=0.3, causal=True, rows=rows)
    np.testing.assert_array_equal(sub, full[:, :, rows])


# ---------------------------------------------------------------------------
# library special case and brute force

@pytest.mark.parametrize("Lq,Lk,causal,alibi,G", [
    (33, 33, False, False, 1), (33, 33, True, False, 1), (17, 40, True, False, 2),
    (29, 29, True, True, 1), (1, 50, True, True, 4), (64, 64, True, False, 8)])
def test_matches_torch_float64_sdpa(Lq, Lk, causal, alibi, G):
    Hkv = 2
    q, k, v = _rand((2, Hkv * G, Lq, 16), 35), _rand((2, Hkv, Lk, 16), 36), _rand((2, Hkv, Lk, 16), 37)
    sl = alibi_slopes(Hkv * G).double().numpy() if alibi else None
    o = oracle.attention(q, k, v, scale=0.25, causal=causal, alibi_slopes=sl)
    np.testing.assert_allclose(o, _sdpa(q, k, v, scale=0.25, causal=causal, slopes=sl),
                               atol=1e-12, rtol=0)


def test_brute_force_tiny_exact_inputs():
    """Every input with entries in {-1, 0, 1} (exact in fp16/bf16), D = 1, Lq = 1."""
    vals = (-1.0, 0.0, 1.0)
    for Lk in (1, 2, 3):
        for combo in itertools.product(vals, repeat=1 + 2 * Lk):
            q = np.array(combo[:1]).reshape(1, 1, 1, 1)
            k = np.array(combo[1:1 + Lk]).reshape(1, 1, Lk, 1)
            v = np.array(combo[1 + Lk:]).reshape(1, 1, Lk, 1)
            o = oracle.attention(q, k, v, scale=1.0)[0, 0, 0, 0]
            s = [q.item() * k[0, 0, j, 0] for j in range(Lk)]
            if Lk == 1:
                expect = v[0, 0, 0, 0]
            elif Lk == 2:
                w0 = 1.0 / (1.0 + math.exp(s[1] - s[0]))
                expect = w0 * v[0, 0, 0, 0] + (1 - w0) * v[0, 0, 1, 0]
            else:
                expect = _sdpa(q, k, v, scale=1.0)[0, 0, 0, 0]
            assert abs(o - expect) < 1e-14


def test_golden_fixtures():
    with open(os.path.join(GOLDEN, "hand_derived.json")) as f:
        cases = json.load(f)["cases"]
    assert len(cases) >= 3
    for c in cases:
        q = np.array(c["q"], dtype=np.float64)[None, None]
        k = np.array(c["k"], dtype=np.float64)[None, None]
        v = np.array(c["v"], dtype=np.float64)[None, None]
        o = oracle.attention(q, k, v, scale=c["scale"], causal=c.get("causal", False))
        np.testing.assert_allclose(o[0, 0], np.array(c["o"]), atol=1e-15, err_msg=c["name"])


def test_softcap_bounds_the_weight_ratio():
    """|cap tanh(x / cap)| <= cap (equal once tanh rounds to 1), so without a bias
    any two visible keys' weights differ by at most e^(2 cap), however large the
    raw scores are."""
    q, k = _rand((1, 2, 9, 8), 33), _rand((1, 2, 30, 8), 34)
    cap = 1.25
    for hq in range(2):
        p = oracle.softmax_probs(q, k, scale=500.0, causal=True, softcap=cap, hq=hq)
        for i in range(9):
            row = p[i, :i + 30 - 9 + 1]
            assert np.all(row > 0) and row.max() / row.min() <= math.exp(2 * cap) * (1 + 1e-12)


# ---------------------------------------------------------------------------
# softmax_probs values (not only their row sums)

def test_softmax_probs_two_keys_logistic():
    """Lk = 2: P[i, 0] = 1 / (1 + e^(s1 - s0)), scores summed by hand."""
    q, k = _rand((1, 2, 5, 7), 61), _rand((1, 1, 2, 7), 62)
    for hq in range(2):
        p = oracle.softmax_probs(q, k, scale=0.45, hq=hq)
        for i in range(5):
            s = [0.45 * math.fsum(q[0, hq, i, d] * k[0, 0, j, d] for d in range(7)) for j in range(2)]
            w0 = 1.0 / (1.0 + math.exp(s[1] - s[0]))
            assert abs(p[i, 0] - w0) <= 1e-13 and abs(p[i, 1] - (1.0 - w0)) <= 1e-13


@pytest.mark.parametrize("Lq,Lk", [(6, 6), (4, 9)])
def test_softmax_probs_causal_scale_zero_uniform(Lq, Lk):
    """scale = 0, causal: row i spreads 1 / (i_abs + 1) over keys 0 .. i_abs."""
    q, k = _rand((1, 1, Lq, 3), 63), _rand((1, 1, Lk, 3), 64)
    p = oracle.softmax_probs(q, k, scale=0.0, causal=True)
    for i in range(Lq):
        ia = i + Lk - Lq
        for j in range(Lk):
            assert p[i, j] == (1.0 / (ia + 1) if j <= ia else 0.0) or abs(p[i, j] - 1.0 / (ia + 1)) < 1e-15


# ---------------------------------------------------------------------------
# sliding window (Window operator of Table tab:operators; causal band of W keys)

@pytest.mark.parametrize("Lq,Lk", [(9, 9), (5, 13), (11, 7)])
def test_window_covering_every_key_is_causal(Lq, Lk):
    q, k, v = _rand((1, 2, Lq, 4), 71), _rand((1, 1, Lk, 4), 72), _rand((1, 1, Lk, 4), 73)
    ref = oracle.attention(q, k, v, scale=0.7, causal=True)
    for W in (Lk, Lk + 3, 10 ** 6):
        np.testing.assert_array_equal(oracle.attention(q, k, v, scale=0.7, causal=True, window=W), ref)


@pytest.mark.parametrize("Lq,Lk", [(8, 8), (5, 12), (10, 6)])
def test_window_of_one_key_selects_its_value(Lq, Lk):
    q, k, v = _rand((2, 2, Lq, 6), 74), _rand((2, 2, Lk, 6), 75), _rand((2, 2, Lk, 6), 76)
    o = oracle.attention(q, k, v, scale=1.3, causal=True, window=1)
    for i in range(Lq):
        ia = i + Lk - Lq
        if ia >= 0:
            np.testing.assert_array_equal(o[:, :, i], v[:, :, ia])
        else:
            assert np.all(o[:, :, i] == 0)


@pytest.mark.parametrize("W", [1, 2, 5, 30])
def test_window_scale_zero_is_band_mean(W):
    Lq, Lk = 12, 20
    q, k, v = _rand((1, 1, Lq, 3), 77), _rand((1, 1, Lk, 3), 78), _rand((1, 1, Lk, 3), 79)
    o = oracle.attention(q, k, v, scale=0.0, causal=True, window=W)
    for i in range(Lq):
        ia = i + Lk - Lq
        band = [v[0, 0, j] for j in range(max(0, ia - W + 1), ia + 1)]
        np.testing.assert_allclose(o[0, 0, i], sum(band) / len(band), atol=1e-14)


def test_window_alibi_scale_zero_geometric_band():
    H, L, W = 3, 15, 4
    q, k, v = _rand((1, H, L, 2), 80), _rand((1, H, L, 2), 81), _rand((1, H, L, 2), 82)
    sl = alibi_slopes(H).double().numpy()
    o = oracle.attention(q, k, v, scale=0.0, causal=True, alibi_slopes=sl, window=W)
    for h in range(H):
        r = math.exp(-sl[h])
        for i in range(L):
            js = range(max(0, i - W + 1), i + 1)
            w = np.array([r ** (i - j) for j in js])
            ref = (w[:, None] * v[0, h, list(js)]).sum(0) / w.sum()
            np.testing.assert_allclose(o[0, h, i], ref, atol=1e-13)


@pytest.mark.parametrize("Lq,Lk,W,G", [(16, 16, 5, 1), (7, 19, 6, 2), (13, 9, 3, 4)])
def test_window_matches_torch_sdpa_with_band_mask(Lq, Lk, W, G):
    """Library special case: PyTorch float64 SDPA with an explicit band mask."""
    Hkv = 2
    q, k, v = _rand((2, Hkv * G, Lq, 8), 83), _rand((2, Hkv, Lk, 8), 84), _rand((2, Hkv, Lk, 8), 85)
    ia = torch.arange(Lq)[:, None] + (Lk - Lq)
    j = torch.arange(Lk)[None, :]
    vis = (j <= ia) & (j > ia - W)
    mask = torch.zeros(Lq, Lk, dtype=torch.float64).masked_fill(~vis, float("-inf"))
    qt, kt, vt = (torch.from_numpy(x) for x in (q, k, v))
    kt, vt = kt.repeat_interleave(G, dim=1), vt.repeat_interleave(G, dim=1)
    ref = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=0.3).numpy()
    rows_seen = vis.any(dim=1).numpy()
    o = oracle.attention(q, k, v, scale=0.3, causal=True, window=W)
    np.testing.assert_allclose(o[:, :, rows_seen], ref[:, :, rows_seen], atol=1e-12)
    assert np.all(o[:, :, ~rows_seen] == 0)


def test_window_needs_the_causal_mask():
    q = _rand((1, 1, 3, 2), 86)
    with pytest.raises(ValueError):
        oracle.attention(q, q, q, scale=1.0, window=2)
