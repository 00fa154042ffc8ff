"""Planted mistakes in the oracle must be caught by its pins (CPU only).

Each mutant is the oracle with one plausible error: a transposed or swapped
operand, a dropped scale, a wrong bias sign, a wrong causal alignment, a wrong
GQA head map, a missing repair factor.  The pins in ``test_oracle_pins`` /
``test_algorithms`` must reject every one of them; this guards against pins
that are too weak to notice a broken oracle.
"""

import math

import numpy as np

import oracle
from oracle import rolling
from paper_2510_08726_amd.workloads import alibi_slopes


def _rand(shape, seed):
    return np.random.Generator(np.random.PCG64(seed)).standard_normal(shape)


def _one_hot_pin(attn):
    D, Lk = 8, 40
    rng = np.random.Generator(np.random.PCG64(7))
    k = rng.standard_normal((1, 1, Lk, D)) * 0.1
    v = rng.standard_normal((1, 1, Lk, D))
    q = np.zeros((1, 1, 1, D))
    q[0, 0, 0, 0] = 1.0
    k[0, 0, Lk - 1, 0] = 40.0
    o = attn(q, k, v, scale=1.0)
    return np.allclose(o[0, 0, 0], v[0, 0, Lk - 1], atol=1e-6)


def _logistic_pin(attn):
    q, k, v = _rand((1, 1, 3, 5), 11), _rand((1, 1, 2, 5), 12), _rand((1, 1, 2, 5), 13)
    o = attn(q, k, v, scale=0.37)
    for i in range(3):
        s = [0.37 * float(q[0, 0, i] @ k[0, 0, j]) for j in range(2)]
        w0 = 1.0 / (1.0 + math.exp(s[1] - s[0]))
        if not np.allclose(o[0, 0, i], w0 * v[0, 0, 0] + (1 - w0) * v[0, 0, 1], atol=1e-12):
            return False
    return True


def _alibi_pin(attn):
    H, L = 2, 7
    q, k, v = _rand((1, H, L, 2), 17), _rand((1, H, L, 2), 18), _rand((1, H, L, 2), 19)
    sl = alibi_slopes(H).double().numpy()
    o = attn(q, k, v, scale=0.0, causal=True, alibi_slopes=sl)
    for h in range(H):
        r = math.exp(-sl[h])
        for i in range(L):
            w = np.array([r ** (i - j) for j in range(i + 1)])
            if not np.allclose(o[0, h, i], (w[:, None] * v[0, h, :i + 1]).sum(0) / w.sum(), atol=1e-12):
                return False
    return True


def _prefix_mean_pin(attn):
    q, k, v = _rand((1, 1, 5, 3), 14), _rand((1, 1, 12, 3), 15), _rand((1, 1, 12, 3), 16)
    o = attn(q, k, v, scale=0.0, causal=True)
    return all(np.allclose(o[0, 0, i], v[0, 0, :i + 8].mean(0), atol=1e-13) for i in range(5))


def _gqa_pin(attn):
    q, k, v = _rand((1, 4, 6, 4), 23), _rand((1, 2, 6, 4), 24), _rand((1, 2, 6, 4), 25)
    o = attn(q, k, v, scale=0.3)
    ref = oracle.attention(q[:, :1], k[:, :1], v[:, :1], scale=0.3)   # hq 0 -> hk 0
    ref1 = oracle.attention(q[:, 1:2], k[:, :1], v[:, :1], scale=0.3)  # hq 1 -> hk 0
    return np.allclose(o[:, :1], ref, atol=1e-13) and np.allclose(o[:, 1:2], ref1, atol=1e-13)


PINS = [_one_hot_pin, _logistic_pin, _alibi_pin, _prefix_mean_pin, _gqa_pin]


def test_true_oracle_passes_every_pin():
    for pin in PINS:
        assert pin(oracle.attention), pin.__name__


def _caught(mutant):
    return any(not pin(mutant) for pin in PINS)


def test_mutant_qv_instead_of_qk_is_caught():
    assert _caught(lambda q, k, v, **kw: oracle.attention(q, v, v, **kw))


def test_mutant_dropped_scale_is_caught():
    assert _caught(lambda q, k, v, scale, **kw: oracle.attention(q, k, v, scale=1.0, **kw))


def test_mutant_alibi_sign_is_caught():
    def m(q, k, v, alibi_slopes=None, **kw):
        sl = None if alibi_slopes is None else -np.asarray(alibi_slopes)
        return oracle.attention(q, k, v, alibi_slopes=sl, **kw)
    assert _caught(m)


def test_mutant_top_left_causal_is_caught():
    def m(q, k, v, causal=False, **kw):
        if not causal:
            return oracle.attention(q, k, v, **kw)
        Lq, Lk = q.shape[2], k.shape[2]
        out = np.zeros(q.shape)
        for i in range(Lq):                      # row i sees keys 0..i (top-left)
            out[:, :, i:i + 1] = oracle.attention(q[:, :, i:i + 1], k[:, :, :i + 1], v[:, :, :i + 1], **kw)
        return out
    assert _caught(m)


def test_mutant_interleaved_gqa_map_is_caught():
    def m(q, k, v, **kw):
        G = q.shape[1] // k.shape[1]
        return oracle.attention(q, np.tile(k, (1, G, 1, 1)), np.tile(v, (1, G, 1, 1)), **kw)
    assert _caught(m)


def test_mutant_missing_repair_factor_is_caught():
    """Rolling update without h (alpha = 1) breaks Theorem 1."""
    q, k, v = _rand((1, 1, 4, 8), 1), _rand((1, 1, 64, 8), 2), _rand((1, 1, 64, 8), 3)
    ref = oracle.attention(q, k, v, scale=0.5)[0, 0]
    saved = rolling._repair
    try:
        rolling._repair = lambda prev, cur: np.ones_like(cur)
        bad = rolling.rolling_update_attention(q, k, v, scale=0.5, block_n=16)
    finally:
        rolling._repair = saved
    assert not np.allclose(bad, ref, atol=1e-6)
    good = rolling.rolling_update_attention(q, k, v, scale=0.5, block_n=16)
    np.testing.assert_allclose(good, ref, atol=1e-12)


# SoftCap score modifier: cap * tanh(scale * q.k / cap), then the bias, then the mask.

def _softcap_saturated_pin(attn):
    """|scale q.k| >> cap: every capped score is +-cap exactly, a closed form in e^cap."""
    cap, Lk = 2.0, 5
    v = _rand((1, 1, Lk, 3), 41)
    q = np.zeros((1, 1, 1, 3))
    q[..., 0] = 1.0
    k = np.zeros((1, 1, Lk, 3))
    k[0, 0, :, 0] = -1e3
    k[0, 0, 0, 0] = 1e3
    o = attn(q, k, v, scale=1.0, softcap=cap)
    w = np.array([math.exp(cap)] + [math.exp(-cap)] * (Lk - 1))
    return np.allclose(o[0, 0, 0], (w[:, None] * v[0, 0]).sum(0) / w.sum(), atol=1e-12)


def _softcap_series_pin(attn):
    """|x| <= 1 << cap: cap tanh(x / cap) = x - x^3/(3 cap^2) + 2 x^5/(15 cap^4) + O(x^7 / cap^6)."""
    cap, Lk = 4.0, 9
    x = np.linspace(-1.0, 1.0, Lk)
    v = _rand((1, 1, Lk, 3), 42)
    q = np.zeros((1, 1, 1, 3))
    q[..., 0] = 1.0
    k = np.zeros((1, 1, Lk, 3))
    k[0, 0, :, 0] = x
    o = attn(q, k, v, scale=1.0, softcap=cap)
    t = x - x ** 3 / (3 * cap ** 2) + 2 * x ** 5 / (15 * cap ** 4)   # remainder < 17 / (315 cap^6) = 1.3e-5
    w = np.exp(t - t.max())
    return np.allclose(o[0, 0, 0], (w[:, None] * v[0, 0]).sum(0) / w.sum(), atol=5e-5)


def _softcap_huge_cap_pin(attn):
    """cap -> infinity gives plain attention."""
    q, k, v = _rand((1, 2, 6, 4), 43), _rand((1, 2, 9, 4), 44), _rand((1, 2, 9, 4), 45)
    o = attn(q, k, v, scale=0.5, causal=True, softcap=1e8)
    return np.allclose(o, oracle.attention(q, k, v, scale=0.5, causal=True), atol=1e-9)


def _softcap_alibi_pin(attn):
    """scale 0 caps nothing (tanh 0 = 0), so the ALiBi geometric closed form holds
    exactly: the bias is added after the cap and the mask comes last."""
    H, L = 2, 7
    q, k, v = _rand((1, H, L, 2), 46), _rand((1, H, L, 2), 47), _rand((1, H, L, 2), 48)
    sl = alibi_slopes(H).double().numpy()
    o = attn(q, k, v, scale=0.0, causal=True, alibi_slopes=sl, softcap=1.5)
    for h in range(H):
        r = math.exp(-sl[h])
        for i in range(L):
            w = np.array([r ** (i - j) for j in range(i + 1)])
            if not np.allclose(o[0, h, i], (w[:, None] * v[0, h, :i + 1]).sum(0) / w.sum(), atol=1e-12):
                return False
    return True


SOFTCAP_PINS = [_softcap_saturated_pin, _softcap_series_pin, _softcap_huge_cap_pin, _softcap_alibi_pin]
_ATT = __import__("sys").modules["oracle.attention"]   # the module (oracle.attention is the function)


def _patched(name, fn):
    """The oracle with one of its module functions replaced by a planted mistake."""
    def mutant(*args, **kw):
        saved = getattr(_ATT, name)
        setattr(_ATT, name, fn)
        try:
            return oracle.attention(*args, **kw)
        finally:
            setattr(_ATT, name, saved)
    return mutant


def test_true_oracle_passes_every_softcap_pin():
    for pin in SOFTCAP_PINS:
        assert pin(oracle.attention), pin.__name__


def _softcap_caught(mutant):
    return any(not pin(mutant) for pin in SOFTCAP_PINS)


def test_mutant_softcap_ignored_is_caught():
    assert _softcap_caught(_patched("_softcap", lambda x, cap: x))


def test_mutant_softcap_missing_outer_cap_is_caught():
    assert _softcap_caught(_patched("_softcap", lambda x, cap: np.tanh(x / cap)))


def test_mutant_softcap_missing_inner_division_is_caught():
    assert _softcap_caught(_patched("_softcap", lambda x, cap: cap * np.tanh(x)))


def _scores_in_order(bias_inside, mask_first):
    base = _ATT.scores

    def scores(q, k, *, scale, causal=False, alibi_slopes=None, softcap=None, window=None, b=0, hq=0,
               rows=None):
        if not softcap:
            return base(q, k, scale=scale, causal=causal, alibi_slopes=alibi_slopes, b=b, hq=hq, rows=rows)
        raw = base(q, k, scale=scale, causal=False, alibi_slopes=alibi_slopes if bias_inside else None,
                   b=b, hq=hq, rows=rows)
        Lq, Lk = q.shape[2], k.shape[2]
        i = np.arange(Lq) if rows is None else np.asarray(rows)
        visible = np.arange(Lk)[None, :] <= i[:, None] + (Lk - Lq)
        if causal and mask_first:
            raw = np.where(visible, raw, -np.inf)
        s = softcap * np.tanh(raw / softcap)
        if alibi_slopes is not None and not bias_inside:
            s = s - float(alibi_slopes[hq]) * (i[:, None] + (Lk - Lq) - np.arange(Lk)[None, :])
        if causal and not mask_first:
            s = np.where(visible, s, -np.inf)
        return s
    return scores


def test_mutant_softcap_bias_inside_the_cap_is_caught():
    assert _softcap_caught(_patched("scores", _scores_in_order(bias_inside=True, mask_first=False)))


def test_mutant_softcap_mask_before_the_cap_is_caught():
    assert _softcap_caught(_patched("scores", _scores_in_order(bias_inside=False, mask_first=True)))


def test_softcap_planted_order_helper_matches_oracle_when_correct():
    """The helper that builds the two order mutants is itself right when given the right order."""
    good = _patched("scores", _scores_in_order(bias_inside=False, mask_first=False))
    assert all(pin(good) for pin in SOFTCAP_PINS)


# ---------------------------------------------------------------------------
# sliding window: the band pins must reject an off-by-one edge, a band on
# the wrong side of the diagonal and a window that is ignored

def _window_one_pin(attn):
    """W = 1: every row with a key at its own position returns that V row."""
    q, k, v = _rand((1, 2, 9, 4), 41), _rand((1, 2, 12, 4), 42), _rand((1, 2, 12, 4), 43)
    o = attn(q, k, v, scale=0.8, causal=True, window=1)
    return all(np.allclose(o[0, h, i], v[0, h, i + 3], atol=1e-13) for h in range(2) for i in range(9))


def _band_mean_pin(attn):
    """scale = 0: row i averages V over keys max(0, i_abs - W + 1) .. i_abs."""
    W = 4
    q, k, v = _rand((1, 1, 7, 3), 44), _rand((1, 1, 10, 3), 45), _rand((1, 1, 10, 3), 46)
    o = attn(q, k, v, scale=0.0, causal=True, window=W)
    for i in range(7):
        ia = i + 3
        band = [v[0, 0, j] for j in range(max(0, ia - W + 1), ia + 1)]
        if not np.allclose(o[0, 0, i], sum(band) / len(band), atol=1e-13):
            return False
    return True


WINDOW_PINS = [_window_one_pin, _band_mean_pin]


def _windowed(edge):
    """Oracle with the band edge replaced: edge(j, i_abs, W) -> visible."""
    base = _ATT.scores

    def scores(q, k, *, scale, causal=False, alibi_slopes=None, softcap=None, window=None, b=0, hq=0,
               rows=None):
        s = base(q, k, scale=scale, causal=causal, alibi_slopes=alibi_slopes, softcap=softcap, b=b, hq=hq,
                 rows=rows)
        if not window:
            return s
        Lq, Lk = q.shape[2], k.shape[2]
        i = (np.arange(Lq) if rows is None else np.asarray(rows))[:, None] + (Lk - Lq)
        return np.where(edge(np.arange(Lk)[None, :], i, int(window)), s, -np.inf)
    return _patched("scores", scores)


def test_true_oracle_passes_every_window_pin():
    for pin in WINDOW_PINS:
        assert pin(oracle.attention), pin.__name__


def test_window_helper_matches_oracle_when_correct():
    good = _windowed(lambda j, i, W: j > i - W)
    assert all(pin(good) for pin in WINDOW_PINS)


def test_mutant_window_off_by_one_is_caught():
    assert any(not pin(_windowed(lambda j, i, W: j >= i - W)) for pin in WINDOW_PINS)


def test_mutant_window_on_the_wrong_side_is_caught():
    assert any(not pin(_windowed(lambda j, i, W: j < i + W)) for pin in WINDOW_PINS)


def test_mutant_window_ignored_is_caught():
    assert any(not pin(_windowed(lambda j, i, W: np.ones_like(j - i, dtype=bool))) for pin in WINDOW_PINS)


# ---------------------------------------------------------------------------
# softmax_probs: a max taken over the wrong axis keeps row sums at 1 but not
# the values, which the Lk = 2 logistic pin of the probabilities checks

def _probs_logistic_pin(probs):
    q, k = _rand((1, 1, 4, 5), 51), _rand((1, 1, 2, 5), 52)
    p = probs(q, k, scale=0.6)
    for i in range(4):
        s = [0.6 * math.fsum(float(q[0, 0, i, d]) * float(k[0, 0, j, d]) for d in range(5)) for j in range(2)]
        if not np.isclose(p[i, 0], 1.0 / (1.0 + math.exp(s[1] - s[0])), atol=1e-13, rtol=0):
            return False
    return True


def test_true_softmax_probs_passes_logistic_pin():
    assert _probs_logistic_pin(oracle.softmax_probs)


def test_mutant_softmax_max_over_wrong_axis_is_caught():
    def probs(q, k, **kw):
        score = oracle.scores(q, k, **kw)
        m = score.max(axis=0, keepdims=True)          # column max instead of row max
        e = np.exp(score - m)
        return e / e.sum(axis=1, keepdims=True)
    p = probs(_rand((1, 1, 4, 5), 51), _rand((1, 1, 2, 5), 52), scale=0.6)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-12)   # row sums do not notice
    assert not _probs_logistic_pin(probs)
