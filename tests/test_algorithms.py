"""The paper's two fusions, run in float64, against the plain definition.

Theorem 1 (rolling update) and Theorem 2 (split-k update) say the repaired
programs compute the same values as the unfused one over the reals; in
float64 they must agree to ~1e-12.  The tag-updating Lemma / Eq.
example-result fix the state after every tile: the repaired running sum equals
the plain prefix sum taken with the current running max.
"""

import math

import numpy as np
import pytest

import oracle
from oracle import rolling, splitk
from paper_2510_08726_amd.workloads import alibi_slopes


def _rand(shape, seed):
    return np.random.Generator(np.random.PCG64(seed)).standard_normal(shape)


CASES = [  # Lq, Lk, Hq, Hkv, causal, alibi
    (40, 40, 2, 2, False, False),
    (40, 40, 2, 2, True, False),
    (23, 57, 4, 2, True, False),
    (37, 37, 4, 1, True, True),
    (1, 77, 4, 2, True, True),
]


@pytest.mark.parametrize("block_n", [1, 3, 16, 32, 64, 200])
@pytest.mark.parametrize("case", CASES)
def test_rolling_update_equals_plain_definition(case, block_n):
    Lq, Lk, Hq, Hkv, causal, alibi = case
    q, k, v = _rand((1, Hq, Lq, 8), 1), _rand((1, Hkv, Lk, 8), 2), _rand((1, Hkv, Lk, 8), 3)
    sl = alibi_slopes(Hq).double().numpy() if alibi else None
    ref = oracle.attention(q, k, v, scale=0.35, causal=causal, alibi_slopes=sl)
    for hq in range(Hq):
        o = rolling.rolling_update_attention(q, k, v, scale=0.35, causal=causal,
                                             alibi_slopes=sl, block_n=block_n, hq=hq)
        np.testing.assert_allclose(o, ref[0, hq], atol=1e-12, rtol=0)


def test_rolling_update_prefix_state_after_every_tile():
    """After tile t the state is plain softmax statistics of the first keys."""
    Lq, Lk, bn = 9, 50, 8
    q, k, v = _rand((1, 1, Lq, 4), 4), _rand((1, 1, Lk, 4), 5), _rand((1, 1, Lk, 4), 6)
    _, states = rolling.rolling_update_attention(q, k, v, scale=0.8, block_n=bn, trace=True)
    s = oracle.scores(q, k, scale=0.8)
    for t, (xmax, xsum, acc) in enumerate(states):
        n = min((t + 1) * bn, Lk)
        m = s[:, :n].max(axis=1, keepdims=True)
        e = np.exp(s[:, :n] - m)
        np.testing.assert_allclose(xmax, m, atol=0)
        np.testing.assert_allclose(xsum, e.sum(axis=1, keepdims=True), rtol=1e-13)
        np.testing.assert_allclose(acc / xsum, oracle.attention(q, k[:, :, :n], v[:, :, :n],
                                                                scale=0.8)[0, 0], atol=1e-13)


def test_motivating_example_prefix_repaired_sums():
    """Eq. example-result: after iteration j, xsum = sum_{j' <= j} exp(x_ij' - m_i<j>)."""
    x = _rand((2, 4), 7) * 3
    # one row of attention scores = x when q = e_0 and k_j = x_j e_0, scale 1
    for i in range(2):
        q = np.zeros((1, 1, 1, 1)) + 1.0
        k = x[i].reshape(1, 1, 4, 1)
        _, states = rolling.rolling_update_attention(q, k, k, scale=1.0, block_n=1, trace=True)
        for j, (xmax, xsum, _) in enumerate(states):
            m = max(x[i, :j + 1])
            assert xmax.item() == m
            assert abs(xsum.item() - sum(math.exp(x[i, jj] - m) for jj in range(j + 1))) < 1e-13


@pytest.mark.parametrize("S", [1, 2, 3, 16, 64, 77, 100])
@pytest.mark.parametrize("case", CASES)
def test_split_k_equals_plain_definition(case, S):
    Lq, Lk, Hq, Hkv, causal, alibi = case
    q, k, v = _rand((2, Hq, Lq, 8), 8), _rand((2, Hkv, Lk, 8), 9), _rand((2, Hkv, Lk, 8), 10)
    sl = alibi_slopes(Hq).double().numpy() if alibi else None
    ref = oracle.attention(q, k, v, scale=0.35, causal=causal, alibi_slopes=sl)
    o = splitk.split_k_attention(q, k, v, scale=0.35, num_splits=S, causal=causal,
                                 alibi_slopes=sl)
    np.testing.assert_allclose(o, ref, atol=1e-12, rtol=0)


def test_split_k_chunks_ragged_and_empty():
    assert splitk.chunk_bounds(10, 4) == [(0, 3), (3, 6), (6, 9), (9, 10)]
    assert splitk.chunk_bounds(10, 6) == [(0, 2), (2, 4), (4, 6), (6, 8), (8, 10), (10, 10)]
    q, k, v = _rand((1, 2, 1, 4), 11), _rand((1, 1, 10, 4), 12), _rand((1, 1, 10, 4), 13)
    o_l, m_l, s_l = splitk.split_local(q, k, v, scale=0.5, num_splits=6)
    assert np.isneginf(m_l[..., 5]).all() and (s_l[..., 5] == 0).all() and (o_l[..., 5, :] == 0).all()
    ref = oracle.attention(q, k, v, scale=0.5)
    np.testing.assert_allclose(splitk.split_global(o_l, m_l, s_l), ref, atol=1e-13)


def test_split_k_global_invariant_under_chunk_permutation():
    q, k, v = _rand((1, 2, 1, 4), 14), _rand((1, 2, 90, 4), 15), _rand((1, 2, 90, 4), 16)
    o_l, m_l, s_l = splitk.split_local(q, k, v, scale=0.5, num_splits=7)
    perm = np.random.Generator(np.random.PCG64(0)).permutation(7)
    a = splitk.split_global(o_l, m_l, s_l)
    b = splitk.split_global(o_l[..., perm, :], m_l[..., perm], s_l[..., perm])
    np.testing.assert_allclose(a, b, atol=1e-14)


def test_split_local_partials_are_plain_chunk_softmax():
    """Each local partial is the unrepaired softmax statistics of its chunk alone."""
    q, k, v = _rand((1, 1, 1, 4), 17), _rand((1, 1, 30, 4), 18), _rand((1, 1, 30, 4), 19)
    o_l, m_l, s_l = splitk.split_local(q, k, v, scale=0.9, num_splits=4)
    s = oracle.scores(q, k, scale=0.9)[0]
    for c, (lo, hi) in enumerate(splitk.chunk_bounds(30, 4)):
        assert m_l[0, 0, 0, c] == s[lo:hi].max()
        np.testing.assert_allclose(o_l[0, 0, 0, c] / s_l[0, 0, 0, c],
                                   oracle.attention(q, k[:, :, lo:hi], v[:, :, lo:hi], scale=0.9)[0, 0, 0],
                                   atol=1e-13)


@pytest.mark.parametrize("S", [1, 3, 16, 77])
@pytest.mark.parametrize("alibi", [False, True])
def test_split_k_with_softcap_equals_plain_definition(S, alibi):
    """Theorem 2 does not depend on the score modifier: with SoftCap (and GQA)
    the repaired split-k program still equals the plain definition."""
    q, k, v = _rand((2, 8, 1, 8), 51) * 3, _rand((2, 2, 77, 8), 52) * 3, _rand((2, 2, 77, 8), 53)
    sl = alibi_slopes(8).double().numpy() if alibi else None
    ref = oracle.attention(q, k, v, scale=0.35, causal=True, alibi_slopes=sl, softcap=2.5)
    o = splitk.split_k_attention(q, k, v, scale=0.35, num_splits=S, causal=True,
                                 alibi_slopes=sl, softcap=2.5)
    np.testing.assert_allclose(o, ref, atol=1e-12, rtol=0)
    plain = oracle.attention(q, k, v, scale=0.35, causal=True, alibi_slopes=sl)
    assert np.abs(ref - plain).max() > 1e-2          # the cap changes the result at these scores


@pytest.mark.parametrize("W,block_n", [(1, 4), (7, 8), (40, 16)])
def test_rolling_update_with_window_equals_plain_definition(W, block_n):
    """Theorem 1 holds for any mask: the rolling update over the windowed scores."""
    q, k, v = _rand((1, 2, 33, 8), 91), _rand((1, 2, 45, 8), 92), _rand((1, 2, 45, 8), 93)
    ref = oracle.attention(q, k, v, scale=0.4, causal=True, window=W)
    for hq in range(2):
        got = rolling.rolling_update_attention(q, k, v, scale=0.4, causal=True, window=W, block_n=block_n, hq=hq)
        np.testing.assert_allclose(got, ref[0, hq], atol=1e-12)
