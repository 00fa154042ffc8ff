"""Pins of the norm oracle (oracle/norms.py) against mathematics: closed forms
of constant rows, exact power-of-two scaling, the stable two-pass form, library
special cases (numpy.linalg.norm, PyTorch's float64 rms_norm), brute force over
tiny integer rows, and the paper's two fusions (rolling update, Theorem 1;
split-k update, Theorem 2).  Planted mistakes in the fused forms are caught."""

import itertools
import math

import numpy as np
import pytest
import torch

from oracle import norms


def _rand(shape, seed, scale=1.0):
    return np.random.Generator(np.random.PCG64(seed)).standard_normal(shape) * scale


@pytest.mark.parametrize("c,M", [(3.0, 100), (-0.5, 7), (0.0, 5), (1e30, 64)])
def test_l2_constant_rows(c, M):
    x = np.full((2, M), c)
    np.testing.assert_allclose(norms.l2_norm(x), abs(c) * math.sqrt(M), rtol=1e-15)


@pytest.mark.parametrize("c,eps", [(2.0, 1e-6), (-3.0, 0.0), (0.25, 1e-3)])
def test_rmsnorm_constant_rows(c, eps):
    y, m = norms.rmsnorm_rowmax(np.full((3, 50), c), eps)
    expect = c / math.sqrt(c * c + eps)
    np.testing.assert_allclose(y, expect, rtol=1e-15)
    np.testing.assert_allclose(m, expect, rtol=1e-15)


def test_l2_power_of_two_scaling_is_exact():
    x = _rand((4, 300), 1)
    for k in (-40, -3, 5, 60):
        np.testing.assert_array_equal(norms.l2_norm(x * 2.0 ** k), norms.l2_norm(x) * 2.0 ** k)


def test_rmsnorm_scale_invariant_without_eps():
    x = _rand((4, 300), 2)
    y, m = norms.rmsnorm_rowmax(x, 0.0)
    y2, m2 = norms.rmsnorm_rowmax(x * 8.0, 0.0)
    np.testing.assert_allclose(y2, y, rtol=1e-14)
    y3, _ = norms.rmsnorm_rowmax(x * -4.0, 0.0)
    np.testing.assert_allclose(y3, -y, rtol=1e-14)
    np.testing.assert_allclose(m, y.max(axis=1), rtol=0)


def test_l2_matches_numpy_linalg_norm():
    x = _rand((9, 1000), 3, 7.0)
    np.testing.assert_allclose(norms.l2_norm(x), np.linalg.norm(x, axis=1), rtol=1e-14)


def test_rmsnorm_matches_torch_float64():
    x = _rand((6, 512), 4)
    y, m = norms.rmsnorm_rowmax(x, 1e-5)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (512,), eps=1e-5).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(m, ref.max(axis=1), rtol=1e-13)


def test_l2_equals_the_stable_two_pass_form():
    """||x|| = m sqrt(sum (x / m)^2), m = max |x| (the form the paper starts from)."""
    x = _rand((5, 777), 5, 1e20)
    m = np.abs(x).max(axis=1)
    np.testing.assert_allclose(norms.l2_norm(x), m * np.sqrt(((x / m[:, None]) ** 2).sum(axis=1)), rtol=1e-14)


def test_l2_brute_force_tiny_integer_rows():
    rows = np.array(list(itertools.product([-2, -1, 0, 1, 2], repeat=3)), dtype=np.float64)
    got = norms.l2_norm(rows)
    for row, g in zip(rows, got):
        assert g == math.sqrt(int(sum(int(v) ** 2 for v in row)))


@pytest.mark.parametrize("block", [1, 3, 8, 64, 5000])
def test_l2_rolling_equals_plain(block):
    """Theorem 1 for the L2 norm: r = max |x|, g = (c/r)^2, h = t (r/r')^2."""
    x = _rand((4, 1003), 6)
    x[1, :500] = 0.0                         # a zero prefix: r stays 0
    x[2] *= np.linspace(0.01, 10, 1003)      # the max grows along the row
    np.testing.assert_allclose(norms.l2_norm_rolling(x, block), norms.l2_norm(x), rtol=1e-13)


@pytest.mark.parametrize("block", [1, 4, 8, 64, 5000])
def test_rmsnorm_rolling_equals_plain(block):
    """Theorem 1 for the RMSNorm row max: r = mean, g = c/sqrt(r+eps), f = max,
    h = t sqrt(r+eps)/sqrt(r'+eps)."""
    x = _rand((4, 999), 7)
    x[3] = -np.abs(x[3])                     # an all-negative row: the max is negative
    _, m = norms.rmsnorm_rowmax(x, 1e-4)
    np.testing.assert_allclose(norms.rmsnorm_rowmax_rolling(x, 1e-4, block), m, rtol=1e-13)


@pytest.mark.parametrize("chunks", [1, 2, 7, 64, 1200])
def test_split_forms_equal_plain(chunks):
    """Theorem 2 for both reductions, including empty trailing chunks."""
    x = _rand((3, 1000), 8)
    np.testing.assert_allclose(norms.l2_norm_split(x, chunks), norms.l2_norm(x), rtol=1e-13)
    _, m = norms.rmsnorm_rowmax(x, 1e-6)
    np.testing.assert_allclose(norms.rmsnorm_rowmax_split(x, 1e-6, chunks), m, rtol=1e-13)


def test_split_local_partials_are_chunk_statistics():
    x = _rand((2, 100), 9)
    r, t = norms.l2_norm_split_local(x, 3, size=40)
    np.testing.assert_allclose(r[0, 1], np.abs(x[0, 40:80]).max(), rtol=0)
    np.testing.assert_allclose(t[1, 2] * r[1, 2] ** 2, (x[1, 80:] ** 2).sum(), rtol=1e-14)
    rr, tt = norms.rmsnorm_split_local(x, 0.5, 4, size=40)
    assert rr[0, 3] == 0.0 and np.isneginf(tt[0, 3])          # the empty fourth chunk
    np.testing.assert_allclose(rr[1, 0] * 100, (x[1, :40] ** 2).sum(), rtol=1e-14)


# planted mistakes in the fused forms

def test_missing_l2_repair_is_caught():
    x = _rand((2, 600), 10)
    x[:, 300:] *= 50.0                       # the max jumps half way
    saved = norms.l2_norm_rolling
    def broken(x, block=8):
        x = np.asarray(x, dtype=np.float64)
        out = []
        for row in x:
            r, t = 0.0, 0.0
            for a in range(0, len(row), block):
                c = row[a:a + block]
                r = max(r, float(np.abs(c).max()))
                t = t + float(((c / r) ** 2).sum())          # no h(t, r, r')
            out.append(r * math.sqrt(t))
        return np.array(out)
    assert np.allclose(saved(x), norms.l2_norm(x), rtol=1e-12)
    assert not np.allclose(broken(x), norms.l2_norm(x), rtol=1e-3)


def test_unsquared_l2_g_is_caught():
    x = _rand((2, 100), 11)
    m = np.abs(x).max(axis=1)
    wrong = m * np.sqrt(np.abs(x / m[:, None]).sum(axis=1))    # g = |c/r| instead of (c/r)^2
    assert not np.allclose(wrong, norms.l2_norm(x), rtol=1e-3)


def test_missing_rms_repair_is_caught():
    x = _rand((2, 600), 12)
    x[:, 300:] *= 20.0
    def broken(x, eps):
        out = []
        for row in np.asarray(x, dtype=np.float64):
            r, t = 0.0, -np.inf
            for a in range(0, len(row), 8):
                c = row[a:a + 8]
                r += float((c * c).sum()) / len(row)
                t = max(t, float((c / math.sqrt(r + eps)).max()))   # no h
            out.append(t)
        return np.array(out)
    _, m = norms.rmsnorm_rowmax(x, 1e-6)
    assert not np.allclose(broken(x, 1e-6), m, rtol=1e-3)
