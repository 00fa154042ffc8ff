"""GPU parity of the single-pass row reductions (norms.h) against the fp64
oracle: the stable L2 norm and RMSNorm with its row max, every dtype, ragged
and empty chunks, the chunk partials element by element, values whose squares
overflow fp32, and the full-size workloads on every row."""

import numpy as np
import pytest
import torch

import paper_2510_08726_amd as pa
from oracle import norms
from paper_2510_08726_amd.workloads import NORM_DTYPES, NORM_WORKLOADS, make_norm_input, NormWorkload
from kernel_cases import NORM_CASES as CASES

pytestmark = pytest.mark.gpu

# fp32 statistics: a few ulps of fp32 per operation over up to 2^17 terms.
RTOL_STAT = 2e-5
# y is rounded to the input type: half an ulp, relative.
RTOL_Y = {"f16": 2.0 ** -11, "bf16": 2.0 ** -8, "f32": 2e-6}

def _x(N, M, dt, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    return torch.from_numpy(rng.standard_normal(size=(N, M), dtype=np.float32)).to(NORM_DTYPES[dt])


def _chunk_size(M, C, dt):
    vec = 4 if dt == "f32" else 8
    per = -(-M // C)
    return -(-per // vec) * vec


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
def test_l2_norm_matches_oracle(case):
    N, M, dt, C = case
    print(f"l2 norm case {case}", flush=True)
    x = _x(N, M, dt, 300 + N)
    xd = x.cuda()
    Cres = C or pa.norm_chunks("l2", N, M, x.dtype)
    ws = torch.empty(pa.norm_workspace_bytes(N, Cres), dtype=torch.uint8, device="cuda")
    out = pa.norm_l2(xd, chunks=C, workspace=ws)
    torch.cuda.synchronize()
    x64 = x.double().numpy()
    np.testing.assert_allclose(out.cpu().double().numpy(), norms.l2_norm(x64), rtol=RTOL_STAT)
    # the local nests, element by element
    r, t = (a.cpu().double().numpy() for a in pa.norm_partials(ws, N, Cres))
    rr, tt = norms.l2_norm_split_local(x64, Cres, size=_chunk_size(M, Cres, dt))
    np.testing.assert_array_equal(r, rr)                  # max |x|: exact
    np.testing.assert_allclose(t, tt, rtol=RTOL_STAT, atol=1e-30)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
def test_rmsnorm_rowmax_matches_oracle(case):
    N, M, dt, C = case
    print(f"rmsnorm case {case}", flush=True)
    eps = 1e-5
    x = _x(N, M, dt, 400 + N)
    xd = x.cuda()
    Cres = C or pa.norm_chunks("rms", N, M, x.dtype)
    ws = torch.empty(pa.norm_workspace_bytes(N, Cres), dtype=torch.uint8, device="cuda")
    y, m = pa.rmsnorm_rowmax(xd, eps=eps, chunks=C, workspace=ws)
    torch.cuda.synchronize()
    x64 = x.double().numpy()
    yr, mr = norms.rmsnorm_rowmax(x64, eps)
    yg = y.cpu().double().numpy()
    assert np.all(np.abs(yg - yr) <= RTOL_Y[dt] * np.abs(yr) + 1e-6)
    np.testing.assert_allclose(m.cpu().double().numpy(), mr, rtol=RTOL_STAT)
    r, t = (a.cpu().double().numpy() for a in pa.norm_partials(ws, N, Cres))
    rr, tt = norms.rmsnorm_split_local(x64, eps, Cres, size=_chunk_size(M, Cres, dt))
    np.testing.assert_allclose(r, rr, rtol=RTOL_STAT, atol=1e-30)
    assert np.array_equal(np.isneginf(t), np.isneginf(tt))
    live = ~np.isneginf(tt)
    np.testing.assert_allclose(t[live], tt[live], rtol=RTOL_STAT)


def test_l2_norm_of_values_whose_squares_overflow_fp32():
    """Entries near 1e30 (squares 1e60, far past fp32): the stable single pass
    still returns the norm (the naive sum of squares would be inf)."""
    x = _x(6, 2048, "f32", 500) * 1e30
    x[2, 100] = 3e37
    out = pa.norm_l2(x.cuda())
    torch.cuda.synchronize()
    got = out.cpu().double().numpy()
    assert np.all(np.isfinite(got))
    assert bool(torch.isinf((x.cuda() * x.cuda()).sum(dim=1)).all())
    np.testing.assert_allclose(got, norms.l2_norm(x.double().numpy()), rtol=RTOL_STAT)


def test_constant_and_zero_rows():
    x = torch.zeros(4, 512, dtype=torch.float32)
    x[1] = 3.0
    x[2] = -0.5
    out = pa.norm_l2(x.cuda())
    y, m = pa.rmsnorm_rowmax(x.cuda(), eps=1e-6)
    torch.cuda.synchronize()
    np.testing.assert_allclose(out.cpu().numpy(), [0.0, 3.0 * 512 ** 0.5, 0.5 * 512 ** 0.5, 0.0], rtol=1e-6)
    np.testing.assert_allclose(m.cpu().numpy(), [0.0, 3.0 / (9.0 + 1e-6) ** 0.5, -0.5 / (0.25 + 1e-6) ** 0.5, 0.0],
                               rtol=1e-6)
    assert torch.all(y[0] == 0) and torch.all(y[3] == 0)


def test_is_deterministic():
    x = _x(16, 10000, "bf16", 600).cuda()
    a = pa.norm_l2(x)
    b = pa.norm_l2(x)
    y1, m1 = pa.rmsnorm_rowmax(x)
    y2, m2 = pa.rmsnorm_rowmax(x)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(y1, y2) and torch.equal(m1, m2)


@pytest.mark.parametrize("name", list(NORM_WORKLOADS))
def test_norm_workload_full(name):
    """The full-size workloads (N 256, M 2^17) on every row and element."""
    w = NORM_WORKLOADS[name]
    print(f"norm workload {name}", flush=True)
    x = make_norm_input(w)
    x64 = x.double().numpy()
    if w.op == "l2":
        out = pa.norm_l2(x.cuda())
        torch.cuda.synchronize()
        np.testing.assert_allclose(out.cpu().double().numpy(), norms.l2_norm(x64), rtol=RTOL_STAT)
    else:
        y, m = pa.rmsnorm_rowmax(x.cuda(), eps=w.eps)
        torch.cuda.synchronize()
        yr, mr = norms.rmsnorm_rowmax(x64, w.eps)
        yg = y.cpu().double().numpy()
        assert np.all(np.abs(yg - yr) <= RTOL_Y[w.dtype] * np.abs(yr) + 1e-6)
        np.testing.assert_allclose(m.cpu().double().numpy(), mr, rtol=RTOL_STAT)
