"""Seeded random sweep of the GPU path against the fp64 oracle: shapes, head
groupings, dtypes and every supported combination of the score and mask
modifiers, drawn per case from a fixed seed (the same cases on every run).
Complements the hand-picked cases of the other GPU tests with corners they
do not name (ragged tiles against ragged chunks, Lq != Lk with a window,
odd split counts with a bias and a cap, rows whose length leaves most lanes
of a one-pass norm idle)."""

import numpy as np
import pytest
import torch

import paper_2510_08726_amd as pa
from gpu_common import MAX_ABS, MEAN_ABS, errors, host32, oracle_fwd
from oracle import norms
from paper_2510_08726_amd.workloads import NORM_DTYPES, alibi_slopes, random_tensors

pytestmark = pytest.mark.gpu

N_CASES = 48


def assert_close_attributed(got, ref, dt, what):
    """The gate of the other parity tests (max-abs <= 1e-2, mean-abs <= 1e-3
    against the fp64 oracle), except that a bf16 output may exceed the max-abs
    gate where the excess is the output type's own quantum: every element past
    the gate must be one of the two bf16 neighbours of the exact value (bf16
    keeps 8 significant bits, so near |O| = 2-4 its spacing is 2^-6 and a
    faithful rounding can already miss by 0.0156).  The mean-abs gate holds
    for every dtype."""
    got = np.asarray(got, dtype=np.float64)
    e = errors(got, ref)
    print(f"{what}: " + " ".join(f"{k}={v:.3e}" for k, v in e.items()), flush=True)
    assert e["mean_abs"] <= MEAN_ABS, (what, e)
    if e["max_abs"] <= MAX_ABS:
        return
    assert dt == "bf16", (what, e)
    d = np.abs(got - ref)
    over = d > MAX_ABS
    ulp = np.exp2(np.floor(np.log2(np.abs(ref[over]))) - 7)   # bf16 spacing at |ref|
    assert np.all(d[over] < ulp), (what, e, "not a faithful bf16 rounding")
    print(f"{what}: {int(over.sum())} element(s) past the max-abs gate, each a bf16 neighbour of the exact value",
          flush=True)


def _prefill_case(i):
    rng = np.random.default_rng(7000 + i)
    D = int(rng.choice([64, 128]))
    dt = str(rng.choice(["f16", "bf16"]))
    Hkv = int(rng.choice([1, 2, 4]))
    G = int(rng.choice([1, 2, 3, 4, 8]))
    B = int(rng.integers(1, 3))
    Lq = int(rng.integers(1, 400))
    Lk = int(rng.integers(1, 400))
    causal = bool(rng.random() < 0.7)
    alibi = bool(rng.random() < 0.35)
    cap = float(rng.uniform(0.5, 8.0)) if causal and not alibi and rng.random() < 0.35 else None
    window = int(rng.integers(1, Lk + 20)) if causal and rng.random() < 0.3 else None
    scale = D ** -0.5 if rng.random() < 0.8 else float(rng.uniform(-0.3, 0.6))
    return dict(B=B, Hq=Hkv * G, Hkv=Hkv, Lq=Lq, Lk=Lk, D=D, dt=dt, causal=causal, alibi=alibi,
                cap=cap, window=window, scale=scale, seed=7000 + i)


def _decode_case(i):
    rng = np.random.default_rng(8000 + i)
    D = int(rng.choice([64, 128]))
    dt = str(rng.choice(["f16", "bf16"]))
    Hkv = int(rng.choice([1, 2, 4]))
    G = int(rng.choice([1, 2, 4, 5, 8, 16, 34]))
    B = int(rng.integers(1, 4))
    Lk = int(rng.integers(1, 5000))
    alibi = bool(rng.random() < 0.35)
    cap = float(rng.uniform(0.5, 8.0)) if rng.random() < 0.35 else None
    S = int(rng.choice([0, 1, 2, 3, 7, 16]))
    scale = D ** -0.5 if rng.random() < 0.8 else float(rng.uniform(-0.3, 0.6))
    return dict(B=B, Hq=Hkv * G, Hkv=Hkv, Lk=Lk, D=D, dt=dt, alibi=alibi, cap=cap, S=S, scale=scale,
                seed=8000 + i)


def _norm_case(i):
    rng = np.random.default_rng(9000 + i)
    dt = str(rng.choice(["f16", "bf16", "f32"]))
    vec = 4 if dt == "f32" else 8
    N = int(rng.integers(1, 300))
    M = vec * int(rng.integers(1, max(2, min(70000, 2_000_000 // N) // vec)))
    C = int(rng.choice([0, 1, 2, 3, 5]))
    return dict(N=N, M=M, dt=dt, C=C, seed=9000 + i)


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_prefill(i):
    c = _prefill_case(i)
    print(f"random prefill {c}", flush=True)
    q, = random_tensors([(c["B"], c["Hq"], c["Lq"], c["D"])], c["dt"], c["seed"])
    k, v = random_tensors([(c["B"], c["Hkv"], c["Lk"], c["D"])] * 2, c["dt"], c["seed"] + 1)
    sl = alibi_slopes(c["Hq"]) if c["alibi"] else None
    dev = torch.device("cuda")
    o = pa.attn_fwd(q.to(dev), k.to(dev), v.to(dev), causal=c["causal"], scale=c["scale"],
                    alibi_slopes=None if sl is None else sl.to(dev), softcap=c["cap"], window=c["window"])
    torch.cuda.synchronize()
    ref = oracle_fwd(q, k, v, scale=c["scale"], causal=c["causal"], slopes=sl, softcap=c["cap"],
                     window=c["window"])
    assert_close_attributed(host32(o), ref, c["dt"], f"random prefill {i}")


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_decode(i):
    c = _decode_case(i)
    print(f"random decode {c}", flush=True)
    q, = random_tensors([(c["B"], c["Hq"], 1, c["D"])], c["dt"], c["seed"])
    k, v = random_tensors([(c["B"], c["Hkv"], c["Lk"], c["D"])] * 2, c["dt"], c["seed"] + 1)
    sl = alibi_slopes(c["Hq"]) if c["alibi"] else None
    dev = torch.device("cuda")
    o = pa.attn_decode(q.to(dev), k.to(dev), v.to(dev), scale=c["scale"],
                       alibi_slopes=None if sl is None else sl.to(dev), softcap=c["cap"], num_splits=c["S"])
    torch.cuda.synchronize()
    # decode is the last query row of causal attention over all Lk keys
    ref = oracle_fwd(q, k, v, scale=c["scale"], causal=True, slopes=sl, softcap=c["cap"])
    assert_close_attributed(host32(o), ref, c["dt"], f"random decode {i}")


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_norms(i):
    c = _norm_case(i)
    print(f"random norms {c}", flush=True)
    rng = np.random.Generator(np.random.PCG64(c["seed"]))
    x = torch.from_numpy(rng.standard_normal(size=(c["N"], c["M"]), dtype=np.float32)).to(NORM_DTYPES[c["dt"]])
    xd = x.cuda()
    out = pa.norm_l2(xd, chunks=c["C"])
    y, m = pa.rmsnorm_rowmax(xd, eps=1e-5, chunks=c["C"])
    torch.cuda.synchronize()
    x64 = x.double().numpy()
    np.testing.assert_allclose(out.cpu().double().numpy(), norms.l2_norm(x64), rtol=2e-5)
    yr, mr = norms.rmsnorm_rowmax(x64, 1e-5)
    rtol_y = {"f16": 2.0 ** -11, "bf16": 2.0 ** -8, "f32": 2e-6}[c["dt"]]
    yg = y.cpu().double().numpy()
    assert np.all(np.abs(yg - yr) <= rtol_y * np.abs(yr) + 1e-6)
    np.testing.assert_allclose(m.cpu().double().numpy(), mr, rtol=2e-5)
