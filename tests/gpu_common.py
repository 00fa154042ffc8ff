"""Helpers shared by the GPU parity tests: run the HIP path, run the oracle on
the same host tensors, and measure the difference."""

import numpy as np
import torch

import oracle
import paper_2510_08726_amd as pa

MAX_ABS = 1e-2    # tolerance of the fused kernels vs the fp64 oracle (fp16/bf16 in,
MEAN_ABS = 1e-3   # fp32 accumulate, output rounded to the input type)


def host64(t):
    """Exact float64 numpy copy of a host or device fp16/bf16/fp32 tensor."""
    return t.detach().to("cpu", torch.float64).numpy()


def host32(t):
    """Exact float32 numpy copy (fp16 and bf16 embed exactly in fp32)."""
    return t.detach().to("cpu", torch.float32).numpy()


def errors(gpu_out, ref):
    d = np.abs(np.asarray(gpu_out, dtype=np.float64) - ref)
    assert np.all(np.isfinite(d)), "non-finite output"
    flat = d.ravel()
    return {
        "max_abs": float(flat.max()),
        "mean_abs": float(flat.mean()),
        "rms": float(np.sqrt(np.mean(flat ** 2))),
        "p90": float(np.percentile(flat, 90)),
        "p99": float(np.percentile(flat, 99)),
    }


def assert_close(gpu_out, ref, what=""):
    e = errors(gpu_out, ref)
    print(f"{what}: " + " ".join(f"{k}={v:.3e}" for k, v in e.items()), flush=True)
    assert e["max_abs"] <= MAX_ABS, (what, e)
    assert e["mean_abs"] <= MEAN_ABS, (what, e)
    return e


def run_fwd(q, k, v, *, scale, causal=False, slopes=None, softcap=None, window=None):
    dev = torch.device("cuda")
    o = pa.attn_fwd(q.to(dev), k.to(dev), v.to(dev), causal=causal, scale=scale,
                    alibi_slopes=None if slopes is None else slopes.to(dev), softcap=softcap,
                    window=window)
    torch.cuda.synchronize()
    return o


def oracle_fwd(q, k, v, *, scale, causal=False, slopes=None, softcap=None, window=None, rows=None,
               heads=None):
    sl = None if slopes is None else host64(slopes)
    return oracle.attention(host32(q), host32(k), host32(v), scale=scale, causal=causal,
                            alibi_slopes=sl, softcap=softcap, window=window, rows=rows, heads=heads)
