"""Seeded synthetic workloads shared by the tests, the bench and the oracle checks.

This module holds no attention arithmetic: it only draws inputs and names the
workload shapes.  Both the GPU path and the oracle receive the same host
tensors from here, so neither can feed the other its inputs.

Recipe: iid N(0, 1) drawn in float32 from ``numpy.random.Generator(PCG64(seed))``
in the order Q, K, V, then rounded once (round-to-nearest-even) to the
workload's storage dtype.  The oracle upcasts exactly to float64.
"""

from dataclasses import dataclass, field
import math

import numpy as np
import torch

DTYPES = {"f16": torch.float16, "bf16": torch.bfloat16}


@dataclass(frozen=True)
class Workload:
    """One attention problem: shapes, dtype, mask/bias flags and seed."""
    name: str
    B: int
    Hq: int
    Hkv: int
    Lq: int
    Lk: int
    D: int
    dtype: str = "f16"
    causal: bool = False
    alibi: bool = False
    decode: bool = False
    seed: int = 0
    num_splits: int = 0
    scale: float = field(default=None)
    softcap: float = 0.0      # SoftCap cap (0: none)
    window: int = 0           # causal sliding window in keys (0: none)

    @property
    def sm_scale(self):
        return 1.0 / math.sqrt(self.D) if self.scale is None else self.scale


# The six shapes the headline metric is quoted on, then ALiBi decode (the MHA
# decode shape with the ALiBi bias) and SoftCap decode (Gemma 2 27B's
# attention: 32 query heads on 16 KV heads of dim 128, logits capped at 50), and
# SoftCap causal prefill with the same heads, and the Window operator with
# Gemma 2 27B's local-attention layers: the same heads, a causal sliding window
# of 4096 keys, L = 8192.
# Prefill: Lq == Lk.  Decode: one query token (Lq = 1) against a KV cache of
# Lk keys.
WORKLOADS = {
    "tiny_noncausal": Workload("tiny_noncausal", 1, 2, 2, 128, 128, 64, "f16",
                               seed=1),
    "causal_mha_prefill": Workload("causal_mha_prefill", 4, 32, 32, 2048, 2048,
                                   128, "f16", causal=True, seed=2),
    "mha_decode": Workload("mha_decode", 8, 32, 32, 1, 8192, 128, "f16",
                           decode=True, seed=3),
    "gqa_causal_prefill": Workload("gqa_causal_prefill", 2, 64, 8, 4096, 4096,
                                   128, "bf16", causal=True, seed=4),
    "alibi_causal_prefill": Workload("alibi_causal_prefill", 4, 16, 16, 4096,
                                     4096, 64, "f16", causal=True, alibi=True,
                                     seed=5),
    "gqa_long_decode": Workload("gqa_long_decode", 16, 32, 8, 1, 32768, 128,
                                "f16", decode=True, seed=6),
    "alibi_decode": Workload("alibi_decode", 8, 32, 32, 1, 8192, 128, "f16",
                             alibi=True, decode=True, seed=7),
    "softcap_decode": Workload("softcap_decode", 16, 32, 16, 1, 8192, 128, "f16",
                               decode=True, seed=8, softcap=50.0),
    "softcap_causal_prefill": Workload("softcap_causal_prefill", 2, 32, 16, 4096, 4096,
                                       128, "f16", causal=True, seed=9, softcap=50.0),
    "window_causal_prefill": Workload("window_causal_prefill", 2, 32, 16, 8192, 8192,
                                      128, "f16", causal=True, seed=10, window=4096),
}


@dataclass(frozen=True)
class NormWorkload:
    """A row reduction of the paper's second workload: X [N, M] of dtype."""
    name: str
    op: str          # "l2" (stable L2 norm) or "rms" (RMSNorm with the row max of y)
    N: int
    M: int
    dtype: str
    seed: int
    eps: float = 1e-6


# The largest shape of the paper's range (N 32..256 rows, M 2^10..2^17
# columns): the L2 norm on fp32 rows (where squares of large entries overflow
# and the stable form matters), RMSNorm on bf16 activations.
NORM_DTYPES = {"f16": torch.float16, "bf16": torch.bfloat16, "f32": torch.float32}
NORM_WORKLOADS = {
    "l2_norm": NormWorkload("l2_norm", "l2", 256, 1 << 17, "f32", seed=11),
    "rmsnorm_rowmax": NormWorkload("rmsnorm_rowmax", "rms", 256, 1 << 17, "bf16", seed=12),
}


def make_norm_input(w: NormWorkload, *, seed=None, device="cpu"):
    """X [N, M]: iid N(0, 1) drawn in float32 from PCG64(seed), rounded once to w.dtype."""
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    x = torch.from_numpy(rng.standard_normal(size=(w.N, w.M), dtype=np.float32)).to(NORM_DTYPES[w.dtype])
    return x.to(device) if device != "cpu" else x


def norm_bytes(op, N, M, elem):
    """Algorithmic HBM bytes of one call: X read once, the [N] fp32 outputs,
    and for RMSNorm the output Y."""
    return N * M * elem * (2 if op == "rms" else 1) + 4 * N


def alibi_slopes(H):
    """ALiBi slopes 2^(-8 h / H) for heads h = 1..H, as float32 (one per head).

    Head index hq (0-based) gets 2^(-8 (hq + 1) / H): the first head has the
    shallowest bias 2^(-8/H) and the last one 2^(-8).
    """
    return torch.tensor([2.0 ** (-8.0 * (h + 1) / H) for h in range(H)],
                        dtype=torch.float32)


def make_inputs(w: Workload, *, seed=None, device="cpu"):
    """Draw (q, k, v, slopes) for workload ``w`` on the host; optionally move them.

    Returns storage-dtype tensors q [B,Hq,Lq,D], k and v [B,Hkv,Lk,D] and the
    float32 slopes [Hq] (None without ALiBi).
    """
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    dt = DTYPES[w.dtype]
    shapes = [(w.B, w.Hq, w.Lq, w.D), (w.B, w.Hkv, w.Lk, w.D), (w.B, w.Hkv, w.Lk, w.D)]
    out = []
    for shp in shapes:
        x = rng.standard_normal(size=shp, dtype=np.float32)
        out.append(torch.from_numpy(x).to(dt))
    slopes = alibi_slopes(w.Hq) if w.alibi else None
    if device != "cpu":
        out = [t.to(device) for t in out]
        slopes = None if slopes is None else slopes.to(device)
    return out[0], out[1], out[2], slopes


def random_tensors(shapes, dtype, seed, device="cpu"):
    """Seeded N(0,1) tensors of the given shapes, rounded to ``dtype``."""
    rng = np.random.Generator(np.random.PCG64(seed))
    dt = DTYPES[dtype] if isinstance(dtype, str) else dtype
    res = []
    for shp in shapes:
        x = rng.standard_normal(size=shp, dtype=np.float32)
        res.append(torch.from_numpy(x).to(dt).to(device))
    return res


def prefill_flops(B, Hq, Lq, Lk, D, causal, window=0):
    """Algorithmic FLOPs: 4 * D per visible (query, key) pair, over all heads.

    Two contractions (Q.K^T and P.V), 2 flops per multiply-add; softmax work
    is not counted.  Causal visibility is bottom-right aligned; a window of W
    keys leaves row i the keys i_abs - W < j <= i_abs.
    """
    if causal:
        off = Lk - Lq
        visible = 0
        for i in range(Lq):
            hi = min(Lk, i + off + 1)
            lo = max(0, i + off + 1 - window) if window else 0
            visible += max(0, hi - lo)
    else:
        visible = Lq * Lk
    return 4 * D * visible * B * Hq


def decode_bytes(B, Hq, Hkv, Lk, D, elem=2):
    """Algorithmic HBM bytes of one decode step: |Q| + |K| + |V| + |O|."""
    return elem * (B * Hq * D * 2 + 2 * B * Hkv * Lk * D)
