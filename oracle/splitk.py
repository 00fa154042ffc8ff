"""Split-k update applied to attention, executed in float64 (test infrastructure).

Section "Split-K Update" (Algorithm 2, Fig. su-result, Eq. su:rewrite): the key
reduction of length Lk is privatised into chunks of ``c = ceil(Lk / S)`` keys
(Section "Reduction Privatization": K reduce iterations, tile size k, then
ceil(K / k) global iterations).  The local nests run per chunk, unrepaired and
independent of each other:

    max_l[j0] = max over the chunk of score
    sum_l[j0] = sum over the chunk of exp(score - max_l[j0])
    o_l[j0]   = sum over the chunk of exp(score - max_l[j0]) * v

and the global nests combine them with the repair function on the right-hand
side of the reducer (Eq. su:rewrite), h(t, r, r') = t * exp(r - r'):

    max_g = max over j0 of max_l[j0]
    sum_g = sum over j0 of exp(max_l[j0] - max_g) * sum_l[j0]
    o     = (sum over j0 of exp(max_l[j0] - max_g) * o_l[j0]) / sum_g

A chunk that holds no visible key (it starts at or past Lk, or is fully
masked) has max_l = -inf, sum_l = 0, o_l = 0 and contributes nothing.  The
decode kernel's workspace partials have exactly the meaning of
(o_l, max_l, sum_l), in natural-log units.
"""

import numpy as np

from .attention import scores as _scores


def chunk_bounds(Lk, num_splits):
    """[start, end) of every chunk: c = ceil(Lk / S); the tail may be short or empty."""
    c = -(-Lk // num_splits)
    return [(min(s * c, Lk), min((s + 1) * c, Lk)) for s in range(num_splits)]


def split_local(q, k, v, *, scale, num_splits, causal=False, alibi_slopes=None,
                softcap=None):
    """Local nests.  Returns (o_l [B,Hq,Lq,S,D], max_l [B,Hq,Lq,S], sum_l [B,Hq,Lq,S])."""
    q = np.asarray(q, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, Hq, Lq, D = q.shape
    Hkv, Lk = k.shape[1], k.shape[2]
    group = Hq // Hkv
    S = num_splits
    o_l = np.zeros((B, Hq, Lq, S, D))
    max_l = np.full((B, Hq, Lq, S), -np.inf)
    sum_l = np.zeros((B, Hq, Lq, S))
    bounds = chunk_bounds(Lk, S)
    for b in range(B):
        for hq in range(Hq):
            score = _scores(q, k, scale=scale, causal=causal,
                            alibi_slopes=alibi_slopes, softcap=softcap, b=b, hq=hq)
            vv = v[b, hq // group]
            for s, (lo, hi) in enumerate(bounds):
                if hi <= lo:
                    continue
                tile = score[:, lo:hi]
                m = tile.max(axis=1)                          # s_max_local
                live = np.isfinite(m)
                safe = np.where(live, m, 0.0)
                e = np.exp(tile - safe[:, None])              # s_sum_local terms
                max_l[b, hq, :, s] = m
                sum_l[b, hq, :, s] = np.where(live, e.sum(axis=1), 0.0)
                o_l[b, hq, :, s] = np.where(live[:, None], e @ vv[lo:hi], 0.0)
    return o_l, max_l, sum_l


def split_global(o_l, max_l, sum_l):
    """Global nests with the repair applied on the right of the reducer.

    Takes the local results for any number of leading axes (..., S, D) /
    (..., S) and returns o (..., D).  All chunks empty gives o = 0.
    """
    max_g = max_l.max(axis=-1, keepdims=True)                 # s_max_global
    live = np.isfinite(max_l)
    with np.errstate(invalid="ignore"):
        w = np.where(live, np.exp(max_l - np.where(np.isfinite(max_g), max_g, 0.0)), 0.0)
    sum_g = (w * sum_l).sum(axis=-1)                          # s_sum_global
    o_g = (w[..., None] * o_l).sum(axis=-2)
    ok = sum_g > 0
    return np.where(ok[..., None], o_g / np.where(ok, sum_g, 1.0)[..., None], 0.0)


def split_k_attention(q, k, v, *, scale, num_splits, causal=False, alibi_slopes=None,
                      softcap=None):
    """Attention by split-k update: local nests then repaired global nests."""
    o_l, max_l, sum_l = split_local(q, k, v, scale=scale, num_splits=num_splits,
                                    causal=causal, alibi_slopes=alibi_slopes,
                                    softcap=softcap)
    return split_global(o_l, max_l, sum_l)
