"""Rolling update applied to attention, executed in float64 (test infrastructure).

This is the algorithm the prefill kernel implements, written the way the paper
states it and nothing more: it exists to pin the algorithm itself against the
plain definition (Theorem 1, "Correctness of the Repaired Program") and to
expose the state after every tile (Lemma "tag-updating", Eq. example-result).

Notation follows Fig. example-ours and the appendix "Privatization":
``xmax_0`` is the producer's result at the previous iteration, ``xmax_1`` at
the current one, ``xsum`` the consumer reduction.  Attention fuses two
consumers into the max producer (Section "Example Operators Amenable to
Neptune Transformations", Attention): the exp-sum and the P.V product.  For
both, g(r, c) = exp(c - r), f = +, and the repair function is
h(t, r, r') = t * exp(r - r') applied to the left-hand side of the reducer
(Eq. fixed-recurrent).  The rolling loop runs over key tiles of ``block_n``
keys; inside a tile the reductions are privatised (appendix "Privatization"):
a local max over the tile, then the global running max.
"""

import numpy as np

from .attention import scores as _scores


def _repair(prev, cur):
    """exp(prev - cur) with the empty-prefix case (both -inf) giving 0."""
    with np.errstate(invalid="ignore"):
        f = np.exp(prev - cur)
    return np.where(np.isneginf(cur), 0.0, f)


def rolling_update_attention(q, k, v, *, scale, causal=False, alibi_slopes=None,
                             window=None, block_n=64, b=0, hq=0, trace=False):
    """Attention of one (batch, query head) by rolling update over key tiles.

    Returns ``o`` [Lq, D] (float64); with ``trace=True`` also a list holding,
    after each tile t, the tuple (xmax, xsum, acc) — the running max, the
    repaired running sum and the repaired unnormalised P.V accumulator.
    """
    v = np.asarray(v, dtype=np.float64)
    group = q.shape[1] // k.shape[1]
    vv = v[b, hq // group]
    score = _scores(q, k, scale=scale, causal=causal, alibi_slopes=alibi_slopes,
                    window=window, b=b, hq=hq)                # [Lq, Lk]
    Lq, Lk = score.shape
    D = vv.shape[1]
    xmax_0 = np.full((Lq, 1), -np.inf)
    xsum = np.zeros((Lq, 1))
    acc = np.zeros((Lq, D))
    states = []
    for j0 in range(0, Lk, block_n):
        tile = score[:, j0:j0 + block_n]
        xmax_1p = tile.max(axis=1, keepdims=True)             # max_local (privatised)
        xmax_1 = np.maximum(xmax_0, xmax_1p)                  # max_global
        safe = np.where(np.isneginf(xmax_1), 0.0, xmax_1)
        e = np.exp(tile - safe)                               # g(xmax_1, c)
        alpha = _repair(xmax_0, xmax_1)                       # h's factor exp(r - r')
        xsum = alpha * xsum + e.sum(axis=1, keepdims=True)
        acc = alpha * acc + e @ vv[j0:j0 + block_n]
        xmax_0 = xmax_1
        if trace:
            states.append((xmax_1.copy(), xsum.copy(), acc.copy()))
    o = np.where(xsum > 0, acc / np.where(xsum > 0, xsum, 1.0), 0.0)
    return (o, states) if trace else o
