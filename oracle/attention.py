"""Plain, unfused float64 attention — the oracle (test infrastructure only).

This module is the checker of the GPU path, never part of it.  It writes out
the definition of attention that the paper states as Eq. attention (appendix
"Additional Example Operators"), with the mask and bias of the operators in
the evaluation's operator table, and nothing else:

    raw scores     r_ij = sum_d q_id k_jd
    modified       z_ij = r_ij * scale (capped by SoftCap, plus the ALiBi bias)
                   where key j is visible to row i, else -inf
    weights        w_ij = exp(z_ij - max_j' z_ij')       (max shift for range)
    output         o_id = sum_j w_ij v_jd / sum_j w_ij

The max shift cancels in the ratio; it only keeps exp in range.  Everything is
float64; the fp16/bf16 inputs are upcast exactly by the caller.  The full
score matrix and the full weight matrix of each (batch, query head) are
materialised: nothing is blocked, fused or reordered.

Readings taken where the paper is silent or garbled (each one is listed in the
design notes):

* Eq. attention prints the first product as q . v; the compute definition
  of Fig. appendix-attention multiplies q by k transposed, which is what is
  used here.
* ``score_mod(p) = p * scale + bias``: the scale multiplies q.k only and the
  bias is added after scaling.  ``scale`` is an argument (1/sqrt(D) in every
  workload).
* Masked entries are -inf whatever the bias is.
* Causal masking is aligned bottom-right: query row i sees key j iff
  j <= i + (Lk - Lq).  With Lq == Lk this is j <= i; with Lq == 1 (decode)
  every key is visible.
* A row that sees no key at all (only possible with causal and Lq > Lk) has
  output 0 instead of the NaN that max over an empty set would give.
* Grouped-query attention maps query head hq to key/value head
  hq // (Hq // Hkv) (contiguous groups).
* ALiBi: bias_ij = -slope[hq] * (i_abs - j) with i_abs = i + (Lk - Lq).  The
  slopes are an input; the oracle takes whatever values the GPU receives.
* Window (the operator table lists it as attention with a windowed mask,
  taken from Gemma 2 27B; the width is not printed): Gemma 2's causal
  sliding window of ``window`` keys.  Row i sees key j iff
  i_abs - window < j <= i_abs; it needs the causal mask.  None or 0 means no
  window.
* SoftCap (the operator table of the evaluation lists it as attention with a
  SoftCap score modifier, GQA heads and the causal mask, taken from Gemma 2
  27B; the paper prints no formula): the scaled product is capped smoothly,
  ``cap * tanh(p * scale / cap)``, before any bias is added and before the
  mask.  ``softcap`` is an argument; None or 0 means no cap.
"""

import numpy as np


def _check(q, k, v, alibi_slopes):
    if q.ndim != 4 or k.ndim != 4 or v.ndim != 4:
        raise ValueError("q, k, v must be [B, H, L, D]")
    B, Hq, Lq, D = q.shape
    Bk, Hkv, Lk, Dk = k.shape
    if k.shape != v.shape or Bk != B or Dk != D:
        raise ValueError("k and v must be [B, Hkv, Lk, D] with q's B and D")
    if Hkv < 1 or Hq % Hkv != 0:
        raise ValueError("Hq must be a multiple of Hkv")
    if alibi_slopes is not None and np.asarray(alibi_slopes).shape != (Hq,):
        raise ValueError("alibi_slopes must have one value per query head")
    return B, Hq, Hkv, Lq, Lk, D


def _softcap(x, cap):
    """The smooth cap of a scaled score: cap * tanh(x / cap), |result| < cap."""
    return cap * np.tanh(x / cap)


def scores(q, k, *, scale, causal=False, alibi_slopes=None, softcap=None, window=None,
           b=0, hq=0, rows=None):
    """Score matrix of one (batch, query head): score_mod(q.k^T) or -inf.

    Returns an array [len(rows), Lk] of float64.  ``rows`` selects query rows
    (default: all of them); each selected row is computed exactly as it would
    be in the full matrix.
    """
    B, Hq, Lq, D = q.shape
    Hkv, Lk = k.shape[1], k.shape[2]
    group = Hq // Hkv
    hk = hq // group
    i = np.arange(Lq) if rows is None else np.asarray(rows, dtype=np.int64)
    qi = np.asarray(q[b, hq], dtype=np.float64)[i]          # [R, D]
    kk = np.asarray(k[b, hk], dtype=np.float64)              # [Lk, D]
    p = qi @ kk.T                                            # raw scores r = q k^T
    i_abs = i[:, None] + (Lk - Lq)                           # bottom-right aligned row index
    j = np.arange(Lk)[None, :]
    score = p * float(scale)
    if softcap:
        score = _softcap(score, float(softcap))
    if alibi_slopes is not None:
        slope = float(np.asarray(alibi_slopes, dtype=np.float64)[hq])
        score = score + (-slope) * (i_abs - j)
    if causal:
        score = np.where(j <= i_abs, score, -np.inf)
    if window:
        if not causal:
            raise ValueError("the sliding window is defined with the causal mask")
        score = np.where(j > i_abs - int(window), score, -np.inf)
    return score


def softmax_probs(q, k, *, scale, causal=False, alibi_slopes=None, softcap=None,
                  window=None, b=0, hq=0, rows=None):
    """Weight matrix w / sum(w) of one (batch, query head), materialised."""
    score = scores(q, k, scale=scale, causal=causal, alibi_slopes=alibi_slopes,
                   softcap=softcap, window=window, b=b, hq=hq, rows=rows)
    m = score.max(axis=1, keepdims=True)                     # row max (shift)
    empty = ~np.isfinite(m)
    m = np.where(empty, 0.0, m)
    e = np.exp(score - m)                                    # unnormalised weights
    s = e.sum(axis=1, keepdims=True)                         # row sum of the weights
    return np.where(empty, 0.0, e / np.where(empty, 1.0, s))


def attention(q, k, v, *, scale, causal=False, alibi_slopes=None, softcap=None,
              window=None, rows=None, heads=None):
    """O = softmax(q.k^T * scale + bias, masked) . v, in float64.

    q: [B, Hq, Lq, D]; k, v: [B, Hkv, Lk, D]; numpy arrays of any real dtype,
    converted to float64 exactly one (batch, head) slice at a time.
    ``alibi_slopes``: None or [Hq] values.  ``softcap``: None/0, or the cap > 0
    of the SoftCap score modifier.  ``window``: None/0, or the width W >= 1
    of the causal sliding window.  ``rows``: optional query-row indices to
    compute (others are skipped, not approximated); ``heads``: optional list
    of (b, hq) pairs to compute.
    Returns float64 [B, Hq, R, D] where R = Lq or len(rows); rows of skipped
    heads are NaN.
    """
    B, Hq, Hkv, Lq, Lk, D = _check(q, k, v, alibi_slopes)
    group = Hq // Hkv
    R = Lq if rows is None else len(rows)
    out = np.full((B, Hq, R, D), np.nan)
    todo = [(b, h) for b in range(B) for h in range(Hq)] if heads is None else heads
    for b, hq in todo:
        score = scores(q, k, scale=scale, causal=causal,
                       alibi_slopes=alibi_slopes, softcap=softcap, window=window,
                       b=b, hq=hq, rows=rows)
        m = score.max(axis=1, keepdims=True)                 # row max (shift)
        empty = ~np.isfinite(m)                              # row sees no key
        m = np.where(empty, 0.0, m)
        e = np.exp(score - m)                                # unnormalised weights
        s = e.sum(axis=1, keepdims=True)                     # row sum of the weights
        o = e @ np.asarray(v[b, hq // group], dtype=np.float64)  # weighted sum of V rows
        o = o / np.where(empty, 1.0, s)                      # divide by the row sum
        out[b, hq] = np.where(empty, 0.0, o)
    return out
