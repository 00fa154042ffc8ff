"""Row reductions of the paper's second workload, in float64 — TEST INFRASTRUCTURE ONLY.

Section "Example Operators Amenable to Neptune Transformations" names two
non-attention operators that the same break-and-repair fusion applies to,
reduced along the rows of an N x M matrix (Section "Experimental
Methodology"):

* the numerically stable L2 norm: ||x|| = m sqrt(sum_i (x_i / m)^2) with
  m = max_i |x_i|.  Fusing the sum into the max reduction gives, in the
  notation of Eq. fixed-recurrent, the producer r = running max |x|, the
  consumer t = running sum, f = +, g(r, c) = (c / r)^2 and the repair
  h(t, r, r') = t (r / r')^2;
* RMSNorm with dynamic scaling: y_i = x_i / sqrt(s + eps), s = mean(x^2),
  followed by the row max m = max_i y_i.  The producer is the mean reduction
  r (the running sum of c^2 / M), the consumer t the running max, f = max,
  g(r, c) = c / sqrt(r + eps) and h(t, r, r') = t sqrt(r + eps) / sqrt(r' + eps).

``l2_norm`` and ``rmsnorm_rowmax`` are the plain definitions (what the GPU is
compared with; the stable form equals ||x|| exactly over the reals, and
float64 squares of any float32 input do not overflow).  The ``*_rolling``
functions execute the fused single pass element block by element block
(appendix "Privatization": a local reduction per block, then the repaired
global update), and the ``*_split`` functions the split-k form (Section
"Split-K Update": independent chunks, then the repaired combine); they exist
to pin the algorithm against the plain definition (Theorems 1 and 2).  No GPU
code imports this module.
"""

import numpy as np


def l2_norm(x):
    """Plain definition: sqrt(sum_i x_i^2) of every row of x [N, M], float64."""
    x = np.asarray(x, dtype=np.float64)
    return np.sqrt((x * x).sum(axis=1))


def rmsnorm_rowmax(x, eps):
    """Plain definition: y = x / sqrt(mean(x^2) + eps) and m = max_i y_i per row.

    Returns (y [N, M], m [N]) in float64.
    """
    x = np.asarray(x, dtype=np.float64)
    s = (x * x).mean(axis=1, keepdims=True)
    y = x / np.sqrt(s + float(eps))
    return y, y.max(axis=1)


def _blocks(M, block):
    return [(j, min(j + block, M)) for j in range(0, M, block)]


def l2_norm_rolling(x, block=8):
    """Single pass over each row: r = running max |x|, t = running sum of
    (c / r)^2, repaired by h(t, r, r') = t (r / r')^2 when r grows."""
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros(x.shape[0])
    for n in range(x.shape[0]):
        r, t = 0.0, 0.0
        for a, b in _blocks(x.shape[1], block):
            c = x[n, a:b]
            r_new = max(r, float(np.abs(c).max()))             # producer: max
            if r_new == 0.0:
                continue                                         # only zeros so far
            t = (t * (r / r_new) ** 2 if r > 0.0 else 0.0) + float(((c / r_new) ** 2).sum())
            r = r_new
        out[n] = r * np.sqrt(t)
    return out


def l2_norm_split_local(x, chunks, size=None):
    """Local nests of the split L2 norm: for every row and chunk of ``size``
    elements (default ceil(M / chunks)), r_c = max |x| and t_c = sum of
    (x / r_c)^2 (both 0 for an empty or all-zero chunk).  Returns (r, t) [N, chunks]."""
    x = np.asarray(x, dtype=np.float64)
    N, M = x.shape
    size = size or -(-M // chunks)
    r = np.zeros((N, chunks))
    t = np.zeros((N, chunks))
    for n in range(N):
        for c in range(chunks):
            seg = x[n, c * size:(c + 1) * size]
            if seg.size and np.abs(seg).max() > 0.0:
                r[n, c] = np.abs(seg).max()
                t[n, c] = ((seg / r[n, c]) ** 2).sum()
    return r, t


def l2_norm_split(x, chunks, size=None):
    """Split-k form: the local nests, then R = max_c r_c and
    T = sum_c h(t_c, r_c, R) = sum_c t_c (r_c / R)^2; the norm is R sqrt(T)."""
    r, t = l2_norm_split_local(x, chunks, size)
    R = r.max(axis=1, keepdims=True)
    safe = np.where(R > 0.0, R, 1.0)
    return np.where(R[:, 0] > 0.0, R[:, 0] * np.sqrt((t * (r / safe) ** 2).sum(axis=1)), 0.0)


def rmsnorm_rowmax_rolling(x, eps, block=8):
    """Row max of RMSNorm in the same pass as the mean: r = running mean
    (sum of c^2 / M), t = running max of c / sqrt(r + eps), repaired by
    h(t, r, r') = t sqrt(r + eps) / sqrt(r' + eps) whenever r grows."""
    x = np.asarray(x, dtype=np.float64)
    N, M = x.shape
    out = np.zeros(N)
    for n in range(N):
        r, t = 0.0, -np.inf
        for a, b in _blocks(M, block):
            c = x[n, a:b]
            r_new = r + float((c * c).sum()) / M                # producer: mean
            t = max(t * np.sqrt(r + eps) / np.sqrt(r_new + eps) if np.isfinite(t) else -np.inf,
                    float((c / np.sqrt(r_new + eps)).max()))
            r = r_new
        out[n] = t
    return out


def rmsnorm_split_local(x, eps, chunks, size=None):
    """Local nests of the split RMSNorm statistics: for every row and chunk,
    r_c = (sum of x^2 over the chunk) / M and t_c = max of x / sqrt(r_c + eps)
    (r_c = 0 and t_c = -inf for an empty chunk).  Returns (r, t) [N, chunks]."""
    x = np.asarray(x, dtype=np.float64)
    N, M = x.shape
    size = size or -(-M // chunks)
    r = np.zeros((N, chunks))
    t = np.full((N, chunks), -np.inf)
    for n in range(N):
        for c in range(chunks):
            seg = x[n, c * size:(c + 1) * size]
            if seg.size:
                r[n, c] = (seg * seg).sum() / M
                t[n, c] = (seg / np.sqrt(r[n, c] + eps)).max()
    return r, t


def rmsnorm_rowmax_split(x, eps, chunks, size=None):
    """Split-k form: the local nests, then r = sum_c r_c and
    m = max_c h(t_c, r_c, r) = max_c t_c sqrt(r_c + eps) / sqrt(r + eps)."""
    rc, tc = rmsnorm_split_local(x, eps, chunks, size)
    r = rc.sum(axis=1, keepdims=True)
    with np.errstate(invalid="ignore"):
        rep = np.where(np.isneginf(tc), -np.inf, tc * np.sqrt(rc + eps) / np.sqrt(r + eps))
    return rep.max(axis=1)
