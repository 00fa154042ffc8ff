"""fp64 CPU oracle for fused attention — TEST INFRASTRUCTURE ONLY.

This package is the checker, not the product.  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  The GPU path (``paper_2510_08726_amd``) never imports it, and it
imports nothing from the GPU path: the two share no code.  The only thing both
consume is the seeded input generator in ``paper_2510_08726_amd.workloads``,
which holds none of the method's arithmetic.

Contents
--------
``attention``      the plain, unfused definition of attention (Eq. attention in
                   the appendix "Additional Example Operators", with the mask
                   and bias of the operator table and the product order of
                   Fig. appendix-attention).  It materialises
                   the full score matrix S and the probability matrix P in
                   float64.  This is what every GPU result is compared with.
``rolling``        the rolling-update algorithm (Section "Rolling Update",
                   Algorithm 1, Eq. fixed-recurrent, and the privatised form of
                   the appendix "Privatization") executed in float64 tile by
                   tile.  Used only to pin the algorithm against the plain
                   definition (Theorem 1) and to expose the per-tile state.
``splitk``         the split-k update algorithm (Section "Split-K Update",
                   Algorithm 2, Fig. su-result, Eq. su:rewrite): local nests per
                   chunk, then the repaired global nest.  Its local-nest outputs
                   have the same meaning as the decode kernel's partials, so the
                   GPU workspace can be compared with them element by element.

``norms``          the row reductions of the paper's second workload (stable
                   L2 norm; RMSNorm and the row max of its output, Section
                   "Example Operators Amenable to Neptune Transformations"):
                   plain definitions, plus their single-pass (rolling) and
                   split-k forms.

Parity status: every function here is pinned by ``tests/test_oracle_pins.py``
and ``tests/test_algorithms.py`` (invariants, closed forms, brute force and
the CPU float64 ``scaled_dot_product_attention`` of PyTorch as a library
special case).  No function is "parity unpinned".
"""

from .attention import attention, scores, softmax_probs  # noqa: F401
from . import norms, rolling, splitk  # noqa: F401
