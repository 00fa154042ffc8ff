"""One small case per compiled kernel instantiation.

``tests/test_kernel_coverage.py`` (CPU) checks that the kernels these cases
dispatch to, as named by the library's own dispatch (attn_fwd_kernels /
attn_decode_kernels), are exactly the kernels in the build;
``tests/test_gpu_variants.py`` runs every case on the GPU against the oracle.
"""

# Prefill: (B, Hq, Hkv, Lq, Lk, D, dtype, causal, alibi, softcap, window).
# The flag combinations are the eight kernels per (head dim, type): plain and
# ALiBi without the mask, causal, causal ALiBi, causal SoftCap, and the
# sliding window alone, with ALiBi and with SoftCap.
_FLAGS = [
    (False, False, None, None),
    (False, True, None, None),
    (True, False, None, None),
    (True, True, None, None),
    (True, False, 2.0, None),
    (True, False, None, 77),
    (True, True, None, 77),
    (True, False, 2.0, 77),
]
PREFILL_VARIANT_CASES = []
for _D in (64, 128):
    for _dt in ("f16", "bf16"):
        for _n, (_c, _a, _cap, _w) in enumerate(_FLAGS):
            # vary the shape a little between cases: GQA groups, Lq != Lk
            _Hq, _Hkv = [(4, 4), (4, 2), (6, 3), (8, 1)][_n % 4]
            _Lq, _Lk = [(300, 300), (257, 410), (333, 333), (150, 150)][(_n + _D // 64) % 4]
            PREFILL_VARIANT_CASES.append((1, _Hq, _Hkv, _Lq, _Lk, _D, _dt, _c, _a, _cap, _w))

# Decode: (B, Hq, Hkv, Lk, D, dtype, alibi, softcap, num_splits).  Query heads
# per KV head: 1 (vector kernel, one head a workgroup), 4 (matrix kernel),
# 34, 36 and 64 (vector kernel with 2, 4 and 8 heads a workgroup).
DECODE_VARIANT_CASES = []
for _D in (64, 128):
    for _dt in ("f16", "bf16"):
        for _Hq, _Hkv in [(4, 4), (8, 2), (34, 1), (36, 1), (64, 1)]:
            for _a in (False, True):
                for _cap in (None, 2.0):
                    _Lk = 333 + 50 * len(DECODE_VARIANT_CASES) % 400
                    DECODE_VARIANT_CASES.append((1, _Hq, _Hkv, _Lk, _D, _dt, _a, _cap, 3))


def case_id(c):
    return "x".join(str(x) for x in c)
