"""One small case per compiled kernel instantiation.

``tests/test_kernel_coverage.py`` (CPU) checks that the kernels these cases
dispatch to, as named by the library's own dispatch (attn_fwd_kernels /
attn_decode_kernels), are exactly the kernels in the build;
``tests/test_gpu_variants.py`` runs every case on the GPU against the oracle,
``tests/test_gpu_norms.py`` every row-reduction case (both operations).
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


# Row reductions: (N, M, dtype, chunks), chunks 0 for the library's choice.
# Every dtype has cases with several chunks per row (chunk partials and a
# second kernel) and with one (a workgroup per row); RMSNorm's one-pass
# kernel at its longest row and one vector past it (then the two kernels run
# with one chunk).
NORM_CASES = [
    (3, 8, "f16", 0),            # one vector per row
    (32, 1024, "bf16", 0),       # the smallest paper shape
    (7, 1000, "f16", 3),         # chunks of 336 elements: the last one short
    (5, 4104, "bf16", 5),        # ragged chunk ends
    (2, 64, "f16", 40),          # more chunks than vectors: empty chunks
    (9, 3000, "f32", 4),
    (4, 4, "f32", 0),
    (64, 1 << 15, "bf16", 0),
    (5, 1000, "f16", 1),         # one chunk: 125 vectors, most lanes idle
    (3, 1 << 17, "bf16", 1),     # the longest row held in registers: 16 vectors every lane
    (2, 1 << 16, "f32", 1),      # the same in fp32
    (2, (1 << 17) + 8, "bf16", 1),   # one vector longer: RMSNorm's two kernels, one chunk
    (300, 2048, "f16", 1),       # more rows than compute units
]


def case_id(c):
    return "x".join(str(x) for x in c)
