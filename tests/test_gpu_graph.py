"""The prefill and the no-allocation decode captured in a HIP graph: every
replay equals the eager call bit for bit, with the program's own eager work
(other calls on the same buffers, synchronisations) between replays.  The
kernels launch on the stream they are given and enqueue no memset, so a
capture records exactly the launches of an eager call."""

import pytest
import torch

import paper_2510_08726_amd as pa
from paper_2510_08726_amd.workloads import alibi_slopes, random_tensors

pytestmark = pytest.mark.gpu

REPLAYS = 4


def _capture(fn):
    """Warm up on a side stream (default priority), then capture fn."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def test_prefill_graph_replays_match_eager():
    print("graph: causal GQA prefill with ALiBi, 2x8/2x300x64 f16", flush=True)
    q, = random_tensors([(2, 8, 300, 64)], "f16", 901, device="cuda")
    k, v = random_tensors([(2, 2, 300, 64)] * 2, "f16", 902, device="cuda")
    sl = alibi_slopes(8).cuda()
    ref = pa.attn_fwd(q, k, v, causal=True, alibi_slopes=sl)
    torch.cuda.synchronize()
    o = torch.empty_like(q)
    g = _capture(lambda: pa.attn_fwd(q, k, v, o, causal=True, alibi_slopes=sl))
    scratch = torch.empty_like(q)
    for r in range(REPLAYS):
        o.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o, ref), f"replay {r}"
        pa.attn_fwd(q, k, v, scratch, causal=False)   # eager work between replays
        torch.cuda.synchronize()


def test_noalloc_decode_graph_replays_match_eager():
    print("graph: attn_decode_noalloc, GQA 4x16/4, Lk 3000, D 128 bf16, SoftCap 5", flush=True)
    q, = random_tensors([(4, 16, 1, 128)], "bf16", 903, device="cuda")
    k, v = random_tensors([(4, 4, 3000, 128)] * 2, "bf16", 904, device="cuda")
    ref = pa.attn_decode_noalloc(q, k, v, softcap=5.0)
    torch.cuda.synchronize()
    o = torch.empty_like(q)
    g = _capture(lambda: pa.attn_decode_noalloc(q, k, v, o, softcap=5.0))
    q2, = random_tensors([(1, 16, 1, 128)], "bf16", 905, device="cuda")
    k2, v2 = random_tensors([(1, 4, 700, 128)] * 2, "bf16", 906, device="cuda")
    for r in range(REPLAYS):
        o.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o, ref), f"replay {r}"
        # eager work between replays that uses the same static workspace
        pa.attn_decode_noalloc(q2, k2, v2)
        torch.cuda.synchronize()
