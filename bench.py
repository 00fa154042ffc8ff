"""Benchmark of the fused attention hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--only NAME] [--no-cpu-baseline]

A step is one call of the library on one batch of the workload: attn_fwd for a
prefill workload (one kernel), attn_decode for a decode workload (split kernel
+ combine kernel).  W untimed steps, then K steps timed with HIP events on the
stream the kernels are launched on, bracketed by device synchronisation.  All
inputs are resident in HBM before the timed region.

The headline line is the causal MHA prefill workload (B=4, H=32, L=2048,
D=128, fp16): `value` is its algorithmic TFLOP/s (4*D per visible query/key
pair).  The decode workloads (B=8, H=32, Lk=8192, D=128; and B=16, Hq=32,
Hkv=8, Lk=32768, D=128) are reported beside it in `decode` and `decode_gqa` as
algorithmic GB/s (|Q|+|K|+|V|+|O|), the ALiBi decode workload (the MHA decode
shape with the ALiBi bias) in `decode_alibi`, the SoftCap decode workload (B=16,
Hq=32, Hkv=16, Lk=8192, D=128, cap 50) in `decode_softcap`, the SoftCap causal
prefill (B=2, Hq=32, Hkv=16, L=4096, D=128, cap 50) in `prefill_softcap`, and
every workload is listed under `workloads`.  `cpu_baseline` is the fp64 oracle timed on this host on a
bounded sample of the headline workload.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_PEAK_TFLOPS = 2500.0    # MI355X dense fp16/bf16 MFMA, published
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, published
HEADLINE = "causal_mha_prefill"
DECODE_HEADLINE = "mha_decode"
DECODE_GQA = "gqa_long_decode"
DECODE_ALIBI = "alibi_decode"
DECODE_SOFTCAP = "softcap_decode"
PREFILL_SOFTCAP = "softcap_causal_prefill"
METRIC = "prefill attn TFLOP/s (% MFMA peak); decode KV-read GB/s (% HBM peak)"
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = {
    "prefill": ["prefill.hip", "kernel_common.h", "launch.h"],
    "decode": ["decode.hip", "kernel_common.h", "launch.h"],
}


def kernel_source_hash(kind):
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kind]:
        with open(os.path.join(ROOT, "paper_2510_08726_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kind, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None
    when it is missing or was taken on a different version of the kernel."""
    path = os.path.join(PROFILES, "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    ent = data.get(f"{kind}:{workload}")
    if not ent or ent.get("source_hash") != kernel_source_hash(kind):
        return None
    return ent.get("traffic_bytes_per_step")


def decode_entry(name, dec):
    """The decode workload's throughput and its HBM roofline (split + combine kernels)."""
    return {
        "workload": name, "value": dec["GB/s"], "unit": "GB/s",
        "ms_per_step": dec["ms_per_step"], "num_splits": dec["num_splits"],
        "roofline": {"bound": "hbm", "achieved": dec["GB/s"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(dec["GB/s"] / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic("decode", name),
                     "per_launch": f"{dec['bytes_per_step']} algorithmic bytes (|Q|+|K|+|V|+|O|), "
                                   "split + combine kernels"},
    }


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--only", default=None, help="run only this workload (for profiler passes)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="budget of the oracle timing sample")
    return ap.parse_args()


def time_steps(fn, steps, warmup):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for _ in range(steps):
        fn()
    end.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    return start.elapsed_time(end) / steps, wall


def run_workload(name, steps, warmup):
    import torch
    import paper_2510_08726_amd as pa
    from paper_2510_08726_amd.workloads import WORKLOADS, make_inputs, prefill_flops, decode_bytes

    w = WORKLOADS[name]
    q, k, v, sl = make_inputs(w, device="cuda")
    o = torch.empty_like(q)
    if w.decode:
        S = w.num_splits or pa.attn_decode_num_splits(w.B, w.Hq, w.Hkv, w.Lk, w.D)
        ws = torch.empty(pa.attn_decode_workspace_bytes(w.B, w.Hq, w.D, S), dtype=torch.uint8,
                         device="cuda")

        def fn():
            pa.attn_decode(q, k, v, o, scale=w.sm_scale, alibi_slopes=sl, softcap=w.softcap or None,
                           num_splits=S, workspace=ws)
        work = decode_bytes(w.B, w.Hq, w.Hkv, w.Lk, w.D)
    else:
        S = None

        def fn():
            pa.attn_fwd(q, k, v, o, causal=w.causal, scale=w.sm_scale, alibi_slopes=sl,
                        softcap=w.softcap or None, window=w.window or None)
        work = prefill_flops(w.B, w.Hq, w.Lq, w.Lk, w.D, w.causal, w.window)
    ms, wall_ms = time_steps(fn, steps, warmup)
    res = {
        "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "Lq": w.Lq, "Lk": w.Lk, "D": w.D, "dtype": w.dtype,
        "causal": w.causal, "alibi": w.alibi, "softcap": w.softcap, "window": w.window,
        "ms_per_step": round(ms, 5),
        "host_wall_ms_per_step": round(wall_ms, 5),
    }
    if w.decode:
        gbs = work / (ms * 1e-3) / 1e9
        res.update({"num_splits": S, "bytes_per_step": work, "GB/s": round(gbs, 1),
                    "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2)})
    else:
        tf = work / (ms * 1e-3) / 1e12
        res.update({"flops_per_step": work, "TFLOP/s": round(tf, 2),
                    "pct_mfma_peak": round(100 * tf / MFMA_PEAK_TFLOPS, 2)})
    del q, k, v, o
    torch.cuda.empty_cache()
    return res


def copy_calibration(mib, steps):
    """A plain device-to-device copy of known size, for scaling HBM counters."""
    import torch
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(steps):
        b.copy_(a)
    torch.cuda.synchronize()


def cpu_baseline(budget_s):
    """The fp64 oracle on whole (batch, head) slices of the headline workload."""
    import numpy as np
    import oracle
    from paper_2510_08726_amd.workloads import WORKLOADS, make_inputs, prefill_flops
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        cores = max([d.get("num_threads", 1) for d in info if d.get("user_api") == "blas"] or [1])
    except Exception:
        cores = 1
    w = WORKLOADS[HEADLINE]
    q, k, v, _ = make_inputs(w)
    qn, kn, vn = (t.float().numpy() for t in (q, k, v))
    heads = [(b, h) for b in range(w.B) for h in range(w.Hq)]
    done = 0
    t0 = time.perf_counter()
    for bh in heads:
        oracle.attention(qn, kn, vn, scale=w.sm_scale, causal=w.causal, heads=[bh])
        done += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    flops = prefill_flops(1, done, w.Lq, w.Lk, w.D, w.causal)
    return {
        "value": round(flops / el / 1e12, 6), "unit": "TFLOP/s", "cores": int(cores),
        "kind": "oracle",
        "sample": f"{done} of {len(heads)} (batch, head) slices of {HEADLINE}, all {w.Lq} query rows "
                  f"each, float64 numpy (BLAS matmul on {cores} threads, exp single-threaded); "
                  f"{el:.1f} s",
        "seconds": round(el, 2),
    }


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build runs on exactly one GPU (no multi-GPU path); "
              "use --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2510_08726_amd as pa
    from paper_2510_08726_amd.workloads import WORKLOADS
    pa.load_library()
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)

    if args.only:
        res = run_workload(args.only, args.steps, args.warmup)
        if args.copy_mib:
            copy_calibration(args.copy_mib, args.steps)
        print(json.dumps({"workload": args.only, **res}), flush=True)
        return

    results = {}
    for name in WORKLOADS:
        results[name] = run_workload(name, args.steps, args.warmup)
        print(f"# {name}: {json.dumps(results[name])}", file=sys.stderr, flush=True)

    head = results[HEADLINE]
    w = WORKLOADS[HEADLINE]
    traffic = measured_traffic("prefill", HEADLINE)
    roofline = {
        "bound": "mfma", "achieved": head["TFLOP/s"], "peak": MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
        "frac": round(head["TFLOP/s"] / MFMA_PEAK_TFLOPS, 4), "traffic": traffic,
        "kernel": "prefill_kernel<128, f16, causal>",
        "per_launch": f"{head['flops_per_step']} algorithmic flops (4*D per visible query/key pair)",
    }
    decode = decode_entry(DECODE_HEADLINE, results[DECODE_HEADLINE])
    decode_gqa = decode_entry(DECODE_GQA, results[DECODE_GQA])
    decode_alibi = decode_entry(DECODE_ALIBI, results[DECODE_ALIBI])
    decode_softcap = decode_entry(DECODE_SOFTCAP, results[DECODE_SOFTCAP])
    ps = results[PREFILL_SOFTCAP]
    prefill_softcap = {
        "workload": PREFILL_SOFTCAP, "value": ps["TFLOP/s"], "unit": "TFLOP/s", "ms_per_step": ps["ms_per_step"],
        "roofline": {"bound": "mfma", "achieved": ps["TFLOP/s"], "peak": MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(ps["TFLOP/s"] / MFMA_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic("prefill", PREFILL_SOFTCAP),
                     "per_launch": f"{ps['flops_per_step']} algorithmic flops (4*D per visible query/key pair)"},
    }
    line = {
        "metric": METRIC, "value": head["TFLOP/s"], "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": HEADLINE, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "Lq": w.Lq, "Lk": w.Lk,
                   "D": w.D, "causal": w.causal, "input": "iid N(0,1) fp16, seed 2"},
        "roofline": roofline,
        "decode": decode,
        "decode_gqa": decode_gqa,
        "decode_alibi": decode_alibi,
        "decode_softcap": decode_softcap,
        "prefill_softcap": prefill_softcap,
        "workloads": results,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
