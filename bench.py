"""Benchmark of the fused attention hot path (and the paper's row reductions) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--only NAME] [--no-cpu-baseline]
                    [--no-errors] [--no-peaks]

A step is one call of the library on one batch of a workload: attn_fwd(_mod)
for a prefill workload (one kernel), attn_decode(_mod) for a decode workload
(split kernel, and the combine kernel with more than one chunk), norm_l2 /
rmsnorm_rowmax for a row reduction (one kernel per row, or split kernel +
combine kernel).  W untimed steps,
continued until at least WARMUP_MS of load has passed (so that the clock has
risen), then K steps timed with HIP events recorded on the stream the kernels
are launched on (the current torch stream, which the binding passes to the
library), bracketed by device synchronisation; `ms_per_step` is their mean.  K more steps, each between
its own pair of events, give `launch_ms` (min and max per step).  All inputs
are resident in HBM before the timed region.

Every workload takes its inputs in turn from copies that span at least
2 GiB, so that no step finds its input in the 256 MB memory-side cache
(Infinity Cache) that the previous steps filled: the rates are those of
inputs read from HBM.  `GB/s_same_input` / `TFLOP/s_same_input` are the
rates with one input read by every step, as a caller that re-reads a
cache-resident tensor would see them.

The headline line is the causal MHA prefill workload (B=4, H=32, L=2048,
D=128, fp16): `value` is its algorithmic TFLOP/s (4*D per visible query/key
pair) and `roofline` its MFMA roofline, against the published dense fp16 peak
and against the peak that an MFMA loop on random operands reaches on the same
GPU in the same run (`achievable`, with the shader clock it held).  Beside it:
the decode workloads as algorithmic GB/s (|Q|+|K|+|V|+|O|) against the HBM
peak and the measured streaming-read rate, the other prefill workloads, the
row reductions, `split_sweep` (decode split counts of the per-head and the
grouped kernel, chunks per row of the row reductions, each beside the
library's choice), error metrics of every workload
against the fp64 oracle (max, mean, RMS, p90, p99 of |GPU - oracle| on a
stated sample), and `cpu_baseline`: the oracle timed on this host.
"""

import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_PEAK_TFLOPS = 2500.0    # MI355X dense fp16/bf16 MFMA, published
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, published
HEADLINE = "causal_mha_prefill"
METRIC = "prefill attn TFLOP/s (% MFMA peak); decode KV-read GB/s (% HBM peak)"
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = {
    "prefill": ["prefill.hip", "kernel_common.h", "launch.h"],
    "decode": ["decode.hip", "kernel_common.h", "launch.h"],
    "norms": ["norms.hip", "kernel_common.h", "launch.h"],
}
# bench-line keys of the workloads reported beside the headline
SIDE = {
    "decode": "mha_decode", "decode_gqa": "gqa_long_decode", "decode_alibi": "alibi_decode",
    "decode_softcap": "softcap_decode", "prefill_gqa": "gqa_causal_prefill",
    "prefill_alibi": "alibi_causal_prefill", "prefill_softcap": "softcap_causal_prefill",
    "prefill_window": "window_causal_prefill",
}
# decode split counts swept beside the library's choice: the per-head kernel
# (MHA decode) and the grouped matrix-unit kernel (long GQA decode)
SWEEPS = {"mha_decode": (1, 2, 4, 8, 32), "gqa_long_decode": (1, 2, 4, 8)}
# chunks per row swept beside the library's choice for the row reductions
NORM_SWEEP = (1, 2, 4, 8, 16, 32)
# minimum warm-up before every timing: after an idle second the GPU needs
# about 100 steps of the causal prefill (tens of ms) to reach its clock
# (measured: 726-734 TFLOP/s after 3 warm-up steps, 842-851 after 300)
WARMUP_MS = 200.0
# input bytes that the workloads rotate through, 8x the memory-side cache, in
# at most MAX_COPIES copies (the tiny workload's inputs stay cache-sized)
COLD_BYTES = 2 << 30
MAX_COPIES = 32


def input_copies(nbytes):
    """Copies of an input of `nbytes` that span COLD_BYTES (2 to MAX_COPIES)."""
    return max(2, min(MAX_COPIES, -(-COLD_BYTES // nbytes)))


def kernel_source_hash(kind):
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kind]:
        with open(os.path.join(ROOT, "paper_2510_08726_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _profile_entry(kind, workload):
    """The committed rocprofv3 counter summary of a workload, or None when it
    is missing or was taken on a different version of the kernels."""
    path = os.path.join(PROFILES, "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    ent = data.get(f"{kind}:{workload}")
    if not ent or ent.get("source_hash") != kernel_source_hash(kind):
        return None
    return ent


def measured_traffic(kind, workload):
    ent = _profile_entry(kind, workload)
    return None if ent is None else ent.get("traffic_bytes_per_step")


def measured_mfma_busy(workload):
    """MFMA-busy fraction of SIMD cycles (SQ_VALU_MFMA_BUSY_CYCLES over
    GRBM_GUI_ACTIVE x SIMDs) from the committed counter profile, or None."""
    ent = _profile_entry("prefill", workload)
    return None if ent is None else ent.get("mfma_busy")


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--only", default=None, help="run only this workload (for profiler passes)")
    ap.add_argument("--splits", type=int, default=0, help="decode split count or norm chunks per row with --only (0: library)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--warmup-ms", type=float, default=WARMUP_MS,
                    help="minimum warm-up load before every timing (0: exactly W steps, for counter passes)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-errors", action="store_true")
    ap.add_argument("--no-peaks", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="budget of the headline oracle timing sample")
    return ap.parse_args()


def time_steps(fn, steps, warmup):
    """Mean ms per launch over `steps` back-to-back launches (HIP events on
    the launch stream around all of them), the host wall time per launch, and
    the min and max of `steps` more launches timed one by one.  `fn` is a
    callable or a list of callables that successive steps take in turn.
    Before them: `warmup` untimed steps, continued in batches until at least
    WARMUP_MS of wall time has passed (the GPU raises its clock only after
    tens of milliseconds of load)."""
    import torch
    fns = list(fn) if isinstance(fn, (list, tuple)) else [fn]
    n = len(fns)
    t0 = time.perf_counter()
    i = 0
    for _ in range(warmup):
        fns[i % n]()
        i += 1
    torch.cuda.synchronize()
    while (time.perf_counter() - t0) * 1e3 < WARMUP_MS:
        for _ in range(20):
            fns[i % n]()
            i += 1
        torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for i in range(steps):
        fns[i % n]()
    end.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for i, (a, b) in enumerate(pairs):
        a.record()
        fns[i % n]()
        b.record()
    torch.cuda.synchronize()
    each = [a.elapsed_time(b) for a, b in pairs]
    return start.elapsed_time(end) / steps, wall, {"min_ms": round(min(each), 5), "max_ms": round(max(each), 5)}


def _error_stats(got, ref):
    import numpy as np
    d = np.abs(np.asarray(got, dtype=np.float64) - ref).ravel()
    return {"max_abs": float(d.max()), "mean_abs": float(d.mean()), "rms": float(np.sqrt(np.mean(d * d))),
            "p90": float(np.percentile(d, 90)), "p99": float(np.percentile(d, 99))}


def attention_errors(w, q, k, v, sl, o):
    """|GPU - oracle| on a sample: prefill, two (batch, head) slices (the first
    and the last) on every row for L <= 4096, else on the first and last row of
    every 32-row block; decode, every row."""
    import numpy as np
    import oracle
    qn, kn, vn = (t.cpu().float().numpy() for t in (q, k, v))
    sln = None if sl is None else sl.cpu().double().numpy()
    og = o.cpu().float().numpy()
    if w.decode:
        ref = oracle.attention(qn, kn, vn, scale=w.sm_scale, causal=True, alibi_slopes=sln,
                               softcap=w.softcap or None)
        return {**_error_stats(og, ref), "sample": "every output row"}
    heads = sorted({(0, 0), (w.B - 1, w.Hq - 1)})
    rows = None
    if w.Lq > 4096:
        rows = sorted({r for r0 in range(0, w.Lq, 32) for r in (r0, min(r0 + 31, w.Lq - 1))})
    ref = oracle.attention(qn, kn, vn, scale=w.sm_scale, causal=w.causal, alibi_slopes=sln,
                           softcap=w.softcap or None, window=w.window or None, rows=rows, heads=heads)
    got = og if rows is None else og[:, :, rows]
    b = [h[0] for h in heads]
    hq = [h[1] for h in heads]
    sample = f"(batch, head) {heads}, " + ("every row" if rows is None else "first/last row of every 32-row block")
    return {**_error_stats(got[b, hq], ref[b, hq]), "sample": sample}


def run_workload(name, steps, warmup, *, splits=0, errors=False):
    import torch
    import paper_2510_08726_amd as pa
    from paper_2510_08726_amd.workloads import WORKLOADS, make_inputs, prefill_flops, decode_bytes

    w = WORKLOADS[name]
    q, k, v, sl = make_inputs(w, device="cuda")
    o = torch.empty_like(q)
    in_bytes = sum(t.numel() * t.element_size() for t in (q, k, v))
    sets = [(q, k, v)] + [(q.clone(), k.clone(), v.clone()) for _ in range(input_copies(in_bytes) - 1)]
    if w.decode:
        S = splits or w.num_splits or pa.attn_decode_num_splits(w.B, w.Hq, w.Hkv, w.Lk, w.D)
        ws = torch.empty(pa.attn_decode_workspace_bytes(w.B, w.Hq, w.D, S), dtype=torch.uint8,
                         device="cuda")
        work = decode_bytes(w.B, w.Hq, w.Hkv, w.Lk, w.D)

        def step(qs, ks, vs):
            return lambda: pa.attn_decode(qs, ks, vs, o, scale=w.sm_scale, alibi_slopes=sl,
                                          softcap=w.softcap or None, num_splits=S, workspace=ws)
        kernels = pa.attn_decode_kernels(w.Hq, w.Hkv, w.D, q.dtype, sl is not None, w.softcap)
        if S == 1:
            kernels = kernels[:1]   # one chunk: the split kernel writes O, no combine runs
    else:
        S = None

        def step(qs, ks, vs):
            return lambda: pa.attn_fwd(qs, ks, vs, o, causal=w.causal, scale=w.sm_scale, alibi_slopes=sl,
                                       softcap=w.softcap or None, window=w.window or None)
        work = prefill_flops(w.B, w.Hq, w.Lq, w.Lk, w.D, w.causal, w.window)
        kernels = pa.attn_fwd_kernels(w.D, q.dtype, w.causal, sl is not None, w.softcap, w.window)
    fn = [step(*t) for t in sets]
    ms, wall_ms, each = time_steps(fn, steps, warmup)
    # One input read by every step (the last calls: o is then set 0's output).
    ms_same = time_steps(fn[0], steps, warmup)[0]
    res = {
        "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "Lq": w.Lq, "Lk": w.Lk, "D": w.D, "dtype": w.dtype,
        "causal": w.causal, "alibi": w.alibi, "softcap": w.softcap, "window": w.window,
        "kernels": kernels, "ms_per_step": round(ms, 5), "launch_ms": each,
        "host_wall_ms_per_step": round(wall_ms, 5), "input_copies": len(sets),
    }
    if w.decode:
        gbs = work / (ms * 1e-3) / 1e9
        res.update({"num_splits": S, "bytes_per_step": work, "GB/s": round(gbs, 1),
                    "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
                    "GB/s_same_input": round(work / (ms_same * 1e-3) / 1e9, 1)})
    else:
        tf = work / (ms * 1e-3) / 1e12
        res.update({"flops_per_step": work, "TFLOP/s": round(tf, 2),
                    "pct_mfma_peak": round(100 * tf / MFMA_PEAK_TFLOPS, 2),
                    "TFLOP/s_same_input": round(work / (ms_same * 1e-3) / 1e12, 2)})
    err = attention_errors(w, q, k, v, sl, o) if errors else None
    del sets, fn
    del q, k, v, o
    torch.cuda.empty_cache()
    return res, err


def run_norm(name, steps, warmup, *, chunks=0, errors=False):
    import numpy as np
    import torch
    import paper_2510_08726_amd as pa
    from paper_2510_08726_amd.workloads import NORM_WORKLOADS, make_norm_input, norm_bytes

    w = NORM_WORKLOADS[name]
    x = make_norm_input(w, device="cuda")
    C = chunks or pa.norm_chunks(w.op, w.N, w.M, x.dtype)
    kernels = pa.norm_kernels(w.op, w.M, x.dtype, C)
    ws = torch.empty(pa.norm_workspace_bytes(w.N, C), dtype=torch.uint8, device="cuda")
    out = torch.empty(w.N, dtype=torch.float32, device="cuda")
    xs = [x] + [x.clone() for _ in range(input_copies(x.numel() * x.element_size()) - 1)]
    if w.op == "l2":
        def step(xi):
            return lambda: pa.norm_l2(xi, out, chunks=C, workspace=ws)
    else:
        y = torch.empty_like(x)

        def step(xi):
            return lambda: pa.rmsnorm_rowmax(xi, y, out, eps=w.eps, chunks=C, workspace=ws)
    fn = [step(xi) for xi in xs]
    ms, wall_ms, each = time_steps(fn, steps, warmup)
    ms_same = time_steps(fn[0], steps, warmup)[0]
    work = norm_bytes(w.op, w.N, w.M, x.element_size())
    gbs = work / (ms * 1e-3) / 1e9
    res = {"op": w.op, "N": w.N, "M": w.M, "dtype": w.dtype, "chunks": C, "kernels": kernels,
           "ms_per_step": round(ms, 5), "launch_ms": each,
           "host_wall_ms_per_step": round(wall_ms, 5), "bytes_per_step": work, "GB/s": round(gbs, 1),
           "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2), "input_copies": len(xs),
           "GB/s_same_input": round(work / (ms_same * 1e-3) / 1e9, 1)}
    del xs, fn
    err = None
    if errors:
        from oracle import norms
        x64 = x.cpu().double().numpy()
        if w.op == "l2":
            err = {**_error_stats(out.cpu().numpy(), norms.l2_norm(x64)), "sample": "every row norm"}
        else:
            yr, mr = norms.rmsnorm_rowmax(x64, w.eps)
            err = {"y": {**_error_stats(y.cpu().float().numpy(), yr), "sample": "every element of y"},
                   "rowmax": {**_error_stats(out.cpu().numpy(), mr), "sample": "every row max"}}
    del x
    torch.cuda.empty_cache()
    return res, err


def achievable_peaks():
    """What this GPU reaches in this run: a streaming read of 2 GiB (the
    decode bound) and the MFMA loop on random fp16 / bf16 operands (the
    prefill bound), with the shader clock the loop held."""
    import torch
    import paper_2510_08726_amd as pa
    out = {}
    buf = torch.empty(2 << 30, dtype=torch.uint8, device="cuda")
    buf.view(torch.float32).normal_()
    sink = pa.peaks_hbm_read(buf)
    torch.cuda.synchronize()
    ms, _, _ = time_steps(lambda: pa.peaks_hbm_read(buf, sink), 10, 2)
    out["hbm_read_GBs"] = round(buf.numel() / (ms * 1e-3) / 1e9, 1)
    out["hbm_read_frac_of_spec"] = round(out["hbm_read_GBs"] / HBM_PEAK_GBS, 4)
    del buf, sink
    ops = torch.randn(pa.peaks_mfma_operand_bytes() // 2, device="cuda")
    iters = 20000
    for dt, key in ((torch.float16, "f16"), (torch.bfloat16, "bf16")):
        o = ops.to(dt)
        t0 = time.perf_counter()
        while (time.perf_counter() - t0) * 1e3 < WARMUP_MS:   # the same warm-up as every workload
            pa.peaks_mfma(dt, iters, o)
            torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        _, ck = pa.peaks_mfma(dt, iters, o)
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e)
        flops = pa.peaks_mfma_waves() * iters * 16 * 32768
        c = ck.cpu().tolist()
        out[f"mfma_{key}_TFLOPs"] = round(flops / (ms * 1e-3) / 1e12, 1)
        out[f"mfma_{key}_frac_of_spec"] = round(out[f"mfma_{key}_TFLOPs"] / MFMA_PEAK_TFLOPS, 4)
        out[f"mfma_{key}_clock_GHz"] = round(c[0] / c[1] * 0.1, 3) if c[1] else None
    out["method"] = ("peaks_hbm_read over 2 GiB (10 launches); peaks_mfma: 32x32x16 MFMAs on operands "
                     "that change every instruction, 2 waves per SIMD, 20000 x 16 per wave, one launch; "
                     f"each after at least {WARMUP_MS:.0f} ms of the same load; clock from s_memtime / s_memrealtime")
    return out


def prefill_roofline(res, name, peaks, kernel):
    tf = res["TFLOP/s"]
    r = {"bound": "mfma", "achieved": tf, "peak": MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
         "frac": round(tf / MFMA_PEAK_TFLOPS, 4), "traffic": measured_traffic("prefill", name),
         "kernel": kernel,
         "per_launch": f"{res['flops_per_step']} algorithmic flops (4*D per visible query/key pair), one launch",
         "mfma_busy_counter": measured_mfma_busy(name)}
    key = "mfma_bf16_TFLOPs" if res["dtype"] == "bf16" else "mfma_f16_TFLOPs"
    if peaks and peaks.get(key):
        r["achievable_peak"] = peaks[key]
        r["frac_achievable"] = round(tf / peaks[key], 4)
    return r


def hbm_roofline(res, kind, name, peaks, what):
    gbs = res["GB/s"]
    r = {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
         "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": measured_traffic(kind, name),
         "per_launch": f"{res['bytes_per_step']} algorithmic bytes ({what})"}
    if peaks and peaks.get("hbm_read_GBs"):
        r["achievable_peak"] = peaks["hbm_read_GBs"]
        r["frac_achievable"] = round(gbs / peaks["hbm_read_GBs"], 4)
    return r


def copy_calibration(mib, steps):
    """A plain device-to-device copy of known size, for scaling HBM counters."""
    import torch
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(steps):
        b.copy_(a)
    torch.cuda.synchronize()


def _host():
    model = platform.processor() or "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        blas = max([d.get("num_threads", 1) for d in info if d.get("user_api") == "blas"] or [1])
    except Exception:
        blas = 1
    return model, os.cpu_count(), int(blas)


def cpu_baseline(budget_s):
    """The fp64 oracle timed on this host: whole (batch, head) slices of the
    headline workload for about `budget_s`, and a bounded sample of every
    other workload, each in its metric's unit."""
    import numpy as np
    import oracle
    from oracle import norms
    from paper_2510_08726_amd.workloads import (WORKLOADS, NORM_WORKLOADS, make_inputs, make_norm_input,
                                                prefill_flops, decode_bytes, norm_bytes)
    model, ncpu, cores = _host()

    def prefill_sample(w, budget, max_slices):
        q, k, v, sl = make_inputs(w)
        qn, kn, vn = (t.float().numpy() for t in (q, k, v))
        sln = None if sl is None else sl.double().numpy()
        heads = [(b, h) for b in range(w.B) for h in range(w.Hq)]
        done, t0 = 0, time.perf_counter()
        for bh in heads[:max_slices]:
            oracle.attention(qn, kn, vn, scale=w.sm_scale, causal=w.causal, alibi_slopes=sln,
                             softcap=w.softcap or None, window=w.window or None, heads=[bh])
            done += 1
            if time.perf_counter() - t0 >= budget:
                break
        el = time.perf_counter() - t0
        flops = prefill_flops(1, done, w.Lq, w.Lk, w.D, w.causal, w.window)
        return flops / el / 1e12, el, f"{done} of {len(heads)} (batch, head) slices, every query row"

    head_tf, head_el, head_sample = prefill_sample(WORKLOADS[HEADLINE], budget_s, 1 << 30)
    per = {}
    for name, w in WORKLOADS.items():
        if name == HEADLINE:
            continue
        if w.decode:
            q, k, v, sl = make_inputs(w)
            b = 1
            qn, kn, vn = (t[:b].float().numpy() for t in (q, k, v))
            t0 = time.perf_counter()
            oracle.attention(qn, kn, vn, scale=w.sm_scale, causal=True,
                             alibi_slopes=None if sl is None else sl.double().numpy(), softcap=w.softcap or None)
            el = time.perf_counter() - t0
            per[name] = {"value": round(decode_bytes(b, w.Hq, w.Hkv, w.Lk, w.D) / el / 1e9, 4), "unit": "GB/s",
                         "sample": f"batch 0 of {w.B}, every head", "seconds": round(el, 2)}
        else:
            tf, el, sample = prefill_sample(w, 2.0, 2)
            per[name] = {"value": round(tf, 6), "unit": "TFLOP/s", "sample": sample, "seconds": round(el, 2)}
    for name, w in NORM_WORKLOADS.items():
        x = make_norm_input(w)[:32].double().numpy()
        t0 = time.perf_counter()
        if w.op == "l2":
            norms.l2_norm(x)
        else:
            norms.rmsnorm_rowmax(x, w.eps)
        el = time.perf_counter() - t0
        per[name] = {"value": round(norm_bytes(w.op, 32, w.M, 2 if w.dtype != "f32" else 4) / el / 1e9, 4),
                     "unit": "GB/s", "sample": f"32 of {w.N} rows", "seconds": round(el, 4)}
    return {
        "value": round(head_tf, 6), "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
        "sample": f"{head_sample} of {HEADLINE}; float64 numpy, BLAS matmul on {cores} threads, exp "
                  f"single-threaded; {head_el:.1f} s",
        "seconds": round(head_el, 2), "cpu_model": model, "nproc": ncpu,
        "per_config": per,
    }


def main():
    global WARMUP_MS
    args = parse()
    WARMUP_MS = args.warmup_ms
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this library runs on exactly one GPU (no multi-GPU path); "
              "use --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2510_08726_amd as pa
    from paper_2510_08726_amd.workloads import WORKLOADS, NORM_WORKLOADS
    pa.load_library()
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)

    if args.only:
        if args.only in NORM_WORKLOADS:
            res, _ = run_norm(args.only, args.steps, args.warmup, chunks=args.splits)
        else:
            res, _ = run_workload(args.only, args.steps, args.warmup, splits=args.splits)
        if args.copy_mib:
            copy_calibration(args.copy_mib, args.steps)
        print(json.dumps({"workload": args.only, **res}), flush=True)
        return

    peaks = None if args.no_peaks else achievable_peaks()
    print(f"# achievable: {json.dumps(peaks)}", file=sys.stderr, flush=True)
    results, errors = {}, {}
    for name in WORKLOADS:
        results[name], errors[name] = run_workload(name, args.steps, args.warmup, errors=not args.no_errors)
        print(f"# {name}: {json.dumps(results[name])}", file=sys.stderr, flush=True)
    for name in NORM_WORKLOADS:
        results[name], errors[name] = run_norm(name, args.steps, args.warmup, errors=not args.no_errors)
        print(f"# {name}: {json.dumps(results[name])}", file=sys.stderr, flush=True)
    sweep = {}
    for wname, splits in SWEEPS.items():
        sweep[wname] = {"library_choice": results[wname]["num_splits"], "splits": {}}
        for S in splits:
            r, _ = run_workload(wname, args.steps, args.warmup, splits=S)
            sweep[wname]["splits"][str(S)] = {
                "GB/s": r["GB/s"], "ms_per_step": r["ms_per_step"],
                "frac": round(r["GB/s"] / HBM_PEAK_GBS, 4),
                "frac_achievable": round(r["GB/s"] / peaks["hbm_read_GBs"], 4) if peaks else None}
    for wname in NORM_WORKLOADS:
        sweep[wname] = {"library_choice": results[wname]["chunks"], "chunks": {}}
        for C in NORM_SWEEP:
            r, _ = run_norm(wname, args.steps, args.warmup, chunks=C)
            sweep[wname]["chunks"][str(C)] = {
                "GB/s": r["GB/s"], "ms_per_step": r["ms_per_step"], "kernels": r["kernels"],
                "frac": round(r["GB/s"] / HBM_PEAK_GBS, 4),
                "frac_achievable": round(r["GB/s"] / peaks["hbm_read_GBs"], 4) if peaks else None}
    print(f"# split sweep: {json.dumps(sweep)}", file=sys.stderr, flush=True)

    head = results[HEADLINE]
    w = WORKLOADS[HEADLINE]
    line = {
        "metric": METRIC, "value": head["TFLOP/s"], "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "warmup_min_ms": WARMUP_MS, "ms_per_step": head["ms_per_step"],
        "launch_ms": head["launch_ms"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": HEADLINE, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "Lq": w.Lq, "Lk": w.Lk,
                   "D": w.D, "causal": w.causal, "input": "iid N(0,1) fp16, seed 2"},
        "roofline": prefill_roofline(head, HEADLINE, peaks, head["kernels"][0]),
    }
    for key, name in SIDE.items():
        r = results[name]
        if WORKLOADS[name].decode:
            entry = {"workload": name, "value": r["GB/s"], "unit": "GB/s", "ms_per_step": r["ms_per_step"],
                     "num_splits": r["num_splits"],
                     "roofline": hbm_roofline(r, "decode", name, peaks, "|Q|+|K|+|V|+|O|, split (+ combine) kernels")}
        else:
            entry = {"workload": name, "value": r["TFLOP/s"], "unit": "TFLOP/s", "ms_per_step": r["ms_per_step"],
                     "roofline": prefill_roofline(r, name, peaks, r["kernels"][0])}
        line[key] = entry
    line["split_sweep"] = sweep
    line["norms"] = {name: {"workload": name, "value": results[name]["GB/s"], "unit": "GB/s",
                            "ms_per_step": results[name]["ms_per_step"],
                            "roofline": hbm_roofline(results[name], "norms", name, peaks,
                                                     "X read once + the [N] fp32 outputs (+ Y written, RMSNorm)")}
                     for name in NORM_WORKLOADS}
    line["achievable"] = peaks
    if not args.no_errors:
        line["errors"] = errors
    line["workloads"] = results
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
