"""Build the gfx950 attention library (libattn.so) in-tree with hipcc.

Every HIP source is compiled for gfx950 only, with packed-fp32 instruction
selection disabled; the host-only C ABI file is compiled as plain C++.  The
library is written next to this file, where the Python binding loads it.
"""

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libattn.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
COMMON = ["-O3", "-std=c++20", "-fPIC", "-I", INCLUDE, "-I", CSRC]
DEVICE = ["-x", "hip", f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wno-unused-command-line-argument"]
# (object name, source, extra flags).  prefill.hip is compiled once per
# (head dim, element type) shard so its instantiations build in parallel.
# Its softmax never needs IEEE NaN handling of max: without it, fmaxf of
# values produced by inline assembly compiles to a plain v_max instead of
# canonicalising both inputs first.  The prefill device assembly is kept
# (-save-temps) for the ISA hazard check in the tests.
UNITS = [(f"prefill{k}", "prefill.hip", ["-fno-honor-nans", f"-DATTN_PREFILL_SHARD={k}", "-save-temps"])
         for k in range(4)] + [("decode", "decode.hip", []), ("attn_api", "attn_api.cpp", [])]


def unit_dir(name):
    """Working directory of one compile (holds its -save-temps files)."""
    return os.path.join(OBJDIR, name)


def prefill_asm_files():
    """Device assembly of the prefill shards written by the last build()."""
    return [os.path.join(unit_dir(f"prefill{k}"), f"prefill-hip-amdgcn-amd-amdhsa-{ARCH}.s") for k in range(4)]


def build(verbose=False):
    """Compile every source (in parallel) and link libattn.so.  Raises on failure."""
    os.makedirs(OBJDIR, exist_ok=True)
    procs = []
    objs = []
    for name, src, flags in UNITS:
        path = os.path.join(CSRC, src)
        obj = os.path.join(OBJDIR, name + ".o")
        objs.append(obj)
        extra = (DEVICE if src.endswith(".hip") else []) + flags
        cmd = [HIPCC, *COMMON, *extra, "-c", path, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        os.makedirs(unit_dir(name), exist_ok=True)
        procs.append((name, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                                             cwd=unit_dir(name))))
    failed = []
    for src, pr in procs:
        out, _ = pr.communicate()
        if pr.returncode != 0:
            failed.append(f"--- {src} ---\n{out}")
        elif verbose and out.strip():
            print(out)
    if failed:
        raise RuntimeError("hipcc failed:\n" + "\n".join(failed))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
