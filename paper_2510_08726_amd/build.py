"""Build the gfx950 attention library (libattn.so) in-tree with hipcc.

Every HIP source is compiled for gfx950 only, with packed-fp32 instruction
selection disabled; the host-only C ABI file is compiled as plain C++.  The
library is written next to this file, where the Python binding loads it.

The prefill kernels keep their long-lived operands in fixed AGPRs (a0..a101)
named by inline assembly.  A kernel that uses AGPRs gets half of its register
budget per file by default (128 VGPRs at two waves per SIMD); the LLVM
function attribute "amdgpu-agpr-alloc" sets the AGPR share instead, but has
no source-level spelling.  So the prefill units run hipcc's own compile steps
(as printed by `hipcc -###`) and set the attribute on every kernel in the
device IR between the front end and the back end, which leaves the kernels
256 - 104 = 152 VGPRs at D = 128 and 256 - 56 = 200 at D = 64.
"""

import os
import re
import shlex
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libattn.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
LLVM_DIS = "/opt/rocm/llvm/bin/llvm-dis"
# AGPRs reserved for the prefill kernels' fixed operands, in the allocation
# granularity of 4, per shard: D = 128 (shards 0, 1) uses a0..a101, D = 64
# (shards 2, 3) a0..a53.
PREFILL_AGPRS = {0: 104, 1: 104, 2: 56, 3: 56}
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
         for k in range(4)] + [("decode", "decode.hip", ["-save-temps"]), ("peaks", "peaks.hip", ["-save-temps"]),
            ("norms", "norms.hip", ["-save-temps"]),
            ("attn_api", "attn_api.cpp", [])]


def unit_dir(name):
    """Working directory of one compile (holds its -save-temps files)."""
    return os.path.join(OBJDIR, name)


def device_asm_files():
    """Device assembly of every kernel unit written by the last build()."""
    return prefill_asm_files() + [os.path.join(unit_dir(u), f"{u}-hip-amdgcn-amd-amdhsa-{ARCH}.s")
                                  for u in ("decode", "peaks", "norms")]


def prefill_asm_files():
    """Device assembly of the prefill shards written by the last build()."""
    return [os.path.join(unit_dir(f"prefill{k}"), f"prefill-hip-amdgcn-amd-amdhsa-{ARCH}.s") for k in range(4)]


def set_agpr_alloc(bc_path, agprs):
    """Rewrite the device IR file `bc_path` (as text IR, which the back end
    reads alike) with "amdgpu-agpr-alloc"=agprs on every kernel."""
    ll = subprocess.run([LLVM_DIS, bc_path, "-o", "-"], capture_output=True, text=True, check=True).stdout
    groups = set(re.findall(r"define [^\n]*amdgpu_kernel void @[^\n]*\) #(\d+)", ll))
    if not groups:
        raise RuntimeError(f"no kernel found in {bc_path}")
    for g in groups:
        ll, n = re.subn(r"(attributes #%s = \{ )" % g, r'\g<1>"amdgpu-agpr-alloc"="%d" ' % agprs, ll)
        if n != 1:
            raise RuntimeError(f"attribute group #{g} not found in {bc_path}")
    with open(bc_path, "w") as f:
        f.write(ll)


def compile_with_agprs(cmd, cwd, agprs):
    """Run the compile steps that `cmd` (a hipcc -c line with -save-temps)
    stands for, setting the AGPR allocation of its device kernels after the
    front end.  Returns (returncode, output)."""
    r = subprocess.run([cmd[0], "-###", *cmd[1:]], cwd=cwd, capture_output=True, text=True)
    if r.returncode != 0:
        return r.returncode, r.stdout + r.stderr
    steps = [shlex.split(line) for line in r.stderr.splitlines() if line.startswith(' "')]
    patched = False
    for a in steps:
        s = subprocess.run(a, cwd=cwd, capture_output=True, text=True)
        if s.returncode != 0:
            return s.returncode, " ".join(a[:3]) + " ...\n" + s.stdout + s.stderr
        if "-emit-llvm-bc" in a and "-triple" in a and a[a.index("-triple") + 1].startswith("amdgcn"):
            set_agpr_alloc(os.path.join(cwd, a[a.index("-o") + 1]), agprs)
            patched = True
    if not patched:
        return 1, "the device front-end step was not found in: " + r.stderr[-2000:]
    return 0, ""


def build(verbose=False):
    """Compile every source (in parallel) and link libattn.so.  Raises on failure."""
    os.makedirs(OBJDIR, exist_ok=True)
    jobs = []
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
        jobs.append((name, src, cmd))

    def run(job):
        name, src, cmd = job
        if src == "prefill.hip":
            return compile_with_agprs(cmd, unit_dir(name), PREFILL_AGPRS[int(name[len("prefill"):])])
        p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, cwd=unit_dir(name))
        return p.returncode, p.stdout

    failed = []
    with ThreadPoolExecutor(max_workers=len(jobs)) as ex:
        for (name, _, _), (rc, out) in zip(jobs, ex.map(run, jobs)):
            if rc != 0:
                failed.append(f"--- {name} ---\n{out}")
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
