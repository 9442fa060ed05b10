"""Build libgca.so (HIP, gfx950) in-tree with hipcc.

``python -m paper_2410_01651_amd.build`` or ``build()`` compiles every source
under ``csrc/`` and links ``paper_2410_01651_amd/libgca.so``.  Objects go to
``paper_2410_01651_amd/_build/``.  Always recompiles (a build check must
compile, not reuse).
"""

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(HERE, "libgca.so")
OBJ_DIR = os.path.join(HERE, "_build")

SOURCES = ["api.cpp", "plan.cpp", "noalloc.hip", "scores.hip", "select.hip", "xattn_fwd.hip", "xattn_decode.hip",
           "xattn_bwd.hip"]
# The attention kernels never rely on NaN semantics: without IEEE mode the
# softmax max needs no operand canonicalisation, and MFMA accumulators in
# ordinary VGPRs need no copies out of the accumulation registers.
PER_SOURCE = {
    "xattn_fwd.hip": ["-mno-amdgpu-ieee", "-fno-honor-nans", "-mllvm", "-amdgpu-mfma-vgpr-form"],
    "xattn_decode.hip": ["-mno-amdgpu-ieee", "-fno-honor-nans", "-mllvm", "-amdgpu-mfma-vgpr-form"],
    "xattn_bwd.hip": ["-mno-amdgpu-ieee", "-fno-honor-nans", "-mllvm", "-amdgpu-mfma-vgpr-form"],
}
ARCH = "gfx950"

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # packed fp32 VALU forms are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libgca)")


def build(verbose: bool = False, jobs: int = 4) -> str:
    cc = hipcc()
    os.makedirs(OBJ_DIR, exist_ok=True)
    procs = []
    objs = []
    for src in SOURCES:
        obj = os.path.join(OBJ_DIR, os.path.splitext(src)[0] + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmd = [cc, *COMMON, *PER_SOURCE.get(src, []), *lang, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        objs.append(obj)
        if len([p for _, p in procs if p.poll() is None]) >= jobs:
            procs[0][1].wait()
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        if p.returncode != 0:
            failed.append((src, text))
        elif verbose and text.strip():
            print(text)
    if failed:
        msg = "\n".join(f"--- {s} ---\n{t}" for s, t in failed)
        raise RuntimeError(f"libgca build failed:\n{msg}")
    tmp = OUT + ".tmp"
    cmd = [cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    if r.returncode != 0:
        raise RuntimeError("libgca link failed:\n" + r.stdout.decode(errors="replace"))
    os.replace(tmp, OUT)
    return OUT


def build_peaks() -> str:
    """The on-device reference-rate probes bench.py reports next to the spec peaks
    (a measurement aid, not part of libgca): peaks/libpeaks.so."""
    src = os.path.join(ROOT, "peaks", "peaks.hip")
    out = os.path.join(ROOT, "peaks", "libpeaks.so")
    cmd = [hipcc(), "-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wno-unused-command-line-argument",
           src, "-o", out + ".tmp"]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    if r.returncode != 0:
        raise RuntimeError("peaks build failed:\n" + r.stdout.decode(errors="replace"))
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
