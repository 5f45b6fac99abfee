"""Build the HIP rollout library for gfx950 in-tree.

    python -m paper_2609_13716_amd.build

compiles every ``csrc/*.hip`` translation unit with hipcc and links them into
``paper_2609_13716_amd/librollout.so`` (the only artefact the Python binding
loads).  Packed float32 instructions are disabled on every device compile.

    python -m paper_2609_13716_amd.build --stamps

builds the instrumented variant ``paper_2609_13716_amd/librollout_stamps.so``
instead (RL_PHASE_STAMPS: per-phase cycle counters in the step loops of the
fused and env-only kernels, read by ``bench.py --phases``); the product
library is never built with them.
"""

import concurrent.futures
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "librollout.so")
OBJDIR = os.path.join(PKG, "_build")
LIB_STAMPS = os.path.join(PKG, "librollout_stamps.so")
OBJDIR_STAMPS = os.path.join(PKG, "_build_stamps")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fno-fast-math", "-ffp-contract=fast-honor-pragmas",
    "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas",
    "-I", INCLUDE, "-I", CSRC,
]


def _compile(src, stamps=False):
    obj = os.path.join(OBJDIR_STAMPS if stamps else OBJDIR, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, *(["-DRL_PHASE_STAMPS"] if stamps else []), "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(line for line in (r.stdout + r.stderr).splitlines()
                     if "packed-fp32-ops" not in line)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{out}")
    return obj, out


def build(verbose=False, stamps=False):
    """Compile and link the library (or, with stamps, its instrumented variant); returns its path.
    Always rebuilds."""
    lib = LIB_STAMPS if stamps else LIB
    os.makedirs(OBJDIR_STAMPS if stamps else OBJDIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        results = list(ex.map(lambda src: _compile(src, stamps), srcs))
    if verbose:
        for _, out in results:
            if out.strip():
                print(out)
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *[o for o, _ in results]]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, stamps="--stamps" in sys.argv))
