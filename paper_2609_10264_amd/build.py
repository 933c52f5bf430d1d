"""Build the HIP libraries behind include/mvk.h for gfx950 with hipcc.

    python -m paper_2609_10264_amd.build

The same sources are built once per field: libmvk.so over 2^31 - 1 and
libmvk_bb.so over BabyBear (15 * 2^27 + 1, macro MVK_FIELD_BABYBEAR).  Always
recompiles.  The translation units of both builds are compiled in parallel,
then each build is linked into one shared object next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmvk.so")
LIB_BB = os.path.join(PKG, "libmvk_bb.so")
ARCH = "gfx950"
# field name -> (library, extra compiler flags)
VARIANTS = {"m31": (LIB, []), "babybear": (LIB_BB, ["-DMVK_FIELD_BABYBEAR"])}

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-core accumulators in VGPRs: with AGPR accumulators the register
    # allocator copies accumulator tiles around every MFMA of the streamed loop
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wall", "-Wno-unused-function",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def sources() -> list[str]:
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def build(verbose: bool = False) -> str:
    """Compile and link every field variant; returns the 2^31 - 1 library's path."""
    cc = hipcc()
    jobs = []
    for name, (_, flags) in VARIANTS.items():
        objdir = os.path.join(PKG, "_build", name)
        os.makedirs(objdir, exist_ok=True)
        for src in sources():
            jobs.append((name, src, os.path.join(objdir, os.path.basename(src).replace(".hip", ".o")), flags))

    def compile_one(job) -> str:
        _, src, obj, flags = job
        cmd = [cc, *HIPCC_FLAGS, *flags, "-c", src, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                        if "packed-fp32-ops" not in l)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src} ({job[0]}):\n{out}")
        if verbose and out.strip():
            print(out, file=sys.stderr)
        return obj

    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_one, jobs))
    for name, (lib, _) in VARIANTS.items():
        mine = [o for o, j in zip(objs, jobs) if j[0] == name]
        tmp = lib + f".tmp{os.getpid()}"
        cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *mine]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed ({name}):\n{r.stdout}{r.stderr}")
        os.replace(tmp, lib)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
