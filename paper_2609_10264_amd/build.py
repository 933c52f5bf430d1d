"""Build the HIP libraries behind include/mvk.h for gfx950 with hipcc.

    python -m paper_2609_10264_amd.build

The same sources are built once per field: libmvk.so over 2^31 - 1 and
libmvk_bb.so over BabyBear (15 * 2^27 + 1, macro MVK_FIELD_BABYBEAR).  Always
recompiles.  The translation units of both builds are compiled in parallel,
then each build is linked into one shared object next to this file.
"""
from __future__ import annotations

import os
import re
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


# Source files whose kernels issue loads through inline assembly (the compiler
# does not know those loads are in flight until the kernel's explicit wait).
ASM_LOAD_SOURCES = ("server_eval.hip",)


def _vregs(tok: str) -> set:
    m = re.match(r"v\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


_VMEM = ("global_", "buffer_", "flat_", "scratch_")  # every vector-memory op counts on vmcnt
_VMEM_LOAD = ("global_load", "buffer_load", "flat_load", "scratch_load")
_VMEM_STORE = ("global_store", "buffer_store", "flat_store", "scratch_store")


def asm_load_hazards(asm_text: str) -> list:
    """Uses of registers that an inline-assembly global_load_dwordx4 of the
    same kernel still targets.  The compiler treats the asm output as ready
    when the asm statement ends, so under register pressure it may

      * copy the register (v_mov*, v_accvgpr*): the copy reads it before the
        load lands;
      * write the register, reusing it for another value (a VALU instruction
        or a compiler-issued load with it as destination): the late load data
        then overwrites that value (a corrupted address, a memory fault);
      * spill it to scratch (a store of it): the spilled copy is stale.

    A load is in flight from its issue until a wait that covers it: every
    vector-memory instruction (load, store, LDS DMA) counts on vmcnt in issue
    order, and `s_waitcnt vmcnt(N)` returns once all but the N most recent
    have completed.  The scan follows the text of each kernel in order (a loop
    body once).  Returns [(kernel, instruction)] for every such use."""
    bad, cur, inasm = [], None, False
    inflight = []  # per vector-memory op in issue order: the registers an asm load of it targets
    for line in asm_text.split("\n"):
        m = re.match(r"^(_Z\S+):", line)
        if m:
            cur, inflight = m.group(1), []
            continue
        if cur is None:
            continue
        if "s_endpgm" in line:
            cur = None
            continue
        if ";;#ASMSTART" in line:
            inasm = True
            continue
        if ";;#ASMEND" in line:
            inasm = False
            continue
        parts = line.strip().split(None, 1)
        if not parts or parts[0].startswith((";", ".")):
            continue
        op, args = parts[0], [a.strip() for a in parts[1].split(",")] if len(parts) > 1 else []
        if op == "s_waitcnt":
            w = re.search(r"vmcnt\((\d+)\)", line)
            if w:
                keep = int(w.group(1))
                inflight = inflight[len(inflight) - keep:] if keep < len(inflight) else inflight
                if keep == 0:
                    inflight = []
            continue
        dests = set().union(*inflight) if inflight else set()
        if op.startswith(_VMEM):
            if not inasm and dests:
                if op.startswith(_VMEM_STORE):
                    # the stored data: scratch/global/flat stores name it second (after the address
                    # or "off"), buffer stores first
                    data = args[0] if op.startswith("buffer_store") else (args[1] if len(args) > 1 else "")
                    if _vregs(data) & dests:
                        bad.append((cur, line.strip()))
                elif op.startswith(_VMEM_LOAD) and args and _vregs(args[0]) & dests:
                    bad.append((cur, line.strip()))
            is_asm_load = inasm and op == "global_load_dwordx4" and bool(args)
            inflight.append(_vregs(args[0]) if is_asm_load else set())
            continue
        if inasm or not dests or not args:
            continue
        if op.startswith("v_mov") or op.startswith("v_accvgpr"):
            if any(_vregs(a) & dests for a in args[1:]):
                bad.append((cur, line.strip()))
                continue
        if op.startswith("v_") and _vregs(args[0]) & dests:
            bad.append((cur, line.strip()))
    return bad


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

    def check_asm(job) -> list:
        # device assembly of a translation unit with inline-assembly loads
        _, src, obj, flags = job
        out = obj.replace(".o", ".s")
        cmd = [cc, *HIPCC_FLAGS, *flags, "--cuda-device-only", "-S", src, "-o", out]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc -S failed for {src}:\n{r.stdout}{r.stderr}")
        with open(out) as f:
            return asm_load_hazards(f.read())

    asm_jobs = [j for j in jobs if os.path.basename(j[1]) in ASM_LOAD_SOURCES]
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_one, jobs))
        hazards = [h for hs in ex.map(check_asm, asm_jobs) for h in hs]
    if hazards:
        lines = "\n".join(f"  {k}: {i}" for k, i in hazards[:20])
        raise RuntimeError(f"registers of in-flight inline-assembly loads are copied, overwritten or spilled "
                           f"({len(hazards)}):\n{lines}")
    for name, (lib, _) in VARIANTS.items():
        mine = [o for o, j in zip(objs, jobs) if j[0] == name]
        tmp = lib + f".tmp{os.getpid()}"
        # -z defs: a symbol that no object defines fails the link, not the first load
        cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Wl,-z,defs", "-o", tmp, *mine]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed ({name}):\n{r.stdout}{r.stderr}")
        os.replace(tmp, lib)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
