"""Build libbranchattn.so (gfx950) in-tree.

    python -m paper_2609_07108_amd.build

Every HIP source is compiled for gfx950 only with packed-FP32 instruction
selection disabled; the result lands in ``paper_2609_07108_amd/_lib``.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(HERE, "_lib")
LIB_NAME = "libbranchattn.so"

HIP_SOURCES = ["plan.hip", "lse_merge.hip", "fwd.hip", "bwd.hip", "rope.hip", "proj.hip", "api.hip"]
HOST_SOURCES = []

ARCH = "gfx950"
COMMON_FLAGS = ["-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function",
                f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]
# -amdgpu-mfma-vgpr-form: MFMA results go to ordinary vector registers.  The
# dK/dV kernel runs one wavefront per SIMD (512 registers) and would
# otherwise get every MFMA accumulator in the accumulation registers, with a
# copy per softmax element; its long-lived dK/dV accumulators are pinned to
# the accumulation registers explicitly instead.
HIP_FLAGS = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wno-inline-asm",
             "-munsafe-fp-atomics", "-mllvm", "-amdgpu-mfma-vgpr-form=1"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    noise = "is not a recognized feature for this target"
    text = "\n".join(l for l in r.stdout.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({' '.join(cmd)}):\n{text}")
    if text.strip():
        print(text, file=sys.stderr)


def compiler_version() -> str:
    r = subprocess.run([hipcc(), "--version"], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    return next((l.strip() for l in r.stdout.splitlines() if "clang version" in l), r.stdout.strip())


# The compiler whose output was last checked by hand as well as by the hazard
# check below.  Another version still builds (the check runs on whatever it
# generates) but says so.
VERIFIED_COMPILER = "AMD clang version 22.0.0git (https://github.com/RadeonOpenCompute/llvm-project roc-7.2.0 26014"


def build(verbose: bool = False, jobs: int = 4) -> str:
    """Compile every source and link the shared library; returns its path.

    The device assembly of every source is kept (``-save-temps``) and run
    through :mod:`hazards`: the inline-assembly MFMAs and direct loads carry
    wait-state requirements that the compiler does not pad, and a build whose
    generated code breaks one is refused."""
    from . import hazards

    os.makedirs(OUT_DIR, exist_ok=True)
    cc = hipcc()
    ver = compiler_version()
    if not ver.startswith(VERIFIED_COMPILER):
        print(f"note: compiler {ver!r} differs from the one the kernels' schedules were last read under; "
              f"relying on the generated-code hazard check", file=sys.stderr)
    tmp = tempfile.mkdtemp(prefix="ba_build_", dir=OUT_DIR)
    try:
        objs, procs = [], []
        for src in HIP_SOURCES + HOST_SOURCES:
            obj = os.path.join(tmp, os.path.splitext(src)[0] + ".o")
            cmd = [cc] + COMMON_FLAGS + (HIP_FLAGS + ["-save-temps=obj"] if src.endswith(".hip") else []) + \
                ["-c", os.path.join(CSRC, src), "-o", obj]
            if verbose:
                print(" ".join(cmd))
            procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
            objs.append(obj)
            if len([p for _, p in procs if p.poll() is None]) >= jobs:
                procs[0][1].wait()
        noise = "is not a recognized feature for this target"
        for cmd, p in procs:
            out, _ = p.communicate()
            text = "\n".join(l for l in out.splitlines() if noise not in l)
            if p.returncode != 0:
                raise RuntimeError(f"compile failed ({' '.join(cmd)}):\n{text}")
            if text.strip():
                print(text, file=sys.stderr)
        errs = []
        for src in HIP_SOURCES:
            asm = os.path.join(tmp, f"{os.path.splitext(src)[0]}-hip-amdgcn-amd-amdhsa-{ARCH}.s")
            if not os.path.exists(asm):
                raise RuntimeError(f"device assembly of {src} missing ({asm}): cannot run the hazard check")
            errs += hazards.check_file(asm)
        if errs:
            raise RuntimeError("hazard check failed on the generated code:\n" + "\n".join(errs[:40]))
        lib_tmp = os.path.join(tmp, LIB_NAME)
        _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", lib_tmp] + objs)
        dst = os.path.join(OUT_DIR, LIB_NAME)
        os.replace(lib_tmp, dst)
        return dst
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
