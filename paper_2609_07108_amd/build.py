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
HIP_FLAGS = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
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


def build(verbose: bool = False, jobs: int = 4) -> str:
    """Compile every source and link the shared library; returns its path."""
    os.makedirs(OUT_DIR, exist_ok=True)
    cc = hipcc()
    tmp = tempfile.mkdtemp(prefix="ba_build_", dir=OUT_DIR)
    try:
        objs, procs = [], []
        for src in HIP_SOURCES + HOST_SOURCES:
            obj = os.path.join(tmp, os.path.splitext(src)[0] + ".o")
            cmd = [cc] + COMMON_FLAGS + (HIP_FLAGS if src.endswith(".hip") else []) + \
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
        lib_tmp = os.path.join(tmp, LIB_NAME)
        _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", lib_tmp] + objs)
        dst = os.path.join(OUT_DIR, LIB_NAME)
        os.replace(lib_tmp, dst)
        return dst
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
