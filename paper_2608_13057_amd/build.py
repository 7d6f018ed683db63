"""Build libtempo_moe.so (the HIP library behind include/tempo_moe.h) for
gfx950 with hipcc, in-tree, next to this file.  Cross-compiles without a GPU.

    python -m paper_2608_13057_amd.build
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libtempo_moe.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # no packed-fp32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]
# MFMA accumulators in VGPRs: the stream-K GEMMs add chunk accumulators with
# VALU, and the AGPR form would copy them back and forth every step.  The
# large-tile GEMM (files ending in _agpr.hip) keeps its 256 accumulator
# registers per lane in AGPRs instead.
VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form"]


def flags_for(src: str):
    return FLAGS if src.endswith("_agpr.hip") else FLAGS + VGPR_FORM


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(CSRC, "*.cpp")))


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every translation unit (in parallel) and link the shared
    library; always rebuilds."""
    with tempfile.TemporaryDirectory(prefix="tempo_build_") as tmp:
        procs = []
        objs = []
        for src in sources():
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            objs.append(obj)
            cmd = [HIPCC, *flags_for(src), "-c", src, "-o", obj]
            if src.endswith(".cpp"):
                cmd = [HIPCC, "-x", "hip", *flags_for(src), "-c", src, "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
            while len([p for _, p in procs if p.poll() is None]) >= jobs:
                procs[0][1].wait(timeout=None) if procs[0][1].poll() is None else None
                for _, p in procs:
                    if p.poll() is None:
                        p.wait()
                        break
        failed = []
        for src, p in procs:
            out = p.communicate()[0].decode(errors="replace")
            out = "\n".join(l for l in out.splitlines() if "packed-fp32-ops" not in l)
            if p.returncode != 0:
                failed.append((src, out))
            elif verbose and out.strip():
                print(out)
        if failed:
            msg = "\n".join(f"--- {s}\n{o}" for s, o in failed)
            raise RuntimeError(f"hipcc failed:\n{msg}")
        tmp_lib = LIB + ".tmp"
        subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp_lib, *objs], check=True)
        os.replace(tmp_lib, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
