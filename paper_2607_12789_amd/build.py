"""Builds ``libavq.so`` (the gfx950 HIP kernels and their C ABI) in-tree.

    python -m paper_2607_12789_amd.build

Every HIP source is compiled with hipcc for gfx950 only, with the packed-fp32
instructions disabled. Device code is compiled without NaN semantics
(``-fno-honor-nans``): the maxima and minima over MFMA results then need no
sNaN-quieting canonicalisation of each operand (one extra VALU instruction per
value in the softmax max and the argmin); host code keeps IEEE semantics.
MFMA results are kept in architectural VGPRs (``-amdgpu-mfma-vgpr-form``): the
assignment kernels compare every product with VALU instructions, which cannot
read accumulation registers, so products left there cost one extra move per
value.
"""
from __future__ import annotations

import os
import subprocess
import sys
from pathlib import Path

PKG = Path(__file__).resolve().parent
ROOT = PKG.parent
CSRC = PKG / "csrc"
LIB = PKG / "libavq.so"
SOURCES = ["avq_api.hip", "avq_assign.hip", "avq_aggregate.hip", "avq_attention.hip",
           "avq_codebook.hip", "avq_order.hip", "avq_pack.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMPILE_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Xarch_device", "-fno-honor-nans",
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
    "-Wall",
]


def build(verbose: bool = False) -> Path:
    """Compile the library; always recompiles."""
    objs = []
    procs = []
    for src in SOURCES:
        obj = CSRC / (Path(src).stem + ".o")
        cmd = [HIPCC, *COMPILE_FLAGS, "-c", str(CSRC / src), "-o", str(obj)]
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        objs.append(obj)
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        # the host pass does not know the packed-fp32 feature; that warning is expected
        lines = [ln for ln in text.splitlines() if "packed-fp32-ops" not in ln]
        if p.returncode != 0:
            failed.append(src)
            sys.stderr.write("\n".join(lines) + "\n")
        elif verbose and lines:
            sys.stderr.write("\n".join(lines) + "\n")
    if failed:
        raise RuntimeError(f"hipcc failed for {failed}")
    tmp = LIB.with_suffix(".so.tmp")
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *map(str, objs), "-o",
                    str(tmp)], check=True)
    os.replace(tmp, LIB)
    for o in objs:
        o.unlink(missing_ok=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
