"""Build libmdnn.so (gfx950) in-tree with hipcc.

    python paper_2011_11188_amd/build.py      # (not -m: that imports the package,
                                              #  which loads the library being rebuilt)

Every source under csrc/ is compiled to an object in _build/ (in parallel),
then linked into paper_2011_11188_amd/libmdnn.so.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import re
import subprocess
import sys
import time

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
OUT_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libmdnn.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
          f"-I{os.path.join(os.path.dirname(PKG), 'include')}"]
# Packed fp32 instructions are disabled for all device code.  MFMA results
# are kept in VGPRs (in-place accumulation), which the kernels are sized for.
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-mllvm", "-amdgpu-mfma-vgpr-form=1"]


RESOURCE_REMARK = "kernel-resource-usage"


def _diagnostics(lines) -> list:
    """Compiler output without the resource-usage remarks (read by _spills)
    and their include-chain and source-excerpt lines, and without the host
    pass's note that it does not know the packed-fp32 target feature."""
    out, pending, in_remark = [], [], False
    for line in lines:
        if not line.strip() or "packed-fp32-ops" in line:
            continue
        if line.startswith("In file included from"):
            pending.append(line)
            continue
        excerpt = re.match(r"^\s*(\d+\s*)?\|", line) is not None
        if RESOURCE_REMARK in line:
            pending, in_remark = [], True
            continue
        if excerpt and in_remark:
            continue
        in_remark = False
        out.extend(pending)
        pending = []
        out.append(line)
    return out + pending


def _spills(lines) -> list:
    """Kernels whose resource-usage remarks report vector registers spilled
    to scratch memory (scalar spills go to vector-register lanes: cheap)."""
    out, name = [], None
    for line in lines:
        if "Function Name:" in line:
            name = line.split("Function Name:")[1].split()[0]
        elif "VGPRs Spill:" in line and name is not None:
            n = int(line.split("Spill:")[1].split()[0])
            if n > 0:
                out.append(f"{name}: {line.split('remark:')[1].split('[')[0].strip()}")
    return out


def _compile(src: str) -> str:
    obj = os.path.join(OUT_DIR, os.path.basename(src) + ".o")
    if src.endswith(".hip"):
        cmd = [HIPCC, "-x", "hip", *DEVICE, *COMMON, f"-Rpass-analysis={RESOURCE_REMARK}", "-c", src, "-o", obj]
    else:
        cmd = [HIPCC, *COMMON, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    lines = (r.stdout + r.stderr).splitlines()
    msgs = "\n".join(_diagnostics(lines))
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{msgs}")
    if msgs:
        print(msgs, file=sys.stderr)
    # a kernel that spills vector registers to scratch has outgrown its budget
    for s in _spills(lines):
        print(f"warning: {os.path.basename(src)}: register spill in {s}", file=sys.stderr)
    return obj


def build(verbose: bool = True) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))
    t0 = time.time()
    workers = min(len(srcs), int(os.environ.get("MDNN_BUILD_JOBS", "8")))
    with cf.ThreadPoolExecutor(max_workers=workers) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB} from {len(srcs)} sources in {time.time() - t0:.1f}s", file=sys.stderr)
    return LIB


if __name__ == "__main__":
    build()
