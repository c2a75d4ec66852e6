"""Build the HIP library libmbp.so in-tree for gfx950 (hipcc cross-compiles; no GPU needed)."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmbp.so")
SOURCES = ["kernels.hip", "engine.hip", "runtime.hip"]
ARCH = os.environ.get("MBP_OFFLOAD_ARCH", "gfx950")

# Packed-FP32 instructions are disabled for all device code: hipcc would otherwise
# emit v_pk_{add,mul,fma}_f32 from ordinary float code.
HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-result",
    # per-kernel registers, scratch and LDS, recorded in _build/kernel_resources.tsv
    "-Rpass-analysis=kernel-resource-usage",
]
RESOURCES = os.path.join(PKG, "_build", "kernel_resources.tsv")
_FIELDS = {"VGPRs": "vgprs", "AGPRs": "agprs", "ScratchSize [bytes/lane]": "scratch",
           "Occupancy [waves/SIMD]": "occupancy", "LDS Size [bytes/block]": "lds"}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False) -> str:
    """Compile every source to an object file, then link the shared library."""
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs, kernels = [], []
    for src in SOURCES:
        obj = os.path.join(objdir, src.replace(".hip", ".o"))
        cmd = [hipcc(), *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", obj]
        kernels += _resources(src, _run(cmd, verbose))
        objs.append(obj)
    with open(RESOURCES, "w") as f:
        f.write("source\tkernel\tvgprs\tagprs\tscratch\toccupancy\tlds\n")
        for k in kernels:
            f.write("\t".join(str(k.get(c, "")) for c in ("source", "kernel", "vgprs", "agprs", "scratch", "occupancy", "lds")) + "\n")
    tmp = LIB + ".tmp"
    _run([hipcc(), "-shared", f"--offload-arch={ARCH}", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


def _resources(src, remarks):
    """The compiler's kernel-resource remarks, one record per kernel."""
    out = []
    for line in remarks:
        if "remark:" not in line:
            continue
        body = line.split("remark:", 1)[1].split(" [-Rpass", 1)[0].strip()
        key, _, val = body.partition(": ")
        if key == "Function Name":
            out.append({"source": src, "kernel": val})
        elif out and key in _FIELDS:
            out[-1][_FIELDS[key]] = int(val)
    return out


def _run(cmd, verbose):
    """Run one build step; returns its resource remarks (other diagnostics are printed
    when verbose)."""
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    lines = [line for line in (r.stderr or "").splitlines() if "packed-fp32-ops" not in line]
    remarks = [line for line in lines if "kernel-resource-usage" in line]
    err = "\n".join(line for line in lines if "kernel-resource-usage" not in line)
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{r.stdout}\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    return remarks


if __name__ == "__main__":
    print(build(verbose=True))
