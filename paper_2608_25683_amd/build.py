"""Build libpsattn.so (host planner + gfx950 HIP kernels) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libpsattn.so")
SOURCES = ["psattn_host.cpp", "psattn_kvcache.cpp", "psattn_sched.cpp", "psattn_fwd.hip", "psattn_bwd.hip", "psattn_layer.hip", "psattn_noalloc.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed fp32 VALU instructions are disabled for all device code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{out}")
    return out


def check_hazards(src, extra_flags=None) -> None:
    """Compiles the device code of one source to assembly and runs the MFMA hazard check on it."""
    from . import hazard_check
    asm = os.path.join(PKG, "_build", os.path.splitext(src)[0] + ".s")
    _run([HIPCC, f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-I", INCLUDE, "-I", CSRC, *DEVICE_FLAGS,
          *(extra_flags or []), "--cuda-device-only", "-S", os.path.join(CSRC, src), "-o", asm])
    bad = {k: v for k, v in hazard_check.check_file(asm).items() if v}
    if bad:
        lines = [f"{k}: {len(v)} violations, first: {v[0]}" for k, v in bad.items()]
        raise RuntimeError("MFMA hazard check failed for " + src + ":\n" + "\n".join(lines))


def build(verbose: bool = False, extra_flags=None) -> str:
    """Compile every source for gfx950, check the kernels' MFMA hazards, link; returns the path."""
    objs = []
    os.makedirs(os.path.join(PKG, "_build"), exist_ok=True)
    for src in SOURCES:
        obj = os.path.join(PKG, "_build", os.path.splitext(src)[0] + ".o")
        cmd = [HIPCC, f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-I", INCLUDE, "-I", CSRC,
               *DEVICE_FLAGS, *(extra_flags or []), "-c", os.path.join(CSRC, src), "-o", obj]
        if src.endswith(".cpp"):
            cmd.insert(1, "-x")
            cmd.insert(2, "hip")
        out = _run(cmd)
        if verbose and out.strip():
            print(out)
        objs.append(obj)
        if src.endswith(".hip"):
            check_hazards(src, extra_flags)
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
