"""Build the HIP library (gfx950) in-tree: paper_1912_03203_amd/libdynconv.so."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "dynconv.hip")
LIB = os.path.join(PKG, "libdynconv.so")
ARCH = "gfx950"

# Packed fp32 instructions are disabled: the compiler may not emit
# v_pk_{add,mul,fma}_f32 for this library.
HIPCC_FLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-result",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build(verbose: bool = False) -> str:
    """Compile the library and, in parallel, its device assembly, which the
    MFMA check (mfma_lint) scans; raises on a compile error or a finding."""
    from . import mfma_lint

    tmp = LIB + ".tmp%d" % os.getpid()
    asm = os.path.join(PKG, "_build", "dynconv_gfx950.s")
    os.makedirs(os.path.dirname(asm), exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc")]
    lib_cmd = [hipcc()] + HIPCC_FLAGS + inc + ["-o", tmp, SRC]
    asm_flags = [f for f in HIPCC_FLAGS if f not in ("-fPIC", "-shared")]
    asm_cmd = [hipcc()] + asm_flags + ["-S", "--offload-device-only"] + inc + ["-o", asm, SRC]
    procs = [subprocess.Popen(c, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)
             for c in (lib_cmd, asm_cmd)]
    outs = [p.communicate() for p in procs]
    for p, (out, err) in zip(procs, outs):
        if p.returncode != 0:
            raise RuntimeError("hipcc failed:\n" + out + err)
    if verbose:
        print(outs[0][0] + outs[0][1])
    with open(asm) as f:
        findings = mfma_lint.check(f.read())
    if findings:
        raise RuntimeError("MFMA result read too early in the generated code:\n" + "\n".join(findings[:20]))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
