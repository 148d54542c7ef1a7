"""Builds libispa.so (gfx950) in-tree with hipcc.

Usage: python -m paper_2607_00712_amd.build
"""

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libispa.so")

SOURCES = ["ispa_abi.cpp", "attn_fast.cpp", "gram_fast.cpp", "proj_fast.cpp", "attn_chunk.hip", "stats.hip",
           "solve.hip", "absorb.hip", "project.hip"]
BUILD = os.path.join(PKG, "_build")
LLVM_BIN = os.environ.get("ROCM_LLVM_BIN", "/opt/rocm/lib/llvm/bin")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-Wall",
    "-Wno-unused-function",
    # keep packed fp32 arithmetic out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE,
    "-I", CSRC,
    "-I", BUILD,
]


def _run(cmd):
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + "\n")
        raise subprocess.CalledProcessError(res.returncode, cmd, res.stdout)


def assemble(module, stem):
    """Generate the assembly of a hand-scheduled kernel (generator `module` in
    csrc), assemble it into a gfx950 code object and write that as a C
    initializer list (_build/<stem>_hsaco.inc) that <stem>.cpp embeds."""
    sys.path.insert(0, CSRC)
    try:
        gen = __import__(module)
    finally:
        sys.path.pop(0)
    os.makedirs(BUILD, exist_ok=True)
    asm = os.path.join(BUILD, stem + ".s")
    obj = os.path.join(BUILD, stem + ".o")
    co = os.path.join(BUILD, stem + ".hsaco")
    with open(asm, "w") as f:
        f.write(gen.generate())
    _run([os.path.join(LLVM_BIN, "clang"), "-x", "assembler", "-target", "amdgcn-amd-amdhsa", "-mcpu=gfx950",
          "-c", asm, "-o", obj])
    _run([os.path.join(LLVM_BIN, "ld.lld"), "-shared", obj, "-o", co])
    data = open(co, "rb").read()
    with open(os.path.join(BUILD, stem + "_hsaco.inc"), "w") as f:
        for i in range(0, len(data), 24):
            f.write(", ".join(str(b) for b in data[i:i + 24]) + ",\n")


def build(verbose=False):
    """Compile every source into libispa.so; raises CalledProcessError on failure."""
    assemble("attn_fast_gen", "attn_fast")   # head_dim-128 chunk attention
    assemble("gram_fast_gen", "gram_fast")   # Gram of widths that are multiples of 256
    assemble("proj_fast_gen", "proj_fast")   # projection (bf16 and W8A8) of widths that are multiples of 256
    srcs = []
    for s in SOURCES:
        p = os.path.join(CSRC, s)
        # hipcc treats .cpp as host C++; the ABI file includes hip_runtime and
        # launches kernels, so compile it as HIP source as well
        srcs += (["-x", "hip", p] if s.endswith(".cpp") else [p])
    tmp = LIB + ".tmp"
    cmd = [HIPCC] + FLAGS + srcs + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(line for line in res.stdout.splitlines()
                    if "packed-fp32-ops" not in line)  # host pass does not know the feature
    if res.returncode != 0:
        sys.stderr.write(out + "\n")
        raise subprocess.CalledProcessError(res.returncode, cmd, out)
    if verbose and out.strip():
        print(out)
    # the host pass can silently drop a kernel's launch stub (the device code
    # still builds): refuse a library with unresolved stubs
    nm = subprocess.run(["nm", "-D", "--undefined-only", tmp], stdout=subprocess.PIPE, text=True)
    missing = [ln for ln in nm.stdout.splitlines() if "__device_stub" in ln]
    if missing:
        os.remove(tmp)
        raise RuntimeError("libispa.so has unresolved kernel stubs:\n" + "\n".join(missing))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
