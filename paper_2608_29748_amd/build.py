"""Builds libretrace.so (the HIP kernels, host runtime and C ABI) for gfx950, in-tree."""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libretrace.so")
BUILD = os.path.join(HERE, "_build")
SOURCES = ["gemm.hip", "gemm_mid.hip", "attn.hip", "misc.hip", "sample.hip", "engine.hip", "validate.cpp"]
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
         # packed fp32 vector ops stay off: hipcc otherwise forms them from float code
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# per-source extras: attention keeps its MFMA accumulators in ordinary VGPRs (the online
# softmax rescales them with vector ALU ops; accumulation registers would be copied)
EXTRA = {"attn.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]}


def _hipcc() -> str:
    return shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [_hipcc(), *FLAGS, *EXTRA.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd = [_hipcc(), "-O2", "-std=c++17", "-fPIC", "-Wall", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


# sources whose kernels hold LDS reads in inline assembly that the compiler's wait
# insertion does not see: their gfx950 assembly is checked (isa_check) on every build
ASM_CHECKED = ["attn.hip"]


def _assembly(src: str) -> str:
    out = os.path.join(BUILD, os.path.splitext(src)[0] + ".s")
    cmd = [_hipcc(), *[f for f in FLAGS if f != "-fPIC"], *EXTRA.get(src, []), "--cuda-device-only", "-S",
           os.path.join(CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return out


def _check_assembly(path: str) -> None:
    try:
        from . import isa_check
    except ImportError:       # run as a script
        import isa_check
    with open(path) as fh:
        asm = fh.read()
    if not isa_check.checked_kernels(asm):
        raise RuntimeError(f"{path}: no kernel with inline-asm LDS reads found (check out of date)")
    bad = isa_check.check(asm)
    if bad:
        raise RuntimeError(f"{path}: registers of untracked LDS reads touched before their wait:\n  "
                           + "\n  ".join(bad[:20]))


STAMP = OUT + ".sha256"


def source_hash() -> str:
    """SHA-256 over the library's sources (kernels, host code, the C ABI header)."""
    import hashlib
    h = hashlib.sha256()
    files = sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".h", ".cpp")))
    for f in files + [os.path.join("..", "..", "include", "retrace.h")]:
        h.update(f.encode())
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    digest = source_hash()
    with cf.ThreadPoolExecutor(8) as ex:
        asms = [ex.submit(_assembly, src) for src in ASM_CHECKED]
        objs = list(ex.map(_compile, SOURCES))
        for f in asms:
            _check_assembly(f.result())
    tmp = OUT + ".tmp"
    cmd = [_hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, OUT)
    with open(STAMP, "w") as fh:     # the sources this library was built from
        fh.write(digest + "\n")
    if verbose:
        print("built", OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
