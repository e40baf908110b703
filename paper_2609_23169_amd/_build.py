"""Builds libultratex.so in-tree with hipcc for gfx950.

Every source is compiled on each call (objects under _build/ next to this
file), then linked into paper_2609_23169_amd/libultratex.so.

`python -m paper_2609_23169_amd._build --sanitize` (or UT_SANITIZE=1) also
builds _build/sanitize/libultratex_sanitize.so: the same kernels, with the
host side of the C ABI (api.cpp: validation, workspace sizing, validate mode)
compiled by g++ under AddressSanitizer and UndefinedBehaviorSanitizer. It is
for CPU runs of the host paths only (README.md gives the command); the GPU
code is never built with a sanitizer.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libultratex.so")
DIAG_OUT = os.path.join(HERE, "libutdiag.so")   # measurement aid (include/ultratex_diag.h)
OBJ = os.path.join(HERE, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SOURCES = ["api.cpp", "trace.cpp", "btd.hip", "block_index.hip", "bsattn_fwd.hip", "bsattn_bwd.hip",
           "topk_mask.hip", "fg_step.hip", "composite.hip"]
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Wall", "-Wno-unused-function",
    # never emit packed-fp32 VALU ops (v_pk_fma_f32 and friends)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in VGPRs: the softmax reads them without AGPR copies
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _compile(src: str) -> str:
    obj = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [HIPCC, *FLAGS, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l and "--hip-link" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{msg}")
    if msg.strip():
        print(msg, file=sys.stderr)
    return obj


GXX = os.environ.get("CXX_HOST", "g++")
SAN = os.path.join(OBJ, "sanitize")
SAN_OUT = os.path.join(SAN, "libultratex_sanitize.so")
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-fno-sanitize-recover=all"]


HOST_SOURCES = ["api.cpp", "trace.cpp"]   # no device code: g++ builds them for the sanitizers


def build_sanitized(objs, verbose: bool = False) -> str:
    """The host sources through g++ with ASan + UBSan, linked with the HIP
    kernel objects."""
    os.makedirs(SAN, exist_ok=True)
    host_objs = []
    for src in HOST_SOURCES:
        obj = os.path.join(SAN, os.path.splitext(src)[0] + ".o")
        cmd = [GXX, "-std=c++17", "-O1", "-g", "-fPIC", "-Wall", *SAN_FLAGS,
               "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
               "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"g++ (sanitized {src}) failed:\n{r.stdout}{r.stderr}")
        host_objs.append(obj)
    host = {os.path.splitext(s)[0] + ".o" for s in HOST_SOURCES}
    kernels = [o for o in objs if os.path.basename(o) not in host]
    cmd = [GXX, "-shared", *SAN_FLAGS, *host_objs, *kernels, "-L/opt/rocm/lib", "-lamdhip64",
           "-Wl,-rpath,/opt/rocm/lib", "-o", SAN_OUT]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized link failed:\n{r.stdout}{r.stderr}")
    if verbose:
        print(f"built {SAN_OUT}")
    return SAN_OUT


def build(verbose: bool = False, sanitize: bool = False) -> str:
    os.makedirs(OBJ, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = OUT + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, OUT)
    if verbose:
        print(f"built {OUT}")
    dobj = _compile("diag_mfma.hip")
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", dobj, "-o", DIAG_OUT + ".tmp"],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link of the diagnostic library failed:\n{r.stdout}{r.stderr}")
    os.replace(DIAG_OUT + ".tmp", DIAG_OUT)
    if verbose:
        print(f"built {DIAG_OUT}")
    if sanitize or os.environ.get("UT_SANITIZE", "0") not in ("", "0"):
        build_sanitized(objs, verbose)
    return OUT


if __name__ == "__main__":
    build(verbose=True, sanitize="--sanitize" in sys.argv)
