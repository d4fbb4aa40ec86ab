"""Build libdlmc.so (HIP kernels for gfx950 + host runtime + C ABI) in-tree."""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libdlmc.so")
BUILD = os.path.join(HERE, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMMON = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
          # packed fp32 VALU forms are kept out of the generated code
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          # a multiply and an add are fused only where the source says fmaf:
          # left to the compiler, the choice depends on the surrounding code,
          # and the same epilogue or softmax expression could round
          # differently in two kernels (tile shapes, block sizes) that must
          # give identical results
          "-ffp-contract=off",
          "-Wno-unused-command-line-argument"]
SOURCES = ["gemm_bf16.hip", "attention.hip", "elementwise.hip", "coding.hip", "ranking.hip", "context.hip",
           "scratch.hip", "model.cpp", "session.cpp", "compress.cpp", "capi.cpp"]
LIBS = ["-lz", "-ldl"]
# per-source flags: attention produces no NaN from finite inputs, so max()
# needs no NaN canonicalisation of the MFMA results (infinities keep their
# meaning: masked keys are -inf)
EXTRA = {"attention.hip": ["-fno-honor-nans"]}


def _code(path: str) -> str:
    """A source file's code: // comments, trailing blanks and empty lines removed."""
    lines = []
    for line in open(path, encoding="utf-8"):
        line = line.split("//", 1)[0].rstrip()
        if line:
            lines.append(line)
    return "\n".join(lines)


def numerics_id() -> int:
    """64-bit identity of the library's arithmetic: a SHA-256 of the code of every
    source and header (comments stripped) and of the compile flags.  Containers
    record it; a build with another identity refuses to decode them, since
    kernels that round differently would replay other decisions."""
    import hashlib
    h = hashlib.sha256()
    files = sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp", ".h")))
    for f in files:
        h.update(f.encode() + b"\0" + _code(os.path.join(CSRC, f)).encode() + b"\0")
    h.update(_code(os.path.join(os.path.dirname(HERE), "include", "dlmc.h")).encode())
    h.update(repr((COMMON, sorted(EXTRA.items()))).encode())
    return int.from_bytes(h.digest()[:8], "little")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, src.rsplit(".", 1)[0] + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    ident = [f"-DDLMC_NUMERICS_ID=0x{numerics_id():016x}ull"] if src == "session.cpp" else []
    cmd = [HIPCC, *COMMON, *EXTRA.get(src, []), *ident, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile of {src} failed:\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = min(len(SOURCES), int(os.environ.get("MAX_JOBS", os.cpu_count() or 4)))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = OUT + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp, *objs, *LIBS]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, OUT)
    if verbose:
        print(f"built {OUT}")
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
