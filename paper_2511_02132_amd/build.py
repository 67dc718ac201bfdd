"""Build libattn_numa.so in-tree with hipcc for gfx950.

``python -m paper_2511_02132_amd.build`` (or ``build()``) always recompiles.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libattn_numa.so")
SOURCES = ["attn_fwd.hip", "attn_fwd_pp.hip", "attn_bwd.hip", "attn_bwd_dq.hip", "attn_calib.hip",
           "attn_abi.cpp"]
# Per-file options.  attn_bwd_dq.hip keeps its matrix-core accumulators in
# ordinary vector registers: the compiler's default (accumulators in AGPRs
# whenever a wave may use more than 256 registers) makes the softmax copy
# them out and back on every tile.
FILE_FLAGS = {"attn_bwd_dq.hip": ["-mllvm", "--amdgpu-mfma-vgpr-form"]}
ARCH = "gfx950"


# The forward kernels and the headers they include: the counter summaries
# under profiles/ describe these, so their hash ties a summary to its code.
KERNEL_SOURCES = ["attn_fwd.hip", "attn_fwd_pp.hip", "attn_device.h", "attn_internal.h"]
# The backward kernels and their headers, for the backward's summaries.
BWD_KERNEL_SOURCES = ["attn_bwd.hip", "attn_bwd_dq.hip", "attn_bwd_common.h", "attn_device.h",
                      "attn_internal.h"]


def code_tokens(text: str) -> str:
    """C++ source without comments and with whitespace runs collapsed: what the
    compiler sees, so an edit to a comment leaves the hash unchanged.  String
    literals are kept as they are (a // or /* inside one is not a comment)."""
    out = []
    i, n = 0, len(text)
    while i < n:
        c = text[i]
        if c == '"' or c == "'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash(names=None) -> str:
    """Short hash of the kernel sources (comments and layout ignored): ties a
    counter summary to the code it measured.  names: the files hashed (default:
    the forward kernels)."""
    import hashlib

    h = hashlib.sha256()
    for name in (names or KERNEL_SOURCES):
        with open(os.path.join(CSRC, name)) as f:
            h.update(code_tokens(f.read()).encode())
    return h.hexdigest()[:16]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libattn_numa.so)")


def compile_flags(name: str = "") -> list:
    """hipcc options for source file `name` (its per-file options included)."""
    return ["--offload-arch=%s" % ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall",
            # packed fp32 VALU ops stay disabled in device code
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", INCLUDE, "-I", CSRC] + FILE_FLAGS.get(os.path.basename(name), [])


def _compile(src: str, obj: str, verbose: bool) -> str:
    cmd = [hipcc(), *compile_flags(src), "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed compiling %s" % src)
    return res.stdout + res.stderr


def build(out: str = LIB, verbose: bool = False) -> str:
    """Compile every source (in parallel, one hipcc per file) and link the library."""
    import concurrent.futures
    import tempfile

    with tempfile.TemporaryDirectory(prefix="attn_build_") as tmpd:
        objs = [os.path.join(tmpd, os.path.splitext(s)[0] + ".o") for s in SOURCES]
        with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as pool:
            logs = list(pool.map(lambda so: _compile(os.path.join(CSRC, so[0]), so[1], verbose),
                                 zip(SOURCES, objs)))
        tmp = out + ".tmp"
        cmd = [hipcc(), "--offload-arch=%s" % ARCH, "-fPIC", "-shared", *objs, "-o", tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stdout + res.stderr)
            raise RuntimeError("hipcc failed linking %s" % out)
        logs.append(res.stdout + res.stderr)
    # Surface warnings, except the host pass's note that it does not know the
    # device-only packed-fp32 feature.
    noise = ("packed-fp32-ops' is not a recognized feature",)
    for line in "".join(logs).splitlines():
        if line.strip() and not any(n in line for n in noise):
            sys.stderr.write(line + "\n")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
