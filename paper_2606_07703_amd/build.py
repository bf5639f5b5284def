"""Build the gfx950 shared library ``libsparse_prefill.so`` in-tree with hipcc.

Every HIP source is compiled for gfx950 only, with packed-fp32 instruction
selection disabled, and linked with the host C ABI layer into one library.
Run ``python -m paper_2606_07703_amd.build`` or call ``build()``.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import re
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libsparse_prefill.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Wno-unused-function", "-I", INCLUDE, "-I", CSRC,
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]

# Per-file additions. The indexer's and the attention kernels' max reductions
# run on MFMA outputs that are never NaN for finite inputs (masked scores are
# -inf); without IEEE mode the compiler drops the quieting pass it otherwise
# puts before every v_max_f32.
NO_IEEE = ["-fno-honor-nans", "-mno-amdgpu-ieee"]
FILE_FLAGS = {
    "indexer_mfma.hip": NO_IEEE,
    "dense_mfma.hip": NO_IEEE,
    "sparse_block_mfma.hip": NO_IEEE,
}


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))


# hipcc's per-kernel resource remarks: kernel names and scratch bytes per lane
RESOURCE_REMARKS = ["-Rpass-analysis=kernel-resource-usage"]


def _scratch_kernels(text: str) -> list:
    """Kernels whose resource remark reports scratch (register spills or
    private arrays): in the hot loops these cost a memory round trip."""
    out, name = [], None
    for ln in text.splitlines():
        if "Function Name:" in ln:
            name = ln.split("Function Name:")[1].split("[")[0].strip()
        elif "ScratchSize [bytes/lane]:" in ln and name:
            n = int(ln.split("ScratchSize [bytes/lane]:")[1].split("[")[0])
            if n:
                out.append((name, n))
    return out


def _compile(src: str) -> tuple:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = ([HIPCC] + CFLAGS + FILE_FLAGS.get(os.path.basename(src), []) + RESOURCE_REMARKS
           + ["-c", src, "-o", obj])
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    text = r.stdout + r.stderr
    # the host pass does not know the packed-fp32 feature; drop that warning
    # and the resource remarks (summarised by build())
    noise = ("is not a recognized feature for this target", "remark:", "kernel-resource-usage")
    context = re.compile(r"^\s*(\d+\s*)?\|")   # source lines and carets quoted by a remark
    msg = "\n".join(ln for ln in text.splitlines()
                    if not any(n in ln for n in noise) and not context.match(ln))
    if msg.strip():
        print(msg, file=sys.stderr)
    return obj, _scratch_kernels(text)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    jobs = min(len(srcs), int(os.environ.get("MAX_JOBS", "8")))
    with cf.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        results = list(ex.map(_compile, srcs))
    objs = [o for o, _ in results]
    scratch = [k for _, ks in results for k in ks]
    if scratch and verbose:
        print("kernels using scratch (bytes/lane): " +
              ", ".join(f"{n} ({b})" for n, b in scratch), file=sys.stderr)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    # A kernel whose host stub was not emitted leaves an undefined symbol that
    # only shows when the library is loaded: load it (in a child process, all
    # symbols resolved now) before it replaces the previous build.
    chk = subprocess.run([sys.executable, "-c",
                          "import ctypes, os, sys; ctypes.CDLL(sys.argv[1], mode=os.RTLD_NOW)", tmp],
                         capture_output=True, text=True)
    if chk.returncode != 0:
        raise RuntimeError(f"built library does not load:\n{chk.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
