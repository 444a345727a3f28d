"""Build libpixelfly.so in-tree with hipcc for gfx950.

    python -m paper_2112_00029_amd.build

Compiles every source under csrc/ (HIP kernels and the C ABI) to objects in
_build/ and links them into paper_2112_00029_amd/libpixelfly.so.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libpixelfly.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# (source, object name, defines): the two GEMM sources are compiled once per
# part (their launchers say which instantiations each part holds) so that
# the template instantiations compile in parallel.
SOURCES = (
    [("layout.cpp", "layout", ()), ("capi.cpp", "capi", ()),
     ("skinny.hip", "skinny", ()), ("attn_kernels.hip", "attn_kernels", ()),
     ("butterfly.hip", "butterfly", ()), ("gemm_tnw.hip", "gemm_tnw", ()),
     ("pairs.hip", "pairs", ())]
    + [("gemm_kernels.hip", f"gemm_kernels_p{p}", (f"PF_GK_PART={p}",)) for p in range(7)]
    + [("gemm_dma.hip", f"gemm_dma_b{b}_{k}", (f"PF_PART_BLK={b}", f"PF_PART_BKN={k}"))
       for b in (32, 64, 128) for k in (0, 1)]
)

# Per-source extra flags.  The attention kernels feed MFMA results straight
# into VALU softmax arithmetic: asking for the VGPR form of MFMA keeps those
# results out of AGPRs (no accvgpr copies) and lowers register use.
SOURCE_FLAGS = {
    "attn_kernels.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}

FLAGS = [
    "-O3", "-fPIC", "-std=c++17", f"--offload-arch={ARCH}",
    # keep the compiler from forming packed-fp32 VALU ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _compile(src: str, build_dir: str = BUILD, defines=(), name=None, part=()) -> str:
    obj = os.path.join(build_dir, (name or os.path.splitext(src)[0]) + ".o")
    cmd = [HIPCC, *FLAGS, *SOURCE_FLAGS.get(src, []), *[f"-D{d}" for d in (*part, *defines)]]
    if src.endswith(".cpp"):
        cmd += ["-x", "hip"]
    cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{out}")
    if out.strip():
        print(out, file=sys.stderr)
    return obj


def build(verbose: bool = True, lib: str = LIB, build_dir: str = BUILD, defines=()) -> str:
    """Compile and link; `defines` are extra -D tuning macros."""
    os.makedirs(build_dir, exist_ok=True)
    # Largest parts first (the NT parts of the direct-to-LDS family).
    order = sorted(SOURCES, key=lambda e: not e[0].startswith("gemm"))
    workers = max(1, min(len(order), os.cpu_count() or 1))
    with cf.ThreadPoolExecutor(max_workers=workers) as ex:
        objs = list(ex.map(lambda e: _compile(e[0], build_dir, defines, e[1], e[2]), order))
    tmp = lib + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    build()
