"""Build libcomfuse.so in place with hipcc for gfx950.

Each translation unit is compiled to an object under ``_build/`` in parallel,
then everything is linked into ``paper_2608_03537_amd/libcomfuse.so``.
Always recompiles (the build check wants a real compile every time).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libcomfuse.so")
ARCH = os.environ.get("CF_OFFLOAD_ARCH", "gfx950")

SOURCES = ["cf_api.cpp", "cf_gemm_registry.cpp", "cf_gemm_inst_v2.hip", "cf_gemm_inst_v1.hip",
           "cf_gemm_inst_wr.hip", "cf_gemm_inst_split.hip", "cf_rows.hip", "cf_b2b.hip", "cf_ffn.hip",
           "cf_noalloc.hip", "cf_mlp.hip", "cf_gemm_inst_kn.hip"]

# -packed-fp32-ops off: hipcc then never forms v_pk_{add,mul,fma}_f32 from
# scalar float code (the host pass warns that it does not know the feature).
CFLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I", os.path.join(ROOT, "include"), "-Wall", "-Wno-unused-function"]


def _hipcc():
    h = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(h):
        raise RuntimeError("hipcc not found")
    return h


# MFMA accumulators stay in VGPRs: every kernel here runs VALU work on its
# accumulator tiles (the row epilogue, GELU, softmax), and accumulators in
# AGPRs would cost a copy each way for every such step.
FILE_FLAGS = {f: ["-mllvm", "-amdgpu-mfma-vgpr-form"]
              for f in ("cf_gemm_inst_v2.hip", "cf_gemm_inst_v1.hip", "cf_gemm_inst_wr.hip", "cf_gemm_inst_split.hip",
                        "cf_gemm_inst_kn.hip",
                        "cf_b2b.hip", "cf_mlp.hip")}
# The GEMM kernels' one atomic (a row-cluster round counter, added by lane 0
# at the start of a tile) returns a value needed only after the main loop.
# LLVM's atomic optimizer rewrites it as a wave-wide reduction and broadcasts
# the result at once, which puts a wait for the atomic's round trip in front
# of the first operand loads.
for _f in ("cf_gemm_inst_v2.hip", "cf_gemm_inst_v1.hip", "cf_gemm_inst_wr.hip", "cf_gemm_inst_split.hip",
           "cf_gemm_inst_kn.hip"):
    FILE_FLAGS[_f] = FILE_FLAGS[_f] + ["-mllvm", "-amdgpu-atomic-optimizer-strategy=None"]


def _compile(src):
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [_hipcc(), *CFLAGS, *FILE_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    errs = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                     if "packed-fp32-ops" not in l and l.strip())
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{errs}")
    return obj, errs


def build(verbose=True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        results = list(ex.map(_compile, SOURCES))
    for obj, msgs in results:
        if msgs and verbose:
            print(msgs, file=sys.stderr)
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp,
           *[o for o, _ in results]]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}", file=sys.stderr)
    return LIB


if __name__ == "__main__":
    build()
