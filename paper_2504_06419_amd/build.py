"""Build the HIP library libspire.so for gfx950 (in-tree, no JIT cache).

Every HIP source is compiled with hipcc for gfx950 with packed-fp32 code
generation disabled (-Xclang -target-feature -Xclang -packed-fp32-ops) and
linked into paper_2504_06419_amd/libspire.so.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libspire.so")
BUILD = os.path.join(HERE, "_build")
ARCH = "gfx950"

SOURCES = ["spire_abi.hip", "plan_combine.hip", "attn_mfma.hip", "attn_staged.hip",
           "attn_generic.hip", "token_verify.hip", "block_verify.hip", "kv_update.hip",
           "feedback_memory.hip", "hbm_probe.hip"]

FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-command-line-argument"]


# Matrix-core kernels: select the MFMA forms that accumulate in ordinary VGPRs.
# With accumulators in AGPRs, every VALU touch of them (the softmax rescale)
# needs AGPR<->VGPR copies, and the compiler hoists those copies out of the
# rarely taken rescale branch into every tile.
MFMA_FLAGS = ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]
SOURCE_FLAGS = {"attn_mfma.hip": MFMA_FLAGS, "attn_staged.hip": MFMA_FLAGS}


def _hipcc():
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build(verbose: bool = False, extra_flags=()) -> str:
    os.makedirs(BUILD, exist_ok=True)
    objs = []

    def compile_one(src):
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        cmd = [_hipcc(), *FLAGS, *SOURCE_FLAGS.get(src, ()), *extra_flags, "-c",
               os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        msgs = "\n".join(ln for ln in (r.stdout + r.stderr).splitlines()
                         if "packed-fp32-ops" not in ln)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{msgs}")
        if verbose and msgs.strip():
            print(msgs)
        return obj

    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = OUT + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(OUT)
