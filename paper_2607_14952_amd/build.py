"""Build the HIP library ``liblongstraw.so`` in-tree for gfx950 with hipcc.

Usage: ``python -m paper_2607_14952_amd.build`` (or ``__graft_entry__.build()``).
Every call recompiles.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "liblongstraw.so")
SOURCES = ["api.hip", "small_kernels.hip", "f32_generic.hip", "fwd_f32_mfma.hip", "fwd_bf16.hip",
           "bwd_bf16.hip",
           "sparse_fwd.hip", "sparse_bwd.hip", "sparse_keys.hip", "dsa_select.hip"]
# Per-source extra flags.  The MFMA kernels keep their accumulators in arch VGPRs
# (AGPRs only as overflow), which avoids VGPR<->AGPR copies of the output tile.
EXTRA = {"fwd_bf16.hip": ["-mllvm", "--amdgpu-mfma-vgpr-form=1"],
         "bwd_bf16.hip": ["-mllvm", "--amdgpu-mfma-vgpr-form=1"],
         "sparse_fwd.hip": ["-mllvm", "--amdgpu-mfma-vgpr-form=1",
                            "-mllvm", "-disable-promote-alloca-to-lds"],
         "sparse_bwd.hip": ["-mllvm", "--amdgpu-mfma-vgpr-form=1",
                            "-mllvm", "-disable-promote-alloca-to-lds"],
         "dsa_select.hip": ["-mllvm", "-disable-promote-alloca-to-lds"]}
ARCH = os.environ.get("LS_OFFLOAD_ARCH", "gfx950")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    "-I", os.path.join(ROOT, "include"),
    # packed fp32 instructions stay off (vector fp32 math is emitted as scalar ops)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False, save_temps: bool = False, out: str = LIB, extra=None) -> str:
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        objs.append(obj)
        flags = list(EXTRA.get(src, [])) if extra is None else list(extra.get(src, []))
        if save_temps:
            flags.append("-save-temps=obj")
        cmds.append([HIPCC, *FLAGS, *flags, "-c", os.path.join(CSRC, src), "-o", obj])
    with ThreadPoolExecutor(min(len(cmds), os.cpu_count() or 4)) as ex:
        outs = list(ex.map(_run, cmds))
    tmp = out + ".tmp"
    outs.append(_run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]))
    os.replace(tmp, out)
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
        print("built", out)
    return out


if __name__ == "__main__":
    build(verbose=True, save_temps="--save-temps" in sys.argv)
