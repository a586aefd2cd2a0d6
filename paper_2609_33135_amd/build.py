"""Build libmpfa.so (HIP kernels for gfx950 + the C ABI) and its data-checking
twin libmpfa_debug.so in-tree with hipcc, plus libmpfa_probe.so, the
measurement probes the benchmark loads (not part of the product library)."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libmpfa.so")

SOURCES = ["api.cpp", "quantize.hip", "prefill.hip", "decode.hip", "mixed.hip", "debug_checks.hip"]
DEBUG_LIB = os.path.join(PKG, "libmpfa_debug.so")
PROBE_LIB = os.path.join(PKG, "libmpfa_probe.so")
# characterization library: the product kernels plus the softmax ablation
# variants of the prefill (outputs meaningless by design; only the benchmark's
# --ablation leg loads it)
ABLATE_LIB = os.path.join(PKG, "libmpfa_ablate.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = os.environ.get("MPFA_CLANG", "/opt/rocm/lib/llvm/bin/clang++")
ARCH = os.environ.get("MPFA_ARCH", "gfx950")

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # packed FP32 instructions are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC, "-Wall", "-Wno-unused-result",
]


# The attention kernels take finite inputs by contract (the debug library checks
# them).  Without NaN semantics fmaxf over MFMA results needs no quieting
# v_max_f32 per operand, which takes about 70 VALU instructions out of every
# 128-key tile of the prefill loop.
EXTRA = {"prefill.hip": ["-fno-honor-nans"], "mixed.hip": ["-fno-honor-nans"],
         # the same for the quantization pass: its max / min reductions need no
         # quieting instruction per loaded value
         "quantize.hip": ["-fno-honor-nans"],
         # the MFMA probe keeps its accumulators in VGPRs: with the AGPR form the
         # compiler copies them between the two register files inside the loop
         "probe.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def _compile(src: str, debug: bool = False, ablate: bool = False) -> str:
    tag = "_debug" if debug else ("_ablate" if ablate else "")
    out = os.path.join(BUILD, os.path.splitext(src)[0] + tag + ".o")
    extra = (["-DMPFA_DEBUG_CHECKS"] if debug else []) + (["-DMPFA_ABLATION_BUILD"] if ablate else []) + \
        EXTRA.get(src, [])
    cmd = [CLANG, "-x", "hip", *COMMON, *extra, "-c", os.path.join(CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{msg}")
    if msg.strip():
        sys.stderr.write(msg + "\n")
    return out


def _link(out: str, objs: list[str]) -> None:
    tmp = out + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    """Compile every source, then link libmpfa.so, libmpfa_debug.so (the same
    kernels; its entry points also check the data they are handed), the
    benchmark's probe library and its characterization library."""
    os.makedirs(BUILD, exist_ok=True)
    jobs = [(s, False, False) for s in SOURCES] + [("api.cpp", True, False), ("probe.hip", False, False),
                                                   ("prefill.hip", False, True)]
    with ThreadPoolExecutor(max_workers=len(jobs)) as ex:
        objs = list(ex.map(lambda j: _compile(*j), jobs))
    kernels = objs[1:len(SOURCES)]
    _link(LIB, [objs[0], *kernels])
    _link(DEBUG_LIB, [objs[len(SOURCES)], *kernels])
    _link(PROBE_LIB, [objs[len(SOURCES) + 1]])
    ablate_prefill = objs[len(SOURCES) + 2]
    _link(ABLATE_LIB, [objs[0], *[ablate_prefill if k.endswith("/prefill.o") else k for k in kernels]])
    if verbose:
        print("built", LIB, DEBUG_LIB, PROBE_LIB, ABLATE_LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
