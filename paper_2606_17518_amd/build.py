"""Compile the HIP sources under csrc/ into libspecgen.so for gfx950.

Objects are built in parallel under _build/ at the repository root and linked
into paper_2606_17518_amd/libspecgen.so; the same kernels with the entry
points built under SPECGEN_DEBUG_CHECKS (every attention block id checked on
the host before launch) into libspecgen_debug.so; the same library with the
bf16 partial kernel built under SPECGEN_TIMELINE (per-slot clock stamps of
every workgroup, for the benchmark's --timeline report) into
libspecgen_timeline.so; and the benchmark's memory-ceiling kernels into
libspecgen_probe.so.  Packed-FP32 instruction
selection is switched off on every device compile.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB_PATH = os.path.join(PKG, "libspecgen.so")
DEBUG_LIB_PATH = os.path.join(PKG, "libspecgen_debug.so")
TIMELINE_LIB_PATH = os.path.join(PKG, "libspecgen_timeline.so")
SOURCES = ["abi.hip", "attn_bf16.hip", "attn_dot.hip", "merge.hip", "kv_import.hip", "kv_append.hip"]
# the benchmark's memory-ceiling kernels, linked into a library of their own
PROBE_SOURCES = ["probe.hip"]
PROBE_LIB_PATH = os.path.join(PKG, "libspecgen_probe.so")
# Per-source device flags: the bf16 attention kernel keeps MFMA accumulators in
# VGPRs and runs without IEEE-mode NaN quieting (masked scores are -inf, never NaN).
EXTRA_FLAGS = {"attn_bf16.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form", "-mno-amdgpu-ieee", "-fno-honor-nans"]}


def _hipcc() -> str:
    for c in (os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc"), shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


def compile_flags() -> list[str]:
    return ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wno-unused-result", "-I", os.path.join(ROOT, "include")]


def build(verbose: bool = False) -> str:
    """Always recompiles every source, then links the shared library."""
    hipcc = _hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)
    flags = compile_flags()

    def one(job: tuple) -> str:
        src, tag, defs = job
        obj = os.path.join(BUILD_DIR, src.replace(".hip", tag + ".o"))
        cmd = [hipcc, *flags, *defs, *EXTRA_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
        if verbose and r.stderr.strip():
            print(r.stderr)
        return obj

    jobs = [(s, "", []) for s in SOURCES + PROBE_SOURCES] + [("abi.hip", "_debug", ["-DSPECGEN_DEBUG_CHECKS"]),
                                                             ("attn_bf16.hip", "_timeline", ["-DSPECGEN_TIMELINE"])]
    with cf.ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 4)) as ex:
        objs = dict(zip([j[0] + j[1] for j in jobs], ex.map(one, jobs)))
    kernels = [objs[s] for s in SOURCES if s != "abi.hip"]
    for lib_path, lib_objs in ((LIB_PATH, [objs["abi.hip"], *kernels]),
                               (DEBUG_LIB_PATH, [objs["abi.hip_debug"], *kernels]),
                               (TIMELINE_LIB_PATH, [objs["abi.hip"], objs["attn_bf16.hip_timeline"],
                                                    *[k for k in kernels if k != objs["attn_bf16.hip"]]]),
                               (PROBE_LIB_PATH, [objs[s] for s in PROBE_SOURCES])):
        tmp = lib_path + ".tmp%d" % os.getpid()
        r = subprocess.run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *lib_objs],
                           capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed:\n{r.stderr}")
        os.replace(tmp, lib_path)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
