"""Build libquartz.so in-tree with hipcc for gfx950.

Every HIP source is compiled with fp contraction off (the quantizer's
products must round to fp32 before the half-even rounding) and without
packed-fp32 instructions; fp32 division stays IEEE (hipcc's default).
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libquartz.so")
SOURCES = ["abi.hip", "quantize_lzs.hip", "pack_weight.hip", "w4a4_gemm.hip", "w4a4_linear.hip",
           "w4a4_gemm_plain.hip", "w4a4_linear_asym.hip", "w4a4_gemm_conv.hip", "scratch.hip",
           "attention.hip", "attention_fused.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build(verbose: bool = False) -> str:
    """Compile every source to an object in parallel (each GEMM output mode is
    its own translation unit), then link libquartz.so."""
    import concurrent.futures
    import tempfile

    noise = "is not a recognized feature for this target"
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    compile_flags = [f for f in HIPCC_FLAGS if f != "-shared"]
    with tempfile.TemporaryDirectory(prefix="quartz_build_") as tmpdir:
        def compile_one(src):
            obj = os.path.join(tmpdir, os.path.splitext(src)[0] + ".o")
            cmd = [hipcc(), *compile_flags, *inc, "-c", "-o", obj, os.path.join(CSRC, src)]
            if verbose:
                print(" ".join(cmd), flush=True)
            res = subprocess.run(cmd, capture_output=True, text=True)
            err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
            return src, obj, res.returncode, err

        workers = max(1, min(len(SOURCES), os.cpu_count() or 1))
        with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as ex:
            results = list(ex.map(compile_one, SOURCES))
        failed = [r for r in results if r[2] != 0]
        for src, _, _, err in results:
            if err.strip() and (verbose or failed):
                sys.stderr.write(f"{src}:\n{err}\n")
        if failed:
            raise RuntimeError("hipcc failed building libquartz.so: " +
                               ", ".join(r[0] for r in failed))
        tmp = LIB + ".tmp"
        cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp,
               *[r[1] for r in results]]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stderr + "\n")
            raise RuntimeError("linking libquartz.so failed")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
