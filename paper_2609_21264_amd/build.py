"""Build step for the HIP library ``libfa.so`` (gfx950).

Run ``python -m paper_2609_21264_amd.build`` (or call :func:`build`). hipcc cross-compiles for gfx950
on any machine with ROCm; no GPU is needed. The library is written next to this file, in-tree.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libfa.so"
LIB_PATH = os.path.join(PKG_DIR, LIB_NAME)
SOURCES = ["fa_api.hip", "fa_fwd_kernel.hip", "fa_lbl_kernel.hip", "fa_decode_kernel.hip"]
# Measurement-only microbenchmarks (measured ceilings), a library of their own.
CEIL_LIB_PATH = os.path.join(PKG_DIR, "libfa_ceilings.so")
CEIL_SOURCES = ["fa_ceilings.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    cand = [os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"]
    for c in cand:
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found: ROCm is required to build libfa.so")


def _device_flags() -> list:
    return [
        f"--offload-arch={ARCH}", "-O3", "-std=c++17",
        # Packed fp32 VALU instructions are kept out of the generated code.
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        # Score MFMAs in VGPR form (the softmax reads them); the P V accumulators are pinned to
        # AGPRs by inline asm in the kernel.
        "-mllvm", "-amdgpu-mfma-vgpr-form=1",
        # The pipelined step is one fully unrolled sequence of MFMA slots; the default limit for
        # "#pragma unroll" stops short of it for the widest head dimension.
        "-mllvm", "-pragma-unroll-threshold=50000",
        # Leading scalar kernel arguments (up to 14 SGPRs) are preloaded by the command processor, so
        # that the fused kernel's first loads do not wait for the argument block.
        "-mllvm", "-amdgpu-kernarg-preload-count=14",
        "-I", INCLUDE, "-I", CSRC,
    ]


def compile_command(out: str, extra=(), sources=SOURCES) -> list:
    return [
        hipcc(), *_device_flags(), "-fPIC", "-shared",
        "-Wall", "-Wno-unused-command-line-argument",
        "-Wl,-rpath,/opt/rocm/lib",
        *extra,
        "-o", out,
        *[os.path.join(CSRC, s) for s in sources],
    ]


def kernel_asm(out: str, source: str = "fa_fwd_kernel.hip") -> None:
    """Write the gfx950 assembly of one kernel translation unit (default: the fused kernel) to `out`,
    for static checks of the generated code; nothing is linked."""
    cmd = [hipcc(), *_device_flags(), "--cuda-device-only", "-S", "-w", "-o", out,
           os.path.join(CSRC, source)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc -S failed:\n" + (res.stdout or "") + (res.stderr or ""))


def _link(path: str, sources, extra, verbose: bool, show: bool) -> None:
    fd, tmp = tempfile.mkstemp(prefix="." + os.path.basename(path) + ".", suffix=".so.tmp", dir=PKG_DIR)
    os.close(fd)
    try:
        cmd = compile_command(tmp, extra, sources)
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        out = (res.stdout or "") + (res.stderr or "")
        # hipcc's host pass does not know the packed-fp32 feature name; that warning is expected.
        lines = [ln for ln in out.splitlines() if "packed-fp32-ops" not in ln or "error" in ln]
        if res.returncode != 0:
            raise RuntimeError("hipcc failed:\n" + "\n".join(lines))
        if verbose or show:
            print("\n".join(lines), flush=True)
        os.replace(tmp, path)
    finally:
        if os.path.exists(tmp):
            os.unlink(tmp)


def build(verbose: bool = False, resource_usage: bool = False) -> str:
    """Compile libfa.so (and the measurement library libfa_ceilings.so) for gfx950 into the package
    directory; returns the path of libfa.so."""
    extra = ["-Rpass-analysis=kernel-resource-usage"] if resource_usage else []
    _link(LIB_PATH, SOURCES, extra, verbose, resource_usage)
    _link(CEIL_LIB_PATH, CEIL_SOURCES, extra, verbose, resource_usage)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose="-v" in sys.argv, resource_usage="--resource-usage" in sys.argv)
    print(LIB_PATH)
