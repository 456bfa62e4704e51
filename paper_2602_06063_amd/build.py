"""Builds libq4nx.so in-tree with hipcc for gfx950.

    python paper_2602_06063_amd/build.py              # the library
    python paper_2602_06063_amd/build.py --sanitize   # host-sanitized copy

Every HIP source is compiled with packed-fp32 instructions disabled (the
compiler otherwise forms v_pk_*_f32 from plain float code).

--sanitize builds _build/libq4nx_asan.so: the same sources with the host code
(packer, validation, launch planning, launchers) instrumented with
AddressSanitizer and UndefinedBehaviorSanitizer; the device code is compiled
as usual (GPU sanitizers are not used).  It is loaded through Q4NX_LIBRARY
with clang's ASan runtime preloaded (asan_runtime()); tests/ runs the host ABI
tests against it on the CPU.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libq4nx.so")
ASAN_LIB = os.path.join(os.path.dirname(HERE), "_build", "libq4nx_asan.so")
ARCH = "gfx950"

SOURCES = ["q4nx_host.cpp", "q4nx_kernels.hip", "q4nx_flowkv.hip"]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def asan_runtime() -> str:
    """Path of the shared ASan runtime of ROCm's clang (to preload)."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    clang = os.path.join(rocm, "llvm", "bin", "clang")
    return subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                          text=True, check=True).stdout.strip()


def build(verbose: bool = False, sanitize: bool = False) -> str:
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    out = ASAN_LIB if sanitize else LIB
    os.makedirs(os.path.dirname(out), exist_ok=True)
    tmp = out + ".tmp"
    opt = ["-O1", "-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all",
           "-shared-libasan"] if sanitize else ["-O3"]
    cmd = [hipcc(), f"--offload-arch={ARCH}"] + opt + ["-std=c++17", "-fPIC", "-shared",
           "-Wall", "-Wno-unused-function", "-pthread",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-o", tmp] + srcs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature and says so.
    noise = "'-packed-fp32-ops' is not a recognized feature for this target (ignoring feature)"
    msgs = [l for l in (r.stdout + r.stderr).splitlines() if noise not in l]
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs))
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv))
