"""Builds the in-tree shared libraries with hipcc for gfx950:
libkvgov.so (the hashing / cache path) and libkvgov_peaks.so (measured-peak
microbenchmarks used by the measurement harness)."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIBS = {
    "libkvgov.so": ["csrc/chains.hip", "csrc/cache.hip", "csrc/radix.hip"],
    "libkvgov_peaks.so": ["csrc/peaks.hip"],
}
OUT = os.path.join(HERE, "libkvgov.so")
ARCH = "gfx950"

FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-Wall",
    # no packed fp32 instructions anywhere in the library
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def build_one(name: str, sources, verbose: bool = False) -> str:
    out = os.path.join(HERE, name)
    tmp = out + ".tmp"
    cmd = [hipcc(), *FLAGS, "-o", tmp, *[os.path.join(HERE, s) for s in sources]]
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "'-packed-fp32-ops' is not a recognized feature"
    msgs = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{' '.join(cmd)}\n{msgs}")
    if verbose and msgs.strip():
        print(msgs, file=sys.stderr)
    os.replace(tmp, out)
    return out


# Host-side AddressSanitizer build of libkvgov (the device code is built as
# usual; only the host validation and bookkeeping are instrumented).  The
# process that loads it must preload the ASan runtime (asan_runtime()).
ASAN_FLAGS = [
    "-O1", "-g",
    "-Xarch_host", "-fsanitize=address",
    "-Xarch_host", "-fno-omit-frame-pointer",
    "-shared-libasan",
]


def build_host_asan(out_dir: str) -> str:
    """Builds libkvgov with host AddressSanitizer into out_dir; returns its path."""
    out = os.path.join(out_dir, "libkvgov_host_asan.so")
    flags = [f for f in FLAGS if f != "-O3"] + ASAN_FLAGS
    cmd = [hipcc(), *flags, "-o", out, *[os.path.join(HERE, s) for s in LIBS["libkvgov.so"]]]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{' '.join(cmd)}\n{res.stderr}")
    return out


def asan_runtime() -> str:
    """Path of the shared ASan runtime of hipcc's clang, or '' if absent."""
    clang = os.path.join(os.path.dirname(os.path.realpath(hipcc())), "..", "llvm", "bin", "clang")
    for c in (clang, "/opt/rocm/llvm/bin/clang"):
        if os.path.exists(c):
            res = subprocess.run([c, "-print-file-name=libclang_rt.asan-x86_64.so"],
                                 capture_output=True, text=True)
            path = res.stdout.strip()
            if res.returncode == 0 and os.path.isabs(path) and os.path.exists(path):
                return path
    return ""


def build(verbose: bool = False) -> str:
    """Builds every library; returns the path of libkvgov.so."""
    for name, sources in LIBS.items():
        build_one(name, sources, verbose)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))
