"""Builds libspecdec.so (gfx950) from csrc/ with hipcc, in place."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libspecdec.so")
SOURCES = ["kernels.hip", "gemm.hip", "sgemv.hip", "scratch.hip", "runtime.cpp"]

# Packed-FP32 VALU forms are turned off for all device code.
HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return "hipcc"


# Host-side AddressSanitizer + UndefinedBehaviorSanitizer (device code is
# built as usual); the sanitizer runtime is linked as a shared library, which
# a host process preloads (LD_PRELOAD) before loading this build.
SANITIZE_FLAGS = [
    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
    "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
    "-shared-libsan", "-g",
]


def build(verbose: bool = False, sanitize: bool = False, out: str = LIB) -> str:
    dest = out
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    tmp = dest + ".tmp"
    extra = SANITIZE_FLAGS if sanitize else []
    cmd = [hipcc(), *HIPCC_FLAGS, *extra, "-I", os.path.join(ROOT, "include"), *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{out}")
    if out.strip() and verbose:
        print(out)
    os.replace(tmp, dest)
    return dest


def sanitizer_runtime() -> str:
    """Path of the compiler's shared AddressSanitizer runtime."""
    r = subprocess.run([hipcc(), "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    if r.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
        raise RuntimeError(f"no shared AddressSanitizer runtime next to {hipcc()}")
    return path


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
