"""In-tree build of libiso.so (hipcc, gfx950)."""
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libiso.so")

SOURCES = ["iso_abi.cpp", "iso_select.hip", "iso_merge.hip", "iso_fused.hip", "iso_spectral.hip", "iso_tsv.hip",
           "iso_noalloc.hip", "iso_ortho.hip"]

HIPFLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off",                  # the value path follows a fixed binary64 rounding sequence
    "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
    "-Wall", "-Wno-unused-result",
]


def build(verbose=False, jobs=8):
    os.makedirs(BUILD, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmd = ["hipcc"] + HIPFLAGS + lang + ["-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"compile failed: {src}\n{r.stdout}\n{r.stderr}")
        return obj

    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB + ".tmp"
    cmd = ["hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    # the streaming calibration kernel of bench.py --calibrate-stream (not part of libiso)
    cal = os.path.join(HERE, "libiso_calibrate.so")
    cmd = ["hipcc"] + HIPFLAGS + ["-shared", "-x", "hip", os.path.join(CSRC, "iso_calibrate.hip"), "-o", cal + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: iso_calibrate.hip\n{r.stdout}\n{r.stderr}")
    os.replace(cal + ".tmp", cal)
    return LIB


# Host-side sanitizer build of the C ABI layer: iso_abi.cpp (argument checks, workspace
# planning, table building) instrumented with AddressSanitizer and UndefinedBehaviorSanitizer,
# linked with the uninstrumented kernel objects of build().  The sanitizer runtime is not linked
# in: it is preloaded into the host process (asan_runtime() below), which the CPU test of the
# ABI does.  Device code is never instrumented.
SANITIZED_LIB = os.path.join(BUILD, "libiso_hostsan.so")
_CLANG_RT = "/opt/rocm/llvm/lib/clang"


def asan_runtime():
    """Path of the clang AddressSanitizer runtime of the ROCm toolchain, or None."""
    if not os.path.isdir(_CLANG_RT):
        return None
    for ver in sorted(os.listdir(_CLANG_RT), reverse=True):
        p = os.path.join(_CLANG_RT, ver, "lib", "linux", "libclang_rt.asan-x86_64.so")
        if os.path.exists(p):
            return p
    return None


def build_host_sanitized(verbose=False):
    """Builds SANITIZED_LIB from the objects of build() (which must have run) and a sanitized
    iso_abi.cpp; returns its path, or None when the toolchain has no ASan runtime."""
    if asan_runtime() is None:
        return None
    obj = os.path.join(BUILD, "iso_abi_hostsan.o")
    cmd = (["hipcc"] + HIPFLAGS
           + ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
              "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer", "-g",
              "-c", os.path.join(CSRC, "iso_abi.cpp"), "-o", obj])
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: iso_abi.cpp (sanitized)\n{r.stdout}\n{r.stderr}")
    objs = [obj] + [os.path.join(BUILD, os.path.splitext(s)[0] + ".o") for s in SOURCES if s != "iso_abi.cpp"]
    tmp = SANITIZED_LIB + ".tmp"
    cmd = ["hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, SANITIZED_LIB)
    return SANITIZED_LIB


if __name__ == "__main__":
    build(verbose=True)
    build_host_sanitized(verbose=True)
