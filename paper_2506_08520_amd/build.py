"""Build step of the HIP library: compiles csrc/*.hip for gfx950 into
libnystra.so inside the package (in-tree, so it travels with the sources).

With NYSTRA_SANITIZE_HOST=1 in the environment the HOST code (the C-ABI layer:
validation, dispatch, launch) is built with AddressSanitizer and
UndefinedBehaviorSanitizer; device code is unchanged.  Such a library is for
the host-only tests, loaded with clang's ASan runtime preloaded:

    NYSTRA_SANITIZE_HOST=1 python paper_2506_08520_amd/build.py
    LD_PRELOAD=$(ls /opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so) \
        ASAN_OPTIONS=detect_leaks=0 python -m pytest tests/test_abi_host.py

Rebuild without the variable afterwards.
"""
import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libnystra.so")
OBJDIR = os.path.join(os.path.dirname(HERE), "_build")
SOURCES = ["abi.hip", "generic.hip", "exact.hip", "tiled.hip", "tiled_large.hip",
           "split.hip", "block.hip"]
ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed-fp32 VALU instructions are kept out of every kernel.  MFMA results
# are written straight to VGPRs (instead of the accumulation registers), which
# spares the copies back and lowers the register count of the tiled kernels.
FLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-Wall", "-Werror",
         "-Wno-unused-function", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-mllvm", "-amdgpu-mfma-vgpr-form=1",
         "-I", os.path.join(os.path.dirname(HERE), "include")]


# Host-side sanitizers (each option marked for the host compilation only).
HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address,undefined",
                 "-Xarch_host", "-fno-sanitize-recover=undefined",
                 "-Xarch_host", "-fno-omit-frame-pointer"]


def _sanitize():
    return HOST_SANITIZE if os.environ.get("NYSTRA_SANITIZE_HOST") == "1" else []


def _compile(src, verbose):
    obj = os.path.join(OBJDIR, src.replace(".hip", ".o"))
    cmd = [HIPCC, *FLAGS, *_sanitize(), "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose=False, jobs=8):
    os.makedirs(OBJDIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *_sanitize()[:2], *objs,
           "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
