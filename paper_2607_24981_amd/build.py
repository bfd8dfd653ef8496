"""Build libilw.so from the HIP sources in csrc/ for gfx950 (in-tree).

    python -m paper_2607_24981_amd.build
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
SO = os.path.join(HERE, "libilw.so")
SOURCES = ["api.hip", "gemm.hip", "ln_gemm.hip", "tail384.hip", "attention.hip", "rowops.hip",
           "deform.hip", "block_tail.hip", "split_conv.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


# Packed-FP32 instructions are disabled for all device code.
FLAGS = ["-O3", f"--offload-arch={ARCH}", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", INCLUDE]


# Per-source device code generation options.  The attention kernel keeps its
# MFMA results in ordinary VGPRs: its int32 scores feed VALU work right away,
# and the accumulation-register form costs one copy per score.
SOURCE_FLAGS = {"attention.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def build(verbose: bool = False) -> str:
    cc = hipcc()
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(objdir, src + ".o")
        cmd = [cc, *FLAGS, *SOURCE_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
        if verbose and r.stderr.strip():
            print(r.stderr, file=sys.stderr)
        return obj

    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = SO + ".tmp"
    subprocess.check_call([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp,
                           *objs])
    os.replace(tmp, SO)
    return SO


# Host-side instrumentation for the sanitizer build: the device code is built
# as usual, only the host pass of the source gets the sanitizers.
SANITIZE_HOST = ("-Xarch_host -fsanitize=address,undefined "
                 "-Xarch_host -fno-sanitize-recover=all "
                 "-Xarch_host -fno-omit-frame-pointer").split()


def build_sanitized(out: str, sources=("api.hip",)) -> str:
    """Link a copy of the library at `out` whose `sources` (by default the
    C ABI layer with all argument validation) have AddressSanitizer and
    UndefinedBehaviorSanitizer in their host code; the other objects are the
    regular ones.  The sanitizer runtime must be preloaded by the process
    that loads it."""
    cc = hipcc()
    objdir = os.path.join(HERE, "_build")
    regular = [os.path.join(objdir, src + ".o") for src in SOURCES if src not in sources]
    if not all(os.path.exists(o) for o in regular):
        build()
    objs = []
    for src in sources:
        obj = out + "." + src + ".o"
        cmd = [cc, *FLAGS, *SOURCE_FLAGS.get(src, []), *SANITIZE_HOST, "-g", "-c",
               os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src} (sanitized):\n{r.stderr}")
        objs.append(obj)
    subprocess.check_call([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out,
                           *objs, *regular])
    return out


def sanitizer_runtime() -> str:
    """Path of the compiler's shared AddressSanitizer runtime (it also carries
    the UndefinedBehaviorSanitizer handlers)."""
    import glob
    root = os.path.dirname(os.path.dirname(os.path.realpath(hipcc())))
    for base in (root, "/opt/rocm"):
        hits = sorted(glob.glob(os.path.join(base, "llvm", "lib", "clang", "*", "lib", "linux",
                                             "libclang_rt.asan-x86_64.so")))
        if hits:
            return hits[-1]
    raise RuntimeError("libclang_rt.asan-x86_64.so not found")


if __name__ == "__main__":
    print(build(verbose=True))
