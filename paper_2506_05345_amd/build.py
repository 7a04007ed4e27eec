"""Build libdms.so (HIP, gfx950 only) in-tree with hipcc."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libdms.so")
SOURCES = ["dms_api.hip", "dms_cache.hip", "dms_decode.hip", "dms_mla.hip", "dms_prefill.hip",
           "dms_quest.hip", "dms_train.hip"]
ARCH = "gfx950"

# Packed fp32 instructions are kept out of every kernel.
GPU_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-fPIC", "-std=c++17", f"--offload-arch={ARCH}", "-Wall",
          "-Wno-unused-function", "-munsafe-fp-atomics"]
# The prefill softmax never forms a NaN (hidden scores are -inf and give exact
# zeros), so its max reductions need no NaN quieting.
PER_SOURCE = {"dms_prefill.hip": ["-fno-honor-nans"], "dms_train.hip": ["-fno-honor-nans"]}


def hipcc() -> str:
    exe = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(exe):
        raise RuntimeError("hipcc not found")
    return exe


def build(verbose: bool = False, extra_flags=()) -> str:
    """Compile every source and link libdms.so; always rebuilds."""
    os.makedirs(BUILD, exist_ok=True)
    cc = hipcc()
    procs = []
    objs = []
    for src in SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        objs.append(obj)
        cmd = [cc, *COMMON, *GPU_FLAGS, *PER_SOURCE.get(src, []), *extra_flags, "-c",
               os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    errors = []
    for src, p in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        # the host pass does not know the gpu-only feature flag; that note is harmless
        text = "\n".join(l for l in text.splitlines() if "packed-fp32-ops" not in l)
        if p.returncode != 0:
            errors.append(f"{src}:\n{text}")
        elif verbose and text.strip():
            print(text)
    if errors:
        raise RuntimeError("hipcc failed:\n" + "\n".join(errors))
    tmp = LIB + ".tmp"
    cmd = [cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout.decode(errors="replace"))
    os.replace(tmp, LIB)
    return LIB


# Host-side sanitizers for the C-ABI layer (argument checks, layout, context):
# AddressSanitizer and UndefinedBehaviorSanitizer instrument the host code of
# dms_api.hip only (the device code and the kernel translation units are
# built as usual); the library then needs the sanitizer runtime preloaded
# (sanitizer_runtime()).
SAN_BUILD = os.path.join(HERE, "_build_san")
SAN_LIB = os.path.join(SAN_BUILD, "libdms_san.so")
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]


def sanitizer_runtime() -> str:
    """The shared AddressSanitizer runtime of hipcc's clang (to preload)."""
    import glob
    root = os.path.dirname(os.path.dirname(os.path.realpath(hipcc())))
    cands = sorted(glob.glob(os.path.join(root, "llvm", "lib", "clang", "*", "lib", "linux",
                                          "libclang_rt.asan-x86_64.so")))
    cands += sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not cands:
        raise RuntimeError("libclang_rt.asan-x86_64.so not found")
    return cands[0]


def build_sanitized(verbose: bool = False) -> str:
    """libdms_san.so: dms_api.hip with host ASan/UBSan, linked with the other
    objects of the regular build (built first if missing)."""
    objs = [os.path.join(BUILD, s.replace(".hip", ".o")) for s in SOURCES if s != "dms_api.hip"]
    if not all(os.path.exists(o) for o in objs):
        build(verbose)
    os.makedirs(SAN_BUILD, exist_ok=True)
    cc = hipcc()
    api = os.path.join(SAN_BUILD, "dms_api.o")
    cmd = [cc, *COMMON, *GPU_FLAGS, *HOST_SAN, "-c", os.path.join(CSRC, "dms_api.hip"), "-o", api]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + r.stdout.decode(errors="replace"))
    tmp = SAN_LIB + ".tmp"
    cmd = [cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *HOST_SAN, "-shared-libasan", api, *objs,
           "-o", tmp]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout.decode(errors="replace"))
    os.replace(tmp, SAN_LIB)
    return SAN_LIB


if __name__ == "__main__":
    if "--sanitize" in sys.argv:
        print(build_sanitized(verbose="-v" in sys.argv))
    else:
        print(build(verbose="-v" in sys.argv))
