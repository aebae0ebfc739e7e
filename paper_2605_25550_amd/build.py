"""Build step of the HIP library: compiles csrc/ for gfx950 with hipcc into
paper_2605_25550_amd/libditmi.so (in-tree, next to the binding)."""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libditmi.so")
OBJDIR = os.path.join(PKG, "_build")
ARCH = "gfx950"

SOURCES = ["gemm_bf16.hip", "gemm_f32.hip", "attention_bf16.hip", "attention_f32.hip", "elementwise.hip", "ditmi.cpp"]
PROBE = os.path.join(PKG, "gemm_probe")

# Packed-fp32 instructions are disabled for every device compile.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def _compile(src: str, extra: list[str]) -> str:
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-result",
           "-Wno-unused-variable", "-I", INCLUDE, "-I", CSRC, *DEVICE_FLAGS, *extra, "-c",
           os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                     if "packed-fp32-ops" not in l and l.strip())
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{msgs}")
    if msgs and os.environ.get("DITMI_BUILD_VERBOSE"):
        print(msgs, file=sys.stderr)
    return obj


def build(extra: list[str] | None = None, jobs: int = 8) -> str:
    """Compile every source and link libditmi.so; returns the library path."""
    os.makedirs(OBJDIR, exist_ok=True)
    extra = list(extra or [])
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, extra), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


def build_probe() -> str:
    """The GEMM timing probe (csrc/gemm_probe.cpp, a measurement tool linked
    against the built library's internal launch functions)."""
    if not os.path.exists(LIB):
        build()
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O2", "-std=c++17", "-I", INCLUDE, "-I", CSRC,
           os.path.join(CSRC, "gemm_probe.cpp"), "-o", PROBE, "-L", PKG, "-lditmi", "-Wl,-rpath,$ORIGIN"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"probe build failed:\n{r.stdout}{r.stderr}")
    return PROBE


MFMA_PROBE = os.path.join(PKG, "mfma_probe")


def build_mfma_probe() -> str:
    """The MFMA throughput and clock probe (csrc/mfma_probe.hip, a
    measurement tool, standalone)."""
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", *DEVICE_FLAGS,
           os.path.join(CSRC, "mfma_probe.hip"), "-o", MFMA_PROBE]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"mfma probe build failed:\n{r.stdout}{r.stderr}")
    return MFMA_PROBE


HBM_PROBE = os.path.join(PKG, "hbm_probe")


def build_hbm_probe() -> str:
    """The HBM bandwidth probe (csrc/hbm_probe.hip, a measurement tool,
    standalone)."""
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", *DEVICE_FLAGS,
           os.path.join(CSRC, "hbm_probe.hip"), "-o", HBM_PROBE]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hbm probe build failed:\n{r.stdout}{r.stderr}")
    return HBM_PROBE


# Host-code sanitizers for the CPU tests of the C ABI: the host side
# (ditmi.cpp: validation, workspace layout, tile planning, launch sequencing)
# is rebuilt with AddressSanitizer and UndefinedBehaviorSanitizer; the kernel
# objects are the regular ones (device code is never sanitized).  The library
# is loaded into a process that preloads the ASan runtime (sanitizer_runtime()).
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
             "-Xarch_host", "-g"]


def sanitizer_runtime() -> str:
    """Path of clang's shared ASan runtime (to preload)."""
    import glob
    root = os.path.dirname(os.path.dirname(os.path.realpath(hipcc())))
    for pat in ("llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so",
                "lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"):
        hits = sorted(glob.glob(os.path.join(root, pat)))
        if hits:
            return hits[-1]
    raise RuntimeError("clang's ASan runtime was not found")


def build_sanitized(out_dir: str) -> str:
    """libditmi.so with the host code under ASan + UBSan, in out_dir."""
    os.makedirs(OBJDIR, exist_ok=True)
    os.makedirs(out_dir, exist_ok=True)
    kernels = [s for s in SOURCES if s != "ditmi.cpp"]
    objs = [os.path.join(OBJDIR, os.path.splitext(s)[0] + ".o") for s in kernels]
    missing = [s for s, o in zip(kernels, objs) if not os.path.exists(o)]
    with cf.ThreadPoolExecutor(max_workers=8) as ex:
        list(ex.map(lambda s: _compile(s, []), missing))
    host = os.path.join(out_dir, "ditmi_san.o")
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O1", "-fPIC", "-std=c++17", "-I", INCLUDE, "-I", CSRC, *DEVICE_FLAGS,
           *SAN_FLAGS, "-c", os.path.join(CSRC, "ditmi.cpp"), "-o", host]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized compile failed:\n{r.stdout}{r.stderr}")
    lib = os.path.join(out_dir, "libditmi.so")
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *SAN_FLAGS, host, *objs, "-o", lib]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized link failed:\n{r.stdout}{r.stderr}")
    return lib


if __name__ == "__main__":
    print(build_probe() if sys.argv[1:] == ["probe"] else build())
