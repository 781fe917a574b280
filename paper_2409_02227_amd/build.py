"""Build libgdy.so in-tree: the GO-Kernel instantiations (HIP, gfx950) and the
host runtime, compiled with hipcc in parallel and linked into one shared
library next to this file."""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libgdy.so")

SOURCES = ["kernels_d_bf16.hip", "kernels_d_f16.hip", "kernels_d_fp8.hip",
           "kernels_bf16.hip", "kernels_f16.hip", "kernels_fp8.hip", "kernels_f32.hip", "kernels_ew.hip", "gdy.cpp"]
ARCH = "gfx950"
# -packed-fp32-ops: keep hipcc from forming packed fp32 ALU ops by itself.
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [_hipcc(), *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd.insert(1, "-x")
        cmd.insert(2, "hip")
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")
    return obj


CEILINGS = os.path.join(HERE, "ceilings")


def build_ceilings() -> str:
    """The stand-alone chip-ceiling probe (csrc/ceilings.hip) as an executable
    next to this file; the profiling harness runs it."""
    tmp = CEILINGS + ".tmp"
    cmd = [_hipcc(), *[f for f in FLAGS if f != "-fPIC"], os.path.join(CSRC, "ceilings.hip"), "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for ceilings.hip:\n{r.stderr}")
    os.replace(tmp, CEILINGS)
    return CEILINGS


EXAMPLES = ("gemm_set", "graph_static")


def build_example() -> list:
    """examples/gemm_set and examples/graph_static: C++ programs that drive
    libgdy through its C-ABI alone (no Python), linked against the in-tree
    library."""
    out = []
    for name in EXAMPLES:
        exe = os.path.join(HERE, "examples", name)
        tmp = exe + ".tmp"
        cmd = [_hipcc(), *[f for f in FLAGS if f != "-fPIC"], os.path.join(HERE, "examples", name + ".cpp"),
               "-L", HERE, "-lgdy", "-Wl,-rpath,$ORIGIN/..", "-o", tmp]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for examples/{name}.cpp:\n{r.stderr}")
        os.replace(tmp, exe)
        out.append(exe)
    return out


def build(jobs: int | None = None) -> str:
    """Compile every source and link libgdy.so (always rebuilds), then build
    the ceiling probe and the C-ABI example programs."""
    os.makedirs(BUILD, exist_ok=True)
    jobs = jobs or min(len(SOURCES), os.cpu_count() or 1)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        probe = ex.submit(build_ceilings)
        objs = list(ex.map(_compile, SOURCES))
        probe.result()
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    build_example()
    return LIB


def build_sanitized() -> str:
    """_build_san/libgdy_san.so: the host runtime (planner, launcher, C-ABI)
    built with clang's AddressSanitizer and UndefinedBehaviorSanitizer on the
    host side only, linked with the kernel objects of the last build().  Load
    it with GDY_LIBRARY=<path> in a process whose LD_PRELOAD starts with the
    ASan runtime (the runtime resolves the sanitizer calls)."""
    san = os.path.join(HERE, "_build_san")
    os.makedirs(san, exist_ok=True)
    obj = os.path.join(san, "gdy.o")
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = [f for f in FLAGS if f != "-O3"] + ["-O1", "-g"]
    cmd = [_hipcc(), "-x", "hip", *flags, *host_san, "-c", os.path.join(CSRC, "gdy.cpp"), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for the sanitizer build:\n{r.stderr}")
    objs = [os.path.join(BUILD, os.path.splitext(x)[0] + ".o") for x in SOURCES if x != "gdy.cpp"]
    missing = [o for o in objs if not os.path.exists(o)]
    if missing:
        raise RuntimeError(f"run build() first: missing {missing}")
    lib = os.path.join(san, "libgdy_san.so")
    r = subprocess.run([_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", lib, obj, *objs],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    return lib


if __name__ == "__main__":
    if "--sanitize" in sys.argv:
        print(build_sanitized())
    else:
        print(build())
