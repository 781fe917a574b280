"""The host runtime (planner, launcher, C-ABI) and the oracle built with
AddressSanitizer and UndefinedBehaviorSanitizer, and the CPU tests that
exercise them run in a child process under those builds (host code only;
no GPU).  Skipped where the compilers or the kernel objects of build() are
missing."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")
SUITES = ["tests/test_library_rules.py", "tests/test_selector.py", "tests/test_plan_properties.py",
          "tests/test_dispatch_map.py", "tests/test_oracle_pins.py", "tests/test_abi_cpu.py",
          "tests/test_tuner_cpu.py"]


def test_cpu_suites_under_asan_and_ubsan():
    if not os.path.exists(CLANG) or not (shutil.which("hipcc") or os.path.exists(os.path.join(ROCM, "bin", "hipcc"))):
        pytest.skip("no clang/hipcc")
    if not os.path.exists(os.path.join(ROOT, "paper_2409_02227_amd", "_build", "kernels_bf16.o")):
        pytest.skip("kernel objects missing: run build() first")
    import oracle
    from paper_2409_02227_amd import build
    lib = build.build_sanitized()
    orc = oracle.build_sanitized()
    rt = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                        text=True).stdout.strip()
    assert os.path.exists(rt), rt
    env = dict(os.environ, LD_PRELOAD=rt + (":" + os.environ["LD_PRELOAD"] if os.environ.get("LD_PRELOAD") else ""),
               ASAN_OPTIONS="detect_leaks=0:verify_asan_link_order=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", GDY_LIBRARY=lib, ORACLE_LIBRARY=orc)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu", "-p", "no:cacheprovider",
                        *SUITES], cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert " passed" in r.stdout
