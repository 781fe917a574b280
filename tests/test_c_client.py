"""The C-ABI without Python: examples/gemm_set.cpp is a C++ program that
allocates with HIP, fills four bf16 GEMMs (one of them with a ragged M, N and
an odd K), runs them with gdy_execute in the selector mode and writes C.
examples/graph_static.cpp runs four GEMMs (two of them split along K) with
gdy_execute, captures gdy_execute_static into a HIP graph and replays it
three times, comparing every replay with the eager call bit for bit.

Its operands are hashed small dyadic values (multiples of 1/8 and 1/16 below
1 in magnitude), so every partial sum of any fp32 accumulation order is exact
and each output is the exact sum rounded once to bf16: the test checks every
element bit for bit against the oracle's fp64 result rounded to nearest even,
and against the oracle's error bound.  The GPU run is a child process; this
process does not touch the GPU for it."""
import os
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "paper_2409_02227_amd", "examples", "gemm_set")
GRAPH_EXE = os.path.join(ROOT, "paper_2409_02227_amd", "examples", "graph_static")
GRAPH_SHAPES = [(16, 1024, 8192), (32, 2048, 8192), (512, 1024, 1024), (1024, 2048, 4096)]  # as in the program
TABLE = os.path.join(ROOT, "paper_2409_02227_amd", "tables", "gfx950.table")
SHAPES = [(512, 1024, 2048), (64, 4096, 1024), (1000, 300, 777), (16, 2048, 8192)]  # as in the program


def _mix(r, c, g, salt):
    """The program's 32-bit hash of (row, column, GEMM, operand), wrapping."""
    u = np.uint32
    h = (r.astype(u) * u(73856093)) ^ (c.astype(u) * u(19349663)) ^ u((g * 83492791) & 0xFFFFFFFF) ^ u(salt)
    h ^= h >> u(13)
    h *= u(0x5bd1e995)
    h ^= h >> u(15)
    return h


def _operands(g, m, n, k):
    """The program's operands of GEMM g as fp32 arrays."""
    i, kk = np.arange(m)[:, None], np.arange(k)[None, :]
    a = ((_mix(i, kk, g, 1) % 13).astype(np.int64) - 6) / 8.0
    kk, j = np.arange(k)[:, None], np.arange(n)[None, :]
    b = ((_mix(kk, j, g, 2) % 11).astype(np.int64) - 5) / 16.0
    return a.astype(np.float32), b.astype(np.float32)


def _bf16_codes_exact(x32):
    """bf16 codes of fp32 values that bf16 holds exactly (the upper halves)."""
    u = x32.view(np.uint32)
    assert not np.any(u & 0xFFFF), "operand not exact in bf16"
    return (u >> 16).astype(np.uint16)


def _bf16_rne(x64):
    """Round fp64 values that fp32 holds exactly to bf16 codes, nearest even."""
    x32 = x64.astype(np.float32)
    assert np.array_equal(x32.astype(np.float64), x64), "sum not exact in fp32"
    u = x32.view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


@pytest.mark.parametrize("exe", [EXE, GRAPH_EXE])
def test_program_is_built_and_free_of_python(exe):
    """The program exists, links libgdy from the package directory and
    neither torch nor Python, and refuses a bad command line before any HIP
    call (so this runs without a GPU)."""
    assert os.path.exists(exe), f"{exe} not built: run __graft_entry__.build()"
    ldd = subprocess.run(["ldd", exe], capture_output=True, text=True, check=True).stdout
    lib = [l for l in ldd.splitlines() if "libgdy.so" in l]
    assert lib and os.path.samefile(lib[0].split("=>")[1].split("(")[0].strip(),
                                    os.path.join(ROOT, "paper_2409_02227_amd", "libgdy.so"))
    assert "torch" not in ldd and "python" not in ldd
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 2 and "usage" in r.stderr


def _check_against_oracle(path, shapes):
    got = np.fromfile(path, dtype=np.uint16)
    assert got.size == sum(m * n for m, n, _ in shapes)
    off = 0
    for g, (m, n, k) in enumerate(shapes):
        a, b = _operands(g, m, n, k)
        ref, bound = oracle.gemm(m, n, k, _bf16_codes_exact(a), "bf16", k, _bf16_codes_exact(b), "bf16", n)
        c = got[off:off + m * n].reshape(m, n)
        off += m * n
        ok, worst = oracle.accept(oracle.decode(c, "bf16").reshape(-1), ref.reshape(-1), bound.reshape(-1), 2.0 ** -7)
        assert ok, f"GEMM {g} ({m}, {n}, {k}): worst ratio {worst:.3g}"
        bad = np.argwhere(c != _bf16_rne(ref))
        assert bad.size == 0, f"GEMM {g} ({m}, {n}, {k}): {len(bad)} elements differ, first {bad[0]}"


@pytest.mark.gpu
def test_program_output_matches_the_oracle(tmp_path):
    out = tmp_path / "c.bin"
    print(f"running {EXE}", flush=True)
    r = subprocess.run([EXE, TABLE, str(out)], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok")
    assert "fallback 0" in r.stdout  # the GO table was loaded
    _check_against_oracle(out, SHAPES)


@pytest.mark.gpu
@pytest.mark.parametrize("mode", ["selector", "default"])
def test_graph_replays_of_the_static_entry_match_the_eager_call(tmp_path, mode):
    out = tmp_path / "c.bin"
    print(f"running {GRAPH_EXE} {mode}", flush=True)
    r = subprocess.run([GRAPH_EXE, TABLE, str(out), mode], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0 and "replays identical" in r.stdout
    assert "0 split GEMMs" not in r.stdout  # split planes live in the static array
    _check_against_oracle(out, GRAPH_SHAPES)
