"""CPU oracle for concurrent independent GEMMs (GOLDYLOC, arXiv 2409.02227).

TEST INFRASTRUCTURE ONLY.  Nothing in the product library imports this
package.  Only the test suite, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may load it.  It shares no code with the HIP
path: the arithmetic lives in ``oracle.c`` (plain C, fp64, built with gcc)
and in ``selector.py`` (plain Python/numpy).

GEMM (Sec. 2.1.2): C = sa*sb * op(A) @ op(B) with A M x K and B giving
the K x N operand; T1/T2 mark transposed use.  ``gemm`` returns the fp64
reference and the error-bound sum |sa*sb| * sum_k |a(i,k) b(k,j)|.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

# oracle-private type codes; must match the enum at the top of oracle.c
_TYPES = {"f16": 0, "bf16": 1, "e4m3fn": 2, "f32": 3, "f64": 4}
_NP_STORAGE = {"f16": np.uint16, "bf16": np.uint16, "e4m3fn": np.uint8,
               "f32": np.float32, "f64": np.float64}

_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so with gcc and OpenMP."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def build_sanitized() -> str:
    """liboracle_san.so: the oracle built with clang's AddressSanitizer and
    UndefinedBehaviorSanitizer (load with ORACLE_LIBRARY=<path> in a process
    whose LD_PRELOAD starts with clang's ASan runtime)."""
    out = os.path.join(_HERE, "liboracle_san.so")
    clang = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "bin", "clang")
    llvm_lib = os.path.join(os.path.dirname(os.path.dirname(clang)), "lib")
    cmd = [clang, "-O1", "-g", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-Wall", "-Wextra",
           "-o", out, _SRC, "-lm", f"-L{llvm_lib}", f"-Wl,-rpath,{llvm_lib}"]
    subprocess.run(cmd, check=True)
    return out


def _load():
    global _lib
    if _lib is None:
        path = os.environ.get("ORACLE_LIBRARY") or _LIB
        if path == _LIB and (not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC)):
            build(force=True)
        lib = ctypes.CDLL(path)
        i64, i32, dbl, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_double, ctypes.c_void_p
        lib.orc_decode.argtypes = [i32, vp, i64, vp]
        lib.orc_decode.restype = i32
        lib.orc_gemm.argtypes = [i64, i64, i64, i32, i32, i32, vp, i64, dbl,
                                 i32, vp, i64, dbl, vp, vp, i64, vp, vp]
        lib.orc_gemm.restype = i32
        lib.orc_gemm_entries.argtypes = [i64, i64, i64, i32, i32, i32, vp, i64, dbl,
                                         i32, vp, i64, dbl, i64, vp, vp, vp, vp]
        lib.orc_gemm_entries.restype = i32
        lib.orc_num_threads.argtypes = []
        lib.orc_num_threads.restype = i32
        _lib = lib
    return _lib


def _ptr(x: np.ndarray | None) -> int | None:
    return None if x is None else x.ctypes.data


def _as_codes(x, dtype: str) -> np.ndarray:
    arr = np.ascontiguousarray(np.asarray(x))
    want = _NP_STORAGE[dtype]
    if arr.dtype != want:
        if arr.dtype.itemsize != np.dtype(want).itemsize:
            raise TypeError(f"{dtype} operand needs {np.dtype(want)} storage, got {arr.dtype}")
        arr = arr.view(want)
    return arr


def decode(codes, dtype: str) -> np.ndarray:
    """Exact fp64 values of an array of encoded elements."""
    arr = _as_codes(codes, dtype)
    out = np.empty(arr.shape, dtype=np.float64)
    rc = _load().orc_decode(_TYPES[dtype], _ptr(arr), arr.size, _ptr(out))
    if rc:
        raise ValueError("orc_decode rejected its arguments")
    return out


def num_threads() -> int:
    return int(_load().orc_num_threads())


def gemm(m, n, k, a, a_type, lda, b, b_type, ldb, trans_a=0, trans_b=0,
         scale_a=1.0, scale_b=1.0, want_bound=True):
    """fp64 reference (and bound) for one GEMM over flat encoded buffers.

    ``a`` and ``b`` are 1-D arrays of codes laid out as the storage reading
    in oracle.c describes; returns (ref, bound) as M x N float64 arrays.
    """
    a = _as_codes(a, a_type).reshape(-1)
    b = _as_codes(b, b_type).reshape(-1)
    ref = np.empty((m, n), dtype=np.float64)
    bound = np.empty((m, n), dtype=np.float64) if want_bound else None
    a_s = np.empty(max(m * k, 1), dtype=np.float64)
    b_s = np.empty(max(k * n, 1), dtype=np.float64)
    _check_extent(m, k, lda, trans_a, a.size, "A")
    _check_extent(k, n, ldb, trans_b, b.size, "B")
    rc = _load().orc_gemm(m, n, k, int(trans_a), int(trans_b),
                          _TYPES[a_type], _ptr(a), lda, float(scale_a),
                          _TYPES[b_type], _ptr(b), ldb, float(scale_b),
                          _ptr(ref), _ptr(bound), n, _ptr(a_s), _ptr(b_s))
    if rc:
        raise ValueError("orc_gemm rejected its arguments")
    return ref, bound


def gemm_entries(m, n, k, a, a_type, lda, b, b_type, ldb, rows, cols,
                 trans_a=0, trans_b=0, scale_a=1.0, scale_b=1.0):
    """fp64 reference and bound for selected (row, col) outputs only."""
    a = _as_codes(a, a_type).reshape(-1)
    b = _as_codes(b, b_type).reshape(-1)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    if rows.shape != cols.shape:
        raise ValueError("rows and cols differ in shape")
    _check_extent(m, k, lda, trans_a, a.size, "A")
    _check_extent(k, n, ldb, trans_b, b.size, "B")
    ref = np.empty(rows.shape, dtype=np.float64)
    bound = np.empty(rows.shape, dtype=np.float64)
    rc = _load().orc_gemm_entries(m, n, k, int(trans_a), int(trans_b),
                                  _TYPES[a_type], _ptr(a), lda, float(scale_a),
                                  _TYPES[b_type], _ptr(b), ldb, float(scale_b),
                                  rows.size, _ptr(rows), _ptr(cols), _ptr(ref), _ptr(bound))
    if rc:
        raise ValueError("orc_gemm_entries rejected its arguments")
    return ref, bound


def add(m, n, a, a_type, lda, b, b_type, ldb):
    """Element-wise A + B over an M x N region (the non-GEMM co-runner of
    Sec. 7.1), in fp64 on the decoded operands; returns (ref, bound) with
    bound = |a| + |b|, the scale a correctly rounded result is judged on."""
    a = _as_codes(a, a_type).reshape(-1)
    b = _as_codes(b, b_type).reshape(-1)
    _check_extent(m, n, lda, 0, a.size, "A")
    _check_extent(m, n, ldb, 0, b.size, "B")
    rows = np.arange(m)[:, None]
    cols = np.arange(n)[None, :]
    va = decode(a[rows * lda + cols], a_type)
    vb = decode(b[rows * ldb + cols], b_type)
    return va + vb, np.abs(va) + np.abs(vb)


def _check_extent(rows, cols, ld, trans, size, name):
    """The flat buffer must hold every element op() touches."""
    if rows == 0 or cols == 0:
        return
    r, c = (cols, rows) if trans else (rows, cols)  # stored shape
    need = (r - 1) * ld + c
    if ld < c or size < need:
        raise ValueError(f"{name}: buffer of {size} elements too small for {r}x{c} with ld={ld}")


def accept(c_values, ref, bound, tau, abs_term=1e-6):
    """Elementwise acceptance |c - ref| <= tau*bound + abs_term.

    Returns (ok, worst_ratio) where worst_ratio is max |c-ref|/(tau*bound+abs).
    """
    c_values = np.asarray(c_values, dtype=np.float64)
    err = np.abs(c_values - ref)
    lim = tau * bound + abs_term
    ok = bool(np.all(err <= lim)) and bool(np.all(np.isfinite(c_values)))
    worst = float(np.max(err / lim)) if err.size else 0.0
    return ok, worst
