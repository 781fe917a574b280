"""ctypes binding of libgdy (include/gdy.h): argument marshalling only.

Every step of the hot path -- validation, features, CD prediction,
grouping, variant binding, launches -- runs inside libgdy.so.  This module
turns Python/torch objects into the C structures and back.  Loading fails
loudly when the library is missing; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgdy.so")

MAX_GEMMS = 256
N_CD = 5
N_FEATURES = 18
CD_CLASSES = (1, 2, 4, 8, 16)

# gdy_dtype
F16, BF16, FP8_E4M3, F32 = 1, 2, 3, 4
# gdy_mode
SEQUENTIAL, DEFAULT, GO, SELECTOR, FORCED, FORCED_GROUPED = 0, 1, 2, 3, 4, 5
CU_PARTITION, CU_PARTITION_GO, CU_PARTITION_RC = 6, 7, 8
GEMM, ADD = 0, 1  # gdy_op
MODES = {"sequential": SEQUENTIAL, "default": DEFAULT, "go": GO,
         "selector": SELECTOR, "forced": FORCED, "forced_grouped": FORCED_GROUPED,
         "cu_partition": CU_PARTITION, "cu_partition_go": CU_PARTITION_GO,
         "cu_partition_rc": CU_PARTITION_RC}
# gdy_create use_cu_masks bits
RC_STREAMS, PARTITION_STREAMS = 1, 2

STATUS = {0: "GDY_OK", 1: "GDY_ERR_INVALID_ARG", 2: "GDY_ERR_UNSUPPORTED", 3: "GDY_ERR_ALIAS",
          4: "GDY_ERR_TOO_MANY", 5: "GDY_ERR_TABLE", 6: "GDY_ERR_HIP", 7: "GDY_ERR_NOMEM"}

EXPORTS = ("gdy_create", "gdy_destroy", "gdy_set_rc", "gdy_plan", "gdy_execute", "gdy_execute_static",
           "gdy_set_timing", "gdy_last_kernel_times", "gdy_kernel_times", "gdy_features", "gdy_dispatch_map",
           "gdy_variant_count",
           "gdy_variant_info", "gdy_variant_find", "gdy_isolated_variant",
           "gdy_catalogue_hash", "gdy_device_cus", "gdy_status_string", "gdy_last_error")


class GemmDesc(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int64), ("n", ctypes.c_int64), ("k", ctypes.c_int64),
                ("a_type", ctypes.c_int32), ("b_type", ctypes.c_int32), ("c_type", ctypes.c_int32),
                ("trans_a", ctypes.c_int32), ("trans_b", ctypes.c_int32),
                ("a", ctypes.c_void_p), ("lda", ctypes.c_int64),
                ("b", ctypes.c_void_p), ("ldb", ctypes.c_int64),
                ("c", ctypes.c_void_p), ("ldc", ctypes.c_int64),
                ("scale_a", ctypes.c_float), ("scale_b", ctypes.c_float),
                ("tenant", ctypes.c_int32), ("variant", ctypes.c_int32),
                ("batch", ctypes.c_int32), ("op", ctypes.c_int32),
                ("stride_a", ctypes.c_int64), ("stride_b", ctypes.c_int64),
                ("stride_c", ctypes.c_int64)]


class Plan(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("cd", ctypes.c_int32), ("n_groups", ctypes.c_int32),
                ("fallback", ctypes.c_int32),
                ("order", ctypes.c_int32 * MAX_GEMMS), ("group_of", ctypes.c_int32 * MAX_GEMMS),
                ("stream_of", ctypes.c_int32 * MAX_GEMMS), ("variant_of", ctypes.c_int32 * MAX_GEMMS),
                ("pred_cd", ctypes.c_int32 * MAX_GEMMS), ("group_size", ctypes.c_int32 * MAX_GEMMS),
                ("n_dispatches", ctypes.c_int32), ("dispatch_of", ctypes.c_int32 * MAX_GEMMS),
                ("split_of", ctypes.c_int32 * MAX_GEMMS)]

    def as_dict(self) -> dict:
        n = self.n
        return {"n": n, "cd": self.cd, "n_groups": self.n_groups, "fallback": self.fallback,
                "order": [x for x in self.order[:n] if x >= 0],
                "group_of": list(self.group_of[:n]), "stream_of": list(self.stream_of[:n]),
                "variant_of": list(self.variant_of[:n]), "pred_cd": list(self.pred_cd[:n]),
                "group_size": list(self.group_size[:self.n_groups]),
                "n_dispatches": self.n_dispatches, "dispatch_of": list(self.dispatch_of[:n]),
                "split_of": list(self.split_of[:n])}


class VariantDesc(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 64), ("dtype", ctypes.c_int32), ("trans_a", ctypes.c_int32),
                ("trans_b", ctypes.c_int32), ("bm", ctypes.c_int32), ("bn", ctypes.c_int32),
                ("bk", ctypes.c_int32), ("waves", ctypes.c_int32), ("mfma", ctypes.c_int32),
                ("lds_bytes", ctypes.c_int32), ("vgprs", ctypes.c_int32),
                ("occupancy", ctypes.c_int32), ("grid_cap_cus", ctypes.c_int32),
                ("direct", ctypes.c_int32), ("kind", ctypes.c_int32)]

    def as_dict(self) -> dict:
        d = {f: getattr(self, f) for f, _ in self._fields_}
        d["name"] = self.name.decode()
        return d


class GdyError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


_lib = None


def load_library(path: str = None) -> ctypes.CDLL:
    """Load libgdy.so (raises if it is missing: no fallback exists).
    GDY_LIBRARY names another build of it (the sanitizer build)."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or os.environ.get("GDY_LIBRARY") or LIB_PATH
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with paper_2409_02227_amd.build.build()")
    lib = ctypes.CDLL(path)
    P, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
    sig = {
        "gdy_create": (i32, [ctypes.POINTER(P), ctypes.c_int, ctypes.c_char_p, i32, i32]),
        "gdy_destroy": (None, [P]),
        "gdy_set_rc": (i32, [P, i32]),
        "gdy_plan": (i32, [P, ctypes.POINTER(GemmDesc), i32, i32, i32, ctypes.POINTER(Plan)]),
        "gdy_execute": (i32, [P, ctypes.POINTER(GemmDesc), i32, i32, i32, P, ctypes.POINTER(Plan)]),
        "gdy_execute_static": (i32, [P, ctypes.POINTER(GemmDesc), i32, i32, i32, P, ctypes.POINTER(Plan)]),
        "gdy_set_timing": (i32, [P, i32]),
        "gdy_last_kernel_times": (i32, [P, ctypes.POINTER(ctypes.c_float),
                                        ctypes.POINTER(ctypes.c_float), i32]),
        "gdy_kernel_times": (i32, [P, i32, ctypes.POINTER(ctypes.c_float),
                                   ctypes.POINTER(ctypes.c_float), i32]),
        "gdy_features": (i32, [P, ctypes.POINTER(GemmDesc), ctypes.POINTER(ctypes.c_double)]),
        "gdy_dispatch_map": (i32, [P, ctypes.POINTER(GemmDesc), i32, i32, i32, i32, i32, ctypes.POINTER(i32),
                                   ctypes.POINTER(i32), ctypes.POINTER(i32), ctypes.POINTER(i32),
                                   ctypes.POINTER(i64)]),
        "gdy_variant_count": (i32, [P]),
        "gdy_variant_info": (i32, [P, i32, ctypes.POINTER(VariantDesc)]),
        "gdy_variant_find": (i32, [P, ctypes.c_char_p]),
        "gdy_isolated_variant": (i32, [P, ctypes.POINTER(GemmDesc)]),
        "gdy_catalogue_hash": (u64, [P]),
        "gdy_device_cus": (i32, [P]),
        "gdy_status_string": (ctypes.c_char_p, [i32]),
        "gdy_last_error": (ctypes.c_char_p, [P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


_TORCH_DTYPE = None


def _dtype_code(t) -> int:
    global _TORCH_DTYPE
    if _TORCH_DTYPE is None:
        import torch
        _TORCH_DTYPE = {torch.float16: F16, torch.bfloat16: BF16, torch.float8_e4m3fn: FP8_E4M3,
                        torch.uint8: FP8_E4M3, torch.float32: F32}
    return _TORCH_DTYPE[t.dtype]


@dataclass
class Add:
    """Element-wise C = A + B over an M x N region: the non-GEMM that co-runs
    with GEMMs (Sec. 7.1).  2-D tensors of one type (bf16, fp16, fp32), or
    3-D strided batches; the last dimension contiguous."""
    a: object
    b: object
    c: object
    tenant: int = 0
    variant: int = -1

    def desc(self) -> GemmDesc:
        a, b, c = self.a, self.b, self.c
        batch = c.shape[0] if c.dim() == 3 else 0
        if batch and any(t.dim() == 3 and t.shape[0] != batch for t in (a, b)):
            raise ValueError("batched operands disagree on the batch size")
        if not batch and (a.dim() == 3 or b.dim() == 3):
            raise ValueError("a batched A or B needs a batched C")

        def mat(t):
            return (t[0], t.stride(0)) if t.dim() == 3 else (t, 0)
        (a2, sa), (b2, sb), (c2, sc) = mat(a), mat(b), mat(c)
        for t in (a2, b2, c2):
            if t.dim() != 2 or (t.shape[1] > 1 and t.stride(1) != 1):
                raise ValueError("operands must be 2-D (or 3-D batches) with a contiguous last dimension")
        m, n = c2.shape
        if tuple(a2.shape) != (m, n) or tuple(b2.shape) != (m, n):
            raise ValueError("add operands must have C's shape")
        d = GemmDesc()
        d.m, d.n, d.k = m, n, 0
        d.a_type, d.b_type, d.c_type = _dtype_code(a), _dtype_code(b), _dtype_code(c)
        d.a, d.lda = a.data_ptr(), max(a2.stride(0), 1)
        d.b, d.ldb = b.data_ptr(), max(b2.stride(0), 1)
        d.c, d.ldc = c.data_ptr(), max(c2.stride(0), 1)
        d.scale_a = d.scale_b = 1.0
        d.tenant, d.variant = int(self.tenant), int(self.variant)
        d.batch, d.op = batch, ADD
        d.stride_a, d.stride_b, d.stride_c = sa, sb, sc
        return d


@dataclass
class Gemm:
    """One GEMM of a submission, from torch device tensors.

    a: M x K (or K x M when trans_a) row-major; b: K x N (or N x K when
    trans_b); c: M x N output.  Strided 2-D views are allowed as long as the
    last dimension is contiguous (ld = stride(0)).  A strided batch
    (B-GEMM) passes 3-D tensors whose first dimension is the batch: C must
    be 3-D; A or B may stay 2-D to be shared by every item (stride 0)."""
    a: object
    b: object
    c: object
    trans_a: int = 0
    trans_b: int = 0
    scale_a: float = 1.0
    scale_b: float = 1.0
    tenant: int = 0
    variant: int = -1

    def desc(self) -> GemmDesc:
        a, b, c = self.a, self.b, self.c
        batch = c.shape[0] if c.dim() == 3 else 0
        if batch and any(t.dim() == 3 and t.shape[0] != batch for t in (a, b)):
            raise ValueError("batched operands disagree on the batch size")
        if not batch and (a.dim() == 3 or b.dim() == 3):
            raise ValueError("a batched A or B needs a batched C")

        def mat(t):  # the 2-D item view and the item stride in elements
            if t.dim() == 3:
                return t[0], t.stride(0)
            return t, 0
        (a2, sa), (b2, sb), (c2, sc) = mat(a), mat(b), mat(c)
        for t in (a2, b2, c2):
            if t.dim() != 2 or (t.shape[1] > 1 and t.stride(1) != 1):
                raise ValueError("operands must be 2-D (or 3-D batches) with a contiguous last dimension")
        m, n = c2.shape
        k = a2.shape[0] if self.trans_a else a2.shape[1]
        am = a2.shape[1] if self.trans_a else a2.shape[0]
        bk, bn = (b2.shape[1], b2.shape[0]) if self.trans_b else (b2.shape[0], b2.shape[1])
        if am != m or bn != n or bk != k:
            raise ValueError(f"shapes disagree: op(A) {am}x{k}, op(B) {bk}x{bn}, C {m}x{n}")
        d = GemmDesc()
        d.m, d.n, d.k = m, n, k
        d.a_type, d.b_type, d.c_type = _dtype_code(a), _dtype_code(b), _dtype_code(c)
        d.trans_a, d.trans_b = int(self.trans_a), int(self.trans_b)
        d.a, d.lda = a.data_ptr(), max(a2.stride(0), 1)
        d.b, d.ldb = b.data_ptr(), max(b2.stride(0), 1)
        d.c, d.ldc = c.data_ptr(), max(c2.stride(0), 1)
        d.scale_a, d.scale_b = float(self.scale_a), float(self.scale_b)
        d.tenant, d.variant = int(self.tenant), int(self.variant)
        d.batch = batch
        d.stride_a, d.stride_b, d.stride_c = sa, sb, sc
        return d


def descs(gemms) -> ctypes.Array:
    """Marshal Gemm objects (or GemmDesc) into a C array once."""
    arr = (GemmDesc * max(len(gemms), 1))()
    for i, g in enumerate(gemms):
        arr[i] = g if isinstance(g, GemmDesc) else g.desc()
    return arr


class Context:
    """A libgdy context on one device (see gdy_create)."""

    def __init__(self, device: int = 0, table: str | None = None, max_streams: int = 16,
                 use_cu_masks: int = 0):
        self.lib = load_library()
        h = ctypes.c_void_p()
        st = self.lib.gdy_create(ctypes.byref(h), device,
                                 table.encode() if table else None, max_streams, int(use_cu_masks))
        if st != 0:
            raise GdyError(st, f"gdy_create failed (see stderr); table={table}")
        self.h = h

    def close(self):
        if getattr(self, "h", None):
            self.lib.gdy_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def last_error(self) -> str:
        """gdy_last_error: the message of the last failure (after creation:
        why a GO table was not used), "" if none."""
        return self.lib.gdy_last_error(self.h).decode()

    def _check(self, st):
        if st != 0:
            raise GdyError(st, self.lib.gdy_last_error(self.h).decode())

    def plan(self, gemms, mode="selector", forced_cd: int = 0) -> dict:
        arr = descs(gemms)
        p = Plan()
        self._check(self.lib.gdy_plan(self.h, arr, len(gemms), _mode(mode), forced_cd, ctypes.byref(p)))
        return p.as_dict()

    def execute(self, gemms, mode="selector", forced_cd: int = 0, stream=None, want_plan=False):
        """Launch a submission on `stream` (torch stream, raw handle or None for
        torch's current stream).  Returns the plan dict when want_plan."""
        arr = descs(gemms)
        handle = _stream_handle(stream)
        p = Plan()
        self._check(self.lib.gdy_execute(self.h, arr, len(gemms), _mode(mode), forced_cd,
                                         handle, ctypes.byref(p)))
        return p.as_dict() if want_plan else None

    def execute_static(self, gemms, mode="selector", forced_cd: int = 0, stream=None, want_plan=False):
        """gdy_execute_static: as execute(), with the split-K planes in the
        library's static device array (no allocation)."""
        arr = descs(gemms)
        handle = _stream_handle(stream)
        p = Plan()
        self._check(self.lib.gdy_execute_static(self.h, arr, len(gemms), _mode(mode), forced_cd,
                                                handle, ctypes.byref(p)))
        return p.as_dict() if want_plan else None

    def execute_descs(self, arr, n, mode, forced_cd, handle):
        """Launch prepared GemmDesc arrays (no per-call marshalling)."""
        self._check(self.lib.gdy_execute(self.h, arr, n, mode, forced_cd, handle, None))

    def set_rc(self, budget_cus: int):
        self._check(self.lib.gdy_set_rc(self.h, budget_cus))

    def set_timing(self, on: bool):
        self._check(self.lib.gdy_set_timing(self.h, int(on)))

    def kernel_times(self, n: int, back: int = 0):
        """(start_ms, end_ms) lists for the GEMMs of a timed submission
        (back = 0: the last one), relative to that submission's start."""
        s = (ctypes.c_float * max(n, 1))()
        e = (ctypes.c_float * max(n, 1))()
        self._check(self.lib.gdy_kernel_times(self.h, back, s, e, n))
        return list(s[:n]), list(e[:n])

    def dispatch_map(self, gemms, mode="selector", forced_cd: int = 0, dispatch: int = 0,
                     max_workgroups: int = 1 << 20) -> dict:
        """gdy_dispatch_map: per workgroup of one dispatch, the member it serves
        (-1: idle), its first work item and stride; per GEMM its item count."""
        arr = descs(gemms)
        n = len(gemms)
        grid = ctypes.c_int32()
        cap = max_workgroups
        gw = (ctypes.c_int32 * cap)()
        fi = (ctypes.c_int32 * cap)()
        st = (ctypes.c_int32 * cap)()
        items = (ctypes.c_int64 * max(n, 1))()
        self._check(self.lib.gdy_dispatch_map(self.h, arr, n, _mode(mode), forced_cd, dispatch, cap,
                                              ctypes.byref(grid), gw, fi, st, items))
        g = min(grid.value, cap)
        return {"grid": grid.value, "gemm": list(gw[:g]), "first": list(fi[:g]), "stride": list(st[:g]),
                "items": list(items[:n])}

    def features(self, gemm) -> list:
        d = gemm if isinstance(gemm, GemmDesc) else gemm.desc()
        out = (ctypes.c_double * N_FEATURES)()
        self._check(self.lib.gdy_features(self.h, ctypes.byref(d), out))
        return list(out)

    def variant_count(self) -> int:
        return int(self.lib.gdy_variant_count(self.h))

    def variant(self, vid: int) -> dict:
        v = VariantDesc()
        self._check(self.lib.gdy_variant_info(self.h, vid, ctypes.byref(v)))
        return v.as_dict()

    def variants(self) -> list:
        return [self.variant(i) for i in range(self.variant_count())]

    def find(self, name: str) -> int:
        return int(self.lib.gdy_variant_find(self.h, name.encode()))

    def isolated_variant(self, gemm) -> int:
        d = gemm if isinstance(gemm, GemmDesc) else gemm.desc()
        return int(self.lib.gdy_isolated_variant(self.h, ctypes.byref(d)))

    def catalogue_hash(self) -> int:
        return int(self.lib.gdy_catalogue_hash(self.h))

    def cus(self) -> int:
        return int(self.lib.gdy_device_cus(self.h))


def _mode(mode) -> int:
    return MODES[mode] if isinstance(mode, str) else int(mode)


def _stream_handle(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if hasattr(stream, "cuda_stream"):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))
