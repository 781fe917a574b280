"""CPU checks of the C-ABI boundary: the built library loads and exports
every function include/gdy.h declares, and the binding's structures match
the header's field order and sizes."""
import ctypes
import os
import re

import pytest

from paper_2409_02227_amd import gdy

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gdy.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gdy_[a-z_]+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(gdy.EXPORTS)


def test_library_loads_and_exports_every_declared_symbol():
    if not os.path.exists(gdy.LIB_PATH):
        pytest.fail("libgdy.so not built: run __graft_entry__.build()")
    lib = ctypes.CDLL(gdy.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} declared in gdy.h but not exported"


def test_struct_layouts_match_header():
    # gdy_gemm: 3 int64, 5 int32, then (ptr, int64) x 3, 2 floats, 2 int32, 2 int32, 3 int64
    assert ctypes.sizeof(gdy.GemmDesc) == 3 * 8 + 5 * 4 + 4 + 6 * 8 + 2 * 4 + 2 * 4 + 2 * 4 + 3 * 8
    assert gdy.GemmDesc.batch.offset == 112 and gdy.GemmDesc.stride_a.offset == 120
    assert gdy.GemmDesc.a.offset == 48
    assert ctypes.sizeof(gdy.Plan) == 4 * 4 + 6 * 4 * gdy.MAX_GEMMS + 4 + 2 * 4 * gdy.MAX_GEMMS
    assert gdy.Plan.dispatch_of.offset == 4 * 4 + 6 * 4 * gdy.MAX_GEMMS + 4
    assert ctypes.sizeof(gdy.VariantDesc) == 64 + 14 * 4
    text = open(HEADER).read()
    assert "#define GDY_MAX_GEMMS 256" in text and "#define GDY_N_FEATURES 18" in text


def test_status_strings_without_device():
    lib = gdy.load_library()
    assert lib.gdy_status_string(0) == b"ok"
    assert lib.gdy_status_string(3).startswith(b"output aliases")
    assert lib.gdy_last_error(None) == b"null context"
    assert lib.gdy_variant_count(None) == 0


def test_binding_layouts_equal_the_c_compilers(tmp_path):
    """Every field offset and struct size of the ctypes binding equals what
    a C compiler makes of include/gdy.h."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    structs = {"gdy_gemm": gdy.GemmDesc, "gdy_plan_t": gdy.Plan, "gdy_variant_desc": gdy.VariantDesc}
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "gdy.h"', "int main(void) {"]
    for cname, py in structs.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in py._fields_:
            lines.append(f'  printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {(a, b): int(c) for a, b, c in (l.split() for l in out if l)}
    for cname, py in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for f, _ in py._fields_:
            assert got[(cname, f)] == getattr(py, f).offset, (cname, f)


def test_binding_rejects_operands_that_disagree():
    """Gemm and Add descriptors are built from tensors only when their shapes,
    batch sizes and last-dimension strides agree: a B of the wrong shape would
    otherwise hand the library extents past its allocation.  CPU tensors:
    building a descriptor touches no device."""
    torch = pytest.importorskip("torch")
    bf = torch.bfloat16
    a, b, c = torch.zeros(8, 16, dtype=bf), torch.zeros(16, 4, dtype=bf), torch.zeros(8, 4, dtype=bf)
    d = gdy.Gemm(a, b, c).desc()
    assert (d.m, d.n, d.k, d.lda, d.ldb, d.ldc) == (8, 4, 16, 16, 4, 4)
    d = gdy.Gemm(a, b.t().contiguous(), c, 0, 1).desc()  # B stored N x K
    assert (d.k, d.ldb, d.trans_b) == (16, 16, 1)
    bad = [gdy.Gemm(a, torch.zeros(15, 4, dtype=bf), c),            # K differs
           gdy.Gemm(a, torch.zeros(16, 5, dtype=bf), c),            # N differs
           gdy.Gemm(torch.zeros(9, 16, dtype=bf), b, c),            # M differs
           gdy.Gemm(a, b, c, 0, 1),                                 # B^T would be 4 x 16
           gdy.Gemm(a, torch.zeros(4, 16, dtype=bf).t(), c),        # last dimension strided
           gdy.Gemm(torch.zeros(2, 8, 16, dtype=bf), torch.zeros(3, 16, 4, dtype=bf),
                    torch.zeros(3, 8, 4, dtype=bf)),                # batch sizes differ
           gdy.Add(c, c.t().contiguous().t(), torch.zeros(8, 4, dtype=bf)),  # strided add operand
           gdy.Add(torch.zeros(2, 8, 4, dtype=bf), c, torch.zeros(3, 8, 4, dtype=bf))]
    for g in bad:
        with pytest.raises(ValueError):
            g.desc()
    e = gdy.Add(c, c, torch.zeros(8, 4, dtype=bf)).desc()
    assert (e.m, e.n, e.k, e.op) == (8, 4, 0, gdy.ADD)
