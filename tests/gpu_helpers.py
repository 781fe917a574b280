"""Helpers for GPU parity tests: run GEMMs through the C-ABI and compare
them with the CPU oracle: |c - ref| <= tau * sum_k |a b| + 1e-6 with
tau = 2^-7 for 16-bit inputs and 2^-3 for fp8 (the stated contract), and
2^-10 for fp32 inputs (derived: an fp32 sum of K <= 16384 products drifts
by at most K * 2^-24 of sum |a b|)."""
import numpy as np
import torch

import oracle
from paper_2409_02227_amd import inputs

TAU = {"bf16": 2.0 ** -7, "f16": 2.0 ** -7, "fp8": 2.0 ** -3, "f32": 2.0 ** -10}
ORC = {"bf16": "bf16", "f16": "f16", "fp8": "e4m3fn", "f32": "f32"}
# element-wise add: half an ulp of the output type, relative to |a| + |b|
TAU_ADD = {"bf16": 2.0 ** -8, "f16": 2.0 ** -11, "f32": 2.0 ** -24}
FULL_LIMIT = 3e8  # multiply-adds the oracle does in full; above: sampled


def out_codes(mat) -> np.ndarray:
    """Output codes (M x N; uint16, or uint32 for fp32 results) copied to the host."""
    c = mat.c.cpu().contiguous()
    if c.dtype == torch.float32:
        return c.view(torch.int32).numpy().view(np.uint32)
    return c.view(torch.int16).numpy().view(np.uint16)


def decode_out(mat) -> np.ndarray:
    out = inputs.OUT[mat.spec.dtype]
    return oracle.decode(out_codes(mat), {"f16": "f16", "bf16": "bf16", "f32": "f32"}[out])


def check(mat, rng=None, samples=8, label=""):
    """Compare one materialised GEMM with the oracle (each item of a strided
    batch against the oracle on that item's operands); returns worst ratio."""
    s = mat.spec
    if s.batch > 0:
        worst = 0.0
        for i in range(s.batch):
            item = _item(mat, i)
            worst = max(worst, check(item, rng, samples, f"{label} item {i}"))
        assert_untouched(mat, label)
        return worst
    dt = ORC[s.dtype]
    got = decode_out(mat)
    if s.m * s.n * s.k <= FULL_LIMIT:
        ref, bound = oracle.gemm(s.m, s.n, s.k, mat.host["a"], dt, s.ld("a"), mat.host["b"], dt,
                                 s.ld("b"), s.trans_a, s.trans_b, mat.scale_a, mat.scale_b)
        ok, worst = oracle.accept(got, ref, bound, TAU[s.dtype])
    else:
        rng = rng or np.random.default_rng(s.seed)
        rows = rng.choice(s.m, size=min(samples, s.m), replace=False)
        cols = rng.choice(s.n, size=min(samples, s.n), replace=False)
        if s.m <= 32:
            rows = np.arange(s.m)
        ok, worst = accept_rows_cols(got[rows], got[:, cols], s.m, s.n, s.k, mat.host["a"], dt, s.ld("a"),
                                     mat.host["b"], dt, s.ld("b"), rows, cols, TAU[s.dtype], s.trans_a,
                                     s.trans_b, mat.scale_a, mat.scale_b)
    assert ok, f"{label} {s.name} ({s.m},{s.n},{s.k},{s.dtype},t{s.trans_a}{s.trans_b}): " \
               f"outside bound, worst ratio {worst:.3g}"
    assert_untouched(mat, label)
    return worst


def rows_cols_ref(m, n, k, a, a_dt, lda, b, b_dt, ldb, rows, cols, ta=0, tb=0, sa=1.0, sb=1.0):
    """Oracle values and bounds of the full rows `rows` (len(rows) x n) and
    the full columns `cols` (m x len(cols)) of C = op(A) op(B).  Each part is
    the oracle's own GEMM over a copy of the stored rows or columns of A or B
    those outputs read (the codes are copied, not changed: every element is
    still the oracle's k-ascending sum), which streams the operands instead
    of walking a column of B per output."""
    rows = np.asarray(rows, dtype=np.int64)
    cols = np.asarray(cols, dtype=np.int64)
    a2 = np.asarray(a).reshape(-1)
    b2 = np.asarray(b).reshape(-1)
    a_st, b_st = _stored(a2, lda), _stored(b2, ldb)
    if ta == 0:  # op(A) row i is stored row i
        ar, lda_r = a_st[rows, :k], k
    else:        # op(A) row i is stored column i of a K x M operand
        ar, lda_r = a_st[:k, rows], len(rows)
    if tb == 0:  # op(B) column j is stored column j of a K x N operand
        bc, ldb_c = b_st[:k, cols], len(cols)
    else:        # op(B) column j is stored row j
        bc, ldb_c = b_st[cols, :k], k
    ref_r, bd_r = oracle.gemm(len(rows), n, k, np.ascontiguousarray(ar).reshape(-1), a_dt, lda_r, b2, b_dt, ldb,
                              ta, tb, sa, sb)
    ref_c, bd_c = oracle.gemm(m, len(cols), k, a2, a_dt, lda, np.ascontiguousarray(bc).reshape(-1), b_dt, ldb_c,
                              ta, tb, sa, sb)
    return ref_r, bd_r, ref_c, bd_c


def _stored(flat, ld):
    """A flat operand as its stored rows of ld elements (a last partial row,
    as a minimal extent ends, is completed with zero codes that no index
    below reaches)."""
    if flat.size % ld:
        full = np.zeros(-(-flat.size // ld) * ld, dtype=flat.dtype)
        full[:flat.size] = flat
        flat = full
    return flat.reshape(-1, ld)


def accept_rows_cols(got_rows, got_cols, m, n, k, a, a_dt, lda, b, b_dt, ldb, rows, cols, tau, ta=0, tb=0,
                     sa=1.0, sb=1.0):
    """oracle.accept over full rows (got_rows: len(rows) x n decoded values)
    and full columns (got_cols: m x len(cols)) of a result."""
    ref_r, bd_r, ref_c, bd_c = rows_cols_ref(m, n, k, a, a_dt, lda, b, b_dt, ldb, rows, cols, ta, tb, sa, sb)
    ok_r, w_r = oracle.accept(got_rows, ref_r, bd_r, tau)
    ok_c, w_c = oracle.accept(got_cols, ref_c, bd_c, tau)
    return ok_r and ok_c, max(w_r, w_c)


def assert_untouched(mat, label=""):
    """C's padding columns (between n and ldc) and the guard rows behind C's
    last row still hold the NaN they were filled with."""
    s = mat.spec
    if s.pad_c:
        pad = mat.c_full[..., s.n:].float()
        assert torch.isnan(pad).all().item(), f"{label} {s.name}: wrote into C padding"
    if mat.c_guard is not None:
        assert torch.isnan(mat.c_guard.float()).all().item(), f"{label} {s.name}: wrote past C's last row"


def _item(mat, i):
    """Item i of a batched GEMM as a single-GEMM Materialized (host codes sliced)."""
    from dataclasses import replace
    s = mat.spec
    single = replace(s, batch=0, pad_item=0, name=f"{s.name}[{i}]")
    host = {}
    for w in ("a", "b"):
        r, _ = s.stored_shape(w)
        off = i * s.item_stride(w)
        host[w] = mat.host[w][off:off + r * s.ld(w)]
    # an item's guard is the next item's rows: the whole batch's guard is checked once
    return inputs.Materialized(single, mat.a[i], mat.b[i], mat.c[i], mat.c_full[i], mat.scale_a,
                               mat.scale_b, host)


def gemm_of(mat, variant=-1):
    from paper_2409_02227_amd import gdy
    return gdy.Gemm(mat.a, mat.b, mat.c, mat.spec.trans_a, mat.spec.trans_b,
                    mat.scale_a, mat.scale_b, mat.spec.tenant, variant)


def reset_outputs(mats):
    for m in mats:
        m.c_full.fill_(float("nan"))
        if m.c_guard is not None:
            m.c_guard.fill_(float("nan"))


def check_add(x, label=""):
    """An element-wise add (inputs.AddInputs) against the oracle: within half
    an output ulp of the exact sum, measured on |a| + |b|; C's padding columns
    untouched."""
    ref, bound = oracle.add(x.m, x.n, x.host["a"], ORC[x.dtype], x.ld, x.host["b"], ORC[x.dtype], x.ld)
    c = x.c.cpu().contiguous()
    codes = c.view(torch.int32).numpy().view(np.uint32) if c.dtype == torch.float32 else \
        c.view(torch.int16).numpy().view(np.uint16)
    got = oracle.decode(codes, ORC[x.dtype])
    ok, worst = oracle.accept(got, ref, bound, TAU_ADD[x.dtype], abs_term=1e-30)
    assert ok, f"{label} add ({x.m},{x.n},{x.dtype}): outside bound, worst ratio {worst:.3g}"
    if x.ld > x.n:
        assert torch.isnan(x.c_full[:, x.n:].float()).all().item(), f"{label}: wrote into C padding"
    if x.c_guard is not None:
        assert torch.isnan(x.c_guard.float()).all().item(), f"{label}: wrote past C's last row"
    return worst
