"""The sampled-check helper of the GPU parity tests (CPU only): the oracle's
full GEMM over the stored rows and columns a set of outputs reads gives, for
every layout and input type, exactly what the oracle's per-entry routine
gives for those outputs (same k-ascending sums, same bounds)."""
import numpy as np
import pytest

import oracle
from paper_2409_02227_amd import inputs

pytest.importorskip("torch")
from tests.gpu_helpers import ORC, accept_rows_cols, rows_cols_ref  # noqa: E402


@pytest.mark.parametrize("dt", ["bf16", "f16", "fp8", "f32"])
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_rows_cols_equal_per_entry_oracle(dt, ta, tb):
    spec = inputs.GemmSpec(37, 45, 29, dt, ta, tb, seed=77, pad_a=3, pad_b=5)
    a, sa = inputs.operand_codes(spec, "a")
    b, sb = inputs.operand_codes(spec, "b")
    rng = np.random.default_rng(3)
    rows = np.sort(rng.choice(spec.m, 5, replace=False))
    cols = np.sort(rng.choice(spec.n, 4, replace=False))
    ref_r, bd_r, ref_c, bd_c = rows_cols_ref(spec.m, spec.n, spec.k, a, ORC[dt], spec.ld("a"), b, ORC[dt],
                                             spec.ld("b"), rows, cols, ta, tb, sa, sb)
    ii = np.repeat(rows, spec.n)
    jj = np.tile(np.arange(spec.n), len(rows))
    e_ref, e_bd = oracle.gemm_entries(spec.m, spec.n, spec.k, a, ORC[dt], spec.ld("a"), b, ORC[dt], spec.ld("b"),
                                      ii, jj, ta, tb, sa, sb)
    assert np.array_equal(ref_r.reshape(-1), e_ref) and np.array_equal(bd_r.reshape(-1), e_bd)
    ii = np.tile(np.arange(spec.m), len(cols))
    jj = np.repeat(cols, spec.m)
    e_ref, e_bd = oracle.gemm_entries(spec.m, spec.n, spec.k, a, ORC[dt], spec.ld("a"), b, ORC[dt], spec.ld("b"),
                                      ii, jj, ta, tb, sa, sb)
    assert np.array_equal(ref_c.T.reshape(-1), e_ref) and np.array_equal(bd_c.T.reshape(-1), e_bd)


def test_accept_rows_cols_catches_one_wrong_element():
    spec = inputs.GemmSpec(40, 33, 21, "bf16", seed=5)
    a, _ = inputs.operand_codes(spec, "a")
    b, _ = inputs.operand_codes(spec, "b")
    full, _ = oracle.gemm(spec.m, spec.n, spec.k, a, "bf16", spec.ld("a"), b, "bf16", spec.ld("b"))
    rows, cols = np.array([0, 17, 39]), np.array([2, 32])
    args = (spec.m, spec.n, spec.k, a, "bf16", spec.ld("a"), b, "bf16", spec.ld("b"), rows, cols, 2.0 ** -7)
    assert accept_rows_cols(full[rows], full[:, cols], *args)[0]
    bad = full.copy()
    bad[39, 32] += 0.5
    assert not accept_rows_cols(bad[rows], bad[:, cols], *args)[0]
