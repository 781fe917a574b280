"""GPU parity of the workloads at their full sizes, in the configurations
bench.py times, against the CPU oracle (|c - ref| <= tau * sum|a b| + 1e-6,
tau = 2^-7 for bf16, 2^-3 for fp8):

  * the tensor-sliced layer share (eight bf16 GEMMs, 463.9 GFLOP): every
    element, in sequential, default, GO and selector mode, and bit-identical
    across the modes that bind the same kernel;
  * the two fp8 tenants under the selector and GO: every element of the
    GEMMs with M <= 256, 16 full rows and 16 full columns of the M = 2048 ones;
  * all 200 heterogeneous submissions the bench times (its device operand
    pools and windows) under the selector: 16 full rows and 16 full columns
    of every GEMM, every element of GEMMs with M <= 32.

Sampled rows and columns are checked against the oracle's full GEMM over the
stored rows of A and columns of B they read (tests.gpu_helpers.rows_cols_ref).
"""
import os

import numpy as np
import pytest

import paper_2409_02227_amd  # noqa: F401  (sets GPU_MAX_HW_QUEUES before HIP starts)

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from paper_2409_02227_amd import gdy, inputs  # noqa: E402
from tests.gpu_helpers import (ORC, TAU, accept_rows_cols, assert_untouched, decode_out, gemm_of,  # noqa: E402
                               out_codes, reset_outputs)

pytestmark = pytest.mark.gpu
TABLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                     "paper_2409_02227_amd", "tables", "gfx950.table")


@pytest.fixture(scope="module")
def wctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = gdy.Context(0, table=TABLE if os.path.exists(TABLE) else None, max_streams=16)
    yield c
    c.close()


def _full_ref(mat):
    s = mat.spec
    return oracle.gemm(s.m, s.n, s.k, mat.host["a"], ORC[s.dtype], s.ld("a"), mat.host["b"], ORC[s.dtype],
                       s.ld("b"), s.trans_a, s.trans_b, mat.scale_a, mat.scale_b)


def _sample(m, n, rows, cols, rng):
    """`rows` full rows (all when m <= 32) and `cols` full columns to check."""
    r = np.arange(m) if m <= 32 else rng.choice(m, size=min(rows, m), replace=False)
    c = rng.choice(n, size=min(cols, n), replace=False)
    return r, c


def test_layer_share_every_element_every_mode(wctx):
    mats = [inputs.materialize(s) for s in inputs.layer_share()]
    refs = [_full_ref(m) for m in mats]
    bits = {}
    for mode in ("sequential", "default", "go", "selector"):
        reset_outputs(mats)
        plan = wctx.execute([gemm_of(m) for m in mats], mode=mode, want_plan=True)
        torch.cuda.synchronize()
        for i, (m, (ref, bound)) in enumerate(zip(mats, refs)):
            ok, worst = oracle.accept(decode_out(m), ref, bound, TAU["bf16"])
            assert ok, f"{mode} {m.spec.name}: worst ratio {worst:.3g}"
            assert_untouched(m, mode)
            key = (i, wctx.variant(plan["variant_of"][i])["name"].rsplit("_c", 1)[0])
            codes = out_codes(m)
            if key in bits:
                assert np.array_equal(bits[key], codes), f"{mode} {m.spec.name}: bits differ"
            bits[key] = codes.copy()
        print(f"layer share {mode}: every element within the bound", flush=True)


@pytest.mark.parametrize("mode", ["selector", "go"])
def test_fp8_tenants(wctx, mode):
    mats = [inputs.materialize(s) for s in inputs.fp8_tenants()]
    reset_outputs(mats)
    wctx.execute([gemm_of(m) for m in mats], mode=mode)
    torch.cuda.synchronize()
    rng = np.random.default_rng(55)
    for m in mats:
        s = m.spec
        got = decode_out(m)
        if s.m <= 256:
            ref, bound = _full_ref(m)
            ok, worst = oracle.accept(got, ref, bound, TAU["fp8"])
        else:
            rows, cols = _sample(s.m, s.n, 16, 16, rng)
            ok, worst = accept_rows_cols(got[rows], got[:, cols], s.m, s.n, s.k, m.host["a"], "e4m3fn",
                                         s.ld("a"), m.host["b"], "e4m3fn", s.ld("b"), rows, cols, TAU["fp8"],
                                         s.trans_a, s.trans_b, m.scale_a, m.scale_b)
        assert ok, f"{mode} {s.name} ({s.m},{s.n},{s.k}): worst ratio {worst:.3g}"
        assert_untouched(m, mode)


@pytest.fixture(scope="module")
def het_pools(wctx):
    a, b = inputs.het_pools(torch)
    a_host = a.view(torch.int16).cpu().numpy().view(np.uint16)
    b_host = b.view(torch.int16).cpu().numpy().view(np.uint16)
    return a, b, a_host, b_host, inputs.het_placed(200)


@pytest.mark.parametrize("chunk", range(10))
def test_heterogeneous_submissions_all_200(wctx, het_pools, chunk):
    a_pool, b_pool, a_host, b_host, placed = het_pools
    rng = np.random.default_rng(400 + chunk)
    for s_idx in range(20 * chunk, 20 * chunk + 20):
        gemms, outs, guards = [], [], []
        for g, oa, ob in placed[s_idx]:
            a = a_pool[oa:oa + g.m * g.k].view(g.m, g.k)
            b = b_pool[ob:ob + g.k * g.n].view(g.k, g.n)
            buf = torch.full(((g.m + inputs.GUARD_ROWS) * g.n,), float("nan"), dtype=torch.bfloat16, device="cuda")
            c = buf[:g.m * g.n].view(g.m, g.n)
            gemms.append(gdy.Gemm(a, b, c))
            outs.append(c)
            guards.append(buf[g.m * g.n:])
        wctx.execute(gemms, mode="selector")
        torch.cuda.synchronize()
        for (g, oa, ob), c in zip(placed[s_idx], outs):
            rows, cols = _sample(g.m, g.n, 16, 16, rng)
            # only the checked rows and columns come back to the host
            c16 = c.view(torch.int16)
            got_r = oracle.decode(c16[torch.from_numpy(rows).cuda()].cpu().numpy().view(np.uint16), "bf16")
            got_c = oracle.decode(c16[:, torch.from_numpy(cols).cuda()].cpu().numpy().view(np.uint16), "bf16")
            ok, worst = accept_rows_cols(got_r, got_c, g.m, g.n, g.k, a_host[oa:oa + g.m * g.k], "bf16", g.k,
                                         b_host[ob:ob + g.k * g.n], "bf16", g.n, rows, cols, TAU["bf16"])
            assert ok, f"submission {s_idx} ({g.m},{g.n},{g.k}): worst ratio {worst:.3g}"
        assert all(torch.isnan(gd.float()).all().item() for gd in guards), f"submission {s_idx}: wrote past C"
    print(f"submissions {20 * chunk}-{20 * chunk + 19}: sampled rows and columns within the bound", flush=True)
