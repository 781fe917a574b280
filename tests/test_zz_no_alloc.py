"""gdy_execute_static (the entry point that allocates nothing: split-K planes
in the library's static device array) against gdy_execute, through the
C-ABI: the same plans and bit-identical outputs, both within the oracle's
bound, on two calls in a row (the second smaller), and a clear refusal of a
plan that needs more than the array holds; and the entry point captured in a
HIP graph (torch.cuda.CUDAGraph on a side stream), every replay bit-identical
to the eager call, with eager work and synchronisations between replays."""
import os

import numpy as np
import pytest

import paper_2409_02227_amd  # noqa: F401  (sets GPU_MAX_HW_QUEUES before HIP starts)

torch = pytest.importorskip("torch")

from paper_2409_02227_amd import gdy, inputs  # noqa: E402
from paper_2409_02227_amd.inputs import GemmSpec  # noqa: E402
from tests.gpu_helpers import check, gemm_of, out_codes, reset_outputs  # noqa: E402

pytestmark = pytest.mark.gpu
TABLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                     "paper_2409_02227_amd", "tables", "gfx950.table")


@pytest.fixture(scope="module")
def sctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = gdy.Context(0, table=TABLE if os.path.exists(TABLE) else None, max_streams=16)
    yield c
    c.close()


def _both(ctx, mats, mode, forced_cd=0, variants=None):
    gemms = [gemm_of(m, -1 if variants is None else variants[i]) for i, m in enumerate(mats)]
    reset_outputs(mats)
    p_ref = ctx.execute(gemms, mode=mode, forced_cd=forced_cd, want_plan=True)
    torch.cuda.synchronize()
    ref = [out_codes(m).copy() for m in mats]
    reset_outputs(mats)
    p_st = ctx.execute_static(gemms, mode=mode, forced_cd=forced_cd, want_plan=True)
    torch.cuda.synchronize()
    assert p_st == p_ref
    for m, r in zip(mats, ref):
        assert np.array_equal(out_codes(m), r), m.spec.name
        check(m, samples=4, label=f"static {mode}")
    return p_st


def test_static_entry_matches_execute_on_two_calls(sctx):
    big = [GemmSpec(16, 1024, 8192, "bf16", seed=9700, name="s0"),
           GemmSpec(32, 2048, 8192, "bf16", seed=9701, name="s1"),
           GemmSpec(64, 1024, 4096, "bf16", seed=9702, name="s2"),
           GemmSpec(512, 1024, 1024, "bf16", seed=9703, name="s3"),
           GemmSpec(20, 100, 3000, "bf16", seed=9704, batch=5, name="s4")]
    small = [GemmSpec(16, 512, 4096, "bf16", seed=9710, name="t0"),
             GemmSpec(8, 256, 2048, "f16", seed=9711, name="t1")]
    for mode in ("selector", "sequential", "default", "go"):
        mats = [inputs.materialize(s) for s in big]
        p = _both(sctx, mats, mode)
        assert any(s > 1 for s in p["split_of"][:len(big)]), (mode, p["split_of"])
        mats = [inputs.materialize(s) for s in small]
        p = _both(sctx, mats, mode)
        assert any(s > 1 for s in p["split_of"][:len(small)]), (mode, p["split_of"])


def test_static_entry_refuses_a_plan_beyond_the_array(sctx):
    # (128, 8192, 4096) on 128 x 128 tiles splits 4 ways into 16 MiB of planes;
    # five in one group need 80 MiB at once, more than the 64 MiB array
    vid = sctx.find("bf16_nn_128x128_w2x2_d2_c0")
    a = torch.zeros(128, 4096, dtype=torch.bfloat16, device="cuda")
    b = torch.zeros(4096, 8192, dtype=torch.bfloat16, device="cuda")
    cs = [torch.zeros(128, 8192, dtype=torch.bfloat16, device="cuda") for _ in range(5)]
    gemms = [gdy.Gemm(a, b, c, variant=vid) for c in cs]
    with pytest.raises(gdy.GdyError) as e:
        sctx.execute_static(gemms, mode="forced_grouped", forced_cd=5)
    assert e.value.status == 2 and "static array" in str(e.value)
    # four fit (64 MiB), and one group after the other reuses the array
    p = sctx.execute_static(gemms[:4], mode="forced_grouped", forced_cd=4, want_plan=True)
    torch.cuda.synchronize()
    assert p["split_of"][:4] == [4] * 4
    p = sctx.execute_static(gemms, mode="forced_grouped", forced_cd=2, want_plan=True)
    torch.cuda.synchronize()
    assert p["n_groups"] == 3 and all(torch.count_nonzero(c).item() == 0 for c in cs)


@pytest.mark.parametrize("mode", ["selector", "default"])
def test_static_entry_in_a_captured_graph(sctx, mode):
    specs = [GemmSpec(16, 1024, 8192, "bf16", seed=9800, name="g0"),    # splits
             GemmSpec(32, 2048, 8192, "bf16", seed=9801, name="g1"),    # splits
             GemmSpec(512, 1024, 1024, "bf16", seed=9802, name="g2"),
             GemmSpec(1024, 4096, 4096, "bf16", seed=9803, name="g3")]  # another kernel
    mats = [inputs.materialize(s) for s in specs]
    gemms = [gemm_of(m) for m in mats]
    reset_outputs(mats)
    plan = sctx.execute_static(gemms, mode=mode, want_plan=True)
    torch.cuda.synchronize()
    print(f"{mode}: {plan['n_groups']} groups, {plan['n_dispatches']} dispatches, splits {plan['split_of'][:4]}",
          flush=True)
    assert any(s > 1 for s in plan["split_of"][:4])
    ref = [out_codes(m).copy() for m in mats]
    for m in mats:
        check(m, samples=4, label=f"eager {mode}")
    side = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    reset_outputs(mats)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=side):
        sctx.execute_static(gemms, mode=mode, stream=side)
    torch.cuda.synchronize()
    other = inputs.materialize(GemmSpec(256, 256, 256, "bf16", seed=9810, name="eager"))
    for rep in range(3):
        reset_outputs(mats)              # a fill kernel per buffer, eager
        sctx.execute([gemm_of(other)], mode="sequential")  # eager library work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for m, r in zip(mats, ref):
            assert np.array_equal(out_codes(m), r), f"replay {rep}: {m.spec.name} differs from the eager call"
    check(other, label="eager between replays")
    del graph
    torch.cuda.synchronize()
