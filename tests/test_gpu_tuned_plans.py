"""GPU parity of the plans the tuned MI355X table gives: heterogeneous
submissions, the attention B-GEMMs and the fp8 tenants under the selector
(with its grouping, shared group kernels, uncapped mixed groups and group
splits).  Each plan must equal the oracle planner's for the same
descriptors, and the outputs meet the oracle's bound on sampled entries."""
import os

import pytest

import paper_2409_02227_amd  # noqa: F401  (sets GPU_MAX_HW_QUEUES before HIP starts)

torch = pytest.importorskip("torch")

from oracle import selector as sel  # noqa: E402
from paper_2409_02227_amd import gdy, inputs  # noqa: E402
from tests.gpu_helpers import check, gemm_of, reset_outputs  # noqa: E402

pytestmark = pytest.mark.gpu
TABLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                     "paper_2409_02227_amd", "tables", "gfx950.table")


@pytest.fixture(scope="module")
def tctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if not os.path.exists(TABLE):
        pytest.skip("no tuned table")
    c = gdy.Context(0, table=TABLE, max_streams=16)
    yield c
    c.close()


def _as_dict(d):
    return {"m": d.m, "n": d.n, "k": d.k, "a_type": d.a_type, "trans_a": d.trans_a,
            "trans_b": d.trans_b, "a": d.a, "b": d.b, "lda": d.lda, "ldb": d.ldb,
            "batch": d.batch, "stride_a": d.stride_a, "stride_b": d.stride_b, "op": d.op}


def _run_and_compare(ctx, mats, label, samples=3):
    reset_outputs(mats)
    gemms = [gemm_of(m) for m in mats]
    plan = ctx.execute(gemms, mode="selector", want_plan=True)
    torch.cuda.synchronize()
    want = sel.plan_selector([_as_dict(g.desc()) for g in gemms], sel.parse_table(TABLE), ctx.variants(),
                             ctx.cus(), 16)
    n = len(mats)
    assert [plan["variant_of"][i] for i in range(n)] == [want["variant_of"][i] for i in range(n)], label
    assert [plan["split_of"][i] for i in range(n)] == [want["split_of"][i] for i in range(n)], label
    for m in mats:
        check(m, samples=samples, label=label)
    return plan


def test_heterogeneous_submissions_selector(tctx):
    plans = []
    for s, sub in enumerate(inputs.config4(count=6)):
        mats = [inputs.materialize(sp) for sp in sub]
        plans.append(_run_and_compare(tctx, mats, f"submission {s}"))
        del mats
    V = tctx.variants()
    # the rules these plans exercise
    assert any(p["n_dispatches"] == 1 and len(p["group_size"]) >= 1 and max(p["group_size"]) > 2 for p in plans)
    assert any(V[v]["grid_cap_cus"] == 0 for p in plans for v in p["variant_of"] if v >= 0)


def test_attention_bgemms_selector(tctx):
    mats = [inputs.materialize(sp) for sp in inputs.config_attn()]
    plan = _run_and_compare(tctx, mats, "attention", samples=4)
    assert plan["n_dispatches"] == 1  # a short group on one kernel


def test_fp8_tenants_selector(tctx):
    mats = [inputs.materialize(sp) for sp in inputs.config5()]
    _run_and_compare(tctx, mats, "fp8 tenants", samples=2)


def test_split_within_a_group(tctx):
    """A group of skinny long-K GEMMs next to short ones: the plan splits the
    long ones only, and every output meets the bound."""
    from paper_2409_02227_amd.inputs import GemmSpec
    specs = [GemmSpec(16, 2048, 8192, "bf16", seed=9300, name="long0"),
             GemmSpec(32, 1024, 8192, "bf16", seed=9301, name="long1"),
             GemmSpec(64, 2048, 1024, "bf16", seed=9302, name="short0"),
             GemmSpec(48, 1024, 1024, "bf16", seed=9303, name="short1")]
    mats = [inputs.materialize(sp) for sp in specs]
    plan = _run_and_compare(tctx, mats, "split in group", samples=6)
    assert plan["split_of"][0] > 1 and plan["split_of"][2] == 1 and plan["split_of"][3] == 1, plan["split_of"]
