"""GPU parity of the plans the tuned MI355X table gives: heterogeneous
submissions, the attention B-GEMMs and the fp8 tenants under the selector
(with its grouping, shared group kernels, uncapped mixed groups and split
GEMMs).  Every output meets the oracle's bound, and every GEMM's bits equal
those of the same GEMM run alone on the variant the plan bound it to: a
variant gives the same bits concurrent and isolated."""
import os

import numpy as np
import pytest

import paper_2409_02227_amd  # noqa: F401  (sets GPU_MAX_HW_QUEUES before HIP starts)

torch = pytest.importorskip("torch")

from paper_2409_02227_amd import gdy, inputs  # noqa: E402
from tests.gpu_helpers import check, gemm_of, out_codes, reset_outputs  # noqa: E402

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


def run_and_check(ctx, mats, label, samples=3, mode="selector"):
    """Run the submission in `mode`, check every output against the oracle,
    then run each GEMM alone on its bound variant (FORCED) and compare bits."""
    reset_outputs(mats)
    gemms = [gemm_of(m) for m in mats]
    plan = ctx.execute(gemms, mode=mode, want_plan=True)
    torch.cuda.synchronize()
    got = [out_codes(m).copy() for m in mats]
    for m in mats:
        check(m, samples=samples, label=label)
    for i, m in enumerate(mats):
        reset_outputs([m])
        alone = ctx.execute([gemm_of(m, plan["variant_of"][i])], mode="forced", want_plan=True)
        torch.cuda.synchronize()
        assert alone["variant_of"][0] == plan["variant_of"][i] and alone["split_of"][0] == plan["split_of"][i]
        assert np.array_equal(out_codes(m), got[i]), f"{label}: gemm {i} bits differ alone"
    return plan


def test_heterogeneous_submissions_selector(tctx):
    plans = []
    for s, sub in enumerate(inputs.het_submissions(count=6)):
        mats = [inputs.materialize(sp) for sp in sub]
        plans.append(run_and_check(tctx, mats, f"submission {s}"))
        del mats
    V = tctx.variants()
    # the rules these plans exercise
    assert any(p["n_dispatches"] == 1 and max(p["group_size"]) > 2 for p in plans)
    assert any(V[v]["grid_cap_cus"] == 0 for p in plans for v in p["variant_of"] if v >= 0)


def test_attention_bgemms_selector(tctx):
    mats = [inputs.materialize(sp) for sp in inputs.attention_bgemms()]
    plan = run_and_check(tctx, mats, "attention", samples=4)
    assert plan["n_dispatches"] == 1  # a short group on one kernel


def test_fp8_tenants_selector(tctx):
    mats = [inputs.materialize(sp) for sp in inputs.fp8_tenants()]
    run_and_check(tctx, mats, "fp8 tenants", samples=2)


def test_split_within_a_group(tctx):
    """A group of skinny long-K GEMMs next to short ones: the long ones split
    (as they would alone), the short ones do not, and every output meets the
    bound with the same bits as alone."""
    from paper_2409_02227_amd.inputs import GemmSpec
    specs = [GemmSpec(16, 2048, 8192, "bf16", seed=9300, name="long0"),
             GemmSpec(32, 1024, 8192, "bf16", seed=9301, name="long1"),
             GemmSpec(64, 2048, 1024, "bf16", seed=9302, name="short0"),
             GemmSpec(48, 1024, 1024, "bf16", seed=9303, name="short1")]
    mats = [inputs.materialize(sp) for sp in specs]
    for mode in ("selector", "go", "default"):
        plan = run_and_check(tctx, mats, f"split in group ({mode})", samples=6, mode=mode)
        assert plan["split_of"][0] > 1 and plan["split_of"][1] > 1, plan["split_of"]
        assert plan["split_of"][2] == 1 and plan["split_of"][3] == 1, plan["split_of"]


def test_deferred_split_group(tctx):
    """Seventeen split GEMMs of 16 MiB of planes each in one group overflow
    the 256 MiB workspace: (128, 8192, 4096) on 128 x 128 tiles has 64 tiles
    and 64 K tiles, so it splits 4 ways into 4 MiB planes.  The seventeenth
    runs in a later group with its own split, so its bits still match the
    GEMM alone."""
    from paper_2409_02227_amd.inputs import GemmSpec
    vid = tctx.find("bf16_nn_128x128_w2x2_d2_c0")
    mats = [inputs.materialize(GemmSpec(128, 8192, 4096, "bf16", seed=9400 + j, name=f"d{j}"))
            for j in range(17)]
    reset_outputs(mats)
    gemms = [gemm_of(m, vid) for m in mats]
    plan = tctx.execute(gemms, mode="forced_grouped", forced_cd=17, want_plan=True)
    torch.cuda.synchronize()
    assert plan["n_groups"] == 2 and plan["group_size"] == [16, 1] and plan["split_of"] == [4] * 17
    got = [out_codes(m).copy() for m in mats]
    for j in (0, 15, 16):
        check(mats[j], samples=4, label=f"deferred {j}")
        reset_outputs([mats[j]])
        tctx.execute([gemms[j]], mode="forced")
        torch.cuda.synchronize()
        assert np.array_equal(out_codes(mats[j]), got[j]), j
