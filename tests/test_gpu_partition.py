"""GPU parity of the CU-Partition modes (Sec. 5.5, Sec. 6.9): GEMMs on
streams with disjoint CU masks, under each kernel choice and partition
count, against the CPU oracle and bit for bit against the same variant run
alone (a CU mask changes where a tile runs, never its sum)."""
import os

import numpy as np
import pytest

import paper_2409_02227_amd  # noqa: F401  (sets GPU_MAX_HW_QUEUES before HIP starts)

torch = pytest.importorskip("torch")

from paper_2409_02227_amd import gdy, inputs  # noqa: E402
from paper_2409_02227_amd.inputs import GemmSpec  # noqa: E402
from tests.gpu_helpers import check, check_add, gemm_of, out_codes, reset_outputs  # noqa: E402

pytestmark = pytest.mark.gpu
TABLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                     "paper_2409_02227_amd", "tables", "gfx950.table")


@pytest.fixture(scope="module")
def pctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = gdy.Context(0, table=TABLE if os.path.exists(TABLE) else None, max_streams=2,
                    use_cu_masks=gdy.PARTITION_STREAMS)
    yield c
    c.close()


def test_partition_modes_parity(pctx):
    specs = [GemmSpec(512, 1024, 768, "bf16", seed=9000, name="p-bf16"),
             GemmSpec(300, 520, 333, "f16", seed=9001, pad_a=3, name="p-f16-ragged"),
             GemmSpec(256, 512, 640, "fp8", seed=9002, name="p-fp8"),
             GemmSpec(192, 256, 130, "f32", seed=9003, name="p-f32"),
             GemmSpec(128, 128, 64, "bf16", 0, 1, seed=9004, batch=6, name="p-bgemm"),
             GemmSpec(640, 256, 1024, "bf16", 1, 0, seed=9005, name="p-tn")]
    mats = [inputs.materialize(s) for s in specs]
    x = inputs.materialize_add(200, 700, "bf16", seed=9006, pad=2)
    for mode in ("cu_partition", "cu_partition_go", "cu_partition_rc"):
        for P in (2, 4, 8):
            label = f"{mode} P={P}"
            print(label, flush=True)
            reset_outputs(mats)
            x.c_full.fill_(float("nan"))
            members = [gemm_of(m) for m in mats] + [gdy.Add(x.a, x.b, x.c)]
            plan = pctx.execute(members, mode=mode, forced_cd=P, want_plan=True)
            torch.cuda.synchronize()
            assert plan["cd"] == P and plan["n_dispatches"] == len(members), label
            assert [plan["stream_of"][i] for i in range(len(members))] == [t % P for t in range(len(members))]
            codes = []
            for m in mats:
                check(m, label=label)
                codes.append(out_codes(m).copy())
            check_add(x, label=label)
            # the same variant alone on the whole GPU gives the same bits
            for i, m in enumerate(mats):
                reset_outputs([m])
                pctx.execute([gemm_of(m, plan["variant_of"][i])], mode="forced", forced_cd=1)
                torch.cuda.synchronize()
                assert np.array_equal(out_codes(m), codes[i]), f"{label}: {m.spec.name} differs alone"


def test_partition_mode_needs_partition_streams(pctx):
    plain = gdy.Context(0, max_streams=2)
    m = inputs.materialize(GemmSpec(64, 64, 64, "bf16", seed=9100, name="np"))
    try:
        with pytest.raises(gdy.GdyError) as e:
            plain.execute([gemm_of(m)], mode="cu_partition", forced_cd=2)
        assert e.value.status == 2
        # planning needs no streams
        assert plain.plan([gemm_of(m)], mode="cu_partition", forced_cd=2)["cd"] == 2
    finally:
        plain.close()
