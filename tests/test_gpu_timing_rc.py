"""GPU tests of the resource constraint and the per-kernel timing calls.

gdy_set_rc (Sec. 4.2.1's RC tuning) moves the launches that go to pool
streams onto streams whose CU mask leaves 128, 64 or 32 CUs, as the tuner's
isolated runs do (GDY_FORCED, forced_cd 1): the same kernel then computes
the same bits, and a GEMM that fills the GPU takes longer on an eighth of
it.  The origin stream (GDY_SEQUENTIAL) is never masked.
gdy_last_kernel_times and gdy_kernel_times (Sec. 5.3's per-kernel runtimes)
report, for each GEMM of a timed submission, its dispatch's interval from the
submission's start; a GEMM that launched nothing reports -1."""
import ctypes
import os
import time

import numpy as np
import pytest

import paper_2409_02227_amd  # noqa: F401  (sets GPU_MAX_HW_QUEUES before HIP starts)

torch = pytest.importorskip("torch")

from paper_2409_02227_amd import gdy  # noqa: E402

pytestmark = pytest.mark.gpu
TABLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                     "paper_2409_02227_amd", "tables", "gfx950.table")


@pytest.fixture(scope="module")
def rctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = gdy.Context(0, table=TABLE if os.path.exists(TABLE) else None, max_streams=4,
                    use_cu_masks=gdy.RC_STREAMS)
    yield c
    c.set_rc(0)
    c.close()


def _operands(m, n, k, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    a = (torch.rand(m, k, device="cuda", generator=g) * 2 - 1).to(torch.bfloat16)
    b = (torch.randn(k, n, device="cuda", generator=g) * 0.05).to(torch.bfloat16)
    return a, b


def _wall(ctx, gemms, mode, reps=10, forced_cd=0):
    for _ in range(2):
        ctx.execute(gemms, mode=mode, forced_cd=forced_cd)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        ctx.execute(gemms, mode=mode, forced_cd=forced_cd)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / reps


def test_rc_pools_compute_the_same_bits_on_fewer_cus(rctx):
    a, b = _operands(4096, 4096, 4096, 41)
    out = {}
    times = {}
    vid = rctx.find("bf16_nn_256x256_w2x4_d2_c0")
    assert vid >= 0
    for rc in (0, 128, 64, 32):
        c = torch.full((4096, 4096), float("nan"), dtype=torch.bfloat16, device="cuda")
        rctx.set_rc(rc)
        gemm = [gdy.Gemm(a, b, c, variant=vid)]
        plan = rctx.execute(gemm, mode="forced", forced_cd=1, want_plan=True)
        torch.cuda.synchronize()
        assert plan["stream_of"][0] == 0  # a pool stream
        out[rc] = c
        times[rc] = _wall(rctx, gemm, "forced", forced_cd=1)
        print(f"rc {rc}: {times[rc] * 1e6:.0f} us", flush=True)
    # the origin stream is not masked: the sequential mode under rc 32 runs at full speed
    seq = _wall(rctx, [gdy.Gemm(a, b, out[0], variant=vid)], "sequential")
    rctx.set_rc(0)
    for rc in (128, 64, 32):
        assert torch.equal(out[rc].view(torch.int16), out[0].view(torch.int16)), f"rc {rc} changed bits"
    assert not torch.isnan(out[0].float()).any()
    # a GEMM of 256 tiles on an eighth of the CUs takes several times longer
    assert times[32] > 2.0 * times[0], times
    assert times[64] > 1.5 * times[0] and times[128] > 1.2 * times[0], times
    assert seq < 0.5 * times[32], (seq, times)


def test_rc_rejects_other_budgets(rctx):
    for bad in (1, 100, 256, -32):
        with pytest.raises(gdy.GdyError):
            rctx.set_rc(bad)
    rctx.set_rc(0)


def test_last_kernel_times_match_the_timing_ring(rctx):
    lib = rctx.lib
    n = 4
    f4 = ctypes.c_float * n
    fresh = gdy.Context(0, max_streams=2)
    try:  # a context without a timed submission has nothing to report
        assert lib.gdy_last_kernel_times(fresh.h, f4(), f4(), n) == 1
    finally:
        fresh.close()
    shapes = [(512, 1024, 2048), (0, 256, 256), (300, 700, 900), (64, 4096, 1024)]
    gemms = []
    for i, (m, nn, k) in enumerate(shapes):
        a, b = _operands(max(m, 1), nn, k, 50 + i)
        a = a[:m]
        gemms.append(gdy.Gemm(a, b, torch.empty(m, nn, dtype=torch.bfloat16, device="cuda")))
    rctx.set_timing(True)
    try:
        for mode in ("sequential", "selector"):
            plan = rctx.execute(gemms, mode=mode, want_plan=True)
            torch.cuda.synchronize()
            s, e = f4(), f4()
            assert lib.gdy_last_kernel_times(rctx.h, s, e, n) == 0
            s, e = np.array(s[:]), np.array(e[:])
            s2, e2 = rctx.kernel_times(n, 0)
            assert np.array_equal(s, np.array(s2, dtype=np.float32)) and np.array_equal(e, np.array(e2, dtype=np.float32))
            print(mode, [f"{x:.3f}-{y:.3f}" for x, y in zip(s, e)], flush=True)
            assert s[1] == -1 and e[1] == -1  # M = 0 launches nothing
            for i in (0, 2, 3):
                assert 0 <= s[i] < e[i] < 50, (mode, i, s[i], e[i])
            # GEMMs that share a dispatch report the same interval
            for i in (0, 2, 3):
                for j in (0, 2, 3):
                    if plan["dispatch_of"][i] == plan["dispatch_of"][j]:
                        assert s[i] == s[j] and e[i] == e[j]
            if mode == "sequential":  # one after another on the origin stream
                order = [i for i in plan["order"][:3]]
                for x, y in zip(order, order[1:]):
                    assert e[x] <= s[y] + 1e-3, (x, y, e[x], s[y])
        assert lib.gdy_last_kernel_times(rctx.h, None, f4(), n) == 1  # NULL pointer
    finally:
        rctx.set_timing(False)
