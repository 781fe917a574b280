"""GPU parity: every GO-Kernel and every execution mode against the CPU
oracle, through the C-ABI (libgdy.so via the ctypes binding).

Bar: |gpu - ref| <= tau * sum_k |a(i,k) b(k,j)| + 1e-6 with tau = 2^-7 for
bf16/fp16 inputs and 2^-3 for fp8 (the stated contract) and 2^-10 for fp32
(derived from K * 2^-24 at K <= 16384); results of one variant are
bit-identical between isolated and concurrent execution.
"""
import itertools
import os

import numpy as np
import pytest

import paper_2409_02227_amd  # noqa: F401  (sets GPU_MAX_HW_QUEUES before HIP starts)

torch = pytest.importorskip("torch")

from paper_2409_02227_amd import gdy, inputs  # noqa: E402
from paper_2409_02227_amd.inputs import GemmSpec  # noqa: E402
from tests.gpu_helpers import check, gemm_of, out_codes, reset_outputs  # noqa: E402

pytestmark = pytest.mark.gpu

DT_NAME = {1: "f16", 2: "bf16", 3: "fp8", 4: "f32"}


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = gdy.Context(0, max_streams=16)
    yield c
    c.close()


def _run(ctx, mats, mode, forced_cd=0, variants=None):
    reset_outputs(mats)
    gemms = [gemm_of(m, -1 if variants is None else variants[i]) for i, m in enumerate(mats)]
    plan = ctx.execute(gemms, mode=mode, forced_cd=forced_cd, want_plan=True)
    torch.cuda.synchronize()
    return plan


def _kernels(ctx):
    """Uncapped variant of every GEMM kernel in the catalogue."""
    return [(i, v) for i, v in enumerate(ctx.variants()) if v["grid_cap_cus"] == 0 and v["kind"] == 0]


def test_every_kernel_ragged_tiles(ctx):
    """Each kernel on a shape spanning several tiles with ragged M, N and K
    tails (K tail inside a 16-byte chunk too)."""
    for vid, v in _kernels(ctx):
        bm, bn, bk = v["bm"], v["bn"], v["bk"]
        dt = DT_NAME[v["dtype"]]
        spec = GemmSpec(2 * bm - 5, bn + 3, {"fp8": bk + 53, "f32": 2 * bk + 7}.get(dt, 2 * bk + 37), dt,
                        v["trans_a"], v["trans_b"], seed=vid, name=v["name"])
        mat = inputs.materialize(spec)
        _run(ctx, [mat], "forced", 1, [vid])
        check(mat, label=v["name"])


def test_every_kernel_aligned_multi_tile(ctx):
    """Each kernel on exact multiples of its tile (vector-load fast path)."""
    for vid, v in _kernels(ctx):
        dt = DT_NAME[v["dtype"]]
        spec = GemmSpec(v["bm"] * 2, v["bn"] * 2, v["bk"] * 3, dt, v["trans_a"], v["trans_b"],
                        seed=1000 + vid, name=v["name"])
        mat = inputs.materialize(spec)
        _run(ctx, [mat], "forced", 1, [vid])
        check(mat, label=v["name"])


@pytest.mark.parametrize("dt,ta,tb", [(d, a, b) for d in ("bf16", "f16", "fp8", "f32")
                                      for a, b in itertools.product([0, 1], [0, 1])])
def test_odd_leading_dims_and_tiny_shapes(ctx, dt, ta, tb):
    """ld > minimal and unaligned (element-wise load path), M = 1, K = 1,
    K below one K tile, and C padding that must stay untouched."""
    shapes = [(1, 1, 1), (1, 77, 300), (5, 3, 1), (33, 65, 17), (130, 70, 200)]
    for i, (m, n, k) in enumerate(shapes):
        spec = GemmSpec(m, n, k, dt, ta, tb, seed=50 + i, pad_a=3, pad_b=5, pad_c=7,
                        name=f"odd{i}")
        mat = inputs.materialize(spec)
        _run(ctx, [mat], "sequential")
        check(mat, label=f"{dt} t{ta}{tb}")


def test_k_zero_writes_zeros_and_empty_is_noop(ctx):
    spec = GemmSpec(40, 50, 0, "bf16", seed=1, name="k0")
    mat = inputs.materialize(spec)
    empty = inputs.materialize(GemmSpec(0, 50, 64, "bf16", seed=2, name="m0"))
    _run(ctx, [mat, empty], "default")
    assert (mat.c.float() == 0).all().item()


def test_grid_caps_are_bit_identical(ctx):
    """A grid cap changes which workgroup runs a tile, never the tile's sum."""
    spec = GemmSpec(700, 900, 650, "bf16", seed=77, name="caps")
    mat = inputs.materialize(spec)
    by_kernel = {}
    for vid, v in enumerate(ctx.variants()):
        if v["dtype"] == 2 and v["trans_a"] == 0 and v["trans_b"] == 0 and v["kind"] == 0:
            by_kernel.setdefault(v["name"].rsplit("_c", 1)[0], []).append(vid)
    for name, vids in by_kernel.items():
        ref = None
        for vid in vids:
            _run(ctx, [mat], "forced", 1, [vid])
            got = out_codes(mat).copy()
            if ref is None:
                check(mat, label=name)
                ref = got
            assert np.array_equal(got, ref), f"{name}: cap variant {vid} differs"


def test_concurrent_equals_isolated_bitwise(ctx):
    """Same variant: isolated, then 8 concurrent on 8 streams, same bits."""
    specs = [GemmSpec(300, 1000, 700, "bf16", seed=200 + i, name=f"c{i}") for i in range(8)]
    mats = [inputs.materialize(s) for s in specs]
    vid = ctx.find("bf16_nn_128x128_w2x2_m32_c0")
    assert vid >= 0
    iso = []
    for m in mats:
        _run(ctx, [m], "forced", 1, [vid])
        iso.append(out_codes(m).copy())
    for rep in range(3):
        _run(ctx, mats, "forced", 8, [vid] * 8)
        for m, ref in zip(mats, iso):
            assert np.array_equal(out_codes(m), ref), f"rep {rep} {m.spec.name} differs"
    check(mats[0])


@pytest.mark.parametrize("mode", ["sequential", "default", "go", "selector"])
def test_square_fp16_and_lstm_gates_full(ctx, mode):
    for specs in (inputs.square_fp16(), inputs.lstm_gates()):
        mats = [inputs.materialize(s) for s in specs]
        plan = _run(ctx, mats, mode)
        assert sorted(plan["order"]) == list(range(len(specs)))
        for m in mats:
            check(m, label=mode)


def test_fp8_tenants_sampled(ctx):
    mats = [inputs.materialize(s) for s in inputs.fp8_tenants()]
    for mode in ("sequential", "default"):
        _run(ctx, mats, mode)
        for m in mats:
            check(m, samples=4, label=mode)


def test_validation_errors(ctx):
    a = torch.zeros(64, 64, dtype=torch.bfloat16, device="cuda")
    b = torch.zeros(64, 64, dtype=torch.bfloat16, device="cuda")
    c = torch.zeros(64, 64, dtype=torch.bfloat16, device="cuda")
    ok = gdy.Gemm(a, b, c)
    with pytest.raises(gdy.GdyError) as e:
        ctx.execute([gdy.Gemm(a, b, a)])  # C aliases A
    assert e.value.status == 3
    with pytest.raises(gdy.GdyError) as e:
        ctx.execute([ok, gdy.Gemm(a, b, c)])  # two GEMMs write the same C
    assert e.value.status == 3
    d = ok.desc()
    d.lda = 10
    with pytest.raises(gdy.GdyError) as e:
        ctx.execute([d])
    assert e.value.status == 1
    d = ok.desc()
    d.c_type = 1
    with pytest.raises(gdy.GdyError) as e:
        ctx.execute([d])
    assert e.value.status == 2
    d = ok.desc()
    d.scale_a = 2.0
    with pytest.raises(gdy.GdyError) as e:
        ctx.execute([d])
    assert e.value.status == 1
    with pytest.raises(gdy.GdyError) as e:
        ctx.execute([ok] * 257)
    assert e.value.status == 4
    d = ok.desc()
    d.variant = 10 ** 6
    with pytest.raises(gdy.GdyError) as e:
        ctx.execute([d], mode="forced", forced_cd=1)
    assert e.value.status == 1
    # nothing was launched by the failed calls: C still zero
    torch.cuda.synchronize()
    assert (c.float() == 0).all().item()


def test_concurrent_kernels_overlap(ctx):
    """With CD > 1 the per-kernel intervals overlap (streams really run
    concurrently; needs GPU_MAX_HW_QUEUES >= the CD).  The GEMMs fill the
    CU slots by their tiles, so none is split into K runs."""
    specs = [GemmSpec(1024, 4096, 8192, "bf16", seed=300 + i, name=f"ov{i}") for i in range(4)]
    mats = [inputs.materialize(s) for s in specs]
    ctx.set_timing(True)
    try:
        best = 0.0
        for _ in range(5):
            plan = _run(ctx, mats, "default")
            assert plan["split_of"] == [1, 1, 1, 1]
            st, en = ctx.kernel_times(4)
            iv = sorted(zip(st, en))
            ov = max(0.0, min(e for _, e in iv) - max(s for s, _ in iv))
            best = max(best, ov)
        print("GPU_MAX_HW_QUEUES", os.environ.get("GPU_MAX_HW_QUEUES"), "overlap ms", best)
        assert best > 0.0, f"kernels never overlapped: {iv}"
    finally:
        ctx.set_timing(False)


def _pad_to(n, mult):
    return (-n) % mult


def test_direct_kernels_ragged_mn(ctx):
    """Each direct kernel (global->LDS copies, transpose reads) on ragged M
    and N, K a whole number of K tiles, leading dimensions padded to 16-byte
    multiples so the direct path is taken (checked in the plan)."""
    for vid, v in _kernels(ctx):
        if not v["direct"]:
            continue
        dt = DT_NAME[v["dtype"]]
        es = 1 if dt == "fp8" else 2
        m, n, k = 2 * v["bm"] - 5, v["bn"] + 3, 2 * v["bk"]
        ta, tb = v["trans_a"], v["trans_b"]
        a_cols = m if ta else k
        b_cols = k if tb else n
        spec = GemmSpec(m, n, k, dt, ta, tb, seed=4000 + vid, name=v["name"],
                        pad_a=_pad_to(a_cols, 16 // es), pad_b=_pad_to(b_cols, 16 // es), pad_c=5)
        mat = inputs.materialize(spec)
        plan = _run(ctx, [mat], "forced", 1, [vid])
        assert plan["variant_of"][0] == vid, f"{v['name']}: direct path not taken"
        check(mat, label=v["name"])


def test_direct_falls_back_when_ineligible(ctx):
    """K not a multiple of the K tile: the plan binds the staged kernel of the
    same tile, which gives a correct result."""
    vid = ctx.find("bf16_nn_128x128_w2x2_d2_c0")
    assert vid >= 0
    spec = GemmSpec(200, 300, 100, "bf16", seed=9, name="fallback")
    mat = inputs.materialize(spec)
    plan = _run(ctx, [mat], "forced", 1, [vid])
    ran = ctx.variant(plan["variant_of"][0])
    assert not ran["direct"] and (ran["bm"], ran["bn"]) == (128, 128)
    check(mat)


def _isolated_codes(ctx, mats, vids):
    out = []
    for m, vid in zip(mats, vids):
        _run(ctx, [m], "forced", 1, [vid])
        out.append(out_codes(m).copy())
    return out


def test_fused_dispatch_mixed_shapes_and_caps(ctx):
    """GEMMs of different shapes (ragged tails, K = 0, one element) and grid
    caps of one kernel share a single dispatch; each GEMM's result equals its
    isolated launch bit for bit and passes the oracle."""
    name = "bf16_nn_128x128_w2x2_m32"
    caps = [ctx.find(f"{name}_c{c}") for c in (0, 32, 128, 64)]
    assert min(caps) >= 0
    shapes = [(300, 1000, 700), (64, 4096, 1024), (5, 77, 33), (513, 129, 256), (1, 1, 1),
              (40, 50, 0), (200, 300, 100), (129, 257, 65)]
    mats = [inputs.materialize(GemmSpec(m, n, k, "bf16", seed=600 + i, name=f"f{i}"))
            for i, (m, n, k) in enumerate(shapes)]
    vids = [caps[i % 4] for i in range(len(mats))]
    iso = _isolated_codes(ctx, mats, vids)
    plan = _run(ctx, mats, "forced_grouped", 0, vids)
    assert plan["n_dispatches"] == 1 and set(plan["dispatch_of"]) == {0}
    assert all(s == -1 for s in plan["stream_of"])
    for m, ref in zip(mats, iso):
        assert np.array_equal(out_codes(m), ref), f"{m.spec.name}: fused differs from isolated"
        check(m, label="fused")


def test_fused_dispatch_direct_kernels(ctx):
    """Direct kernels (global->LDS copies) fused: 16-byte aligned operands,
    K whole K tiles, ragged M and N."""
    for dt in ("bf16", "fp8"):
        vid = ctx.find(f"{dt}_nn_128x128_w2x2_d2_c0")
        assert vid >= 0
        bk = ctx.variant(vid)["bk"]
        es = 1 if dt == "fp8" else 2
        shapes = [(300, 1000, 4 * bk), (64, 520, bk), (257, 136, 2 * bk), (128, 128, 3 * bk)]
        mats = []
        for i, (m, n, k) in enumerate(shapes):
            mats.append(inputs.materialize(GemmSpec(
                m, n, k, dt, 0, 0, seed=700 + i, name=f"fd{i}", pad_a=_pad_to(k, 16 // es),
                pad_b=_pad_to(n, 16 // es), pad_c=3)))
        vids = [vid] * len(mats)
        iso = _isolated_codes(ctx, mats, vids)
        plan = _run(ctx, mats, "forced_grouped", 0, vids)
        assert plan["n_dispatches"] == 1 and all(v == vid for v in plan["variant_of"])
        for m, ref in zip(mats, iso):
            assert np.array_equal(out_codes(m), ref), f"{dt} {m.spec.name}: fused differs"
            check(m, label=f"fused direct {dt}")


def test_fused_dispatch_chunks_and_kernel_split(ctx):
    """20 GEMMs of one kernel make two dispatches (16 + 4, the second on a
    pool stream); a group with two kernels makes one dispatch per kernel."""
    vid = ctx.find("bf16_nn_64x128_w1x4_m32_c0")
    other = ctx.find("bf16_nn_128x128_w2x2_m32_c0")
    assert vid >= 0 and other >= 0
    mats = [inputs.materialize(GemmSpec(100 + 7 * i, 200 + 3 * i, 96, "bf16", seed=800 + i,
                                        name=f"ch{i}")) for i in range(20)]
    iso = _isolated_codes(ctx, mats, [vid] * 20)
    plan = _run(ctx, mats, "forced_grouped", 0, [vid] * 20)
    assert plan["n_dispatches"] == 2
    assert plan["dispatch_of"] == [0] * 16 + [1] * 4
    assert plan["stream_of"] == [-1] * 16 + [0] * 4
    for m, ref in zip(mats, iso):
        assert np.array_equal(out_codes(m), ref), f"{m.spec.name}: chunked dispatch differs"
    check(mats[0])
    check(mats[19])
    # two kernels alternating in groups of 4: two dispatches per group
    vids = [vid if i % 2 == 0 else other for i in range(8)]
    sub = mats[:8]
    iso = _isolated_codes(ctx, sub, vids)
    plan = _run(ctx, sub, "forced_grouped", 4, vids)
    assert plan["n_groups"] == 2 and plan["n_dispatches"] == 4
    assert plan["dispatch_of"] == [0, 1, 0, 1, 2, 3, 2, 3]
    for m, ref in zip(sub, iso):
        assert np.array_equal(out_codes(m), ref), f"{m.spec.name}: split dispatch differs"
    # two GEMMs on two kernels: the second dispatch forks to a pool stream
    big = [inputs.materialize(GemmSpec(4096, 4096, 1024, "bf16", seed=900 + i, name=f"big{i}"))
           for i in range(2)]
    vids = [vid, other]
    iso = _isolated_codes(ctx, big, vids)
    plan = _run(ctx, big, "forced_grouped", 0, vids)
    assert plan["dispatch_of"] == [0, 1] and plan["stream_of"] == [-1, 0]
    for m, ref in zip(big, iso):
        assert np.array_equal(out_codes(m), ref), f"{m.spec.name}: forked dispatch differs"
        check(m, samples=4, label="forked")


@pytest.mark.parametrize("dt", ["fp8", "f16"])
def test_subnormal_inputs(ctx, dt):
    """A holds only positive subnormal codes, B positive normal codes: every
    product comes from a subnormal input and ref equals the bound, so a
    kernel that flushed subnormal inputs to zero would fail the bound.  Every
    uncapped kernel of the dtype and layout (staged and direct)."""
    m, n, k = 96, 160, 256
    rng = np.random.default_rng(11)
    if dt == "fp8":
        a_codes = rng.integers(0x01, 0x08, size=m * k).astype(np.uint8)   # (j/8) 2^-6
        b_codes = rng.integers(0x30, 0x48, size=k * n).astype(np.uint8)   # 0.5 .. 3.75
    else:
        a_codes = rng.integers(0x0001, 0x0400, size=m * k).astype(np.uint16)  # < 2^-14
        b_codes = rng.integers(0x3800, 0x4400, size=k * n).astype(np.uint16)  # 0.5 .. 4
    spec = GemmSpec(m, n, k, dt, 0, 0, seed=0, name=f"subnormal_{dt}")
    mat = inputs.from_codes(spec, a_codes, b_codes)
    ran = 0
    for vid, v in _kernels(ctx):
        if DT_NAME[v["dtype"]] != dt or v["trans_a"] or v["trans_b"]:
            continue
        plan = _run(ctx, [mat], "forced", 1, [vid])
        assert plan["variant_of"][0] == vid, f"{v['name']}: a different kernel ran"
        check(mat, label=f"subnormal {v['name']}")
        ran += 1
    assert ran > 0


def test_direct_kernels_k_depths(ctx):
    """Each direct kernel at K-tile counts 1, 2, S-1, S, S+1 and 2S+1 for its
    ring of S stages (prologue, ring wrap and last-tile paths of the main
    loop), ragged M and N, 16-byte aligned rows."""
    for vid, v in _kernels(ctx):
        if not v["direct"]:
            continue
        dt = DT_NAME[v["dtype"]]
        es = 1 if dt == "fp8" else 2
        stages = int(v["name"].split("_d")[-1].split("_")[0].rstrip("h"))
        m, n = v["bm"] + 5, v["bn"] + 3
        for nk in sorted({1, 2, max(stages - 1, 1), stages, stages + 1, 2 * stages + 1}):
            k = nk * v["bk"]
            ta, tb = v["trans_a"], v["trans_b"]
            a_cols = m if ta else k
            b_cols = k if tb else n
            spec = GemmSpec(m, n, k, dt, ta, tb, seed=5000 + 7 * vid + nk, name=f"{v['name']}_nk{nk}",
                            pad_a=_pad_to(a_cols, 16 // es), pad_b=_pad_to(b_cols, 16 // es))
            mat = inputs.materialize(spec)
            plan = _run(ctx, [mat], "forced", 1, [vid])
            assert plan["variant_of"][0] == vid, f"{v['name']}: direct path not taken"
            check(mat, label=f"{v['name']} nk={nk}")


def test_f32_concurrent_and_selector_modes(ctx):
    """fp32 GEMMs (the paper's full-precision case) in every execution mode:
    the fused and stream launches of one variant give the isolated bits."""
    specs = [GemmSpec(300 + 37 * i, 520 - 41 * i, 384 + 64 * i, "f32", i % 2, (i // 2) % 2,
                      seed=950 + i, name=f"f32_{i}") for i in range(4)]
    mats = [inputs.materialize(s) for s in specs]
    for mode in ("sequential", "default", "go", "selector"):
        _run(ctx, mats, mode)
        for m in mats:
            check(m, label=f"f32 {mode}")
    vid = ctx.find("f32_nn_128x128_w2x2_m32_c0")
    assert vid >= 0
    same = [inputs.materialize(GemmSpec(200, 300, 100 + 50 * i, "f32", seed=960 + i, name=f"f32s{i}"))
            for i in range(4)]
    iso = _isolated_codes(ctx, same, [vid] * 4)
    for mode, cd in (("forced", 4), ("forced_grouped", 4)):
        _run(ctx, same, mode, cd, [vid] * 4)
        for m, ref in zip(same, iso):
            assert np.array_equal(out_codes(m), ref), f"{mode}: {m.spec.name} differs"


# --------------------------------------------------------------------------
# strided batched GEMMs (B-GEMMs, Sec. 6.7)
# --------------------------------------------------------------------------

def test_bgemm_every_dtype_layout_and_family(ctx):
    """Ragged batched GEMMs in every dtype and layout on one staged and one
    direct kernel, item strides 16-byte aligned (direct path taken) and not
    (vector loads off, staged kernel bound); each item against the oracle."""
    for vid, v in _kernels(ctx):
        if (v["bm"], v["bn"]) != (128, 128) or v["name"].endswith(("_d4_c0",)):
            continue
        dt = DT_NAME[v["dtype"]]
        es = {"fp8": 1, "f32": 4}.get(dt, 2)
        ta, tb = v["trans_a"], v["trans_b"]
        m, n, k = 150, 133, 2 * v["bk"]
        a_cols, b_cols = (m if ta else k), (k if tb else n)
        for pad_item in (16 // es * 3, 1):
            spec = GemmSpec(m, n, k, dt, ta, tb, seed=7000 + vid + pad_item, batch=5,
                            pad_item=pad_item, pad_a=_pad_to(a_cols, 16 // es),
                            pad_b=_pad_to(b_cols, 16 // es), name=f"{v['name']}_b5p{pad_item}")
            mat = inputs.materialize(spec)
            plan = _run(ctx, [mat], "forced", 1, [vid])
            ran = ctx.variant(plan["variant_of"][0])
            if v["direct"]:
                assert ran["direct"] == (pad_item != 1), f"{v['name']} pad {pad_item}: {ran['name']}"
            check(mat, label=f"bgemm {v['name']} pad {pad_item}")


def test_bgemm_items_equal_single_gemms_bitwise(ctx):
    """Each item of a batch gives the bits of the same GEMM run alone."""
    vid = ctx.find("bf16_nn_128x128_w2x2_d2_c0")
    assert vid >= 0
    spec = GemmSpec(200, 264, 128, "bf16", seed=7100, batch=6, pad_item=64, name="bits")
    mat = inputs.materialize(spec)
    _run(ctx, [mat], "forced", 1, [vid])
    batched = out_codes(mat).copy()
    from tests.gpu_helpers import _item
    for i in range(spec.batch):
        single = _item(mat, i)
        # copies so that the single GEMM owns its operands
        alone = inputs.from_codes(single.spec, single.host["a"], single.host["b"])
        _run(ctx, [alone], "forced", 1, [vid])
        assert np.array_equal(out_codes(alone), batched[i]), f"item {i} differs"


def test_bgemm_heterogeneous_concurrent_modes(ctx):
    """Four attention-score B-GEMMs of different sequence lengths (Q K^T per
    head, K stored SL x 64 and used transposed) in every execution mode."""
    specs = [GemmSpec(sl, sl, 64, "bf16", 0, 1, seed=7200 + sl, batch=8, name=f"attn{sl}")
             for sl in (128, 200, 384, 512)]
    mats = [inputs.materialize(s) for s in specs]
    for mode in ("sequential", "default", "go", "selector"):
        plan = _run(ctx, mats, mode)
        assert sorted(plan["order"]) == [0, 1, 2, 3]
        for m in mats:
            check(m, label=f"bgemm {mode}")


def test_bgemm_shared_operand_and_validation(ctx):
    """A B operand shared by every item (stride 0); overlapping C items and
    a negative batch are rejected before anything runs."""
    batch, m, n, k = 4, 96, 160, 128
    spec = GemmSpec(m, n, k, "bf16", seed=7300, batch=batch, name="shared")
    mat = inputs.materialize(spec)
    b2 = mat.b[0]  # every item uses item 0's B
    reset_outputs([mat])
    ctx.execute([gdy.Gemm(mat.a, b2, mat.c)], mode="sequential")
    torch.cuda.synchronize()
    from tests.gpu_helpers import _item
    for i in range(batch):
        it = _item(mat, i)
        it.host["b"] = mat.host["b"][:k * n]
        check(it, label=f"shared B item {i}")
    d = gdy.Gemm(mat.a, mat.b, mat.c).desc()
    d.stride_c = m * n - 1  # items of C would overlap
    with pytest.raises(gdy.GdyError) as e:
        ctx.execute([d])
    assert e.value.status == 3
    d = gdy.Gemm(mat.a, mat.b, mat.c).desc()
    d.batch = -2
    with pytest.raises(gdy.GdyError) as e:
        ctx.execute([d])
    assert e.value.status == 1


# --------------------------------------------------------------------------
# Split-K: skinny GEMMs with a long K run each tile as several K runs
# --------------------------------------------------------------------------

def test_split_k_every_small_tile_kernel(ctx):
    """Every kernel with tiles up to 128x128 on a GEMM of three tiles and a
    long K (whole K tiles, and a ragged K tail for staged kernels): the plan
    splits it; the result meets the oracle's bound, repeats bit for bit, and
    is bit-identical fused with another GEMM (the split count depends on the
    GEMM and its kernel only)."""
    for vid, v in _kernels(ctx):
        if v["bm"] * v["bn"] > 128 * 128:
            continue
        dt = DT_NAME[v["dtype"]]
        for tail in (0, 0 if v["direct"] else 17):
            # ragged M and N tails that keep 16-byte rows (direct kernels stay direct)
            spec = GemmSpec(max(v["bm"] - 16, 8), 2 * v["bn"] + 16, 64 * v["bk"] + tail, dt, v["trans_a"],
                            v["trans_b"], seed=5000 + vid + tail, name=v["name"])
            mat = inputs.materialize(spec)
            other = inputs.materialize(GemmSpec(v["bm"], v["bn"], v["bk"] * 2, dt, v["trans_a"], v["trans_b"],
                                                seed=5500 + vid, name="other"))
            label = f"{v['name']} K={spec.k}"
            plan = _run(ctx, [mat], "forced", 1, [vid])
            assert plan["split_of"][0] > 1, label
            check(mat, label=label)
            ref = out_codes(mat).copy()
            _run(ctx, [mat], "forced", 1, [vid])
            assert np.array_equal(out_codes(mat), ref), f"{label}: repeat differs"
            alone = plan["split_of"][0]
            plan = _run(ctx, [other, mat], "forced_grouped", 0, [vid, vid])
            assert plan["n_dispatches"] == 1 and plan["split_of"][1] == alone, label
            assert np.array_equal(out_codes(mat), ref), f"{label}: fused differs"
            check(other, label=label + " co-runner")


def test_split_k_batched_and_modes(ctx):
    """A strided batch of skinny GEMMs and a set of skinny GEMMs in every
    execution mode: split plans, oracle bound, bits equal across modes that
    bind the same kernel (a grid cap changes where a tile runs, never its
    bits; the split count follows the GEMM and its kernel)."""
    b = inputs.materialize(GemmSpec(20, 100, 3000, "bf16", seed=5900, batch=5, name="bsplit"))
    plan = _run(ctx, [b], "sequential")
    assert plan["split_of"][0] > 1
    check(b, label="batched split")
    specs = [GemmSpec(16, 1024, 4096, "bf16", seed=5901 + i, name=f"skinny{i}") for i in range(3)]
    specs.append(GemmSpec(64, 2048, 2048, "f16", seed=5905, name="skinny-f16"))
    mats = [inputs.materialize(sp) for sp in specs]
    seen = {}
    for mode in ("sequential", "default", "go", "selector"):
        plan = _run(ctx, mats, mode)
        assert any(s > 1 for s in plan["split_of"]), mode
        for i, m in enumerate(mats):
            check(m, label=f"{mode} {m.spec.name}")
            key = (i, ctx.variant(plan["variant_of"][i])["name"].rsplit("_c", 1)[0])
            if key in seen:
                assert np.array_equal(seen[key], out_codes(m)), f"{mode} {m.spec.name}"
            seen[key] = out_codes(m).copy()


# --------------------------------------------------------------------------
# GEMM + non-GEMM co-runs (Sec. 7.1): the element-wise add
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
def test_add_every_type_and_edge(ctx, dt):
    """Element-wise adds of every supported type: one element, ragged rows
    and columns with padded leading dimensions (element-wise loads), and
    aligned ones (vector loads)."""
    from tests.gpu_helpers import check_add
    for i, (m, n, pad) in enumerate(((1, 1, 0), (37, 300, 3), (64, 4096, 0), (257, 1030, 8))):
        x = inputs.materialize_add(m, n, dt, seed=8000 + i, pad=pad)
        ctx.execute([gdy.Add(x.a, x.b, x.c)], mode="sequential")
        torch.cuda.synchronize()
        check_add(x, label=f"{dt} {m}x{n}+{pad}")


def test_gemm_add_corun_every_mode(ctx):
    """A GEMM and an add of its output size (plus a second add, fused with the
    first) in every execution mode; every output against the oracle."""
    from tests.gpu_helpers import check_add
    g = inputs.materialize(GemmSpec(512, 1024, 768, "bf16", seed=8100, name="corun"))
    adds = [inputs.materialize_add(512, 1024, "bf16", seed=8101 + i) for i in range(2)]
    for mode in ("sequential", "default", "go", "selector"):
        reset_outputs([g])
        for x in adds:
            x.c_full.fill_(float("nan"))
        plan = ctx.execute([gemm_of(g)] + [gdy.Add(x.a, x.b, x.c) for x in adds], mode=mode,
                           want_plan=True)
        torch.cuda.synchronize()
        assert sorted(plan["order"]) == [0, 1, 2]
        ew = [ctx.variant(plan["variant_of"][i])["kind"] for i in range(3)]
        assert ew == [0, 1, 1], (mode, ew)
        check(g, label=f"corun {mode}")
        for x in adds:
            check_add(x, label=f"corun {mode}")
    # in one group both adds ride in the GEMM's dispatch: one launch, no second stream
    plan = ctx.plan([gdy.Add(x.a, x.b, x.c) for x in adds] + [gemm_of(g)], mode="go")
    assert plan["n_dispatches"] == 1 and plan["order"][:3] == [2, 0, 1], plan["order"][:3]
    assert plan["dispatch_of"][0] == plan["dispatch_of"][1] == plan["dispatch_of"][2]
    # a group of adds only keeps the add kernel, both adds in one dispatch
    plan = ctx.plan([gdy.Add(x.a, x.b, x.c) for x in adds], mode="go")
    assert plan["n_dispatches"] == 1


def test_add_fused_into_every_gemm_kernel(ctx):
    """An add rides in the dispatch of every GEMM kernel (staged and direct,
    every block size): adds of each type, ragged, with unaligned rows, or a
    strided batch; GEMM and add against the oracle, and the add's bits equal
    to those of its own kernel."""
    from tests.gpu_helpers import check_add
    V = ctx.variants()
    ew = {DT_NAME[v["dtype"]]: i for i, v in enumerate(V) if v["kind"] == 1 and v["grid_cap_cus"] == 0}
    cases = ((1, 1, 0, "bf16", 0), (37, 300, 3, "f16", 0), (70, 1030, 0, "f32", 0),
             (257, 4100, 8, "bf16", 0), (96, 520, 0, "f16", 3), (40, 136, 5, "f32", 4))
    for j, (vid, v) in enumerate(_kernels(ctx)):
        dt = DT_NAME[v["dtype"]]
        spec = GemmSpec(v["bm"] * 2, v["bn"] * 2, v["bk"] * 3, dt, v["trans_a"], v["trans_b"],
                        seed=1000 + vid, name=v["name"])
        mat = inputs.materialize(spec)
        m, n, pad, adt, items = cases[j % len(cases)]
        x = inputs.materialize_add(m * max(items, 1), n, adt, seed=8300 + j, pad=pad)

        def add_of(variant):
            if items:
                a, b, c = (t.unflatten(0, (items, m)) for t in (x.a, x.b, x.c))
                return gdy.Add(a, b, c, variant=variant)
            return gdy.Add(x.a, x.b, x.c, variant=variant)
        reset_outputs([mat])
        plan = ctx.execute([add_of(ew[adt]), gemm_of(mat, vid)], mode="forced_grouped",
                           want_plan=True)
        torch.cuda.synchronize()
        label = f"{v['name']} + add {adt} {m}x{n}+{pad} items {items}"
        assert plan["n_dispatches"] == 1 and plan["order"][:2] == [1, 0], label
        assert ctx.variant(plan["variant_of"][1])["kind"] == 0, label
        check(mat, label=label)
        check_add(x, label=label)
        fused = x.c_full.clone()
        x.c_full.fill_(float("nan"))
        ctx.execute([add_of(-1)], mode="sequential")
        torch.cuda.synchronize()
        raw = torch.int32 if adt == "f32" else torch.int16
        assert torch.equal(fused.view(raw), x.c_full.view(raw)), f"{label}: fused bits differ"


def test_add_validation(ctx):
    x = inputs.materialize_add(32, 64, "bf16", seed=8200)
    d = gdy.Add(x.a, x.b, x.c).desc()
    d.k = 5
    with pytest.raises(gdy.GdyError) as e:
        ctx.execute([d])
    assert e.value.status == 1
    d = gdy.Add(x.a, x.b, x.c).desc()
    d.c_type = 1  # mixed types
    with pytest.raises(gdy.GdyError) as e:
        ctx.execute([d])
    assert e.value.status == 2
    d = gdy.Add(x.a, x.b, x.c).desc()
    d.op = 7
    with pytest.raises(gdy.GdyError) as e:
        ctx.execute([d])
    assert e.value.status == 1
