"""The seeded workload generators (no GPU): each workload has the shapes,
types and value ranges it is stated to have, the same seed gives the same
specs and operand codes, and every heterogeneous GEMM's windows lie inside
the device pools without overlapping the other windows of its submission."""
import numpy as np

from paper_2409_02227_amd import inputs


def test_square_lstm_and_layer_share_shapes():
    assert [(s.m, s.n, s.k, s.dtype) for s in inputs.square_fp16()] == [(256, 256, 256, "f16")] * 2
    assert [(s.m, s.n, s.k, s.dtype) for s in inputs.lstm_gates()] == [(64, 4096, 1024, "bf16")] * 4
    ls = inputs.layer_share()
    assert [(s.m, s.n, s.k) for s in ls] == [(m, n, k) for _, m, n, k in inputs.LAYER_SHARE_SHAPES] * 2
    assert len({s.seed for s in ls}) == 8  # each GEMM draws its own operands


def test_heterogeneous_submissions_ranges():
    subs = inputs.het_submissions()
    assert len(subs) == 200
    sizes = {1024, 2048, 4096, 8192}
    for sub in subs:
        assert 2 <= len(sub) <= 16
        for s in sub:
            assert 16 <= s.m <= 4096 and s.n in sizes and s.k in sizes and s.dtype == "bf16"
    ms = np.array([s.m for sub in subs for s in sub])
    # log-uniform M: about half of the GEMMs below the geometric middle, 256
    assert 0.4 < np.mean(ms < 256) < 0.6
    assert [[(s.m, s.n, s.k) for s in sub] for sub in inputs.het_submissions(count=5)] == \
        [[(s.m, s.n, s.k) for s in sub] for sub in subs[:5]]


def test_fp8_tenants_composition():
    specs = inputs.fp8_tenants()
    assert len(specs) == 32 and {s.dtype for s in specs} == {"fp8"}
    for t in (0, 1):
        mine = sorted((s.m, s.n) for s in specs if s.tenant == t)
        # each tenant: every (M, N = K) combination twice
        assert mine == sorted([(m, nk) for m in (1, 32, 256, 2048) for nk in (4096, 8192)] * 2)
    assert all(s.n == s.k for s in specs)


def test_attention_bgemms_are_batched_and_transposed():
    specs = inputs.attention_bgemms()
    assert [(s.m, s.n, s.k, s.batch, s.trans_b) for s in specs] == \
        [(sl, sl, 64, 64, 1) for sl in (128, 256, 384, 512)]


def test_operand_codes_are_deterministic_and_in_range():
    spec = inputs.lstm_gates()[0]
    a1, sa1 = inputs.operand_codes(spec, "a")
    a2, sa2 = inputs.operand_codes(spec, "a")
    b1, _ = inputs.operand_codes(spec, "b")
    assert np.array_equal(a1, a2) and sa1 == sa2 == 1.0 and not np.array_equal(a1[:1024], b1[:1024])
    import torch
    av = torch.from_numpy(a1.view(np.int16)).view(torch.bfloat16).float().numpy()
    assert a1.size == spec.m * spec.ld("a") and av.min() >= -1 and av.max() <= 1  # A ~ U[-1, 1]
    fp = inputs.fp8_tenants()[0]
    codes, scale = inputs.operand_codes(fp, "a")
    vals = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().numpy()
    assert codes.dtype == np.uint8 and np.abs(vals).max() <= 448 and 2 ** -4 / 448 <= scale <= 2 ** 4 / 448


def test_heterogeneous_windows_fit_the_pools_and_stay_disjoint():
    for sub in inputs.het_placed(200):
        spans_a, spans_b = [], []
        for g, oa, ob in sub:
            assert oa % 256 == 0 and ob % 256 == 0
            assert 0 <= oa and oa + g.m * g.k <= inputs.HET_A_ELEMS
            assert 0 <= ob and ob + g.k * g.n <= inputs.HET_B_ELEMS
            spans_a.append((oa, oa + g.m * g.k))
            spans_b.append((ob, ob + g.k * g.n))
        for spans in (spans_a, spans_b):
            spans.sort()
            assert all(e0 <= s1 for (_, e0), (s1, _) in zip(spans, spans[1:])), "windows overlap"
