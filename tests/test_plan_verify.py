"""Host-side replay of planned launches (ks_plan_verify): every global access
of every thread stays in bounds, every LDS cell the MFMA reads was written,
and every element of Y is written exactly once (the row sets of the paper's
Section 4.1 partition the output, so no two workgroups may touch one element).
Runs on the CPU; nothing is enqueued."""
import pytest

import paper_2405_15013_amd as ks
from shapes import DMA_ROW_GROUP_SHAPES, DMA_SHAPES


def sweep_patterns():
    return [(a, b, c, d) for a in (1, 2, 4, 8) for b in (16, 32, 48, 64, 96, 128) for c in (16, 32, 48, 64, 96, 128)
            for d in (1, 2, 4, 8, 16) if a * b * d <= 8192 and a * c * d <= 8192]


CONFIGS = ([(2, 4, 4, 2)] + [(2 ** (l - 1), 2, 2, 2 ** (10 - l)) for l in range(1, 11)]
           + [(1, 32, 32, 32), (32, 32, 32, 1), (6, 64, 16, 8), (6, 16, 64, 8)])


@pytest.mark.parametrize("pattern", sweep_patterns()[::23])
@pytest.mark.parametrize("batch", [48, 1000, 4096])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sweep_plans(pattern, batch, layout, dtype):
    st, rep = ks.ks_plan_verify(*pattern, batch, layout, dtype)
    assert st == 0, "%s B=%d %s %s: %s [%s]" % (pattern, batch, layout, dtype, rep,
                                                ks.ks_plan_describe(*pattern, batch, layout, dtype))


@pytest.mark.parametrize("pattern", CONFIGS)
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_config_plans_small_batch(pattern, layout, dtype):
    for batch in (1, 32, 104, 256):
        st, rep = ks.ks_plan_verify(*pattern, batch, layout, dtype)
        assert st == 0, "%s B=%d %s %s: %s" % (pattern, batch, layout, dtype, rep)


@pytest.mark.parametrize("pattern,batch", [((1, 32, 32, 32), 16384), ((6, 64, 16, 8), 25088),
                                           ((6, 16, 64, 8), 25088), ((1, 2, 2, 512), 4096)])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
def test_full_size_plans(pattern, batch, layout):
    st, rep = ks.ks_plan_verify(*pattern, batch, layout, "bf16")
    assert st == 0, rep


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
def test_all_sweep_plans_ragged_batch(dtype, layout):
    """Every sweep pattern, a batch that leaves a partial tile in both layouts."""
    bad = []
    for pattern in sweep_patterns():
        st, rep = ks.ks_plan_verify(*pattern, 72, layout, dtype)
        if st != 0:
            bad.append((pattern, rep))
    assert not bad, bad[:5]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("batch,every", [(72, 1), (1000, 5)])
def test_all_sweep_plans_staged(dtype, layout, batch, every):
    """The LDS-staged kernel on every sweep pattern (forced): bounds, LDS cells
    written before they are read, every operand element the right X value,
    every output written once."""
    bad = []
    ks.ks_force_variant(4)
    try:
        for pattern in sweep_patterns()[::every]:
            st, rep = ks.ks_plan_verify(*pattern, batch, layout, dtype)
            if st != 0 and not (rep == "no plan" and layout == "bsl" and batch % (16 // (4 if dtype == "f32" else 2))):
                bad.append((pattern, rep))
    finally:
        ks.ks_force_variant(None)
    assert not bad, bad[:5]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("batch,every", [(72, 1), (1000, 7), (25088, 97)])
def test_all_sweep_plans_dma(dtype, batch, every):
    """The LDS-DMA kernel (forced) on every batch-size-first sweep pattern:
    every DMA lane fills one unit of the stage from an in-bounds address, every
    swizzled operand read holds the right X value, every output written once.
    It must accept every pattern of the sweep."""
    bad = []
    ks.ks_force_variant(6)
    try:
        for pattern in sweep_patterns()[::every]:
            st, rep = ks.ks_plan_verify(*pattern, batch, "bsf", dtype)
            if st != 0:
                bad.append((pattern, rep))
            else:
                assert "name=dma" in ks.ks_plan_describe(*pattern, batch, "bsf", dtype)
    finally:
        ks.ks_force_variant(None)
    assert not bad, bad[:5]


def test_sweep_plans_use_mfma_kernels():
    """The whole sweep runs on the MFMA kernels (aligned buffers): LDS-DMA for
    batch-size-first with d >= 4 or at least 8 MB of X and Y, and for
    batch-size-last in fp32, or in 16-bit types with b a power of two from 32
    and c of 32 or 64; register-direct otherwise."""
    for pattern in sweep_patterns()[::7]:
        for layout in ("bsf", "bsl"):
            for dtype in ("f32", "bf16", "f16"):
                desc = ks.ks_plan_describe(*pattern, 4096, layout, dtype)
                a, b, c, d = pattern
                big = 4096 * (a * c * d + a * b * d) * (4 if dtype == "f32" else 2) >= 8 << 20
                if layout == "bsf":
                    dma = d >= 4 or big
                else:
                    dma = dtype == "f32" or (b in (32, 64, 128) and c in (32, 64))
                want = "name=dma" if dma else "name=direct"
                assert want in desc, (pattern, layout, dtype, desc)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("batch,every", [(72, 3), (1000, 7), (25088, 97)])
def test_all_sweep_plans_dma_bsl(dtype, batch, every):
    """The batch-size-last LDS-DMA kernel (forced) on the batch-size-last sweep
    patterns it accepts (c a multiple of its stage: 16 for fp32, 32 for 16-bit
    types; the batch a multiple of the vector): DMA units in bounds and each
    written once per stage, every operand read the X value its products need,
    every output written once.  It must accept every such pattern."""
    bad = []
    ks.ks_force_variant(6)
    try:
        for pattern in sweep_patterns()[::every]:
            a, b, c, d = pattern
            if c % (16 if dtype == "f32" else 32) or batch % (4 if dtype == "f32" else 8):
                continue
            st, rep = ks.ks_plan_verify(*pattern, batch, "bsl", dtype)
            if st != 0:
                bad.append((pattern, rep))
            else:
                assert "kernel=ks_dma_bsl_kernel" in ks.ks_plan_describe(*pattern, batch, "bsl", dtype)
    finally:
        ks.ks_force_variant(None)
    assert not bad, bad[:5]


@pytest.mark.parametrize("variant", [0, 1, 2, 3, 4, 5, 6])
def test_forced_variants(variant):
    """Every variant that accepts a shape produces a valid launch for it."""
    ks.ks_force_variant(variant)
    try:
        for pattern, layout in [((2, 4, 4, 2), "bsl"), ((2, 4, 4, 2), "bsf"), ((1, 16, 16, 4), "bsf"),
                                ((1, 16, 16, 4), "bsl"), ((3, 32, 48, 2), "bsf")]:
            st, rep = ks.ks_plan_verify(*pattern, 64, layout, "f32")
            assert st in (0, 5), rep
            if st == 5:
                assert rep == "no plan", rep
    finally:
        ks.ks_force_variant(None)


def test_dma_row_group_plans_covered():
    """The GPU parity shapes of the DMA kernel reach every (MT, NT, stage
    length, strided) plan its planner makes on sweep-like patterns at batch
    4096, and each of those plans passes the replay."""
    def key(p, dt):
        f = dict(kv.split("=", 1) for kv in ks.ks_plan_describe(*p, 4096, "bsf", dt).split())
        return (dt, f["waves_m"], f["nt"], f["lch"], f["unroll"])
    have = {key(p, dt) for p in DMA_ROW_GROUP_SHAPES + DMA_SHAPES for dt in ("f32", "bf16")}
    want = {key(p, dt) for p in [(a, b, c, d) for a in (1, 2, 4, 8) for b in (16, 32, 64, 128) for c in (16, 32, 64)
                                  for d in (1, 2, 4, 8, 16) if a * b * d <= 8192 and a * c * d <= 8192]
            for dt in ("f32", "bf16")}
    assert want <= have, sorted(want - have)
    for p in DMA_ROW_GROUP_SHAPES:
        for dt in ("f32", "bf16"):
            for batch in (4096, 4000):
                st, rep = ks.ks_plan_verify(*p, batch, "bsf", dt)
                assert st == 0, (p, dt, batch, rep)


ODD = [(1, 24, 24, 8), (1, 17, 33, 3), (2, 48, 80, 2), (6, 64, 16, 8), (1, 64, 64, 1), (3, 20, 40, 1), (1, 100, 36, 2),
       (4, 16, 17, 2), (1, 33, 16, 5)]


@pytest.mark.parametrize("pattern", ODD)
@pytest.mark.parametrize("batch", [1, 37, 1001, 4096, 25087])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_no_generic_plan_for_large_blocks(pattern, batch, layout, dtype):
    """Blocks with b or c above 16 always get an MFMA kernel (the masked one
    when b or c is not a multiple of 16 or the batch is not a multiple of the
    vector), whose host replay passes at every access width the planner may
    pick for less aligned buffers."""
    desc = ks.ks_plan_describe(*pattern, batch, layout, dtype)
    assert "name=generic" not in desc, desc
    if batch <= 4096:
        st, rep = ks.ks_plan_verify(*pattern, batch, layout, dtype)
        assert st == 0, (desc, rep)


@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("batch", [4096, 1001])
def test_fp8_sweep_plans(layout, batch):
    """Host replay of the FP8 kernel's plan (access width up to 8 in both
    layouts) over every sweep pattern: coverage, padding, alignment."""
    for pattern in sweep_patterns()[::15] + [(6, 64, 16, 8), (6, 16, 64, 8), (1, 17, 33, 3), (4, 48, 32, 16)]:
        st, rep = ks.ks_plan_verify(*pattern, batch, layout, "fp8")
        assert st == 0, "%s B=%d %s: %s" % (pattern, batch, layout, rep)
        assert "name=fp8" in ks.ks_plan_describe(*pattern, batch, layout, "fp8")


def test_fp8_bsf_uses_full_rows_when_d_is_8():
    desc = ks.ks_plan_describe(6, 64, 16, 8, 25088, "bsf", "fp8")
    assert "vec=8" in desc, desc
