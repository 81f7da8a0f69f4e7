"""Host-side checks of the fused chain path (no GPU): which chains run fused,
the workspace they need, and a replay of the fused kernel's accesses
(ks_chain_verify) over chain shapes, batches, layouts and storage types."""
import pytest

import paper_2405_15013_amd as ks

P0 = 1 << 44


def butterfly(L):
    return [(2 ** (l - 1), 2, 2, 2 ** (L - l)) for l in range(1, L + 1)]


def factors(pats):
    return [(p, P0 + q * (1 << 30)) for q, p in enumerate(pats)]


CHAINS = {
    "butterfly1024": butterfly(10),
    "butterfly512": butterfly(9),
    "butterfly32": butterfly(5),
    "butterfly16": butterfly(4),
    "butterfly8": butterfly(3),
    "butterfly2": butterfly(1) * 2,
    "deformable": [(2, 3, 4, 1), (1, 8, 6, 1), (3, 2, 2, 1)],      # b != c: two LDS buffers
    "radix4": [(1, 4, 4, 16), (4, 4, 4, 4), (16, 4, 4, 1)],
    "mixed": [(4, 8, 8, 2), (8, 2, 2, 4), (2, 4, 3, 8), (6, 4, 4, 2)],
    "wide_inplace": [(1, 2, 2, 1024), (1024, 2, 2, 1)],            # width 2048: 160 KB of LDS, not fused
    # square blocks of one size in {16, 32, 48, 64}: the MFMA form
    "monarch1024": [(1, 32, 32, 32), (32, 32, 32, 1)],
    "monarch256": [(1, 16, 16, 16), (16, 16, 16, 1)],
    "square48": [(16, 48, 48, 1), (1, 48, 48, 16), (4, 48, 48, 4)],
    "square64": [(2, 64, 64, 8), (16, 64, 64, 1)],
    "square_wide": [(1, 16, 16, 128), (128, 16, 16, 1)],           # width 2048: 160 KB, one buffer
}


@pytest.mark.parametrize("name", sorted(CHAINS))
@pytest.mark.parametrize("layout", ["bsl", "bsf"])
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("batch", [1, 15, 16, 17, 100, 4096])
def test_fused_chain_replay(name, layout, dtype, batch):
    f = factors(CHAINS[name])
    desc = ks.ks_chain_describe(f, batch, layout, dtype)
    st, rep = ks.ks_chain_verify(f, batch, layout, dtype)
    assert st == 0, (desc, rep)
    if desc.startswith("fused"):
        assert rep == "ok"
        assert desc.startswith("fused-mfma") == name.startswith(("monarch", "square"))
    else:
        assert rep == "not fused"
    if name.startswith(("monarch", "square")):
        # batch-size-first: tiles of 16 columns; batch-size-last only fp32 with
        # tiles of 32 columns (blocks up to 32, width up to 1024)
        pats = CHAINS[name]
        wide = pats[0][1] <= 32 and pats[0][0] * pats[0][1] * pats[0][3] <= 1024
        if dtype == "f32" and wide:
            assert desc.startswith("fused-mfma") and desc.endswith("cols=32"), desc
        elif layout == "bsf":
            assert desc.startswith("fused-mfma") and desc.endswith("cols=16"), desc
        else:
            assert desc.startswith("unfused"), desc


def test_which_chains_fuse():
    bf = factors(butterfly(10))
    for layout in ("bsl", "bsf"):
        for dtype in ("f32", "bf16"):
            desc = ks.ks_chain_describe(bf, 4096, layout, dtype)
            # the dyadic butterfly of size 16 .. 1024: two register passes of 32 rows
            assert desc.startswith("fused-bfly ") and "passes=2 groups=32,32 " in desc, desc
            assert ks.ks_chain_workspace_bytes(bf, 4096, dtype) == 0
    assert ks.ks_chain_describe(factors(butterfly(9)), 64, "bsl", "f32").startswith("fused-bfly ")
    assert ks.ks_chain_describe(factors(butterfly(4)), 64, "bsl", "f32").startswith("fused-bfly ")
    # shorter butterflies and other small-block chains: radix passes
    assert ks.ks_chain_describe(factors(butterfly(3)), 64, "bsl", "f32").startswith("fused factors=3")
    assert ks.ks_chain_describe(factors(CHAINS["radix4"]), 64, "bsl", "f32").startswith("fused factors=3")
    # Monarch factors (32 x 32 blocks) run fused on the MFMAs, in one LDS
    # buffer, batch-size-first; batch-size-last factor by factor
    mon = factors([(1, 32, 32, 32), (32, 32, 32, 1)])
    for dtype in ("f32", "bf16", "f16"):
        desc = ks.ks_chain_describe(mon, 16384, "bsf", dtype)
        if dtype == "f32":  # fp32: tiles of 32 columns (144 KB of LDS)
            assert desc.startswith("fused-mfma ") and "inplace=1" in desc and "lds=147456 " in desc and "cols=32" in desc, desc
        else:
            assert desc.startswith("fused-mfma ") and "inplace=1" in desc and "lds=81920 " in desc and "cols=16" in desc, desc
        desc = ks.ks_chain_describe(mon, 16384, "bsl", dtype)
        if dtype == "f32":
            assert desc.startswith("fused-mfma ") and "lds=147456 " in desc and desc.endswith("grid=512 block=512 cols=32"), desc
            assert ks.ks_chain_workspace_bytes(mon, 16384, dtype) == 0
        else:
            # batch-size-last 16-bit chains run factor by factor; the workspace
            # query has no layout and answers for that run
            assert desc.startswith("unfused"), desc
            assert ks.ks_chain_workspace_bytes(mon, 16384, dtype) == 1024 * 16384 * 2
    # blocks that are not all square of one size in {16, 32, 48, 64}, or that
    # mix small and large blocks, run factor by factor
    for pats in ([(1, 32, 16, 32), (32, 16, 32, 1)], [(1, 96, 96, 8), (8, 96, 96, 1)],
                 [(1, 24, 24, 8), (8, 24, 24, 1)], [(1, 32, 32, 4), (16, 2, 2, 4)],
                 [(2, 64, 64, 8), (16, 64, 64, 1), (4, 16, 16, 16)]):
        assert ks.ks_chain_describe(factors(pats), 256, "bsf", "f32").startswith("unfused"), pats
    # MFMA form of width 4096 needs 320 KB of LDS: not fused
    assert ks.ks_chain_describe(factors([(1, 64, 64, 64), (64, 64, 64, 1)]), 64, "bsf", "f32").startswith("unfused")
    assert ks.ks_chain_describe(factors(CHAINS["square_wide"]), 64, "bsf", "f32").startswith("fused-mfma")
    # width 2048 with 16 fp32 columns needs 160 KB of LDS: not fused
    assert ks.ks_chain_describe(factors(CHAINS["wide_inplace"]), 64, "bsl", "f32").startswith("unfused")
    # a single factor is not a chain to fuse
    assert ks.ks_chain_describe(factors(butterfly(1)), 64, "bsl", "f32").startswith("unfused")


def test_fusion_can_be_switched_off_per_thread():
    bf = factors(butterfly(10))
    ks.ks_force_chain_fusion(0)
    try:
        assert ks.ks_chain_describe(bf, 4096, "bsl", "f32").startswith("unfused")
        assert ks.ks_chain_workspace_bytes(bf, 4096, "f32") == 2 * 1024 * 4096 * 4
    finally:
        ks.ks_force_chain_fusion(None)
    assert ks.ks_chain_describe(bf, 4096, "bsl", "f32").startswith("fused")
    # a forced kernel variant also runs chains factor by factor
    ks.ks_force_variant(0)
    try:
        assert ks.ks_chain_describe(bf, 4096, "bsl", "f32").startswith("unfused")
    finally:
        ks.ks_force_variant(None)
