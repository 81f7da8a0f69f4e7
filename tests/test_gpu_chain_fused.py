"""GPU parity of the fused chain kernel (ks_chain on chains of small-block
factors, and batch-size-first of square blocks of one size in 16 .. 64 on the MFMAs):
against the fp64 oracle chain, against the factor-by-factor path on
the same inputs, on aligned and offset buffers (16-byte and element access),
full and ragged batch tiles, both layouts, every storage type; bit-exact on
the Hadamard chain."""
import numpy as np
import pytest

import oracle
import paper_2405_15013_amd as ks
from paper_2405_15013_amd import inputs
from parity_util import TOL, from_device, nan_tensor, rel_err, to_device

pytestmark = pytest.mark.gpu


def butterfly(L):
    return [(2 ** (l - 1), 2, 2, 2 ** (L - l)) for l in range(1, L + 1)]


CHAINS = {
    "butterfly1024": butterfly(10),
    "butterfly512": butterfly(9),
    "butterfly64": butterfly(6),
    "butterfly16": butterfly(4),
    "butterfly8": butterfly(3),
    "deformable": [(2, 3, 4, 1), (1, 8, 6, 1), (3, 2, 2, 1)],
    "radix4": [(1, 4, 4, 16), (4, 4, 4, 4), (16, 4, 4, 1)],
    "mixed": [(4, 8, 8, 2), (8, 2, 2, 4), (2, 4, 3, 8), (6, 4, 4, 2)],
    # square blocks of one size in {16, 32, 48, 64} (the MFMA form)
    "monarch1024": [(1, 32, 32, 32), (32, 32, 32, 1)],
    "monarch256": [(1, 16, 16, 16), (16, 16, 16, 1)],
    "square48": [(16, 48, 48, 1), (1, 48, 48, 16), (4, 48, 48, 4)],
    "square64": [(2, 64, 64, 8), (16, 64, 64, 1)],
    "square_wide": [(1, 16, 16, 128), (128, 16, 16, 1)],  # width 2048: 160 KB of LDS, one workgroup per CU
}


def run_chain(pats, x, kvs, batch, dtype, layout, fused=True, x_offset=0, y_offset=0, k_offset=0):
    import torch
    M = pats[0][0] * pats[0][1] * pats[0][3]
    xflat = inputs.to_layout(x, layout).reshape(-1)
    xd = to_device(np.concatenate([np.zeros(x_offset, dtype=xflat.dtype), xflat]), dtype)[x_offset:]
    factors = [(p, to_device(np.concatenate([np.zeros(k_offset, dtype=k.dtype), k.reshape(-1)]), dtype)[k_offset:])
               for p, k in zip(pats, kvs)]
    yd = nan_tensor((y_offset + batch * M,), dtype)[y_offset:]
    ks.ks_force_chain_fusion(None if fused else 0)
    try:
        desc = ks.ks_chain_describe(factors, batch, layout, dtype)
        # the MFMA form (square blocks of 16 .. 64) fuses batch-size-first, and
        # batch-size-last in fp32 with 32-column tiles (blocks up to 32, width
        # up to 1024)
        small = max(max(p[1], p[2]) for p in pats) <= 8
        wide = pats[0][1] <= 32 and pats[0][0] * pats[0][1] * pats[0][3] <= 1024
        fuses = fused and (small or layout == "bsf" or (dtype == "f32" and wide))
        assert desc.startswith("fused" if fuses else "unfused"), desc
        need = ks.ks_chain_workspace_bytes(factors, batch, dtype)
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device="cuda")
        ks.ks_chain(factors, xd, yd, batch, layout, dtype, ws, need)
        torch.cuda.synchronize()
    finally:
        ks.ks_force_chain_fusion(None)
    y = from_device(yd, dtype).reshape((batch, M) if layout == "bsf" else (M, batch))
    return inputs.from_layout(y, layout)


def chain_case(name, batch, dtype, cfg=41):
    pats = CHAINS[name]
    x = inputs.make_x(cfg, pats[-1], batch, dtype)
    kvs = [inputs.make_kv(cfg, p, batch, dtype, dist="normal_c", factor=f) for f, p in enumerate(pats)]
    y64 = oracle.chain(pats, [inputs.to_f64(k, dtype) for k in kvs], inputs.to_f64(x, dtype), batch, "bsf")
    return pats, x, kvs, y64


@pytest.mark.parametrize("name", sorted(CHAINS))
@pytest.mark.parametrize("layout", ["bsl", "bsf"])
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("batch", [1, 17, 4096])
def test_fused_chain_against_oracle(name, layout, dtype, batch):
    pats, x, kvs, y64 = chain_case(name, batch, dtype)
    print("fused chain %s B=%d %s %s" % (name, batch, dtype, layout), flush=True)
    y = run_chain(pats, x, kvs, batch, dtype, layout)
    assert np.all(np.isfinite(y)), "unwritten outputs"
    assert rel_err(y, y64) <= TOL[dtype]


@pytest.mark.parametrize("name", ["butterfly1024", "mixed", "monarch1024", "square48"])
@pytest.mark.parametrize("layout", ["bsl", "bsf"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fused_chain_offset_buffers(name, layout, dtype):
    """Buffers shifted off 16-byte alignment: the element-wise load/store path;
    factor values shifted by one element: the element-wise value fetch."""
    batch = 100
    pats, x, kvs, y64 = chain_case(name, batch, dtype, cfg=42)
    y = run_chain(pats, x, kvs, batch, dtype, layout, x_offset=1, y_offset=3)
    assert rel_err(y, y64) <= TOL[dtype]
    y = run_chain(pats, x, kvs, batch, dtype, layout, k_offset=1)
    assert rel_err(y, y64) <= TOL[dtype]


@pytest.mark.parametrize("name", ["butterfly1024", "monarch1024"])
@pytest.mark.parametrize("layout", ["bsl", "bsf"])
def test_fused_and_factor_by_factor_agree(name, layout):
    batch = 4096
    pats, x, kvs, y64 = chain_case(name, batch, "f32", cfg=43)
    yf = run_chain(pats, x, kvs, batch, "f32", layout, fused=True)
    yu = run_chain(pats, x, kvs, batch, "f32", layout, fused=False)
    assert rel_err(yf, y64) <= TOL["f32"] and rel_err(yu, y64) <= TOL["f32"]


@pytest.mark.parametrize("layout", ["bsl", "bsf"])
def test_monarch_chain_of_permutations_is_exact(layout):
    """Blocks that are permutation matrices: every output is one input value,
    moved through fp32 LDS and the MFMAs with exact products and zero sums."""
    batch = 1000
    pats = CHAINS["monarch1024"]
    x = inputs.make_x(5, pats[-1], batch, "f32")
    rng = np.random.default_rng(11)
    kvs = []
    for p in pats:
        nb = p[0] * p[3]
        kv = np.zeros((nb, p[1], p[2]), dtype=np.float32)
        for q in range(nb):
            kv[q, np.arange(p[1]), rng.permutation(p[2])] = 1.0
        kvs.append(kv)
    y = run_chain(pats, x, kvs, batch, "f32", layout)
    y64 = oracle.chain(pats, [k.astype(np.float64) for k in kvs], x.astype(np.float64), batch, "bsf")
    np.testing.assert_array_equal(y, y64)


@pytest.mark.parametrize("layout", ["bsl", "bsf"])
@pytest.mark.parametrize("fused", [True, False])
def test_hadamard_chain_bit_exact_both_paths(layout, fused):
    import scipy.linalg
    batch = 4096
    pats = butterfly(10)
    x = inputs.make_x(2, pats[-1], batch, "f32", dist="sign")
    h2 = np.array([[1, 1], [1, -1]], dtype=np.float32)
    kvs = [np.broadcast_to(h2, (p[0] * p[3], 2, 2)).copy() for p in pats]
    y = run_chain(pats, x, kvs, batch, "f32", layout, fused=fused)
    H = scipy.linalg.hadamard(1024).astype(np.float64)
    np.testing.assert_array_equal(y, x.astype(np.float64) @ H)
