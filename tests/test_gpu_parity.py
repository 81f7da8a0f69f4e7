"""GPU parity: the HIP path (through the C ABI) against the fp64 CPU oracle on
the same seeded inputs, for every workload family of the benchmark and the
edge cases of the method.  Outputs are pre-filled with NaN so that an element
a kernel fails to write shows up as an infinite error."""
import zlib

import numpy as np
import pytest

import oracle
import paper_2405_15013_amd as ks
from paper_2405_15013_amd import inputs
from parity_util import TOL, case, from_device, nan_tensor, oracle_y, rel_err, to_device, torch_dtype
from shapes import DMA_ROW_GROUP_SHAPES, DMA_SHAPES, MFMA_SHAPES

pytestmark = pytest.mark.gpu

VARIANTS = {"generic": 0, "valu_bsl": 1, "valu_bsf": 2, "direct": 3, "staged": 4, "dma": 6}


def run_gpu(pattern, x_logical, kv, batch, dtype, layout, variant=None, x_offset=0, y_offset=0):
    """Lay out X, run ks_matmul on the device, return Y in logical (batch, M) order.
    x_offset / y_offset shift the buffers by that many elements (alignment tests)."""
    import torch
    a, b, c, d = pattern
    M = a * b * d
    xd_full = to_device(np.concatenate([np.zeros(x_offset, dtype=x_logical.dtype),
                                        inputs.to_layout(x_logical, layout).reshape(-1)]), dtype)
    xd = xd_full[x_offset:]
    kd = to_device(kv, dtype)
    yd_full = nan_tensor((y_offset + batch * M,), dtype)
    yd = yd_full[y_offset:]
    ks.ks_force_variant(variant)
    try:
        ks.ks_matmul(a, b, c, d, kd, xd, yd, batch, layout, dtype)
    finally:
        ks.ks_force_variant(None)
    torch.cuda.synchronize()
    y = from_device(yd, dtype)
    y = y.reshape((batch, M) if layout == "bsf" else (M, batch))
    return inputs.from_layout(y, layout)


def check(pattern, batch, dtype, layout, cfg=0, variant=None, xdist="normal", kdist="uniform_c", tol=None, **kw):
    x, kv, _, _ = case(cfg, pattern, batch, dtype, xdist, kdist)
    y = run_gpu(pattern, x, kv, batch, dtype, layout, variant=variant, **kw)
    y64 = oracle_y(cfg, pattern, batch, dtype, xdist, kdist)
    err = rel_err(y, y64)
    assert err <= (TOL[dtype] if tol is None else tol), "pattern %s batch %d %s %s variant %s: rel err %.3e" % (
        pattern, batch, dtype, layout, variant, err)
    return err


# --- tiny: (2,4,4,2), B = 32, K is 16 x 16 with 64 nonzeros ------------------

@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("variant", [None, "generic", "valu"])
def test_tiny(layout, dtype, variant):
    v = None if variant is None else (0 if variant == "generic" else (1 if layout == "bsl" else 2))
    check((2, 4, 4, 2), 32, dtype, layout, cfg=1, variant=v, kdist="normal")


# --- butterfly factors for N = 1024, B = 4096 --------------------------------

BUTTERFLY = [(2 ** (l - 1), 2, 2, 2 ** (10 - l)) for l in range(1, 11)]


@pytest.mark.parametrize("pattern", BUTTERFLY)
@pytest.mark.parametrize("layout", ["bsl", "bsf"])
def test_butterfly_single(pattern, layout):
    check(pattern, 4096, "f32", layout, cfg=2, kdist="normal")


@pytest.mark.parametrize("layout", ["bsl", "bsf"])
def test_butterfly_chain(layout):
    import torch
    batch = 4096
    pats = BUTTERFLY
    x = inputs.make_x(2, pats[-1], batch, "f32")
    kvs = [inputs.make_kv(2, p, batch, "f32", dist="normal", factor=f) for f, p in enumerate(pats)]
    kds = [to_device(k, "f32") for k in kvs]
    xd = to_device(inputs.to_layout(x, layout), "f32")
    y = ks.chain(xd, [(p, k) for p, k in zip(pats, kds)], layout=layout)
    torch.cuda.synchronize()
    y = inputs.from_layout(from_device(y, "f32"), layout)
    y64 = oracle.chain(pats, [inputs.to_f64(k, "f32") for k in kvs], x.astype(np.float64), batch, "bsf")
    assert rel_err(y, y64) <= TOL["f32"]


@pytest.mark.parametrize("layout", ["bsl", "bsf"])
def test_butterfly_chain_hadamard_bit_exact(layout):
    """All blocks [[1,1],[1,-1]] and inputs in {-1,0,1}: every intermediate is a
    small integer, exact in fp32, so the result must equal X H exactly."""
    import scipy.linalg
    import torch
    batch = 4096
    pats = BUTTERFLY
    x = inputs.make_x(2, pats[-1], batch, "f32", dist="sign")
    h2 = np.array([[1, 1], [1, -1]], dtype=np.float32)
    kds = [to_device(np.broadcast_to(h2, (p[0] * p[3], 2, 2)).copy(), "f32") for p in pats]
    xd = to_device(inputs.to_layout(x, layout), "f32")
    y = ks.chain(xd, list(zip(pats, kds)), layout=layout)
    torch.cuda.synchronize()
    y = inputs.from_layout(from_device(y, "f32"), layout)
    H = scipy.linalg.hadamard(1024).astype(np.float64)
    np.testing.assert_array_equal(y, x.astype(np.float64) @ H)


# --- Monarch factors for N = 1024, B = 16384 ---------------------------------

MONARCH = [(1, 32, 32, 32), (32, 32, 32, 1)]


@pytest.mark.parametrize("pattern", MONARCH)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
def test_monarch_single(pattern, dtype, layout):
    check(pattern, 16384, dtype, layout, cfg=3, kdist="normal_c")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
def test_monarch_chain(dtype, layout):
    import torch
    batch = 16384
    x = inputs.make_x(3, MONARCH[-1], batch, dtype)
    kvs = [inputs.make_kv(3, p, batch, dtype, dist="normal_c", factor=f) for f, p in enumerate(MONARCH)]
    xd = to_device(inputs.to_layout(x, layout), dtype)
    y = ks.chain(xd, [(p, to_device(k, dtype)) for p, k in zip(MONARCH, kvs)], layout=layout)
    torch.cuda.synchronize()
    y = inputs.from_layout(from_device(y, dtype).reshape(y.shape), layout)
    y64 = oracle.chain(MONARCH, [inputs.to_f64(k, dtype) for k in kvs], inputs.to_f64(x, dtype), batch, "bsf")
    assert rel_err(y, y64) <= TOL[dtype]


# --- Transformer-MLP-shaped layers, B = 25088 --------------------------------

MLP = [(6, 64, 16, 8), (6, 16, 64, 8)]


@pytest.mark.parametrize("pattern", MLP)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
def test_mlp(pattern, dtype, layout):
    check(pattern, 25088, dtype, layout, cfg=4)


# --- edge cases ---------------------------------------------------------------

@pytest.mark.parametrize("pattern", [(3, 5, 7, 2), (1, 17, 33, 3), (2, 1, 1, 5), (5, 3, 2, 1), (1, 20, 12, 1),
                                     (2, 16, 16, 3), (1, 48, 32, 5), (4, 32, 16, 1)])
@pytest.mark.parametrize("batch", [1, 37, 130])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
def test_odd_shapes(pattern, batch, layout):
    check(pattern, batch, "f32", layout, cfg=5)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("pattern", [(2, 4, 4, 2), (1, 32, 32, 4), (2, 2, 2, 8)])
def test_unaligned_buffers(dtype, layout, pattern):
    check(pattern, 64, dtype, layout, cfg=6, x_offset=1, y_offset=3)


@pytest.mark.parametrize("layout", ["bsf", "bsl"])
def test_empty_batch(layout):
    import torch
    kd = to_device(np.ones((4, 3, 3), dtype=np.float32), "f32")
    x = torch.empty(0, device="cuda")
    y = torch.empty(0, device="cuda")
    assert ks.ks_matmul(2, 3, 3, 2, kd, x, y, 0, layout, "f32") == 0


# --- the pattern sweep (every 13th pattern), sampled at full batch ------------

def sweep_patterns():
    return [(a, b, c, d) for a in (1, 2, 4, 8) for b in (16, 32, 48, 64, 96, 128) for c in (16, 32, 48, 64, 96, 128)
            for d in (1, 2, 4, 8, 16) if a * b * d <= 8192 and a * c * d <= 8192]


SWEEP_SAMPLE = sweep_patterns()[::13]


def check_sampled(pattern, batch, dtype, layout, cfg, nsample=4096, variant=None):
    """Run the full-size product on the GPU; compare a seeded sample of outputs
    (always including the first and last batch rows) with the oracle, computed
    one by one."""
    a, b, c, d = pattern
    M = a * b * d
    x, kv, x64, kv64 = case(cfg, pattern, batch, dtype, "normal", "normal")
    y = run_gpu(pattern, x, kv, batch, dtype, layout, variant=variant)
    rng = np.random.default_rng(zlib.crc32(repr((pattern, batch, dtype, layout)).encode()))
    bi = np.concatenate([rng.integers(0, batch, nsample), np.zeros(M // 4 + 1, np.int64),
                         np.full(M // 4 + 1, batch - 1)])
    mi = np.concatenate([rng.integers(0, M, nsample), rng.integers(0, M, 2 * (M // 4 + 1))])
    y64 = oracle.entries(pattern, kv64, x64, batch, "bsf", bi, mi)
    assert np.all(np.isfinite(y)), "unwritten (NaN) outputs"
    err = rel_err(y[bi, mi], y64)
    assert err <= TOL[dtype], "%s B=%d %s %s: sampled rel err %.3e" % (pattern, batch, dtype, layout, err)


@pytest.mark.parametrize("pattern", SWEEP_SAMPLE)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
def test_sweep_sample_b4096(pattern, dtype, layout):
    check_sampled(pattern, 4096, dtype, layout, cfg=7)


@pytest.mark.parametrize("pattern", SWEEP_SAMPLE[::3])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
def test_sweep_sample_b25088(pattern, dtype, layout):
    check_sampled(pattern, 25088, dtype, layout, cfg=7)


@pytest.mark.parametrize("pattern", SWEEP_SAMPLE)
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
def test_sweep_ragged_batch_full(pattern, dtype, layout):
    """Batches that leave a partial batch tile: full comparison."""
    batch = 104 if dtype == "f32" else 120  # multiples of the 16-byte vector width, not of the tile
    check(pattern, batch, dtype, layout, cfg=8, kdist="normal")



@pytest.mark.parametrize("pattern", MFMA_SHAPES)
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("batch", [256, 72, 68])
def test_direct_forced(pattern, dtype, layout, batch):
    """The register-direct MFMA kernel on every j-vector mode (d = 1, 2, 4 and
    d > 4), c % 32 == 16 tails of the 16-bit path, and ragged batches (68: the
    16-bit batch-size-last path with 4 instead of 8 batch entries per lane)."""
    check(pattern, batch, dtype, layout, cfg=11, variant=VARIANTS["direct"], kdist="normal")


@pytest.mark.parametrize("pattern", [s for s in MFMA_SHAPES if s[3] <= 16])
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("batch", [256, 72, 1000])
def test_staged_forced(pattern, dtype, layout, batch):
    """The LDS-staged MFMA kernel: the same shapes, ragged batches, several
    stages of l (c up to 128) and the 16-bit c % 32 == 16 tail."""
    if layout == "bsl" and batch % (4 if dtype == "f32" else 8):
        pytest.skip("BSL staging needs the batch to be a multiple of a 16-byte unit")
    check(pattern, batch, dtype, layout, cfg=12, variant=VARIANTS["staged"], kdist="normal")




@pytest.mark.parametrize("pattern", DMA_SHAPES)
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("batch", [256, 72, 1000])
def test_dma_forced(pattern, dtype, batch):
    """The LDS-DMA kernel (batch-size-first, d in {4, 8, 16}): strided and
    contiguous j-vectors, one to eight stages of l (the 1-, 2- and 3-stage
    tails of its pipeline), the 16-bit c % 32 == 16 lane depth, ragged
    batches."""
    check(pattern, batch, dtype, "bsf", cfg=14, variant=VARIANTS["dma"], kdist="normal")


@pytest.mark.parametrize("pattern", DMA_ROW_GROUP_SHAPES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("batch", [4096, 4000])
def test_dma_row_groups(pattern, dtype, batch):
    """The LDS-DMA kernel with several 16-row groups per wavefront (each K
    operand reused for 32 or 64 batch rows), full and ragged last tiles."""
    check(pattern, batch, dtype, "bsf", cfg=16, variant=VARIANTS["dma"], kdist="normal")


@pytest.mark.parametrize("pattern", [(6, 64, 16, 8), (2, 128, 128, 16), (8, 16, 128, 4)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_dma_full_batch(pattern, dtype):
    """The LDS-DMA kernel at the full batch of 25088 rows (thousands of tiles,
    XCD remap)."""
    check(pattern, 25088, dtype, "bsf", cfg=15, variant=VARIANTS["dma"], kdist="normal")


# Batch-size-last DMA kernel: b covers MT = 1..4 (fp32) and the RS/KGW splits,
# c gives 1, 2, 3 and 8 stages of 16 (fp32) or 1, 2, 4 of 32 (16-bit).
DMA_BSL_SHAPES = [(1, 16, 16, 1), (2, 32, 32, 4), (1, 48, 48, 2), (3, 64, 64, 1), (1, 96, 128, 2),
                  (1, 128, 96, 1), (2, 64, 32, 8)]


@pytest.mark.parametrize("pattern", DMA_BSL_SHAPES)
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("batch", [64, 200, 1000])
def test_dma_bsl_forced(pattern, dtype, batch):
    """The batch-size-last LDS-DMA kernel forced: every M-tile count and
    batch-group split the planner can pick, one to eight stages of l, batches
    that end inside a tile (columns beyond the batch read clamped units and
    are not stored)."""
    a, b, c, d = pattern
    if dtype != "f32" and c % 32:
        pytest.skip("16-bit stages hold 32 values of l")
    check(pattern, batch, dtype, "bsl", cfg=17, variant=VARIANTS["dma"], kdist="normal")


@pytest.mark.parametrize("pattern", [(8, 96, 64, 8), (1, 128, 128, 16), (4, 16, 64, 8)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_dma_bsl_full_batch(pattern, dtype):
    """The batch-size-last LDS-DMA kernel at the full batch of 25088 entries
    (thousands of tiles, XCD remap)."""
    check(pattern, 25088, dtype, "bsl", cfg=18, variant=VARIANTS["dma"], kdist="normal")


@pytest.mark.parametrize("pattern", [(1, 32, 32, 32), (6, 64, 16, 8), (4, 96, 48, 2)])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
def test_every_kernel_family_against_oracle(pattern, layout):
    """The generic, register-direct, LDS-staged and LDS-DMA (batch-size-first
    with d <= 16, and batch-size-last) kernels, each forced on the same inputs
    and each compared with the fp64 oracle."""
    names = ["generic", "direct"]
    if layout == "bsl" or pattern[3] <= 16:  # BSF staging takes d <= 16 (at most 4 j-groups per tile)
        names.append("staged")
    if layout == "bsl" or pattern[3] in (1, 2, 4, 8, 16):
        names.append("dma")
    for name in names:
        check(pattern, 512, "f32", layout, cfg=10, variant=VARIANTS[name], kdist="normal")


def test_wrappers_reject_mismatched_tensors():
    """matmul() and chain() check sizes, dtypes, devices and contiguity on the
    host: the C ABI sees raw pointers only, so a mismatch must never reach it."""
    import torch
    dev = "cuda"
    kv = torch.randn(2 * 2 * 4 * 4, device=dev)
    x = torch.randn(16, 32, device=dev)  # BSL (N, batch), N = 16
    assert ks.matmul(x, kv, (2, 4, 4, 2), "bsl").shape == (16, 32)
    with pytest.raises(ValueError):
        ks.matmul(x, kv[:-1], (2, 4, 4, 2), "bsl")                      # K too small
    with pytest.raises(TypeError):
        ks.matmul(x, kv.to(torch.bfloat16), (2, 4, 4, 2), "bsl")        # K dtype
    with pytest.raises(ValueError):
        ks.matmul(x, kv, (2, 4, 4, 2), "bsl", out=torch.empty(16, 31, device=dev))  # out too small
    with pytest.raises(TypeError):
        ks.matmul(x, kv, (2, 4, 4, 2), "bsl", out=torch.empty(16, 32, device=dev, dtype=torch.float16))
    with pytest.raises(ValueError):
        ks.matmul(x, kv, (2, 4, 4, 2), "bsl", out=torch.empty(32, 16, device=dev).t())  # not contiguous
    with pytest.raises(ValueError):
        ks.matmul(torch.randn(15, device=dev), kv, (2, 4, 4, 2), "bsl")  # not a multiple of N
    with pytest.raises(ValueError):
        ks.matmul(x, kv, (2, 4, 4, 2), "bsf")                           # (16, 32) is not (batch, 16)
    f = [((1, 4, 4, 4), torch.randn(64, device=dev)), ((4, 4, 4, 1), torch.randn(64, device=dev))]
    assert ks.chain(x, f, "bsl").shape == (16, 32)
    with pytest.raises(ValueError):
        ks.chain(x, [f[0], ((4, 4, 4, 1), torch.randn(63, device=dev))], "bsl")
    with pytest.raises(ValueError):
        ks.chain(x, [f[0], ((4, 4, 3, 1), torch.randn(48, device=dev))], "bsl")  # X width 12 != 16
    with pytest.raises(ValueError):
        ks.chain(x, [((1, 4, 4, 2), torch.randn(32, device=dev)), f[1]], "bsl")  # 8 != 16


MASKED_CASES = [((1, 64, 64, 1), 25087, "bsl"), ((1, 24, 24, 8), 4096, "bsl"), ((1, 24, 24, 8), 4096, "bsf"),
                ((6, 64, 16, 8), 25087, "bsl"), ((6, 64, 16, 8), 25090, "bsl"), ((1, 100, 36, 2), 1001, "bsf"),
                ((3, 20, 40, 1), 37, "bsl"), ((4, 16, 17, 2), 130, "bsf"), ((1, 33, 16, 5), 1001, "bsl")]


@pytest.mark.parametrize("case_", MASKED_CASES, ids=[str(c) for c in MASKED_CASES])
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_masked_kernel(case_, dtype):
    """The masked MFMA kernel (zero-padded tiles, narrow accesses): b or c not
    a multiple of 16, batch-size-last batches that are not a multiple of the
    vector; the whole output against the oracle."""
    pattern, batch, layout = case_
    desc = ks.ks_plan_describe(*pattern, batch, layout, dtype)
    assert "name=masked" in desc, desc
    check(pattern, batch, dtype, layout, cfg=17, kdist="normal")


@pytest.mark.parametrize("pattern", [(1, 32, 32, 4), (6, 64, 16, 8), (1, 24, 24, 8)])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("offsets", [(1, 3), (2, 2), (4, 0)])
def test_offset_buffers_run_masked(pattern, layout, dtype, offsets):
    """Buffers shifted off 16-byte alignment by 1, 2 or 4 elements: the masked
    kernel at the access width their alignment allows."""
    check(pattern, 256, dtype, layout, cfg=18, x_offset=offsets[0], y_offset=offsets[1], kdist="normal")


# --- bias + GELU epilogue (ks_matmul_bias_act) --------------------------------

EPI_CASES = [("generic", (2, 4, 4, 2), "bsl", 40), ("valu_bsl", (2, 4, 4, 2), "bsl", 64),
             ("valu_bsf", (4, 2, 2, 8), "bsf", 50), ("direct", (6, 64, 16, 8), "bsl", 256),
             ("direct", (2, 48, 80, 2), "bsf", 72), ("staged", (1, 32, 32, 32), "bsf", 100),
             ("dma", (6, 64, 16, 8), "bsf", 1000), ("dma", (4, 48, 96, 4), "bsf", 72),
             ("dma", (2, 64, 64, 4), "bsl", 200), ("dma", (1, 128, 32, 2), "bsl", 1000),
             ("masked", (1, 24, 24, 8), "bsl", 100), ("masked", (1, 100, 36, 2), "bsf", 37),
             (None, (6, 64, 16, 8), "bsl", 25088), (None, (6, 16, 64, 8), "bsf", 25088)]
VARIANTS["masked"] = 7


@pytest.mark.parametrize("case_", EPI_CASES, ids=["%s-%s-%s-%d" % c for c in EPI_CASES])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("epi", ["bias", "bias_gelu", "gelu"])
def test_bias_gelu_epilogue(case_, dtype, epi):
    """Y = act(X K^T + bias) from every kernel family's epilogue against the
    oracle's matmul followed by its bias/GELU step."""
    import torch
    variant, pattern, layout, batch = case_
    a, b, c, d = pattern
    M = a * b * d
    x, kv, x64, kv64 = case(19, pattern, batch, dtype, "normal", "normal")
    bias = inputs.round_to(np.random.default_rng(M + batch).standard_normal(M), dtype) if epi != "gelu" else None
    act = "gelu" if "gelu" in epi else None
    xd = to_device(inputs.to_layout(x, layout), dtype)
    kd = to_device(kv, dtype)
    bd = to_device(bias, dtype) if bias is not None else None
    yd = nan_tensor((batch * M,), dtype)
    ks.ks_force_variant(None if variant is None else VARIANTS[variant])
    try:
        desc = ks.ks_plan_describe(a, b, c, d, batch, layout, dtype)
        ks.ks_matmul_bias_act(a, b, c, d, kd, bd, act, xd, yd, batch, layout, dtype)
    finally:
        ks.ks_force_variant(None)
    torch.cuda.synchronize()
    y = inputs.from_layout(from_device(yd, dtype).reshape((batch, M) if layout == "bsf" else (M, batch)), layout)
    y64 = oracle.bias_act(oracle.matmul(pattern, kv64, x64, batch, "bsf"),
                          None if bias is None else inputs.to_f64(bias, dtype), "bsf", act)
    err = rel_err(y, y64)
    assert err <= TOL[dtype], "%s %s: rel err %.3e [%s]" % (case_, epi, err, desc)


def test_bias_act_rejects_bad_arguments():
    import torch
    kd = torch.ones(64, device="cuda")
    x = torch.ones(16, 8, device="cuda")
    y = torch.empty(16, 8, device="cuda")
    assert ks.ks_matmul_bias_act(2, 4, 4, 2, kd, None, 2, x, y, 8, "bsl", "f32", check=False) == 5  # unknown act
    assert ks.ks_matmul_bias_act(2, 4, 4, 2, kd, y, 0, x, y, 8, "bsl", "f32", check=False) == 4     # bias aliases Y


# Calls whose last workgroup has wavefronts past the last work item (the item
# count is not a multiple of the wavefronts per workgroup): those wavefronts
# run the last item's loads and MFMAs and must store nothing; and DMA tiles
# that end past the batch (their rows or columns beyond it are loaded from
# clamped addresses and not stored).
SPARE_WAVE_CASES = [((1, 16, 16, 1), 72, "f32", "bsf", "direct"), ((1, 16, 16, 1), 200, "bf16", "bsl", "direct"),
                    ((3, 48, 32, 1), 40, "bf16", "bsf", "direct"), ((1, 32, 16, 2), 40, "f32", "bsf", "direct"),
                    ((1, 40, 24, 1), 100, "f32", "bsl", "masked"), ((1, 100, 36, 2), 37, "bf16", "bsf", "masked"),
                    ((6, 64, 16, 8), 1000, "f32", "bsf", "dma"), ((2, 64, 64, 4), 200, "f32", "bsl", "dma"),
                    ((1, 64, 64, 4), 1000, "bf16", "bsl", "dma")]


@pytest.mark.parametrize("case_", SPARE_WAVE_CASES, ids=["%s-%d-%s-%s" % c[:4] for c in SPARE_WAVE_CASES])
def test_spare_waves_store_nothing(case_):
    """Y between two guard regions of a sentinel value: the guards are intact
    after the call (nothing is written before or after Y) and Y matches the
    oracle, for plans whose last workgroup has spare wavefronts or whose last
    DMA tile ends past the batch."""
    import torch
    pattern, batch, dtype, layout, name = case_
    a, b, c, d = pattern
    M = a * b * d
    desc = ks.ks_plan_describe(*pattern, batch, layout, dtype)
    assert "name=%s" % name in desc, desc
    x, kv, _, _ = case(19, pattern, batch, dtype, "normal", "normal")
    xd = to_device(inputs.to_layout(x, layout).reshape(-1), dtype)
    kd = to_device(kv, dtype)
    guard, sentinel = 4096, -7.5  # exact in every storage type
    buf = torch.full((guard + batch * M + guard,), sentinel, dtype=torch_dtype(dtype), device="cuda")
    y_view = buf[guard:guard + batch * M]
    y_view.fill_(float("nan"))
    ks.ks_matmul(a, b, c, d, kd, xd, y_view, batch, layout, dtype)
    torch.cuda.synchronize()
    host = buf.float().cpu().numpy()
    assert np.all(host[:guard] == sentinel) and np.all(host[guard + batch * M:] == sentinel), "write outside Y"
    y = from_device(y_view, dtype).reshape((batch, M) if layout == "bsf" else (M, batch))
    err = rel_err(inputs.from_layout(y, layout), oracle_y(19, pattern, batch, dtype, "normal", "normal"))
    assert err <= TOL[dtype], err
