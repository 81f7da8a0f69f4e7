"""GPU parity of the FP8 path (KS_FP8_E4M3: X and K_values in OCP E4M3, Y in
bfloat16, fp32 accumulation on the fp8 MFMAs) against the fp64 oracle on the
same E4M3-rounded inputs; whole outputs NaN-prefilled."""
import numpy as np
import pytest

import oracle
import paper_2405_15013_amd as ks
from paper_2405_15013_amd import inputs
from parity_util import TOL, from_device, nan_tensor, rel_err, to_device

pytestmark = pytest.mark.gpu


def run_fp8(pattern, batch, layout, cfg=51, bias=False, act=None, x_offset=0, y_offset=0):
    import torch
    a, b, c, d = pattern
    M = a * b * d
    x = inputs.make_x(cfg, pattern, batch, "fp8")
    kv = inputs.make_kv(cfg, pattern, batch, "fp8", dist="normal")
    bv = inputs.round_to(np.random.default_rng(M).standard_normal(M), "bf16") if bias else None
    xflat = inputs.to_layout(x, layout).reshape(-1)
    xd = to_device(np.concatenate([np.zeros(x_offset, np.uint8), xflat]), "fp8")[x_offset:]
    yd = nan_tensor((y_offset + batch * M,), "bf16")[y_offset:]
    desc = ks.ks_plan_describe(a, b, c, d, batch, layout, "fp8")
    assert "name=fp8" in desc, desc
    ks.ks_matmul_bias_act(a, b, c, d, to_device(kv, "fp8"), None if bv is None else to_device(bv, "bf16"), act,
                          xd, yd, batch, layout, "fp8")
    torch.cuda.synchronize()
    y = inputs.from_layout(from_device(yd, "bf16").reshape((batch, M) if layout == "bsf" else (M, batch)), layout)
    y64 = oracle.matmul(pattern, inputs.to_f64(kv, "fp8"), inputs.to_f64(x, "fp8"), batch, "bsf")
    if bias or act:
        y64 = oracle.bias_act(y64, None if bv is None else inputs.to_f64(bv, "bf16"), "bsf", act)
    assert np.all(np.isfinite(y)), "unwritten outputs"
    err = rel_err(y, y64)
    assert err <= TOL["fp8"], "%s B=%d %s: rel err %.3e [%s]" % (pattern, batch, layout, err, desc)


SHAPES = [(1, 64, 64, 1), (6, 64, 16, 8), (6, 16, 64, 8), (1, 32, 32, 32), (32, 32, 32, 1), (2, 128, 128, 4),
          (8, 16, 96, 2), (4, 48, 32, 16), (1, 24, 24, 8), (1, 17, 33, 3),
          (2, 17, 24, 8), (3, 48, 8, 8),  # d = 8 row runs with padded k rows / c = 8
          (2, 20, 8, 4), (3, 18, 16, 2)]  # per-lane runs: padded k rows (b = 20), b not a multiple of 4


@pytest.mark.parametrize("pattern", SHAPES)
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("batch", [4096, 1001])
def test_fp8_against_oracle(pattern, layout, batch):
    run_fp8(pattern, batch, layout)


@pytest.mark.parametrize("pattern", [(6, 64, 16, 8), (6, 16, 64, 8)])
@pytest.mark.parametrize("layout", ["bsf", "bsl"])
def test_fp8_mlp_full_batch(pattern, layout):
    run_fp8(pattern, 25088, layout, cfg=52)


@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("epi", [(True, None), (True, "gelu")])
def test_fp8_bias_gelu(layout, epi):
    run_fp8((6, 64, 16, 8), 4096, layout, cfg=53, bias=epi[0], act=epi[1])


@pytest.mark.parametrize("layout", ["bsf", "bsl"])
@pytest.mark.parametrize("offsets", [(1, 1), (2, 4), (4, 0)])
def test_fp8_offset_buffers(layout, offsets):
    run_fp8((1, 32, 32, 4), 512, layout, cfg=54, x_offset=offsets[0], y_offset=offsets[1])


def test_fp8_chain_unsupported():
    import torch
    f = [((1, 4, 4, 4), torch.zeros(64, dtype=torch.uint8, device="cuda")),
         ((4, 4, 4, 1), torch.zeros(64, dtype=torch.uint8, device="cuda"))]
    assert ks.ks_chain(f, 1 << 40, 2 << 40, 8, "bsl", "fp8", None, 0, check=False) == 5
