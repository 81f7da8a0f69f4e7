"""ks_chain_noalloc (the chain entry point that allocates nothing: its
intermediates live in the library's fixed per-GPU scratch array) against
ks_chain with a caller workspace, through the C ABI, on the same inputs:
two calls in a row, the second on a smaller input, each output compared with
ks_chain's and with the fp64 oracle."""
import numpy as np
import pytest

import oracle
import paper_2405_15013_amd as ks
from paper_2405_15013_amd import inputs
from parity_util import TOL, from_device, nan_tensor, rel_err, to_device

pytestmark = pytest.mark.gpu

BUTTERFLY = [(2 ** (l - 1), 2, 2, 2 ** (10 - l)) for l in range(1, 11)]
MONARCH = [(1, 32, 32, 32), (32, 32, 32, 1)]


def _run_both(pats, batch, dtype, layout, cfg):
    import torch
    x = inputs.make_x(cfg, pats[-1], batch, dtype)
    kvs = [inputs.make_kv(cfg, p, batch, dtype, dist="normal_c", factor=f) for f, p in enumerate(pats)]
    factors = [(p, to_device(k, dtype)) for p, k in zip(pats, kvs)]
    xd = to_device(inputs.to_layout(x, layout), dtype)
    M = pats[0][0] * pats[0][1] * pats[0][3]
    need = ks.ks_chain_workspace_bytes(factors, batch, dtype)
    assert 0 < need <= ks.ks_chain_noalloc_max_workspace()
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    y_ref = nan_tensor((batch * M,), dtype)
    ks.ks_chain(factors, xd, y_ref, batch, layout, dtype, ws, need)
    y_na = nan_tensor((batch * M,), dtype)
    ks.ks_chain_noalloc(factors, xd, y_na, batch, layout, dtype)
    torch.cuda.synchronize()
    a = from_device(y_na, dtype)
    b = from_device(y_ref, dtype)
    assert np.all(np.isfinite(a)), "unwritten outputs"
    # Same kernels on the same inputs: the results must agree exactly.
    np.testing.assert_array_equal(a, b)
    shape = (batch, M) if layout == "bsf" else (M, batch)
    y64 = oracle.chain(pats, [inputs.to_f64(k, dtype) for k in kvs], inputs.to_f64(x, dtype), batch, "bsf")
    assert rel_err(inputs.from_layout(a.reshape(shape), layout), y64) <= TOL[dtype]


@pytest.mark.parametrize("layout", ["bsl", "bsf"])
def test_noalloc_matches_workspace_chain_two_calls(layout):
    # The butterfly chain would run fused (no intermediates in memory): run
    # chains factor by factor on this thread, so both calls use the array.
    ks.ks_force_chain_fusion(0)
    try:
        # first call: butterfly 10-chain at batch 4096 (two 16 MiB intermediates)
        _run_both(BUTTERFLY, 4096, "f32", layout, cfg=31)
        # second call, smaller: Monarch 2-chain at batch 520 in bf16 (the array
        # still holds the first call's intermediates)
        _run_both(MONARCH, 520, "bf16", layout, cfg=32)
    finally:
        ks.ks_force_chain_fusion(None)


def test_noalloc_rejects_chains_beyond_the_scratch_size():
    import torch
    kds = [torch.zeros(p[0] * p[1] * p[2] * p[3], device="cuda") for p in MONARCH]
    batch = 32768  # one intermediate of 128 MiB
    # factor by factor (the fused Monarch chain needs no intermediates), so the
    # call is rejected before any launch
    ks.ks_force_chain_fusion(0)
    try:
        assert ks.ks_chain_workspace_bytes(list(zip(MONARCH, kds)), batch, "f32") == 128 << 20
        st = ks.ks_chain_noalloc(list(zip(MONARCH, kds)), 1 << 40, 2 << 40, batch, "bsl", "f32", check=False)
    finally:
        ks.ks_force_chain_fusion(None)
    assert ks.STATUS_NAMES[st] == "KS_ERR_SCRATCH_LIMIT"
