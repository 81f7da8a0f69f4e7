"""Host-only checks of the C ABI (no GPU needed): the library loads, exports
every function include/ks.h declares, and rejects bad arguments before
enqueueing anything (every rejected call below returns without touching the
HIP runtime, so these run on a machine without a GPU)."""
import ctypes
import os
import re

import pytest

import paper_2405_15013_amd as ks

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# Stand-in device addresses: never dereferenced, because every call below is
# rejected (or has batch 0) before anything is enqueued.
P0 = 1 << 44
P1 = P0 + (1 << 40)
P2 = P0 + (2 << 40)


def header_functions():
    with open(os.path.join(ROOT, "include", "ks.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ks_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = ks.load_library()
    declared = header_functions()
    assert set(declared) == set(ks.EXPORTED_SYMBOLS)
    for name in declared:
        assert hasattr(lib, name), name
        assert ctypes.cast(getattr(lib, name), ctypes.c_void_p).value


def test_status_strings():
    for code, name in ks.STATUS_NAMES.items():
        assert ks.ks_status_string(code).startswith(name)


@pytest.mark.parametrize("pattern", [(0, 2, 2, 2), (2, 0, 2, 2), (2, 2, -1, 2), (2, 2, 2, 0),
                                     (1 << 40, 1 << 40, 2, 2)])
def test_invalid_pattern(pattern):
    st = ks.ks_matmul(*pattern, P0, P1, P2, 8, ks.BSL, ks.F32, stream=0, check=False)
    assert ks.STATUS_NAMES[st] == "KS_ERR_INVALID_PATTERN"


def test_invalid_args():
    assert ks.ks_matmul(2, 2, 2, 2, P0, P1, P2, -1, ks.BSL, ks.F32, stream=0, check=False) == 2
    assert ks.ks_matmul(2, 2, 2, 2, None, P1, P2, 8, ks.BSL, ks.F32, stream=0, check=False) == 2
    assert ks.ks_matmul(2, 2, 2, 2, P0, None, P2, 8, ks.BSL, ks.F32, stream=0, check=False) == 2
    assert ks.ks_matmul(2, 2, 2, 2, P0, P1, None, 8, ks.BSL, ks.F32, stream=0, check=False) == 2


def test_unsupported_layout_dtype_and_size():
    assert ks.ks_matmul(2, 2, 2, 2, P0, P1, P2, 8, 7, ks.F32, stream=0, check=False) == 5
    assert ks.ks_matmul(2, 2, 2, 2, P0, P1, P2, 8, ks.BSL, 9, stream=0, check=False) == 5
    # batch * N >= 2^31 elements
    assert ks.ks_matmul(1, 64, 64, 1, P0, P1, P2, 1 << 25, ks.BSL, ks.F32, stream=0, check=False) == 5


def test_empty_batch_is_ok_without_buffers():
    assert ks.ks_matmul(2, 3, 4, 5, P0, None, None, 0, ks.BSF, ks.BF16, stream=0, check=False) == 0


def test_alias_detected():
    # Y overlapping X, and Y overlapping the packed values.
    assert ks.ks_matmul(2, 4, 4, 2, P0, P1, P1 + 64, 32, ks.BSL, ks.F32, stream=0, check=False) == 4
    assert ks.ks_matmul(2, 4, 4, 2, P0, P1, P0 + 4, 32, ks.BSL, ks.F32, stream=0, check=False) == 4


@pytest.fixture
def factor_by_factor():
    """Chains below run factor by factor (no fused kernel), so their
    workspace checks apply; every call is rejected before any launch."""
    ks.ks_force_chain_fusion(0)
    yield
    ks.ks_force_chain_fusion(None)


def test_chain_errors(factor_by_factor):
    f_ok = [((1, 4, 4, 4), P0), ((4, 4, 4, 1), P0 + 4096)]
    f_bad = [((1, 4, 4, 4), P0), ((1, 3, 3, 1), P0 + 4096)]
    assert ks.ks_chain_workspace_bytes(f_bad, 8, ks.F32) == 0
    assert ks.ks_chain(f_bad, P1, P2, 8, ks.BSL, ks.F32, None, 0, stream=0, check=False) == 3
    need = ks.ks_chain_workspace_bytes(f_ok, 8, ks.F32)
    assert need >= 16 * 8 * 4
    assert ks.ks_chain(f_ok, P1, P2, 8, ks.BSL, ks.F32, None, 0, stream=0, check=False) == 6
    assert ks.ks_chain(f_ok, P1, P2, 8, ks.BSL, ks.F32, P0 + (3 << 40), need - 1, stream=0, check=False) == 6
    # workspace overlapping X
    assert ks.ks_chain(f_ok, P1, P2, 8, ks.BSL, ks.F32, P1 + 16, need, stream=0, check=False) == 4
    assert ks.ks_chain([], P1, P2, 8, ks.BSL, ks.F32, None, 0, stream=0, check=False) == 2
    # three factors need two ping-pong buffers
    f3 = [((1, 4, 4, 4), P0), ((4, 4, 4, 1), P0 + 4096), ((2, 4, 4, 2), P0 + 8192)]
    assert ks.ks_chain_workspace_bytes(f3, 8, ks.F32) == 2 * need


def test_chain_empty_batch_ok():
    f_ok = [((1, 4, 4, 4), P0), ((4, 4, 4, 1), P0 + 4096)]
    assert ks.ks_chain(f_ok, None, None, 0, ks.BSL, ks.F32, None, 0, stream=0, check=False) == 0


def test_plan_describe_picks_expected_families():
    # butterfly factor, batch-size-last -> VALU streaming kernel
    assert "name=valu_bsl" in ks.ks_plan_describe(4, 2, 2, 128, 4096, "bsl", "f32")
    assert "name=valu_bsf" in ks.ks_plan_describe(4, 2, 2, 128, 4096, "bsf", "f32")
    # large odd blocks run on the masked MFMA kernel (zero-padded tiles)
    assert "name=masked" in ks.ks_plan_describe(1, 17, 19, 3, 64, "bsf", "f32")
    assert ks.ks_plan_describe(1, 4, 4, 1, 0, "bsf", "f32") == "empty"


def test_wrappers_reject_host_tensors():
    """The tensor-level wrappers take device tensors only (there is no CPU
    path); the check runs before the library is called."""
    import torch
    with pytest.raises(ValueError):
        ks.matmul(torch.randn(16, 8), torch.randn(64), (2, 4, 4, 2), "bsl")
    with pytest.raises(ValueError):
        ks.chain(torch.randn(16, 8), [((2, 4, 4, 2), torch.randn(64))], "bsl")


def test_chain_noalloc_host_errors(factor_by_factor):
    """ks_chain_noalloc checks its arguments like ks_chain, and rejects chains
    whose intermediates exceed its fixed scratch array, before touching the
    GPU."""
    f_ok = [((1, 4, 4, 4), P0), ((4, 4, 4, 1), P0 + 4096)]
    f_bad = [((1, 4, 4, 4), P0), ((1, 3, 3, 1), P0 + 4096)]
    assert ks.ks_chain_noalloc_max_workspace() == 64 << 20
    assert ks.ks_chain_noalloc(f_bad, P1, P2, 8, ks.BSL, ks.F32, stream=0, check=False) == 3
    assert ks.ks_chain_noalloc(f_ok, None, None, 0, ks.BSL, ks.F32, stream=0, check=False) == 0
    # 16 x (1 << 21) fp32 intermediates: 128 MiB > 64 MiB
    st = ks.ks_chain_noalloc(f_ok, P1, P2, 1 << 21, ks.BSL, ks.F32, stream=0, check=False)
    assert ks.STATUS_NAMES[st] == "KS_ERR_SCRATCH_LIMIT"
