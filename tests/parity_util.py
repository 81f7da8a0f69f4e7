"""Helpers for the GPU parity tests: move seeded storage arrays to the device,
bring results back as exact float64, and measure errors against the oracle."""
import functools

import numpy as np

import oracle
from paper_2405_15013_amd import inputs

# Normwise tolerance max|Y - Y64| / max|Y64| against the fp64 oracle: fp32
# storage with fp32 accumulation, and 16-bit storage with fp32 accumulation
# (one final rounding to a 2^-8 / 2^-11 ulp format dominates).
TOL = {"f32": 1e-5, "bf16": 1e-2, "f16": 1e-2, "fp8": 1e-2}  # fp8: E4M3 inputs, bf16 output


def torch_dtype(dtype):
    import torch
    return {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]


def to_device(arr, dtype, device="cuda"):
    import torch
    a = np.ascontiguousarray(arr)
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    if dtype == "fp8":
        return torch.from_numpy(a.view(np.uint8)).to(device).view(torch.float8_e4m3fn)
    return torch.from_numpy(a).to(device)


def from_device(t, dtype):
    import torch
    if dtype == "bf16":
        bits = t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        return inputs.to_f64(bits, "bf16")
    return t.detach().cpu().numpy().astype(np.float64)


def nan_tensor(shape, dtype, device="cuda"):
    import torch
    return torch.full(shape, float("nan"), dtype=torch_dtype(dtype), device=device)


def rel_err(y, y64):
    y = np.asarray(y, dtype=np.float64)
    y64 = np.asarray(y64, dtype=np.float64)
    if y64.size == 0:
        return 0.0
    scale = np.max(np.abs(y64))
    if scale == 0:
        scale = 1.0
    diff = np.abs(y - y64)
    if np.isnan(diff).any():
        return float("inf")
    return float(np.max(diff) / scale)


@functools.lru_cache(maxsize=16)
def case(cfg, pattern, batch, dtype, xdist="normal", kdist="uniform_c"):
    """Seeded storage arrays (logical X, packed Kv) plus their exact float64 views."""
    x = inputs.make_x(cfg, pattern, batch, dtype, dist=xdist)
    kv = inputs.make_kv(cfg, pattern, batch, dtype, dist=kdist)
    return x, kv, inputs.to_f64(x, dtype), inputs.to_f64(kv, dtype)


@functools.lru_cache(maxsize=16)
def oracle_y(cfg, pattern, batch, dtype, xdist="normal", kdist="uniform_c"):
    """fp64 oracle result (logical (batch, M) order) for `case(...)`."""
    _, _, x64, kv64 = case(cfg, pattern, batch, dtype, xdist, kdist)
    return oracle.matmul(pattern, kv64, x64, batch, "bsf")
