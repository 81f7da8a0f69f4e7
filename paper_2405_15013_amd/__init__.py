"""MI355X (gfx950) Kronecker-sparse matrix multiplication.

Python binding of libks.so.  The functions named like the C ABI
(``ks_matmul``, ``ks_chain``, ...) only marshal arguments; every step of the
computation runs in the library's HIP kernels.  PyTorch is used for device
buffers and streams only.  If libks.so is missing the first call raises
``RuntimeError``; there is no CPU fallback.

Semantics (paper Section 1, Definition 2.1, Section 2.2 layouts): for a KS
factor K of pattern (a, b, c, d) with packed values ``K_values`` of shape
(a*d, b, c), ``ks_matmul`` computes Y = X K^T for a batch in batch-size-first
(X: (batch, a*c*d)) or batch-size-last (X: (a*c*d, batch)) layout.
"""
import ctypes
import os

__all__ = [
    "BSF", "BSL", "F32", "BF16", "F16", "FP8", "KsError",
    "ks_matmul", "ks_chain", "ks_chain_workspace_bytes", "ks_chain_noalloc", "ks_chain_noalloc_max_workspace",
    "ks_status_string",
    "ks_last_hip_error", "ks_plan_describe", "ks_force_variant", "ks_plan_verify",
    "ks_chain_describe", "ks_force_chain_fusion", "ks_chain_verify", "ks_matmul_bias_act",
    "ACT_NONE", "ACT_GELU", "matmul", "chain", "library_path", "load_library", "EXPORTED_SYMBOLS",
]

BSF, BSL = 0, 1
F32, BF16, F16, FP8 = 0, 1, 2, 3
ACT_NONE, ACT_GELU = 0, 1

KS_OK = 0
STATUS_NAMES = {
    0: "KS_OK", 1: "KS_ERR_INVALID_PATTERN", 2: "KS_ERR_INVALID_ARG", 3: "KS_ERR_DIM_MISMATCH",
    4: "KS_ERR_ALIAS", 5: "KS_ERR_UNSUPPORTED", 6: "KS_ERR_WORKSPACE", 7: "KS_ERR_HIP",
    8: "KS_ERR_SCRATCH_LIMIT",
}

# Every function declared in include/ks.h.
EXPORTED_SYMBOLS = (
    "ks_matmul", "ks_chain_workspace_bytes", "ks_chain", "ks_chain_noalloc", "ks_chain_noalloc_max_workspace",
    "ks_status_string", "ks_last_hip_error", "ks_plan_describe", "ks_force_variant", "ks_plan_verify",
    "ks_chain_describe", "ks_force_chain_fusion", "ks_chain_verify", "ks_matmul_bias_act",
)

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libks.so")
_lib = None


class KsError(RuntimeError):
    """A libks call returned a status other than KS_OK."""

    def __init__(self, status, where):
        self.status = int(status)
        self.name = STATUS_NAMES.get(self.status, str(status))
        msg = "%s failed: %s" % (where, ks_status_string(self.status))
        if self.status == 7:
            msg += " (hipError_t %d)" % ks_last_hip_error()
        super().__init__(msg)


class _Factor(ctypes.Structure):
    _fields_ = [("a", ctypes.c_int64), ("b", ctypes.c_int64), ("c", ctypes.c_int64),
                ("d", ctypes.c_int64), ("K_values", ctypes.c_void_p)]


def library_path():
    return _LIB_PATH


def load_library():
    """Load libks.so (raises RuntimeError if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError("libks.so is not built (expected at %s); run "
                           "`python -m paper_2405_15013_amd.build`" % _LIB_PATH)
    # libks.so and PyTorch must share one HIP runtime (the buffers and streams
    # passed in are PyTorch's).  PyTorch bundles its own libamdhip64 under the
    # same soname, and whichever is loaded first serves both, so PyTorch is
    # loaded before the library.
    import torch  # noqa: F401
    lib = ctypes.CDLL(_LIB_PATH)
    i64, vp, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    lib.ks_matmul.argtypes = [i64, i64, i64, i64, vp, vp, vp, i64, ci, ci, vp]
    lib.ks_matmul.restype = ci
    lib.ks_matmul_bias_act.argtypes = [i64, i64, i64, i64, vp, vp, ci, vp, vp, i64, ci, ci, vp]
    lib.ks_matmul_bias_act.restype = ci
    lib.ks_chain_workspace_bytes.argtypes = [ctypes.POINTER(_Factor), ci, i64, ci]
    lib.ks_chain_workspace_bytes.restype = ctypes.c_size_t
    lib.ks_chain.argtypes = [ctypes.POINTER(_Factor), ci, vp, vp, i64, ci, ci, vp, ctypes.c_size_t, vp]
    lib.ks_chain.restype = ci
    lib.ks_chain_noalloc.argtypes = [ctypes.POINTER(_Factor), ci, vp, vp, i64, ci, ci, vp]
    lib.ks_chain_noalloc.restype = ci
    lib.ks_chain_noalloc_max_workspace.argtypes = []
    lib.ks_chain_noalloc_max_workspace.restype = ctypes.c_size_t
    lib.ks_chain_describe.argtypes = [ctypes.POINTER(_Factor), ci, i64, ci, ci, ctypes.c_char_p, ctypes.c_size_t]
    lib.ks_chain_describe.restype = ci
    lib.ks_chain_verify.argtypes = [ctypes.POINTER(_Factor), ci, i64, ci, ci, ctypes.c_char_p, ctypes.c_size_t]
    lib.ks_chain_verify.restype = ci
    lib.ks_force_chain_fusion.argtypes = [ci]
    lib.ks_force_chain_fusion.restype = None
    lib.ks_status_string.argtypes = [ci]
    lib.ks_status_string.restype = ctypes.c_char_p
    lib.ks_last_hip_error.argtypes = []
    lib.ks_last_hip_error.restype = ci
    lib.ks_plan_describe.argtypes = [i64, i64, i64, i64, i64, ci, ci, ctypes.c_char_p, ctypes.c_size_t]
    lib.ks_plan_describe.restype = ci
    lib.ks_force_variant.argtypes = [ci]
    lib.ks_force_variant.restype = None
    lib.ks_plan_verify.argtypes = [i64, i64, i64, i64, i64, ci, ci, ctypes.c_char_p, ctypes.c_size_t]
    lib.ks_plan_verify.restype = ci
    _lib = lib
    return lib


def _code(v, table, what):
    if isinstance(v, str):
        key = v.lower()
        if key not in table:
            raise ValueError("unknown %s %r" % (what, v))
        return table[key]
    return int(v)


_LAYOUTS = {"bsf": BSF, "bsl": BSL}
_DTYPES = {"f32": F32, "fp32": F32, "float32": F32, "bf16": BF16, "bfloat16": BF16, "f16": F16, "fp16": F16,
           "float16": F16, "fp8": FP8, "e4m3": FP8, "float8_e4m3fn": FP8}


def _ptr(t):
    """Device pointer of a tensor (or an int / None passed through)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def ks_status_string(status):
    return load_library().ks_status_string(int(status)).decode()


def ks_last_hip_error():
    return int(load_library().ks_last_hip_error())


def ks_force_variant(variant):
    load_library().ks_force_variant(-1 if variant is None else int(variant))


def ks_plan_describe(a, b, c, d, batch, layout, dtype):
    buf = ctypes.create_string_buffer(512)
    st = load_library().ks_plan_describe(a, b, c, d, batch, _code(layout, _LAYOUTS, "layout"),
                                         _code(dtype, _DTYPES, "dtype"), buf, 512)
    if st != KS_OK:
        raise KsError(st, "ks_plan_describe")
    return buf.value.decode()


def ks_plan_verify(a, b, c, d, batch, layout, dtype):
    """Host-side replay of the planned launch; returns (status, report)."""
    buf = ctypes.create_string_buffer(512)
    st = load_library().ks_plan_verify(a, b, c, d, batch, _code(layout, _LAYOUTS, "layout"),
                                       _code(dtype, _DTYPES, "dtype"), buf, 512)
    return int(st), buf.value.decode()


def ks_matmul(a, b, c, d, K_values, X, Y, batch, layout, dtype, stream=None, check=True):
    """C-ABI ks_matmul: tensors (or raw device pointers) are passed as pointers."""
    st = load_library().ks_matmul(a, b, c, d, _ptr(K_values), _ptr(X), _ptr(Y), batch,
                                  _code(layout, _LAYOUTS, "layout"), _code(dtype, _DTYPES, "dtype"),
                                  _stream(stream))
    if check and st != KS_OK:
        raise KsError(st, "ks_matmul")
    return st


_ACTS = {"none": ACT_NONE, "gelu": ACT_GELU}


def ks_matmul_bias_act(a, b, c, d, K_values, bias, act, X, Y, batch, layout, dtype, stream=None, check=True):
    """C-ABI ks_matmul_bias_act: Y = act(X K^T + bias) (bias may be None)."""
    st = load_library().ks_matmul_bias_act(a, b, c, d, _ptr(K_values), _ptr(bias),
                                           _code(act if act is not None else "none", _ACTS, "activation"),
                                           _ptr(X), _ptr(Y), batch, _code(layout, _LAYOUTS, "layout"),
                                           _code(dtype, _DTYPES, "dtype"), _stream(stream))
    if check and st != KS_OK:
        raise KsError(st, "ks_matmul_bias_act")
    return st


def _factor_array(factors):
    arr = (_Factor * len(factors))()
    for q, f in enumerate(factors):
        (a, b, c, d), kv = f
        arr[q] = _Factor(a, b, c, d, _ptr(kv))
    return arr


def ks_chain_workspace_bytes(factors, batch, dtype):
    """factors: sequence of ((a, b, c, d), K_values) in product order."""
    arr = _factor_array(factors)
    return int(load_library().ks_chain_workspace_bytes(arr, len(factors), batch, _code(dtype, _DTYPES, "dtype")))


def ks_chain(factors, X, Y, batch, layout, dtype, workspace, workspace_bytes, stream=None, check=True):
    """C-ABI ks_chain: Y = X (K_1 ... K_L)^T, factors in product order."""
    arr = _factor_array(factors)
    st = load_library().ks_chain(arr, len(factors), _ptr(X), _ptr(Y), batch, _code(layout, _LAYOUTS, "layout"),
                                 _code(dtype, _DTYPES, "dtype"), _ptr(workspace), int(workspace_bytes),
                                 _stream(stream))
    if check and st != KS_OK:
        raise KsError(st, "ks_chain")
    return st


def ks_chain_noalloc(factors, X, Y, batch, layout, dtype, stream=None, check=True):
    """C-ABI ks_chain_noalloc: ks_chain with the intermediates in the
    library's fixed per-GPU scratch array (no workspace argument)."""
    arr = _factor_array(factors)
    st = load_library().ks_chain_noalloc(arr, len(factors), _ptr(X), _ptr(Y), batch,
                                         _code(layout, _LAYOUTS, "layout"), _code(dtype, _DTYPES, "dtype"),
                                         _stream(stream))
    if check and st != KS_OK:
        raise KsError(st, "ks_chain_noalloc")
    return st


def ks_chain_describe(factors, batch, layout, dtype):
    """How ks_chain runs these factors: 'fused ...' or 'unfused ...'."""
    arr = _factor_array(factors)
    buf = ctypes.create_string_buffer(256)
    st = load_library().ks_chain_describe(arr, len(factors), batch, _code(layout, _LAYOUTS, "layout"),
                                          _code(dtype, _DTYPES, "dtype"), buf, 256)
    if st != KS_OK:
        raise KsError(st, "ks_chain_describe")
    return buf.value.decode()


def ks_chain_verify(factors, batch, layout, dtype):
    """Host replay of the fused chain kernel's accesses; returns (status, report)."""
    arr = _factor_array(factors)
    buf = ctypes.create_string_buffer(256)
    st = load_library().ks_chain_verify(arr, len(factors), batch, _code(layout, _LAYOUTS, "layout"),
                                        _code(dtype, _DTYPES, "dtype"), buf, 256)
    return int(st), buf.value.decode()


def ks_force_chain_fusion(mode):
    """mode 0: run chains factor by factor on this thread; None: automatic."""
    load_library().ks_force_chain_fusion(-1 if mode is None else int(mode))


def ks_chain_noalloc_max_workspace():
    return int(load_library().ks_chain_noalloc_max_workspace())


_TORCH_DTYPE_CODES = None


def _dtype_of(t):
    global _TORCH_DTYPE_CODES
    import torch
    if _TORCH_DTYPE_CODES is None:
        _TORCH_DTYPE_CODES = {torch.float32: F32, torch.bfloat16: BF16, torch.float16: F16,
                              torch.float8_e4m3fn: FP8}
    if t.dtype not in _TORCH_DTYPE_CODES:
        raise TypeError("unsupported dtype %s" % t.dtype)
    return _TORCH_DTYPE_CODES[t.dtype]


def _check_tensor(t, name):
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def _check_values(kv, pattern, dtype, device, name="K_values"):
    """The packed values of a factor: a*d*b*c contiguous elements of the
    storage dtype on the same device (the library reads exactly that many)."""
    a, b, c, d = pattern
    _check_tensor(kv, name)
    if kv.dtype != dtype:
        raise TypeError("%s has dtype %s, expected %s" % (name, kv.dtype, dtype))
    if kv.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, kv.device, device))
    if kv.numel() != a * b * c * d:
        raise ValueError("%s has %d elements, pattern %s needs a*b*c*d = %d"
                         % (name, kv.numel(), tuple(pattern), a * b * c * d))


def _check_batch(X, N, lay):
    """Batch size of an input of width N in layout `lay` (2-D tensors must
    have the layout's shape; flat ones any multiple of N)."""
    if X.numel() % N:
        raise ValueError("X has %d elements, not a multiple of N = %d" % (X.numel(), N))
    batch = X.numel() // N
    want = (batch, N) if lay == BSF else (N, batch)
    if X.dim() == 2 and tuple(X.shape) != want:
        raise ValueError("X has shape %s, expected %s" % (tuple(X.shape), want))
    if X.dim() not in (1, 2):
        raise ValueError("X must be 1-D or 2-D, got %d dimensions" % X.dim())
    return batch


def _check_out(out, shape, X, dtype=None):
    """A caller-supplied output: contiguous, of the output dtype (X's unless
    given) and X's device, with exactly batch*M elements (the library writes
    all of them)."""
    _check_tensor(out, "out")
    dtype = X.dtype if dtype is None else dtype
    if out.dtype != dtype:
        raise TypeError("out has dtype %s, expected %s" % (out.dtype, dtype))
    if out.device != X.device:
        raise ValueError("out is on %s, expected %s" % (out.device, X.device))
    n = shape[0] * shape[1]
    if out.numel() != n or (out.dim() == 2 and tuple(out.shape) != tuple(shape)):
        raise ValueError("out has shape %s, expected %s" % (tuple(out.shape), tuple(shape)))


def matmul(X, K_values, pattern, layout="bsl", out=None, bias=None, act=None):
    """Allocate Y (unless `out` is given) and run ks_matmul, or
    ks_matmul_bias_act when `bias` (a*b*d values) or `act` ("gelu") is given.
    X is (batch, a*c*d) for BSF or (a*c*d, batch) for BSL; K_values is
    (a*d, b, c) or flat; all share one dtype and device.  Every argument is
    checked on the host before the call (the C ABI sees only pointers)."""
    import torch
    a, b, c, d = (int(v) for v in pattern)
    lay = _code(layout, _LAYOUTS, "layout")
    _check_tensor(X, "X")
    dt = _dtype_of(X)
    _check_values(K_values, (a, b, c, d), X.dtype, X.device)
    N, M = a * c * d, a * b * d
    batch = _check_batch(X, N, lay)
    shape = (batch, M) if lay == BSF else (M, batch)
    ydtype = torch.bfloat16 if dt == FP8 else X.dtype  # FP8 inputs give bf16 outputs
    if out is None:
        out = torch.empty(shape, dtype=ydtype, device=X.device)
    else:
        _check_out(out, shape, X, ydtype)
    if bias is None and act is None:
        ks_matmul(a, b, c, d, K_values, X, out, batch, lay, dt)
        return out
    if bias is not None:
        _check_tensor(bias, "bias")
        if bias.dtype != ydtype or bias.device != X.device:
            raise TypeError("bias must have the output's dtype (%s) and X's device" % ydtype)
        if bias.numel() != M:
            raise ValueError("bias has %d elements, the output has a*b*d = %d features" % (bias.numel(), M))
    ks_matmul_bias_act(a, b, c, d, K_values, bias, act, X, out, batch, lay, dt)
    return out


def chain(X, factors, layout="bsl", out=None, workspace=None):
    """Y = X (K_1 ... K_L)^T; factors = [((a,b,c,d), K_values), ...] in product
    order (K_L is applied first).  Checks every factor's values, the input
    width, `out` and the workspace size on the host before the call."""
    import torch
    lay = _code(layout, _LAYOUTS, "layout")
    if len(factors) < 1:
        raise ValueError("a chain needs at least one factor")
    _check_tensor(X, "X")
    dt = _dtype_of(X)
    pats = [tuple(int(v) for v in p) for p, _ in factors]
    for q, (p, kv) in enumerate(factors):
        _check_values(kv, pats[q], X.dtype, X.device, "K_values of factor %d" % q)
    for q in range(len(pats) - 1):
        a0, b0, c0, d0 = pats[q]
        a1, b1, c1, d1 = pats[q + 1]
        if a0 * c0 * d0 != a1 * b1 * d1:
            raise ValueError("factors %d and %d do not compose: a*c*d = %d, next a*b*d = %d"
                             % (q, q + 1, a0 * c0 * d0, a1 * b1 * d1))
    (a1, b1, c1, d1), (aL, bL, cL, dL) = pats[0], pats[-1]
    N, M = aL * cL * dL, a1 * b1 * d1
    batch = _check_batch(X, N, lay)
    ws_bytes = ks_chain_workspace_bytes(factors, batch, dt)
    if workspace is None:
        if ws_bytes > 0:
            workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=X.device)
    else:
        _check_tensor(workspace, "workspace")
        if workspace.device != X.device:
            raise ValueError("workspace is on %s, expected %s" % (workspace.device, X.device))
    shape = (batch, M) if lay == BSF else (M, batch)
    if out is None:
        out = torch.empty(shape, dtype=X.dtype, device=X.device)
    else:
        _check_out(out, shape, X)
    ws_avail = workspace.numel() * workspace.element_size() if workspace is not None else 0
    ks_chain(factors, X, out, batch, lay, dt, workspace, ws_avail)
    return out
