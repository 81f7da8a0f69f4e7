"""CPU oracle for Kronecker-sparse matrix multiplication (fp64).

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(``paper_2405_15013_amd``) never imports, links or runs anything here, and this
package imports nothing from it.

The arithmetic lives in ``ks_oracle.c`` (plain C, fp64, OpenMP); this module
only marshals numpy arrays to it.  See the header of ``ks_oracle.c`` for the
definition it evaluates (paper Section 1, Definition 2.1, Section 4.1 index
sets, Section 2.2 layouts, Appendix B.1 Table 5 chain order).

Parity status: every function here is pinned by ``tests/test_oracle_pins.py``
(brute-force dense products built with numpy's ``kron``, the dense-GEMM and
diagonal special cases, the Sylvester-Hadamard closed form for butterfly
chains, the adjoint identity, the Figure 4 index sets, and for the bias/GELU
epilogue the normal CDF of scipy.stats at sample points).
"""
import ctypes
import os
import subprocess

import numpy as np

BSF = 0
BSL = 1

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ks_oracle.c")
_LIB = os.path.join(_HERE, "libks_oracle.so")
_lib = None


def build(force=False):
    """Compile ks_oracle.c into libks_oracle.so next to it (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        i64, p = ctypes.c_int64, ctypes.c_void_p
        lib.kso_matmul.argtypes = [i64, i64, i64, i64, p, p, p, i64, ctypes.c_int, ctypes.c_int]
        lib.kso_matmul.restype = ctypes.c_int
        lib.kso_entries.argtypes = [i64, i64, i64, i64, p, p, i64, ctypes.c_int, p, p, i64, p]
        lib.kso_entries.restype = ctypes.c_int
        lib.kso_dense.argtypes = [i64, i64, i64, i64, p, p]
        lib.kso_dense.restype = ctypes.c_int
        lib.kso_chain.argtypes = [ctypes.c_int, p, p, p, p, i64, ctypes.c_int, ctypes.c_int]
        lib.kso_chain.restype = ctypes.c_int
        lib.kso_bias_act.argtypes = [p, p, i64, i64, ctypes.c_int, ctypes.c_int]
        lib.kso_bias_act.restype = ctypes.c_int
        lib.kso_max_threads.argtypes = []
        lib.kso_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _f64(arr):
    return np.ascontiguousarray(arr, dtype=np.float64)


def _ptr(arr):
    return arr.ctypes.data_as(ctypes.c_void_p)


def threads():
    """Number of host threads the oracle runs on."""
    return int(_load().kso_max_threads())


def _layout_code(layout):
    if layout in (BSF, "bsf", "BSF"):
        return BSF
    if layout in (BSL, "bsl", "BSL"):
        return BSL
    raise ValueError("unknown layout %r" % (layout,))


def matmul(pattern, kv, x, batch, layout, nthreads=0):
    """Y = X K^T for one factor.  ``kv`` is (a*d, b, c); ``x`` is laid out as
    (batch, N) for BSF or (N, batch) for BSL; the result has the same layout."""
    a, b, c, d = (int(v) for v in pattern)
    lay = _layout_code(layout)
    kv64, x64 = _f64(kv), _f64(x)
    assert kv64.size == a * d * b * c, "Kv has %d values, pattern needs %d" % (kv64.size, a * b * c * d)
    assert x64.size == batch * a * c * d
    shape = (batch, a * b * d) if lay == BSF else (a * b * d, batch)
    y = np.empty(shape, dtype=np.float64)
    rc = _load().kso_matmul(a, b, c, d, _ptr(kv64), _ptr(x64), _ptr(y), batch, lay, nthreads)
    if rc != 0:
        raise ValueError("kso_matmul rejected its arguments (%d)" % rc)
    return y


def entries(pattern, kv, x, batch, layout, beta_idx, m_idx):
    """Y[beta_idx[t], m_idx[t]] for every t, each computed from the definition."""
    a, b, c, d = (int(v) for v in pattern)
    lay = _layout_code(layout)
    kv64, x64 = _f64(kv), _f64(x)
    bi = np.ascontiguousarray(beta_idx, dtype=np.int64)
    mi = np.ascontiguousarray(m_idx, dtype=np.int64)
    assert bi.shape == mi.shape
    out = np.empty(bi.shape, dtype=np.float64)
    rc = _load().kso_entries(a, b, c, d, _ptr(kv64), _ptr(x64), batch, lay, _ptr(bi), _ptr(mi), bi.size, _ptr(out))
    if rc != 0:
        raise ValueError("kso_entries rejected its arguments (%d)" % rc)
    return out


def dense(pattern, kv):
    """The dense (a*b*d) x (a*c*d) matrix K, zeros off the KS support."""
    a, b, c, d = (int(v) for v in pattern)
    kv64 = _f64(kv)
    k = np.empty((a * b * d, a * c * d), dtype=np.float64)
    rc = _load().kso_dense(a, b, c, d, _ptr(kv64), _ptr(k))
    if rc != 0:
        raise ValueError("kso_dense rejected its arguments (%d)" % rc)
    return k


def chain(patterns, kvs, x, batch, layout, nthreads=0):
    """Y = X (K_1 ... K_L)^T, factors listed in product order (K_L applied
    first), fp64 intermediates."""
    lay = _layout_code(layout)
    n = len(patterns)
    pat = np.ascontiguousarray(np.array(patterns, dtype=np.int64).reshape(n, 4))
    kv64 = [_f64(k) for k in kvs]
    ptrs = (ctypes.c_void_p * n)(*[k.ctypes.data for k in kv64])
    x64 = _f64(x)
    a, b, c, d = (int(v) for v in pat[0])
    shape = (batch, a * b * d) if lay == BSF else (a * b * d, batch)
    y = np.empty(shape, dtype=np.float64)
    rc = _load().kso_chain(n, _ptr(pat), ctypes.cast(ptrs, ctypes.c_void_p), _ptr(x64), _ptr(y), batch, lay, nthreads)
    if rc == -2:
        raise ValueError("chain factors have incompatible dimensions")
    if rc != 0:
        raise ValueError("kso_chain rejected its arguments (%d)" % rc)
    return y


def bias_act(y, bias, layout, act):
    """act(Y + bias) elementwise per output feature m (bias: M values or
    None; act: None/"none" or "gelu"), returning a new fp64 array in the same
    layout as y ((batch, M) for BSF, (M, batch) for BSL)."""
    lay = _layout_code(layout)
    out = np.array(y, dtype=np.float64, copy=True, order="C")
    M = out.shape[1] if lay == BSF else out.shape[0]
    batch = out.shape[0] if lay == BSF else out.shape[1]
    b = None if bias is None else _f64(bias)
    assert b is None or b.size == M
    a = {None: 0, "none": 0, "gelu": 1}[act]
    rc = _load().kso_bias_act(_ptr(out), None if b is None else _ptr(b), M, batch, lay, a)
    if rc != 0:
        raise ValueError("kso_bias_act rejected its arguments (%d)" % rc)
    return out
