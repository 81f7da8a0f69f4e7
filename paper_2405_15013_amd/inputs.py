"""Seeded synthetic inputs for Kronecker-sparse matmul.

This module only draws numbers and arranges them in memory; it holds none of
the method's arithmetic.  Both the HIP path's tests/benchmark and the CPU oracle
consume what it returns, so both sides always see the same values.

Distributions follow the paper's benchmark set-up (Appendix E.1): inputs X are
i.i.d. N(0, 1) and the nonzeros of K are i.i.d. uniform on [-1/sqrt(c), 1/sqrt(c)].
Values are drawn in float64 and rounded to the storage dtype with
round-to-nearest-even (float64 -> float32 -> bfloat16/float16; float64 ->
FP8 E4M3 with saturation at +-448), so the rounded values are exactly
representable in every wider format.

Streams: numpy PCG64 seeded with SeedSequence([BASE_SEED, cfg, a, b, c, d,
batch, tensor]); tensor 0 is X and tensor 1 + f is the packed values of
factor f.
"""
import numpy as np

BASE_SEED = 20240523

DTYPES = ("f32", "bf16", "f16", "fp8")


def _e4m3_table():
    """The 256 values of the OCP FP8 E4M3 ("E4M3FN") encoding: sign, 4-bit
    exponent with bias 7, 3-bit mantissa, subnormals at exponent 0, no
    infinities, NaN at codes 0x7F and 0xFF; largest finite value 448."""
    vals = np.empty(256, dtype=np.float64)
    for code in range(256):
        s, e, m = code >> 7, (code >> 3) & 15, code & 7
        if e == 15 and m == 7:
            v = np.nan
        elif e == 0:
            v = m * 2.0 ** -9
        else:
            v = (1 + m / 8.0) * 2.0 ** (e - 7)
        vals[code] = -v if s else v
    return vals


E4M3_VALUES = _e4m3_table()
E4M3_MAX = 448.0


def e4m3_from_f64(x64):
    """Round to the nearest E4M3 value (ties to the even code), saturating to
    +-448; returns the 8-bit codes as uint8.  NaN inputs give code 0x7F."""
    x = np.asarray(x64, dtype=np.float64)
    pos = E4M3_VALUES[:127]  # codes 0 .. 126: 0, then increasing positive values
    a = np.minimum(np.abs(x), E4M3_MAX)
    hi = np.clip(np.searchsorted(pos, a, side="left"), 0, 126)
    lo = np.clip(hi - 1, 0, 126)
    dlo, dhi = a - pos[lo], pos[hi] - a
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo).astype(np.uint8)
    code = np.where(np.signbit(x) & (code != 0), code | 0x80, code).astype(np.uint8)
    return np.where(np.isnan(x), np.uint8(0x7F), code).astype(np.uint8)


def generator(cfg, pattern, batch, tensor):
    a, b, c, d = (int(v) for v in pattern)
    ss = np.random.SeedSequence([BASE_SEED, int(cfg), a, b, c, d, int(batch), int(tensor)])
    return np.random.Generator(np.random.PCG64(ss))


def bf16_bits_from_f32(x32):
    """Round float32 values to bfloat16 (round-to-nearest-even); returns the
    raw 16-bit patterns as uint16."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    is_nan = np.isnan(np.ascontiguousarray(x32, dtype=np.float32))
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    r = np.where(is_nan, np.uint16(0x7FC0), r)
    return r.astype(np.uint16)


def f32_from_bf16_bits(bits):
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_to(x64, dtype):
    """float64 array -> storage array: float32, uint16 (bfloat16 bits) or float16."""
    x32 = np.asarray(x64, dtype=np.float64).astype(np.float32)
    if dtype == "f32":
        return x32
    if dtype == "bf16":
        return bf16_bits_from_f32(x32)
    if dtype == "f16":
        return x32.astype(np.float16)
    if dtype == "fp8":
        return e4m3_from_f64(x64)
    raise ValueError("unknown dtype %r" % (dtype,))


def to_f64(arr, dtype):
    """Storage array -> exact float64 values."""
    if dtype == "bf16":
        return f32_from_bf16_bits(arr).astype(np.float64)
    if dtype == "fp8":
        return E4M3_VALUES[np.asarray(arr, dtype=np.uint8)]
    return np.asarray(arr).astype(np.float64)


def draw(rng, shape, dist, c=1):
    """float64 samples.  dist: 'normal' N(0,1); 'uniform_c' U[-1/sqrt(c), 1/sqrt(c)];
    'normal_c' N(0,1)/sqrt(c); 'sign' uniform on {-1, 0, 1}; 'ones'."""
    if dist == "normal":
        return rng.standard_normal(shape)
    if dist == "uniform_c":
        lim = 1.0 / np.sqrt(c)
        return rng.uniform(-lim, lim, size=shape)
    if dist == "normal_c":
        return rng.standard_normal(shape) / np.sqrt(c)
    if dist == "sign":
        return rng.integers(-1, 2, size=shape).astype(np.float64)
    if dist == "ones":
        return np.ones(shape)
    raise ValueError("unknown distribution %r" % (dist,))


def make_x(cfg, pattern, batch, dtype, dist="normal"):
    """Logical input batch: (batch, a*c*d) in storage dtype."""
    a, b, c, d = (int(v) for v in pattern)
    rng = generator(cfg, pattern, batch, 0)
    return round_to(draw(rng, (batch, a * c * d), dist), dtype)


def make_kv(cfg, pattern, batch, dtype, dist="uniform_c", factor=0):
    """Packed nonzeros of one factor: (a*d, b, c) in storage dtype."""
    a, b, c, d = (int(v) for v in pattern)
    rng = generator(cfg, pattern, batch, 1 + factor)
    return round_to(draw(rng, (a * d, b, c), dist, c=c), dtype)


def to_layout(x_logical, layout):
    """(batch, width) logical matrix -> memory order of the given layout
    ('bsf': unchanged; 'bsl': transposed to (width, batch))."""
    if layout in ("bsf", 0):
        return np.ascontiguousarray(x_logical)
    if layout in ("bsl", 1):
        return np.ascontiguousarray(np.asarray(x_logical).T)
    raise ValueError("unknown layout %r" % (layout,))


def from_layout(y, layout):
    """Memory order of the given layout -> (batch, width) logical matrix."""
    if layout in ("bsf", 0):
        return np.asarray(y)
    return np.asarray(y).T
