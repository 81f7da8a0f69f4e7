"""Shapes shared by the GPU parity tests and the host-side plan checks."""

# Register-direct / staged / streaming MFMA kernels: every j-vector mode
# (d = 1, 2, 4 and d > 4), c % 32 == 16 tails of the 16-bit path.
MFMA_SHAPES = [(1, 32, 32, 32), (32, 32, 32, 1), (6, 64, 16, 8), (6, 16, 64, 8), (2, 48, 80, 2), (1, 128, 16, 16),
               (8, 16, 128, 4), (3, 96, 48, 1), (1, 16, 112, 8), (2, 64, 128, 2)]

# LDS-DMA kernel (batch-size-first, d in {1, 2, 4, 8, 16}): strided and
# contiguous j-vectors, one to eight stages of l.
DMA_SHAPES = ([s for s in MFMA_SHAPES if s[3] <= 16]
              + [(2, 128, 128, 16), (4, 48, 96, 4), (1, 32, 48, 16), (1, 16, 32, 8), (3, 64, 80, 4), (2, 96, 16, 16),
                 (1, 16, 16, 1), (2, 32, 48, 2), (8, 128, 96, 1)])

# Batch 4096 shapes whose DMA plans take 2 or 4 row groups per wavefront (NT),
# 16x16x16 stages of 16-bit types with c % 32 == 0, strided and contiguous, and
# whose register-direct plans take 2 or 4 M-tiles per wavefront (d = 1).
DMA_ROW_GROUP_SHAPES = [(1, 128, 16, 16), (4, 128, 32, 4), (2, 128, 32, 8), (8, 128, 16, 4), (8, 128, 32, 4),
                        (4, 128, 16, 4), (2, 64, 64, 16), (4, 128, 16, 8), (4, 128, 64, 1), (8, 64, 32, 2),
                        (2, 48, 64, 1), (8, 128, 16, 2), (1, 16, 16, 4), (1, 16, 32, 4), (1, 64, 32, 8),
                        (1, 128, 32, 4), (1, 128, 16, 1), (2, 128, 16, 1)]


def sweep_patterns():
    """The benchmark's pattern sweep: a in {1,2,4,8}, b, c in
    {16,32,48,64,96,128}, d in {1,2,4,8,16}, a*b*d <= 8192 and a*c*d <= 8192
    (700 patterns)."""
    return [(a, b, c, d) for a in (1, 2, 4, 8) for b in (16, 32, 48, 64, 96, 128) for c in (16, 32, 48, 64, 96, 128)
            for d in (1, 2, 4, 8, 16) if a * b * d <= 8192 and a * c * d <= 8192]


BUTTERFLY = [(2 ** (l - 1), 2, 2, 2 ** (10 - l)) for l in range(1, 11)]
MONARCH = [(1, 32, 32, 32), (32, 32, 32, 1)]
MLP = [(6, 64, 16, 8), (6, 16, 64, 8)]


def bench_points():
    """Every (pattern, batch, dtype, layout) single-factor call the benchmark
    makes: the 5600 sweep points, then the tiny, butterfly, Monarch and
    Transformer-MLP workloads (the chains run the same factors), then the FP8
    calls."""
    pts = [(p, batch, dtype, layout) for dtype in ("f32", "bf16") for batch in (4096, 25088)
           for layout in ("bsf", "bsl") for p in sweep_patterns()]
    pts += [((2, 4, 4, 2), 32, "f32", layout) for layout in ("bsf", "bsl")]
    pts += [(p, 4096, "f32", layout) for p in BUTTERFLY for layout in ("bsf", "bsl")]
    pts += [(p, 16384, dtype, layout) for p in MONARCH for dtype in ("f32", "bf16") for layout in ("bsf", "bsl")]
    pts += [(p, 25088, dtype, layout) for p in MLP for dtype in ("f32", "bf16") for layout in ("bsf", "bsl")]
    # FP8 (E4M3 inputs, bf16 outputs): the MLP layers and every 7th sweep pattern
    pts += [(p, 25088, "fp8", layout) for p in MLP for layout in ("bsf", "bsl")]
    pts += [(p, batch, "fp8", layout) for batch in (4096, 25088) for layout in ("bsf", "bsl")
            for p in sweep_patterns()[::7]]
    return pts
