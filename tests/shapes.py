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
