// Planner and launcher of the register-direct MFMA kernels (ks_direct.h).
//
// A plan fixes the vector width V (along the batch in BSL: 8 elements for
// 16-bit storage when the batch allows it, else 4; the j-run min(d, 4) in
// BSF), the number MT of 16-row M-tiles per wavefront,
// and the wavefronts per workgroup.  MT trades X re-reads (b / (16*MT)
// wavefronts read the same X tile) against registers and parallelism.
#include "ks_direct_index.h"
#include "ks_internal.h"
#include "ks_masked_index.h"

namespace ks {

hipError_t launch_direct_f32(const Problem& p, const DirectTile& t, int V, bool strided, int mt, unsigned grid,
                             hipStream_t s);
hipError_t launch_direct_bf16(const Problem& p, const DirectTile& t, int V, bool strided, int mt, unsigned grid,
                              hipStream_t s);
hipError_t launch_direct_f16(const Problem& p, const DirectTile& t, int V, bool strided, int mt, unsigned grid,
                             hipStream_t s);
hipError_t launch_direct_f32_epi(const Problem& p, const DirectTile& t, int V, bool strided, int mt, unsigned grid,
                                 hipStream_t s);
hipError_t launch_direct_bf16_epi(const Problem& p, const DirectTile& t, int V, bool strided, int mt, unsigned grid,
                                  hipStream_t s);
hipError_t launch_direct_f16_epi(const Problem& p, const DirectTile& t, int V, bool strided, int mt, unsigned grid,
                                 hipStream_t s);
hipError_t launch_masked_f32(const Problem& p, const MaskedTile& t, int V, unsigned grid, hipStream_t s);
hipError_t launch_masked_bf16(const Problem& p, const MaskedTile& t, int V, unsigned grid, hipStream_t s);
hipError_t launch_masked_f16(const Problem& p, const MaskedTile& t, int V, unsigned grid, hipStream_t s);

// Largest MT instantiated for (storage size, layout, V); keep in sync with
// direct_mt_max() in ks_direct.h.
static int mt_max(int esize, int layout, int V) {
  return esize == 4 ? ((layout == BSL || V <= 2) ? 4 : 2) : ((layout == BSL || V <= 2) ? 4 : 2);
}

DirectTile direct_tile(const Problem& p, const Plan& pl) {
  DirectTile t;
  const int V = pl.vec, MT = pl.waves_m;
  t.kgroups = p.b / (16 * MT);
  t.jgroups = p.layout == BSL ? p.d : p.d / V;
  const int span = p.layout == BSL ? 16 * V : 16;
  t.nbt = (p.batch + span - 1) / span;
  t.items = t.nbt * p.a * t.jgroups * t.kgroups;
  t.waves = (int)pl.block / 64;
  div_magic((uint32_t)t.kgroups, &t.mkg, &t.skg);
  div_magic((uint32_t)t.nbt, &t.mnbt, &t.snbt);
  div_magic((uint32_t)t.jgroups, &t.mjg, &t.sjg);
  return t;
}

bool plan_direct(const Problem& p, bool al16, Plan* pl) {
  if (!al16 || p.b % 16 || p.c % 16) return false;
  const int s = p.dtype == F32 ? 4 : 2;
  const int vec = 4;  // kDirectVec in ks_direct.h
  int V;
  bool strided = false;
  if (p.layout == BSL) {
    // 16-bit storage: 8 batch entries per lane (16-byte loads and stores)
    // when the batch allows it (kDirectVecBsl16 in ks_direct.h).
    V = (s == 2 && p.batch % 8 == 0) ? 8 : vec;
    if (p.batch % V) return false;
  } else {
    V = p.d < vec ? p.d : vec;
    if (V != 1 && V != 2 && V != 4) return false;
    if (p.d % V) return false;
    strided = V < p.d;
  }
  const int kt = p.b / 16;  // M-tiles per block
  const int span = p.layout == BSL ? 16 * V : 16;
  const int64_t nbt = (p.batch + span - 1) / span;
  const int64_t per_k = nbt * p.a * (p.layout == BSL ? p.d : p.d / V);
  // Largest MT that still leaves >= 768 wavefronts (three per CU); otherwise
  // the MT giving the most wavefronts.  Fewer k-groups mean fewer re-reads of
  // each X tile, which measured worth more than extra wavefronts down to
  // about three per CU.
  int best = 0;
  for (int mt = mt_max(s, p.layout, V); mt >= 1; --mt) {
    if (kt % mt) continue;
    best = mt;
    if (per_k * (kt / mt) >= 768) break;
  }
  const int64_t items = per_k * (kt / best);
  // Four wavefronts per workgroup at every size: consecutive items (the
  // k-groups of one X tile first) share a CU's caches, and spreading small
  // problems over more, smaller workgroups measured slower.
  const int waves = 4;
  const int64_t grid = (items + waves - 1) / waves;
  if (items > 0x7fffffff || grid > 0x7fffffff) return false;
  pl->variant = V_DIRECT;
  pl->vec = V;
  pl->unroll = strided ? 1 : 0;
  pl->waves_m = best;
  pl->waves_n = kt / best;
  pl->bt = span;
  pl->jg = p.layout == BSL ? 1 : V;
  pl->lds_bytes = 0;
  pl->block = 64u * waves;
  pl->grid = (unsigned)grid;
  pl->xcd_remap = 0;
  return true;
}

// Masked register-direct kernel (ks_masked.h): blocks larger than the VALU
// kernels take (b or c > 16) that the other MFMA kernels cannot run.  The
// access width V is the widest the layout, the batch (BSL) or d (BSF) and the
// buffers' alignment allow (up to 16 bytes along the batch in BSL, up to 4
// consecutive j in BSF), 8-byte pieces only for 16-bit BSL.
int masked_vec(const Problem& p) {
  const int s = p.dtype == F32 ? 4 : 2;
  const int vmax = p.layout == BSL ? 16 / s : 4;
  int V = vmax;
  for (; V > 1; V /= 2) {
    if (p.layout == BSL && p.batch % V) continue;
    if (p.layout == BSF && p.d % V) continue;
    if (V * s >= 8 && p.align % (V * s)) continue;  // vector accesses need their alignment
    // 8-byte pieces measured slower than element pieces here except for
    // 16-bit batch-size-last runs (e.g. fp32 BSF (6,64,16,8) at batch 25088:
    // 2.0 ms with 8-byte pieces, 0.68 ms with 4-byte ones)
    if (V * s == 8 && !(p.layout == BSL && s == 2)) continue;
    break;
  }
  return V;
}

bool plan_masked(const Problem& p, Plan* pl) {
  if (p.b <= 16 && p.c <= 16 && (p.b % 16 || p.c % 16)) return false;  // the VALU kernels' blocks
  const int V = masked_vec(p);
  const MaskedTile t = masked_tile(p, V);
  const int64_t items = (int64_t)t.nbt * p.a * t.jgroups * t.kgroups;
  if (items > 0x7fffffff - 3) return false;
  pl->variant = V_MASKED;
  pl->vec = V;
  pl->unroll = 0;
  pl->waves_m = 1;
  pl->waves_n = t.kgroups;
  pl->bt = p.layout == BSL ? 16 * V : 16;
  pl->jg = p.layout == BSL ? 1 : V;
  pl->lds_bytes = 0;
  pl->block = 256;
  pl->grid = (unsigned)((items + 3) / 4);
  pl->xcd_remap = 0;
  return true;
}

hipError_t launch_masked(const Problem& p, const Plan& pl, hipStream_t s) {
  const MaskedTile t = masked_tile(p, pl.vec);
  switch (p.dtype) {
    case F32: return launch_masked_f32(p, t, pl.vec, pl.grid, s);
    case BF16: return launch_masked_bf16(p, t, pl.vec, pl.grid, s);
    case F16: return launch_masked_f16(p, t, pl.vec, pl.grid, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_direct(const Problem& p, const Plan& pl, hipStream_t s) {
  const DirectTile t = direct_tile(p, pl);
  const bool strided = pl.unroll != 0;
  if (has_epilogue(p)) {
    switch (p.dtype) {
      case F32: return launch_direct_f32_epi(p, t, pl.vec, strided, pl.waves_m, pl.grid, s);
      case BF16: return launch_direct_bf16_epi(p, t, pl.vec, strided, pl.waves_m, pl.grid, s);
      case F16: return launch_direct_f16_epi(p, t, pl.vec, strided, pl.waves_m, pl.grid, s);
      default: return hipErrorInvalidValue;
    }
  }
  switch (p.dtype) {
    case F32: return launch_direct_f32(p, t, pl.vec, strided, pl.waves_m, pl.grid, s);
    case BF16: return launch_direct_bf16(p, t, pl.vec, strided, pl.waves_m, pl.grid, s);
    case F16: return launch_direct_f16(p, t, pl.vec, strided, pl.waves_m, pl.grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ks
