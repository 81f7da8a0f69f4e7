// Planner and launcher of the LDS-staged MFMA kernels (ks_staged.h).
//
// A plan fixes the vector width V (4 along the batch in BSL, min(d, 4) of j
// in BSF), the M-tiles per wavefront MT, and how the W <= 8 wavefronts of a
// tile split the work: JG j-groups (BSF: d / V) x KGW k-groups x RS row/column
// groups, with W = 4 (8 when d / V = 8: eight j-groups).  Larger tiles cut
// the re-reads of K and X but leave fewer workgroups resident per CU, which
// measured slower.  Preferred: enough tiles for the chip, then the fewest
// re-reads of X, then the largest MT.  A stage of X is at most 256 16-byte
// units per wavefront (4 per thread) and a workgroup needs two stage buffers
// of LDS.
#include "ks_staged_index.h"
#include "ks_internal.h"

namespace ks {

hipError_t launch_staged_f32(const Problem& p, const StagedTile& t, int V, bool strided, int mt, int cps,
                             hipStream_t s);
hipError_t launch_staged_bf16(const Problem& p, const StagedTile& t, int V, bool strided, int mt, int cps,
                              hipStream_t s);
hipError_t launch_staged_f16(const Problem& p, const StagedTile& t, int V, bool strided, int mt, int cps,
                             hipStream_t s);
#define KS_DMA_DECL(T, M) \
  hipError_t launch_dma_##T##_##M(const Problem& p, const StagedTile& t, int mt, int lp, hipStream_t s);
KS_DMA_DECL(f32, v4s) KS_DMA_DECL(f32, v4c) KS_DMA_DECL(f32, v2) KS_DMA_DECL(f32, v1)
KS_DMA_DECL(bf16, v4s) KS_DMA_DECL(bf16, v4c) KS_DMA_DECL(bf16, v2) KS_DMA_DECL(bf16, v1)
KS_DMA_DECL(f16, v4s) KS_DMA_DECL(f16, v4c) KS_DMA_DECL(f16, v2) KS_DMA_DECL(f16, v1)
#undef KS_DMA_DECL
hipError_t launch_dma_bsl_f32(const Problem& p, const StagedTile& t, int mt, hipStream_t s);
hipError_t launch_dma_bsl_bf16(const Problem& p, const StagedTile& t, int mt, hipStream_t s);
hipError_t launch_dma_bsl_f16(const Problem& p, const StagedTile& t, int mt, hipStream_t s);

namespace {
constexpr int kUnitsPerWave = 256;  // 64 threads x kStagedUnitsPerThread (ks_staged.h)
constexpr int kMaxLds = 128 * 1024;  // kStagedMaxLds (ks_staged.h)

// Largest MT instantiated; keep in sync with direct_mt_max() in ks_direct.h.
int mt_max(int esize, int layout, int V) {
  (void)esize;
  return (layout == BSL || V <= 2) ? 4 : 2;
}
}  // namespace

StagedTile staged_tile_of(const Problem& p, const Plan& pl) {
  StagedTile t;
  const int S = p.dtype == F32 ? 4 : 2, V = pl.vec, MT = pl.waves_m;
  t.W = (int)pl.block / 64;
  t.RS = pl.rs;
  t.JG = p.layout == BSL ? 1 : p.d / V;
  t.KGW = pl.kgw;
  t.kgt = p.b / (16 * MT * t.KGW);
  t.NT = (pl.variant == V_DMA) ? pl.nt : 1;
  const int span = p.layout == BSL ? 16 * V * t.RS : 16 * t.RS * t.NT;
  t.nbt = (p.batch + span - 1) / span;
  t.tiles = t.nbt * p.a * (p.layout == BSL ? p.d : 1) * t.kgt;
  t.LCH = pl.lch;
  if (p.layout == BSL) {
    t.pitch = 16 * V * t.RS * S;
    t.stage = t.LCH * t.pitch;
  } else {
    t.pitch = t.LCH * p.d * S + 16;
    t.stage = 16 * t.RS * t.pitch;
  }
  t.remap = pl.xcd_remap;
  t.ypitch = 0;
  t.UR = 0;
  t.UD = 0;
  t.lUR = t.lRS = t.lJG = t.lUY = 0;
  t.mkgt = t.mnbt = t.md = 0;
  t.skgt = t.snbt = t.sd = 0;
  t.lds = 2 * t.stage;
  auto log2i = [](int v) { int l = 0; while ((1 << l) < v) ++l; return l; };
  if (pl.variant == V_DMA && p.layout == BSL) {
    // Stage rows of UR = 16*RS units (16*V*RS batch entries, V*esize = 16
    // bytes), one per value of l; three stage buffers or one per stage.
    t.UR = 16 * V * t.RS * S / 16;
    t.pitch = t.UR * 16;
    t.stage = t.LCH * t.pitch;
    t.UD = t.stage / 16 / (64 * t.W);
    t.lds = dma_stage_buffers(p.c / t.LCH) * t.stage;
    t.lUR = log2i(t.UR);
    t.lRS = log2i(t.RS);
    div_magic((uint32_t)t.kgt, &t.mkgt, &t.skgt);
    div_magic((uint32_t)t.nbt, &t.mnbt, &t.snbt);
    div_magic((uint32_t)p.d, &t.md, &t.sd);
    return t;
  }
  if (pl.variant == V_DMA) {
    // Unpadded, swizzled rows of UR units; three stage buffers, or one per
    // stage when there are fewer stages (dma_stage_buffers).
    t.UR = t.LCH * p.d * S / 16;
    t.pitch = t.UR * 16;
    t.stage = 16 * t.RS * t.NT * t.pitch;
    t.UD = t.stage / 16 / (64 * t.W);
    t.lds = dma_stage_buffers(p.c / t.LCH) * t.stage;
    t.lUR = log2i(t.UR);
    t.lRS = log2i(t.RS);
    t.lJG = log2i(t.JG);
    t.lUY = log2i(MT * t.KGW * p.d * S);  // 16-byte units per output tile row
    div_magic((uint32_t)t.kgt, &t.mkgt, &t.skgt);
    div_magic((uint32_t)t.nbt, &t.mnbt, &t.snbt);
  }
  if (p.layout == BSF) {
    t.ypitch = 16 * MT * t.KGW * p.d * S + 16;
    const int ytile = 16 * t.RS * t.NT * t.ypitch;
    if (ytile > t.lds) t.lds = ytile;
  }
  return t;
}

bool plan_staged(const Problem& p, bool al16, Plan* pl) {
  if (!al16 || p.b % 16 || p.c % 16) return false;
  const int S = p.dtype == F32 ? 4 : 2;
  const int UE = 16 / S, CH = S == 4 ? 16 : 32;
  int V, JG;
  bool strided = false;
  if (p.layout == BSL) {
    V = 4;
    if (p.batch % UE) return false;
    JG = 1;
  } else {
    V = p.d < 4 ? p.d : 4;
    if ((V != 1 && V != 2 && V != 4) || p.d % V) return false;
    strided = V < p.d;
    JG = p.d / V;
    if (JG > 8) return false;
  }
  const int lch = (p.layout == BSF && CH * p.d * S < 128) ? 2 * CH : CH;
  const int KT = p.b / 16;
  bool found = false;
  int64_t best_tiles = 0;
  int best_kgt = 0, best_mt = 0, best_kgw = 0, best_rs = 0;
  for (int mt = mt_max(S, p.layout, V); mt >= 1; --mt) {
    if (KT % mt) continue;
    const int kgroups = KT / mt;
    for (int kgw = 1; kgw <= 8; ++kgw) {
      if (kgroups % kgw || kgw * JG > 8) continue;
      for (int rs = 1; rs * kgw * JG <= 8; rs *= 2) {
        const int w = rs * kgw * JG;
        // Four wavefronts per tile (smaller tiles keep more workgroups resident
        // per CU); eight only when there are eight j-groups.
        if (w != (JG > 4 ? 8 : 4)) continue;
        const int64_t units = p.layout == BSL ? (int64_t)lch * (16 * V * rs * S / 16)
                                              : (int64_t)16 * rs * (lch * p.d * S / 16);
        if (units > (int64_t)kUnitsPerWave * w) continue;
        const int kgt = kgroups / kgw;
        const int span = p.layout == BSL ? 16 * V * rs : 16 * rs;
        const int64_t tiles = (int64_t)((p.batch + span - 1) / span) * p.a * (p.layout == BSL ? p.d : 1) * kgt;
        if (tiles > 0x7fffffff) continue;
        // LDS: two stages, and the BSF output tile
        const int64_t pitch = p.layout == BSL ? (int64_t)16 * V * rs * S : (int64_t)lch * p.d * S + 16;
        const int64_t stage = p.layout == BSL ? lch * pitch : 16 * rs * pitch;
        int64_t lds = 2 * stage;
        if (p.layout == BSF) {
          const int64_t ytile = 16 * rs * ((int64_t)16 * mt * kgw * p.d * S + 16);
          if (ytile > lds) lds = ytile;
        }
        if (lds > kMaxLds) continue;
        // Enough tiles (4 per CU) first, then the fewest re-reads of X, then
        // the largest MT.
        const int64_t tcap = tiles < 1024 ? tiles : 1024;
        const int64_t bcap = best_tiles < 1024 ? best_tiles : 1024;
        bool better = !found;
        if (!better) {
          if (tcap != bcap) better = tcap > bcap;
          else if (kgt != best_kgt) better = kgt < best_kgt;
          else better = mt > best_mt;
        }
        if (better) {
          found = true;
          best_tiles = tiles;
          best_kgt = kgt;
          best_mt = mt;
          best_kgw = kgw;
          best_rs = rs;
        }
      }
    }
  }
  if (!found) return false;
  pl->variant = V_STAGED;
  pl->vec = V;
  pl->unroll = strided ? 1 : 0;
  pl->waves_m = best_mt;
  pl->waves_n = best_kgt;
  pl->jg = JG;
  pl->rs = best_rs;
  pl->kgw = best_kgw;
  pl->lch = lch;
  pl->cps = lch / CH;
  pl->bt = p.layout == BSL ? 16 * V * best_rs : 16 * best_rs;
  pl->block = 64u * (unsigned)(best_rs * best_kgw * JG);
  pl->grid = (unsigned)best_tiles;
  pl->xcd_remap = (best_kgt > 1 && best_tiles % 8 == 0) ? 1 : 0;
  const StagedTile t = staged_tile_of(p, *pl);
  if (t.lds > kMaxLds) return false;
  pl->lds_bytes = t.lds;
  return true;
}

// LDS-DMA kernel (ks_dma.h): batch-size-first, d in {1, 2, 4, 8, 16}
// (V = min(d, 4) j values per lane: d / V j-groups), four wavefronts per tile, one MFMA chunk
// per stage (16 values of l for fp32; 32, or 16 when c % 32 == 16, for 16-bit
// types), a stage of 2, 4 or 8 DMA instructions per wavefront, three stage
// buffers, NT groups of 16 rows per wavefront (MT * NT <= 4).
struct DmaChoice {
  int lp, mt, nt, kgw, rs, kgt;
  int64_t tiles, lds;
};
// Preference: at most 64 KB of LDS (two workgroups per CU; see dma_lds_pref
// for the one exception), then enough tiles
// for one per CU (256), then the deeper MFMA (LP: 16x16x32 steps for 16-bit
// types when c allows), then the most batch rows per K operand (NT: K is read
// from L2 once per 16*NT rows), then the fewest re-reads of X (k-group
// tiles), then the largest MT.  Asking for more
// tiles than CUs (smaller tiles, more k-group tiles) measured slower over the
// pattern sweep: the extra K and X re-reads cost more than the parallelism.
constexpr int64_t kDmaLdsPref = 64 * 1024;
constexpr int64_t kDmaTileTarget = 256;
// fp32 with d = 16, b >= 64 and c >= 48: the 64 KB preference would leave
// 16-row tiles (four j-groups take the four wavefronts) whose stages hold too
// few MFMAs to cover the next stage's K loads; 32-row tiles in up to 128 KB
// measured 4-18 % faster (median per c) there, and slower with one or two
// stages (c <= 32), where there is no next stage to cover.
int64_t dma_lds_pref(const Problem& p) {
  return (p.dtype == F32 && p.d >= 16 && p.b >= 64 && p.c >= 48) ? 128 * 1024 : kDmaLdsPref;
}
bool dma_better(const DmaChoice& c, const DmaChoice& b, int64_t lds_pref) {
  if ((c.lds <= lds_pref) != (b.lds <= lds_pref)) return c.lds <= lds_pref;
  const int64_t tc = c.tiles < kDmaTileTarget ? c.tiles : kDmaTileTarget;
  const int64_t tb = b.tiles < kDmaTileTarget ? b.tiles : kDmaTileTarget;
  if (tc != tb) return tc > tb;
  if (c.lp != b.lp) return c.lp > b.lp;
  if (c.nt != b.nt) return c.nt > b.nt;
  if (c.kgt != b.kgt) return c.kgt < b.kgt;
  return c.mt > b.mt;
}
// Batch-size-last DMA kernel (ks_dma_bsl.h): one 16-byte unit of V = 16 /
// esize batch entries per lane column, stages of CH = 16 (fp32) or 32 (16-bit)
// values of l, four wavefronts per tile as RS batch groups x KGW = 4 / RS
// k-groups, MT <= 4 (fp32) or 2 (16-bit).  Preference: enough tiles for one
// per CU, then the fewest k-group tiles (each re-reads X), then the smallest
// MT (the widest batch range per tile).  Fitted on every feasible (MT, RS) of
// the sampled sweep points (fp32 batch 25088: sweep median 0.549, mean regret
// against the per-point best 1.026; "largest MT" instead: regret 1.05).
bool plan_dma_bsl(const Problem& p, bool al16, Plan* pl) {
  if (!al16 || p.layout != BSL || p.b % 16) return false;
  const int S = p.dtype == F32 ? 4 : 2, V = 16 / S, LP = S == 4 ? 4 : 8, CH = 4 * LP, W = 4;
  if (p.c % CH || p.batch % V) return false;
  const int KT = p.b / 16, mtmax = S == 4 ? 4 : 2;
  bool found = false;
  int best_mt = 0, best_rs = 0, best_kgt = 0;
  int64_t best_tiles = 0;
  for (int mt = 1; mt <= mtmax; ++mt) {
    if (KT % mt) continue;
    const int kgroups = KT / mt;
    for (int rs = 1; rs <= W; rs *= 2) {
      const int kgw = W / rs;
      if (kgroups % kgw) continue;
      const int kgt = kgroups / kgw, span = 16 * V * rs;
      const int64_t tiles = (int64_t)((p.batch + span - 1) / span) * p.a * p.d * kgt;
      if (tiles > 0x7fffffff) continue;
      const int64_t lds = (int64_t)dma_stage_buffers(p.c / CH) * CH * 16 * rs * 16;
      if (lds > kMaxLds) continue;
      const int64_t tc = tiles < kDmaTileTarget ? tiles : kDmaTileTarget;
      const int64_t tb = best_tiles < kDmaTileTarget ? best_tiles : kDmaTileTarget;
      bool better = !found;
      if (!better) {
        if (tc != tb) better = tc > tb;
        else if (kgt != best_kgt) better = kgt < best_kgt;
        else better = mt < best_mt;
      }
      if (better) {
        found = true;
        best_mt = mt;
        best_rs = rs;
        best_kgt = kgt;
        best_tiles = tiles;
      }
    }
  }
  if (!found) return false;
  pl->variant = V_DMA;
  pl->vec = V;
  pl->unroll = 0;
  pl->waves_m = best_mt;
  pl->waves_n = best_kgt;
  pl->jg = 1;
  pl->rs = best_rs;
  pl->kgw = W / best_rs;
  pl->nt = 1;
  pl->lch = CH;
  pl->cps = LP;
  pl->bt = 16 * V * best_rs;
  pl->block = 64u * W;
  pl->grid = (unsigned)best_tiles;
  pl->xcd_remap = (best_kgt > 1 && best_tiles % 8 == 0) ? 1 : 0;
  const StagedTile t = staged_tile_of(p, *pl);
  if (t.lds > kMaxLds || t.UD * 64 * W * 16 != t.stage) return false;
  pl->lds_bytes = t.lds;
  return true;
}

bool plan_dma(const Problem& p, bool al16, Plan* pl) {
  if (p.layout == BSL) return plan_dma_bsl(p, al16, pl);
  if (!al16 || p.layout != BSF || p.b % 16 || p.c % 16) return false;
  if (p.d != 1 && p.d != 2 && p.d != 4 && p.d != 8 && p.d != 16) return false;
  const int S = p.dtype == F32 ? 4 : 2;
  const int V = p.d < 4 ? p.d : 4, JG = p.d / V, W = 4;
  const int KT = p.b / 16;
  bool found = false;
  DmaChoice best{};
  // 16-bit types: 16x16x32 MFMAs (LP = 8, stages of 32 values of l) when
  // c % 32 == 0, or 16x16x16 (LP = 4, stages of 16: half the stage size).
  for (int LP = (S == 2 && p.c % 32 == 0) ? 8 : 4; LP >= 4; LP /= 2) {
    const int CH = 4 * LP, UR = CH * p.d * S / 16;
    for (int mt = 2; mt >= 1; --mt) {
      if (KT % mt) continue;
      const int kgroups = KT / mt;
      for (int nt = 1; nt * mt <= 4; nt *= 2) {
        for (int kgw = 1; kgw * JG <= W; ++kgw) {
          if (kgroups % kgw || W % (kgw * JG)) continue;
          const int rs = W / (kgw * JG);
          const int64_t units = (int64_t)16 * rs * nt * UR;
          if (units % (64 * W)) continue;
          const int64_t ud = units / (64 * W);
          if (ud != 2 && ud != 4 && ud != 8) continue;
          const int64_t stage = units * 16;
          const int64_t ytile = 16 * rs * nt * ((int64_t)16 * mt * kgw * p.d * S + 16);
          const int64_t sbuf = dma_stage_buffers(p.c / CH) * stage;
          const int64_t lds = sbuf > ytile ? sbuf : ytile;
          if (lds > kMaxLds) continue;
          const int kgt = kgroups / kgw;
          const int span = 16 * rs * nt;
          const int64_t tiles = (int64_t)((p.batch + span - 1) / span) * p.a * kgt;
          if (tiles > 0x7fffffff) continue;
          const DmaChoice c{LP, mt, nt, kgw, rs, kgt, tiles, lds};
          if (!found || dma_better(c, best, dma_lds_pref(p))) {
            found = true;
            best = c;
          }
        }
      }
    }
  }
  if (!found) return false;
  pl->variant = V_DMA;
  pl->vec = V;
  pl->unroll = p.d > V ? 1 : 0;
  pl->waves_m = best.mt;
  pl->waves_n = best.kgt;
  pl->jg = JG;
  pl->rs = best.rs;
  pl->kgw = best.kgw;
  pl->nt = best.nt;
  pl->lch = 4 * best.lp;
  pl->cps = best.lp;  // MFMA lane depth (4 or 8 values of l per lane group)
  pl->bt = 16 * best.rs * best.nt;
  pl->block = 64u * W;
  pl->grid = (unsigned)best.tiles;
  pl->xcd_remap = (best.kgt > 1 && best.tiles % 8 == 0) ? 1 : 0;
  const StagedTile t = staged_tile_of(p, *pl);
  if (t.lds > kMaxLds || t.UD * 64 * W * 16 != t.stage) return false;
  pl->lds_bytes = t.lds;
  return true;
}

hipError_t launch_dma(const Problem& p, const Plan& pl, hipStream_t s) {
  const StagedTile t = staged_tile_of(p, pl);
  if (p.layout == BSL) {
    switch (p.dtype) {
      case F32: return launch_dma_bsl_f32(p, t, pl.waves_m, s);
      case BF16: return launch_dma_bsl_bf16(p, t, pl.waves_m, s);
      case F16: return launch_dma_bsl_f16(p, t, pl.waves_m, s);
      default: return hipErrorInvalidValue;
    }
  }
  const int mode = pl.unroll ? 0 : (pl.vec == 4 ? 1 : (pl.vec == 2 ? 2 : 3));  // v4s, v4c, v2, v1
  if ((pl.unroll && pl.vec != 4) || (!pl.unroll && pl.vec != p.d)) return hipErrorInvalidValue;
#define KS_DMA_CALL(T)                                                 \
  switch (mode) {                                                      \
    case 0: return launch_dma_##T##_v4s(p, t, pl.waves_m, pl.cps, s);  \
    case 1: return launch_dma_##T##_v4c(p, t, pl.waves_m, pl.cps, s);  \
    case 2: return launch_dma_##T##_v2(p, t, pl.waves_m, pl.cps, s);   \
    default: return launch_dma_##T##_v1(p, t, pl.waves_m, pl.cps, s);  \
  }
  switch (p.dtype) {
    case F32: KS_DMA_CALL(f32)
    case BF16: KS_DMA_CALL(bf16)
    case F16: KS_DMA_CALL(f16)
    default: return hipErrorInvalidValue;
  }
#undef KS_DMA_CALL
}

hipError_t launch_staged(const Problem& p, const Plan& pl, hipStream_t s) {
  const StagedTile t = staged_tile_of(p, pl);
  const bool strided = pl.unroll != 0;
  switch (p.dtype) {
    case F32: return launch_staged_f32(p, t, pl.vec, strided, pl.waves_m, pl.cps, s);
    case BF16: return launch_staged_bf16(p, t, pl.vec, strided, pl.waves_m, pl.cps, s);
    case F16: return launch_staged_f16(p, t, pl.vec, strided, pl.waves_m, pl.cps, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ks
