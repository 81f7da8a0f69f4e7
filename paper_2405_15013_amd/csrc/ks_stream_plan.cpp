// Planner and launcher of the streaming MFMA kernels (ks_stream.h).
//
// Same vector width V as the register-direct kernels and the largest MT that
// leaves at least 8 tiles per SIMD.  The number of wavefronts is one resident
// round of the kernel instance, known only on the device: the launcher asks
// the runtime for it; the plan records a stand-in round of 2048 wavefronts
// (2 per SIMD), which is what the host verifier replays (the partition of the
// tiles into equal shares is valid for any number of wavefronts).
#include "ks_stream_index.h"

namespace ks {

#define KS_STREAM_DECL(NAME)                                                                                   \
  hipError_t NAME(const Problem& p, const StreamTile& t, int V, bool strided, int mt, unsigned grid, \
                  hipStream_t s);
KS_STREAM_DECL(launch_stream_f32_bsl)
KS_STREAM_DECL(launch_stream_f32_bsf)
KS_STREAM_DECL(launch_stream_bf16_bsl)
KS_STREAM_DECL(launch_stream_bf16_bsf)
KS_STREAM_DECL(launch_stream_f16_bsl)
KS_STREAM_DECL(launch_stream_f16_bsf)
#undef KS_STREAM_DECL

namespace {
constexpr int64_t kRoundStandIn = 2048;

// Largest MT instantiated; keep in sync with direct_mt_max() in ks_direct.h.
int mt_max(int layout, int V) { return (layout == BSL || V <= 2) ? 4 : 2; }
}  // namespace

StreamTile stream_tile_of(const Problem& p, const Plan& pl) {
  StreamTile t;
  const int V = pl.vec, MT = pl.waves_m;
  t.kgroups = p.b / (16 * MT);
  t.jgroups = p.layout == BSL ? p.d : p.d / V;
  const int span = p.layout == BSL ? 16 * V : 16;
  t.nbt = (p.batch + span - 1) / span;
  t.tiles = t.kgroups * t.nbt * t.jgroups * p.a;
  t.waves = 4;
  t.nwaves = (int)pl.grid * 4 < t.tiles ? (int)pl.grid * 4 : t.tiles;
  return t;
}

bool plan_stream(const Problem& p, bool al16, Plan* pl) {
  if (!al16 || p.b % 16 || p.c % 16) return false;
  const int vec = 4;  // kDirectVec in ks_direct.h
  int V;
  bool strided = false;
  if (p.layout == BSL) {
    V = vec;
    if (p.batch % V) return false;
  } else {
    V = p.d < vec ? p.d : vec;
    if ((V != 1 && V != 2 && V != 4) || p.d % V) return false;
    strided = V < p.d;
  }
  const int kt = p.b / 16;
  const int span = p.layout == BSL ? 16 * V : 16;
  const int64_t nbt = (p.batch + span - 1) / span;
  const int64_t per_k = nbt * p.a * (p.layout == BSL ? p.d : p.d / V);  // tiles per k-group
  int mt = 1;
  for (int m = mt_max(p.layout, V); m >= 1; --m) {
    if (kt % m) continue;
    mt = m;
    if (per_k * (kt / m) >= 8 * 1024) break;
  }
  const int64_t tiles = per_k * (kt / mt);
  if (tiles > 0x7fffffff) return false;
  const int64_t nwaves = tiles < kRoundStandIn ? tiles : kRoundStandIn;
  pl->variant = V_STREAM;
  pl->vec = V;
  pl->unroll = strided ? 1 : 0;
  pl->waves_m = mt;
  pl->waves_n = kt / mt;
  pl->bt = (int)((tiles + nwaves - 1) / nwaves);  // tiles per wavefront (stand-in round)
  pl->jg = p.layout == BSL ? 1 : V;
  pl->lds_bytes = 0;
  pl->block = 256;
  pl->grid = (unsigned)((nwaves + 3) / 4);
  pl->xcd_remap = 0;
  return true;
}

hipError_t launch_stream(const Problem& p, const Plan& pl, hipStream_t s) {
  const StreamTile t = stream_tile_of(p, pl);
  const bool strided = pl.unroll != 0;
  const bool bsl = p.layout == BSL;
  switch (p.dtype) {
    case F32:
      return bsl ? launch_stream_f32_bsl(p, t, pl.vec, strided, pl.waves_m, pl.grid, s)
                 : launch_stream_f32_bsf(p, t, pl.vec, strided, pl.waves_m, pl.grid, s);
    case BF16:
      return bsl ? launch_stream_bf16_bsl(p, t, pl.vec, strided, pl.waves_m, pl.grid, s)
                 : launch_stream_bf16_bsf(p, t, pl.vec, strided, pl.waves_m, pl.grid, s);
    case F16:
      return bsl ? launch_stream_f16_bsl(p, t, pl.vec, strided, pl.waves_m, pl.grid, s)
                 : launch_stream_f16_bsf(p, t, pl.vec, strided, pl.waves_m, pl.grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ks
