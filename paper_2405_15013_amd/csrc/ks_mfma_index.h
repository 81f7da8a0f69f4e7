// Index arithmetic of the MFMA kernel, shared by the kernel itself and by the
// host-side plan verifier (ks_plan_verify), so both walk exactly the same
// addresses.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

#include "ks_internal.h"

#define KS_HD __host__ __device__ __forceinline__

namespace ks {

// Loader modes (how the X tile is laid out in global memory).
enum LoadMode : int {
  LM_BSL = 0,       // c rows, each BT contiguous batch columns
  LM_BSF_RUNS = 1,  // per batch row, c runs of JG contiguous j (JG a multiple of VEC)
  LM_BSF_SEG = 2    // per batch row, one contiguous segment of c*d elements (JG == d)
};

struct MfmaTile {
  int bt;     // batch vectors per tile (multiple of 16*MT)
  int jg;     // j values per tile
  int njg;    // d / jg
  int nbt;    // number of batch tiles
  int mode;   // LoadMode
  int remap;  // XCD-aware tile order
  int vec;    // elements per 16-byte chunk
};

constexpr int kMaxChunks = 16;  // 16-byte X chunks per thread per tile

// Workgroup w runs on XCD w % 8; give each XCD a contiguous range of logical
// tiles so that tiles sharing cache lines run on the same L2 (g % 8 == 0).
KS_HD int xcd_remap(int w, int g) { return (w & 7) * (g >> 3) + (w >> 3); }

struct TileCoord {
  int i, j0, beta0;
};

KS_HD TileCoord tile_coord(const Problem& p, const MfmaTile& t, int block, int grid) {
  const int tile = t.remap ? xcd_remap(block, grid) : block;
  const int jgi = tile % t.njg;
  const int rest = tile / t.njg;
  TileCoord tc;
  tc.i = rest % p.a;
  tc.j0 = jgi * t.jg;
  tc.beta0 = (rest / p.a) * t.bt;
  return tc;
}

// LDS row pitch of Xs[jj][beta][l] in elements (16 bytes of padding).
KS_HD int x_pitch(const Problem& p, const MfmaTile& t) { return p.c + t.vec; }
// Number of 16-byte chunks in an X tile.
KS_HD int x_chunks(const Problem& p, const MfmaTile& t) { return (p.c * t.bt * t.jg) / t.vec; }

// Chunk q of the X tile: offset (elements) of its first element in X, or -1
// when it lies beyond the batch (then the tile is zero-filled there).  Within a
// group of 16 consecutive chunks l varies fastest (BSL, BSF runs), so the
// transposing LDS writes of a wavefront hit distinct banks.
KS_HD int64_t x_chunk_src(const Problem& p, const MfmaTile& t, const TileCoord& tc, int q) {
  const int c = p.c, d = p.d, V = t.vec;
  if (p.layout == BSL) {
    const int nv = t.bt / V;
    const int l = (q / (16 * nv)) * 16 + (q & 15);
    const int beta = tc.beta0 + ((q >> 4) % nv) * V;
    if (beta >= p.batch) return -1;
    return (int64_t)(tc.i * c * d + l * d + tc.j0) * p.batch + beta;
  }
  if (t.mode == LM_BSF_RUNS) {
    const int nv = t.jg / V;
    const int l = ((q / (16 * nv)) % (c >> 4)) * 16 + (q & 15);
    const int v = (q >> 4) % nv;
    const int beta = tc.beta0 + q / (nv * c);
    if (beta >= p.batch) return -1;
    return (int64_t)beta * p.N + tc.i * c * d + l * d + tc.j0 + v * V;
  }
  const int nv = (c * d) / V;
  const int beta = tc.beta0 + q / nv;
  if (beta >= p.batch) return -1;
  return (int64_t)beta * p.N + tc.i * c * d + (q % nv) * V;
}

// LDS element index in Xs of element e (< vec) of chunk q.
KS_HD int x_chunk_lds(const Problem& p, const MfmaTile& t, int q, int e) {
  const int c = p.c, V = t.vec, P = x_pitch(p, t);
  if (p.layout == BSL) {
    const int nv = t.bt / V;
    const int l = (q / (16 * nv)) * 16 + (q & 15);
    return (((q >> 4) % nv) * V + e) * P + l;
  }
  if (t.mode == LM_BSF_RUNS) {
    const int nv = t.jg / V;
    const int l = ((q / (16 * nv)) % (c >> 4)) * 16 + (q & 15);
    const int v = (q >> 4) % nv;
    const int beta = q / (nv * c);
    return ((v * V + e) * t.bt + beta) * P + l;
  }
  const int nv = (c * p.d) / V;
  const int f = (q % nv) * V + e;
  const int l = f / p.d, jj = f - (f / p.d) * p.d;
  return (jj * t.bt + q / nv) * P + l;
}

// BSF epilogue: pitch of Ys[beta][k*JG + jj] and the destination of chunk q.
KS_HD int y_pitch(const Problem& p, const MfmaTile& t) { return p.b * t.jg + t.vec; }
KS_HD int y_chunks(const Problem& p, const MfmaTile& t) { return t.bt * ((p.b * t.jg) / t.vec); }
KS_HD int64_t y_chunk_dst(const Problem& p, const MfmaTile& t, const TileCoord& tc, int q, int* lds) {
  const int segv = (p.b * t.jg) / t.vec;
  const int beta = q / segv;
  const int e0 = (q - beta * segv) * t.vec;
  *lds = beta * y_pitch(p, t) + e0;
  if (tc.beta0 + beta >= p.batch) return -1;
  const int col = tc.i * p.b * p.d + (e0 / t.jg) * p.d + tc.j0 + (e0 % t.jg);
  return (int64_t)(tc.beta0 + beta) * p.M + col;
}

// Work item `it` of a tile: (jj, m-group, n-group).
struct Item {
  int jj, mgi, ngi;
};
KS_HD int mfma_items(const Problem& p, const MfmaTile& t, int MT, int NT) {
  return t.jg * (t.bt / (16 * MT)) * ((p.b >> 4) / NT);
}
KS_HD Item mfma_item(const Problem& p, const MfmaTile& t, int MT, int NT, int it) {
  const int ngroups = (p.b >> 4) / NT;
  const int mgroups = t.bt / (16 * MT);
  Item r;
  r.ngi = it % ngroups;
  const int r2 = it / ngroups;
  r.mgi = r2 % mgroups;
  r.jj = r2 / mgroups;
  return r;
}

}  // namespace ks
