// Index arithmetic of the LDS-staged MFMA kernels (ks_staged.h), shared by the
// kernels and by the host-side plan verifier (ks_plan_verify).
//
// A workgroup of W wavefronts owns one tile: the X values a set of W work
// items share (paper Section 4.1, Algorithm 2: output-stationary, every output
// written once).  The reduction over l is walked in stages of LCH values; the
// workgroup loads a stage of X with coalesced 16-byte loads (consecutive
// threads take consecutive 16-byte units of a contiguous run of memory) into a
// double-buffered LDS tile, and each wavefront reads its MFMA operands from
// LDS.
//
//  * batch-size-first: a tile is 16*RS batch rows of one i, all d values of j
//    and KGW k-groups.  Stage rows are the runs X[beta, i*c*d + ls*d ..
//    (ls + nl)*d) (all j of nl values of l, contiguous); LDS row r holds batch
//    row beta0 + r with a 16-byte pad per row (bank spread).
//  * batch-size-last: a tile is 16*V*RS batch entries of one (i, j) and KGW
//    k-groups.  Stage rows are the input rows of l = ls .. ls + nl - 1, each
//    16*V*RS contiguous batch entries.
//
// Wavefront w of the tile takes rs = w % RS, jg = (w / RS) % JG and
// kgw = w / (RS * JG) (W = RS * JG * KGW <= 8), i.e. the work item
// (rows or columns group rs, j-group jg, k-group kt*KGW + kgw).  In the
// batch-size-first DMA kernel a wavefront's rows group is NT consecutive
// groups of 16 rows (tile rows 16*RS*NT), so each K operand it loads serves
// 16*NT rows.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

#include "ks_divide.h"
#include "ks_internal.h"

#define KS_HD __host__ __device__ __forceinline__

namespace ks {

struct StagedTile {
  int W;         // wavefronts per workgroup: RS * JG * KGW
  int RS;        // 16-row (BSF) or 16*V-column (BSL) groups per tile
  int JG;        // j-groups per tile (BSF: d / V; BSL: 1)
  int KGW;       // k-groups per tile
  int kgt;       // k-group tiles: b / (16 * MT * KGW)
  int nbt;       // batch tiles
  int tiles;     // nbt * a * (BSL ? d : 1) * kgt
  int LCH;       // l values per stage (a multiple of 16)
  int pitch;     // LDS row pitch, bytes
  int stage;     // LDS bytes of one stage buffer
  int remap;     // XCD-aware tile order (tiles % 8 == 0)
  int ypitch;    // BSF: LDS row pitch of the staged output tile, bytes
  int lds;       // LDS bytes per workgroup: max(2 * stage, BSF output tile)
  // LDS-DMA kernel (ks_dma.h) only, 0 otherwise:
  int UR;        // 16-byte units per stage row (LCH * d * esize / 16, a power of two)
  int UD;        // DMA instructions (64 units each) per wavefront per stage
  int NT;        // batch-size-first: 16-row groups per wavefront (1 except in the DMA kernel)
  // DMA kernel: log2 of the power-of-two sizes, and multiply-shift constants
  // for the divisions of the tile decode (div_fast, ks_divide.h).
  int lUR, lRS, lJG, lUY;
  uint32_t mkgt, mnbt, md;
  int skgt, snbt, sd;
};



struct STile {
  int i, j, kt, bt;  // j: BSL only
};

// Workgroup g runs on XCD g % 8; give each XCD a contiguous range of logical
// tiles so that tiles sharing X (neighbouring k-group tiles) share an L2.
KS_HD int staged_remap(int g, int tiles) { return (g & 7) * (tiles >> 3) + (g >> 3); }

// Tile order: k-group tile fastest, then the batch tile (tiles running
// together read neighbouring rows or runs of X and share K), then j (BSL),
// then i.
KS_HD STile staged_tile(const Problem& p, const StagedTile& t, int block) {
  const int tile = t.remap ? staged_remap(block, t.tiles) : block;
  STile s;
  int rest = tile;
  s.kt = rest % t.kgt;
  rest /= t.kgt;
  s.bt = rest % t.nbt;
  rest /= t.nbt;
  if (p.layout == BSL) {
    s.j = rest % p.d;
    rest /= p.d;
  } else {
    s.j = 0;
  }
  s.i = rest;
  return s;
}

// Number of batch entries a tile spans.
KS_HD int staged_span(const Problem& p, const StagedTile& t, int V) {
  return p.layout == BSL ? 16 * V * t.RS : 16 * t.RS * t.NT;
}

// ---- stage loads ----------------------------------------------------------
// Stage rows and 16-byte units per row for a stage of nl values of l.
KS_HD int staged_rows(const Problem& p, const StagedTile& t, int nl) {
  return p.layout == BSL ? nl : 16 * t.RS * t.NT;
}
KS_HD int staged_units_per_row(const Problem& p, const StagedTile& t, int V, int esize, int nl) {
  return p.layout == BSL ? (16 * V * t.RS * esize) / 16 : (nl * p.d * esize) / 16;
}
// Element offset in X of unit v of stage row r (stage starting at l = ls);
// rows or columns beyond the batch read the last valid one instead.
KS_HD int64_t staged_x_unit(const Problem& p, const StagedTile& t, const STile& s, int V, int esize, int ls, int r,
                            int v) {
  const int ue = 16 / esize;  // elements per unit
  const int c = p.c, d = p.d;
  if (p.layout == BSL) {
    int beta = s.bt * 16 * V * t.RS + v * ue;
    if (beta >= p.batch) beta = p.batch - ue;
    const int64_t row = (int64_t)s.i * c * d + (int64_t)(ls + r) * d + s.j;
    return row * p.batch + beta;
  }
  int beta = s.bt * 16 * t.RS * t.NT + r;
  if (beta >= p.batch) beta = p.batch - 1;
  return (int64_t)beta * p.N + (int64_t)s.i * c * d + (int64_t)ls * d + (int64_t)v * ue;
}
// LDS byte offset of unit v of stage row r within a stage buffer.
KS_HD int staged_lds_unit(const StagedTile& t, int r, int v) { return r * t.pitch + v * 16; }

// ---- operand reads from LDS -----------------------------------------------
// Work item of wavefront w in tile s.
struct SItem {
  int rs, jg, kgw;
  int j0, k0, beta0;
};
KS_HD SItem staged_item(const Problem& p, const StagedTile& t, const STile& s, int V, int MT, int w) {
  SItem it;
  it.rs = w % t.RS;
  it.jg = (w / t.RS) % t.JG;
  it.kgw = w / (t.RS * t.JG);
  it.k0 = (s.kt * t.KGW + it.kgw) * 16 * MT;
  if (p.layout == BSL) {
    it.j0 = s.j;
    it.beta0 = s.bt * 16 * V * t.RS + it.rs * 16 * V;
  } else {
    it.j0 = it.jg * V;
    it.beta0 = (s.bt * t.RS + it.rs) * 16 * t.NT;
  }
  return it;
}
// A lane's operand block of an MFMA chunk at l = l0 (relative to the stage
// start) is LP x V elements (flat t*V + e), read as pieces of PE elements:
// piece q at LDS byte offset base + q * qstride (+ l0 * lstride).
//   BSL:            row LP*g + q (l), columns 16*V*rs + V*n .. + V;
//   BSF strided:    row 16*rs + n, elements (LP*g + q)*d + j0 .. + V;
//   BSF contiguous: row 16*rs + n, elements (LP*g)*d + q*PE .. + PE (V == d).
KS_HD int staged_op_base(const Problem& p, const StagedTile& t, const SItem& it, int LP, int V, int esize, int n,
                         int g) {
  if (p.layout == BSL) return (LP * g) * t.pitch + (it.rs * 16 * V + V * n) * esize;
  return (it.rs * 16 + n) * t.pitch + ((LP * g) * p.d + it.j0) * esize;
}
KS_HD int staged_op_lstride(const Problem& p, const StagedTile& t, int esize) {
  return p.layout == BSL ? t.pitch : p.d * esize;
}
KS_HD int staged_op_qstride(const Problem& p, const StagedTile& t, bool strided, int pe, int esize) {
  if (p.layout == BSL) return t.pitch;
  return strided ? p.d * esize : pe * esize;
}

// ---- batch-size-first output tile ------------------------------------------
// In BSF the tile's outputs of a batch row are the contiguous run
// Y[beta, i*b*d + kb*d .. i*b*d + (kb + KR)*d) with kb = kt*KGW*16*MT and
// KR = 16*MT*KGW (all j of KR consecutive k).  The wavefronts write their
// accumulators into an LDS copy of the tile (row r at r * ypitch) and the
// workgroup stores it with coalesced 16-byte units ("structured epilogue").
KS_HD int staged_y_kr(const StagedTile& t, int MT) { return 16 * MT * t.KGW; }
// LDS byte offset of output element (row r, k, j) of the tile.
KS_HD int staged_y_lds(const Problem& p, const StagedTile& t, const STile& s, int MT, int esize, int r, int k, int j) {
  const int kb = s.kt * t.KGW * 16 * MT;
  return r * t.ypitch + ((k - kb) * p.d + j) * esize;
}
// 16-byte units per row of the output tile and the Y offset (elements) of
// unit v of tile row r, or -1 beyond the batch.
KS_HD int staged_y_units_per_row(const Problem& p, const StagedTile& t, int MT, int esize) {
  return staged_y_kr(t, MT) * p.d * esize / 16;
}
KS_HD int64_t staged_y_unit(const Problem& p, const StagedTile& t, const STile& s, int MT, int esize, int r, int v) {
  const int beta = s.bt * 16 * t.RS * t.NT + r;
  if (beta >= p.batch) return -1;
  const int kb = s.kt * t.KGW * 16 * MT;
  return (int64_t)beta * p.M + (int64_t)s.i * p.b * p.d + (int64_t)kb * p.d + (int64_t)v * (16 / esize);
}

// ---- LDS-DMA stages (ks_dma.h) ---------------------------------------------
// Batch-size-first (the batch-size-last form follows further down).  A stage buffer holds 16*RS*NT rows of UR 16-byte
// units with no padding; logical unit v of row r sits at physical unit
// v ^ swizzle(r) of that row, which puts the same logical unit of 16
// consecutive rows (what an operand read touches) at 16 distinct 16-byte
// positions of a 256-byte bank line: swizzle(r) = r mod 16 for rows of 16
// units or more, else the row's index among the rows sharing a position,
// (r * UR / 16) mod UR.  DMA instruction m of wavefront w writes the 64
// consecutive physical units (m*W + w)*64 + lane, so each lane loads the
// logical unit that lands there.
KS_HD int dma_swizzle(const StagedTile& t, int r) {
  const int wide = r & 15;
  const int narrow = (int)((((uint32_t)r * (uint32_t)t.UR) >> 4) & (uint32_t)(t.UR - 1));
  return t.UR >= 16 ? wide : narrow;  // both computed: a select, not a branch
}
// Physical unit P of a stage buffer -> row r and logical unit v.
KS_HD void dma_unit_of(const StagedTile& t, int P, int* r, int* v) {
  *r = P / t.UR;
  *v = (P % t.UR) ^ dma_swizzle(t, *r);
}
// Physical unit written by lane `lane` of DMA instruction m of wavefront w.
KS_HD int dma_phys_unit(const StagedTile& t, int m, int w, int lane) { return (m * t.W + w) * 64 + lane; }
// LDS byte offset (within a stage buffer) of logical byte b of row r.
KS_HD int dma_lds_byte(const StagedTile& t, int r, int b) {
  return (r * t.UR + ((b >> 4) ^ dma_swizzle(t, r))) * 16 + (b & 15);
}
// Byte (within its stage row) of piece q of chunk l0 for lane (n, g), item it
// (the operand layout of staged_op_base: strided pieces of V elements at
// stride d, contiguous pieces of PE elements).
KS_HD int dma_op_byte(const Problem& p, const SItem& it, int LP, int V, bool strided, int pe, int esize, int l0, int g,
                      int q) {
  if (strided) return ((l0 + LP * g + q) * p.d + it.j0) * esize;
  return ((l0 + LP * g) * p.d + it.j0) * esize + q * pe * esize;
}

// Stage buffers the DMA kernel uses for nst stages of l: three (stage s is
// multiplied while s+1 and s+2 are in flight), or one per stage when there
// are fewer; with one or two stages no DMA targets the third buffer, so it is
// not allocated (more workgroups fit in a CU's LDS).
KS_HD int dma_stage_buffers(int nst) { return nst < 3 ? nst : 3; }

// Logical tile of workgroup `block` in the DMA kernels: the XCD remap when
// t.remap is set, else the identity, selected without a branch (both forms
// computed), so that the tile count arrives with the other kernel arguments
// instead of in a second round of scalar loads behind the test of t.remap.
KS_HD uint32_t dma_tile_index(const StagedTile& t, int block) {
  const uint32_t rm = (uint32_t)staged_remap(block, t.tiles);
  const uint32_t mask = 0u - (uint32_t)(t.remap != 0);
  return (rm & mask) | ((uint32_t)block & ~mask);
}

// Tile and work item of the DMA kernel: staged_tile and staged_item computed
// with the multiply-shift divisions and the power-of-two shifts above (the
// plan verifier checks both against the plain forms for every tile).
KS_HD STile dma_tile(const StagedTile& t, int block) {
  const uint32_t tile = dma_tile_index(t, block);
  STile s;
  const uint32_t q1 = div_fast(tile, t.mkgt, t.skgt);
  s.kt = (int)(tile - q1 * (uint32_t)t.kgt);
  const uint32_t q2 = div_fast(q1, t.mnbt, t.snbt);
  s.bt = (int)(q1 - q2 * (uint32_t)t.nbt);
  s.j = 0;
  s.i = (int)q2;
  return s;
}
KS_HD SItem dma_item(const StagedTile& t, const STile& s, int V, int MT, int w) {
  SItem it;
  it.rs = w & (t.RS - 1);
  it.jg = (w >> t.lRS) & (t.JG - 1);
  it.kgw = w >> (t.lRS + t.lJG);
  it.k0 = (s.kt * t.KGW + it.kgw) * 16 * MT;
  it.j0 = it.jg * V;
  it.beta0 = (s.bt * t.RS + it.rs) * 16 * t.NT;
  return it;
}
// Physical unit P of a stage buffer -> row r and logical unit v (UR a power of two).
KS_HD void dma_unit_of_fast(const StagedTile& t, int P, int* r, int* v) {
  *r = (int)((uint32_t)P >> t.lUR);
  *v = (int)(((uint32_t)P & (uint32_t)(t.UR - 1)) ^ (uint32_t)dma_swizzle(t, *r));
}

// Output tile of the DMA kernel: LDS byte offset of the lane's first output
// (row group 0, M-tile 0, r = 0); output (u, mt, r) is u*16*ypitch +
// (16*mt + r)*d*esize further.  Y element offset of output-tile row `row`
// relative to the tile's first row, and that first row's offset.
KS_HD int dma_y_lds_lane(const Problem& p, const StagedTile& t, const SItem& it, int MT, int esize, int n, int g) {
  return (16 * t.NT * it.rs + n) * t.ypitch + ((it.kgw * 16 * MT + 4 * g) * p.d + it.j0) * esize;
}
KS_HD int64_t dma_y_tile_base(const Problem& p, const StagedTile& t, const STile& s, int MT) {
  return (int64_t)s.bt * 16 * t.RS * t.NT * p.M + (int64_t)s.i * p.b * p.d + (int64_t)s.kt * t.KGW * 16 * MT * p.d;
}
KS_HD int dma_y_row(const Problem& p, int row, int v, int esize) { return row * p.M + v * (16 / esize); }

// ---- LDS-DMA stages, batch-size-last (ks_dma_bsl.h) --------------------------
// A tile is 16*V*RS consecutive batch entries (V = 16 / esize: one 16-byte
// unit per lane column) of one (i, j), and KGW k-groups of 16*MT rows; the
// four wavefronts take rs = w % RS, kgw = w / RS.  A stage buffer holds the
// input rows of CH consecutive values of l, each the tile's UR = 16*RS units
// of one row of X (unpadded: the sixteen lanes of an operand read take one
// row's 256 contiguous bytes).  DMA instruction m of wavefront w writes the
// 64 physical units (m*W + w)*64 + lane: stage row P / UR, unit P % UR.
KS_HD void dma_bsl_unit_of(const StagedTile& t, int P, int* r, int* v) {
  *r = (int)((uint32_t)P >> t.lUR);
  *v = (int)((uint32_t)P & (uint32_t)(t.UR - 1));
}
// X element offset of unit v of stage row r, relative to the stage's first
// row: the unit holds batch entries bt*16*V*RS + V*v .. + V of row
// i*c*d + (ls + r)*d + j (the stage and i parts, (i*c*d + ls*d) * batch, are
// added by the kernel as pointer steps).  Units beyond the batch read the
// last unit of the row instead (the batch is a multiple of V).
KS_HD int dma_bsl_src(const Problem& p, const StagedTile& t, const STile& s, int V, int r, int v) {
  int beta = s.bt * 16 * V * t.RS + V * v;
  if (beta >= p.batch) beta = p.batch - V;
  return (r * p.d + s.j) * p.batch + beta;
}
// LDS byte offset (within a stage buffer) of operand piece q of lane (n, g):
// stage row LP*g + q (value l of the MFMA chunk), the lane's unit 16*rs + n.
KS_HD int dma_bsl_op_byte(const StagedTile& t, const SItem& it, int LP, int n, int g, int q) {
  return ((LP * g + q) * t.UR + 16 * it.rs + n) * 16;
}
// Tile and work item with multiply-shift divisions (staged_tile and
// staged_item for batch-size-last; the verifier compares them).
KS_HD STile dma_bsl_tile(const Problem& p, const StagedTile& t, int block) {
  const uint32_t tile = dma_tile_index(t, block);
  STile s;
  const uint32_t q1 = div_fast(tile, t.mkgt, t.skgt);
  s.kt = (int)(tile - q1 * (uint32_t)t.kgt);
  const uint32_t q2 = div_fast(q1, t.mnbt, t.snbt);
  s.bt = (int)(q1 - q2 * (uint32_t)t.nbt);
  const uint32_t q3 = div_fast(q2, t.md, t.sd);
  s.j = (int)(q2 - q3 * (uint32_t)p.d);
  s.i = (int)q3;
  return s;
}
KS_HD SItem dma_bsl_item(const StagedTile& t, const STile& s, int V, int MT, int w) {
  SItem it;
  it.rs = w & (t.RS - 1);
  it.jg = 0;
  it.kgw = w >> t.lRS;
  it.k0 = (s.kt * t.KGW + it.kgw) * 16 * MT;
  it.j0 = s.j;
  it.beta0 = s.bt * 16 * V * t.RS + it.rs * 16 * V;
  return it;
}

}  // namespace ks
