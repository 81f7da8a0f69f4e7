// Index arithmetic of the register-direct MFMA kernels (ks_direct.h), shared by
// the kernels and by the host-side plan verifier (ks_plan_verify), so that both
// walk exactly the same addresses.
//
// Work decomposition (output-stationary, paper Section 4.1, Algorithm 2): one
// wavefront owns one item = (batch tile, i, j or j-group, k-group) and produces
//     Yt[k][beta] = sum_l Kv[i*d + j][k][l] * X[beta, i*c*d + l*d + j]
// for 16*MT output rows k of block (i, j), for all l < c, writing every output
// exactly once.  Lanes are (n, g) = (lane % 16, lane / 16), the MFMA operand
// layout: a lane's B operand holds the l values LPL*g .. LPL*g + LPL-1 of one
// chunk for "column" n, its accumulators the outputs k = 4g .. 4g+3.
//
//  * batch-size-last: column n is a group of V consecutive batch entries
//    (one 16-byte vector of a row of X or Y); the wave tile is 16*V batch
//    entries of one j.
//  * batch-size-first: column n is one batch row; the lane reads V consecutive
//    j (a 16-byte vector or less) per l, the wave tile is 16 batch rows of a
//    j-group of V consecutive j.  When V == d the lane's LPL x V block of
//    a row of X is contiguous ("contiguous" mode), else (V < d) it is LPL
//    vectors at stride d ("strided" mode).
//
// Each MFMA chain e < V owns one accumulator per M-tile: in BSL chain e is the
// batch entry V*n + e, in BSF it is block j0 + e.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

#include "ks_divide.h"
#include "ks_internal.h"

#define KS_HD __host__ __device__ __forceinline__

namespace ks {

struct DirectTile {
  int kgroups;   // b / (16*MT)
  int jgroups;   // BSL: d (one j per item); BSF: d / V
  int nbt;       // batch tiles (16*V entries in BSL, 16 rows in BSF)
  int items;     // nbt * a * jgroups * kgroups
  int waves;     // wavefronts per workgroup (1, 2 or 4)
  uint32_t mkg, mnbt, mjg;  // multiply-shift constants of the item decode (ks_divide.h)
  int skg, snbt, sjg;
};

struct DItem {
  int i, j0, k0, beta0;
};

// Reductions lengths with a specialised kernel instance (the chunk loop fully
// unrolled, loads issued several chunks ahead): c / CH full chunks of
// CH = 16 (fp32) or 32 (16-bit) values of l, plus a 16-value tail for 16-bit
// storage when c % 32 == 16.  Other c use the runtime-length kernel.
KS_HD bool direct_c_specialised(int esize, int c, int* nch, bool* tail) {
  if (esize == 4) {
    *nch = c / 16;
    *tail = false;
    return c % 16 == 0 && (*nch == 1 || *nch == 2 || *nch == 3 || *nch == 4 || *nch == 6 || *nch == 8);
  }
  *nch = c / 32;
  *tail = c % 32 == 16;
  return c % 16 == 0 && (c == 16 || c == 32 || c == 48 || c == 64 || c == 96 || c == 128);
}

// Item order: k-group fastest (items sharing X are neighbours, in the same
// workgroup when possible), then the batch tile (wavefronts running together
// stream neighbouring runs of the same rows of X and Y and share a K block),
// then j-group, then i.
KS_HD DItem direct_item(const Problem& p, const DirectTile& t, int V, int MT, int item) {
  DItem it;
  int rest = item;
  const int kg = rest % t.kgroups;
  rest /= t.kgroups;
  const int bt = rest % t.nbt;
  rest /= t.nbt;
  const int jg = rest % t.jgroups;
  it.i = rest / t.jgroups;
  it.k0 = kg * 16 * MT;
  if (p.layout == BSL) {
    it.j0 = jg;
    it.beta0 = bt * 16 * V;
  } else {
    it.j0 = jg * V;
    it.beta0 = bt * 16;
  }
  return it;
}

// direct_item with the divisions done by multiply and shift (the kernels'
// form; the plan verifier checks it against direct_item for every item).
KS_HD DItem direct_item_fast(const Problem& p, const DirectTile& t, int V, int MT, int item) {
  DItem it;
  const uint32_t q1 = div_fast((uint32_t)item, t.mkg, t.skg);
  const int kg = item - (int)q1 * t.kgroups;
  const uint32_t q2 = div_fast(q1, t.mnbt, t.snbt);
  const int bt = (int)q1 - (int)q2 * t.nbt;
  const uint32_t q3 = div_fast(q2, t.mjg, t.sjg);
  const int jg = (int)q2 - (int)q3 * t.jgroups;
  it.i = (int)q3;
  it.k0 = kg * 16 * MT;
  if (p.layout == BSL) {
    it.j0 = jg;
    it.beta0 = bt * 16 * V;
  } else {
    it.j0 = jg * V;
    it.beta0 = bt * 16;
  }
  return it;
}

// ---- X loads ----------------------------------------------------------------
// A lane's chunk block is LPL x V elements, flat index t*V + e (t: the l offset
// LPL*g + t within the chunk, e: chain).  It is loaded as pieces of PE
// contiguous elements; piece q covers flat indices [q*PE, (q+1)*PE).
//   BSL / BSF strided:  pieces are the LPL rows t (PE = V);
//   BSF contiguous:     the block is contiguous, PE = min(LPL*V, 16 bytes).
// The offset of piece q of the chunk starting at l0 is
//     base + l0 * lstride + q * qstride
// with a per-lane base and strides that are uniform over the wavefront.  A
// lane whose column lies beyond the batch reads the last column instead (in
// bounds; its outputs are never stored), so the loads need no branches.
KS_HD int direct_x_piece_elems(int layout, bool strided, int LPL, int V, int esize) {
  if (layout == BSL || strided) return V;
  const int all = LPL * V, vec = 16 / esize;
  return all < vec ? all : vec;
}
KS_HD int direct_x_pieces(int layout, bool strided, int LPL, int V, int esize) {
  return (LPL * V) / direct_x_piece_elems(layout, strided, LPL, V, esize);
}
// Elements between consecutive l of one column.
KS_HD int64_t direct_x_lstride(const Problem& p) { return p.layout == BSL ? (int64_t)p.d * p.batch : p.d; }
KS_HD int64_t direct_x_qstride(const Problem& p, bool strided, int LPL, int V, int esize) {
  if (p.layout == BSL || strided) return direct_x_lstride(p);
  return direct_x_piece_elems(p.layout, strided, LPL, V, esize);
}
// True when the lane's column holds real batch entries (its outputs are stored).
KS_HD bool direct_lane_valid(const Problem& p, const DItem& it, int V, int n) {
  return p.layout == BSL ? it.beta0 + V * n < p.batch : it.beta0 + n < p.batch;
}
KS_HD int64_t direct_x_base(const Problem& p, const DItem& it, int LPL, int V, int n, int g) {
  const int c = p.c, d = p.d;
  if (p.layout == BSL) {
    int beta = it.beta0 + V * n;
    if (beta >= p.batch) beta = p.batch - V;
    const int64_t row = (int64_t)it.i * c * d + (int64_t)(LPL * g) * d + it.j0;
    return row * p.batch + beta;
  }
  int beta = it.beta0 + n;
  if (beta >= p.batch) beta = p.batch - 1;
  return (int64_t)beta * p.N + (int64_t)it.i * c * d + (int64_t)(LPL * g) * d + it.j0;
}
KS_HD int64_t direct_x_off(const Problem& p, const DItem& it, bool strided, int LPL, int V, int esize, int l0,
                           int n, int g, int q) {
  return direct_x_base(p, it, LPL, V, n, g) + (int64_t)l0 * direct_x_lstride(p) +
         (int64_t)q * direct_x_qstride(p, strided, LPL, V, esize);
}

// ---- K loads ----------------------------------------------------------------
// A operand of M-tile mt, chain e: LPL contiguous values of row k of block
// (i, j), starting at l = l0 + LPL*g (lane (m, g), m = lane % 16).
// Written as base + mt * 16*c + e * b*c + l0 (chain e is block j0 + e in BSF).
KS_HD int64_t direct_k_base(const Problem& p, const DItem& it, int LPL, int m, int g) {
  return ((int64_t)(it.i * p.d + it.j0) * p.b + it.k0 + m) * p.c + LPL * g;
}
KS_HD int64_t direct_k_off(const Problem& p, const DItem& it, int LPL, int l0, int m, int g, int mt, int e) {
  const int eb = p.layout == BSL ? 0 : e;
  return direct_k_base(p, it, LPL, m, g) + (int64_t)mt * 16 * p.c + (int64_t)eb * p.b * p.c + l0;
}

// ---- Y stores ---------------------------------------------------------------
// Per M-tile a lane holds 4 x V outputs (r = 0..3: k = k0 + 16*mt + 4g + r;
// e: chain), flat index r*V + e, stored as pieces of PE contiguous elements.
//   BSL / BSF strided: pieces are the 4 values of r (PE = V);
//   BSF contiguous:    the 4*V outputs are contiguous, PE = min(4V, 16 bytes).
KS_HD int direct_y_piece_elems(int layout, bool strided, int V, int esize) {
  if (layout == BSL || strided) return V;
  const int all = 4 * V, vec = 16 / esize;
  return all < vec ? all : vec;
}
KS_HD int direct_y_pieces(int layout, bool strided, int V, int esize) {
  return (4 * V) / direct_y_piece_elems(layout, strided, V, esize);
}
// Per-lane base (mt = 0, q = 0) and uniform strides of the output pieces:
//     off = base + mt * mstride + q * qstride.
KS_HD int64_t direct_y_base(const Problem& p, const DItem& it, int V, int n, int g) {
  const int b = p.b, d = p.d;
  const int kb = it.k0 + 4 * g;
  if (p.layout == BSL) {
    const int64_t row = (int64_t)it.i * b * d + (int64_t)kb * d + it.j0;
    return row * p.batch + it.beta0 + V * n;
  }
  return (int64_t)(it.beta0 + n) * p.M + (int64_t)it.i * b * d + (int64_t)kb * d + it.j0;
}
KS_HD int64_t direct_y_mstride(const Problem& p) { return p.layout == BSL ? (int64_t)16 * p.d * p.batch : 16 * p.d; }
KS_HD int64_t direct_y_qstride(const Problem& p, bool strided, int V, int esize) {
  if (p.layout == BSL) return (int64_t)p.d * p.batch;
  if (strided) return p.d;
  return direct_y_piece_elems(p.layout, strided, V, esize);
}
// Offset of output piece q of M-tile mt, or -1 when the lane's column lies
// beyond the batch (nothing stored).
KS_HD int64_t direct_y_off(const Problem& p, const DItem& it, bool strided, int V, int esize, int mt, int n, int g,
                           int q) {
  if (!direct_lane_valid(p, it, V, n)) return -1;
  return direct_y_base(p, it, V, n, g) + (int64_t)mt * direct_y_mstride(p) +
         (int64_t)q * direct_y_qstride(p, strided, V, esize);
}

}  // namespace ks
