// Host-side plan verifier: replays, on the CPU, the address arithmetic every
// thread of the planned launch would perform, and checks that all global reads
// and writes stay inside their tensors, that every MFMA operand element a lane
// reads (from memory or from an LDS stage written in the same stage) is the X
// value the product needs, and that every element of Y is written exactly once
// (the partition property of the row/col index sets, paper Section 4.1).
// Nothing is enqueued on a GPU.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/ks.h"
#include "ks_internal.h"
#include "ks_direct_index.h"
#include "ks_masked_index.h"
#include "ks_staged_index.h"

namespace ks {

// Defined in ks_direct_plan.cpp and ks_staged_plan.cpp.
DirectTile direct_tile(const Problem& p, const Plan& pl);
StagedTile staged_tile_of(const Problem& p, const Plan& pl);

// Defined in ks_host.cpp.
bool plan_for_verify(int64_t a, int64_t b, int64_t c, int64_t d, int64_t batch, int layout, int dtype, Problem* p,
                     Plan* pl, ks_status_t* st);

namespace {

struct Checker {
  const Problem& p;
  int64_t xsize, ysize, ksize;
  std::vector<uint8_t> cover;
  std::string err;
  explicit Checker(const Problem& pp)
      : p(pp),
        xsize((int64_t)pp.batch * pp.N),
        ysize((int64_t)pp.batch * pp.M),
        ksize((int64_t)pp.a * pp.d * pp.b * pp.c),
        cover((size_t)ysize, 0) {}
  bool fail(const char* what, int64_t v) {
    if (err.empty()) {
      char buf[200];
      snprintf(buf, sizeof buf, "%s (value %lld)", what, (long long)v);
      err = buf;
    }
    return false;
  }
  bool read_x(int64_t off, int n) { return (off >= 0 && off + n <= xsize) ? true : fail("X read out of bounds", off); }
  bool read_k(int64_t off, int n) { return (off >= 0 && off + n <= ksize) ? true : fail("Kv read out of bounds", off); }
  bool write_y(int64_t off, int n) {
    if (off < 0 || off + n > ysize) return fail("Y write out of bounds", off);
    for (int e = 0; e < n; ++e) cover[(size_t)(off + e)]++;
    return true;
  }
  bool coverage() {
    for (size_t q = 0; q < cover.size(); ++q)
      if (cover[q] != 1) return fail(cover[q] ? "Y element written more than once" : "Y element never written", (int64_t)q);
    return true;
  }
};

bool verify_generic(Checker& ck, const Plan& pl) {
  const int64_t total = (int64_t)ck.p.batch * ck.p.M;
  const int64_t stride = (int64_t)pl.grid * pl.block;
  for (int64_t idx = 0; idx < total && idx < stride; ++idx)
    for (int64_t q = idx; q < total; q += stride) ck.write_y(q, 1);
  return ck.err.empty();
}

bool verify_valu_bsl(Checker& ck, const Plan& pl) {
  const Problem& p = ck.p;
  const int V = pl.vec, U = pl.unroll, nvec = p.batch / V;
  for (int ij = 0; ij < p.a * p.d; ++ij) {
    const int i = ij / p.d, j = ij % p.d;
    ck.read_k((int64_t)ij * p.b * p.c, p.b * p.c);
    for (unsigned gx = 0; gx < pl.grid; ++gx)
      for (int tid = 0; tid < 256; ++tid)
        for (int u = 0; u < U; ++u) {
          const int v = (int)gx * 256 * U + tid + u * 256;
          if (v >= nvec) continue;
          for (int l = 0; l < p.c; ++l) ck.read_x((int64_t)(i * p.c * p.d + j + l * p.d) * p.batch + (int64_t)v * V, V);
          for (int k = 0; k < p.b; ++k) ck.write_y((int64_t)(i * p.b * p.d + j + k * p.d) * p.batch + (int64_t)v * V, V);
        }
  }
  if (nvec * V != p.batch) ck.fail("batch not a multiple of the vector width", p.batch);
  return ck.err.empty();
}

bool verify_valu_bsf(Checker& ck, const Plan& pl) {
  const Problem& p = ck.p;
  const int V = pl.vec, nj = p.d / V, per_row = p.a * nj;
  if (nj * V != p.d) ck.fail("d not a multiple of the vector width", p.d);
  const int64_t total = (int64_t)p.batch * per_row;
  for (int64_t t = 0; t < (int64_t)pl.grid * 256; ++t) {
    if (t >= total) break;
    const int beta = (int)(t / per_row), r = (int)(t % per_row);
    const int i = r / nj, j0 = (r % nj) * V;
    for (int l = 0; l < p.c; ++l) ck.read_x((int64_t)beta * p.N + i * p.c * p.d + j0 + l * p.d, V);
    ck.read_k(((int64_t)i * p.d + j0) * p.b * p.c, V * p.b * p.c);
    for (int k = 0; k < p.b; ++k) ck.write_y((int64_t)beta * p.M + i * p.b * p.d + j0 + k * p.d, V);
  }
  return ck.err.empty();
}

// X element (offset) that flat element f = t*V + e of a lane's operand block
// must hold: l = l0 + LP*g + t and column e (batch V*n + e in BSL, j0 + e in
// BSF), from the definition of the product (Section 4.1 index sets).
int64_t expected_x(const Problem& p, const DItem& it, int V, int LP, int l0, int n, int g, int f) {
  const int t = f / V, e = f % V;
  const int64_t l = l0 + LP * g + t;
  if (p.layout == BSL)
    return ((int64_t)it.i * p.c * p.d + l * p.d + it.j0) * p.batch + it.beta0 + V * n + e;
  return (int64_t)(it.beta0 + n) * p.N + (int64_t)it.i * p.c * p.d + l * p.d + it.j0 + e;
}

// X and K reads and Y writes of one register-direct work item, for the
// chunks (l0, values of l per lane group) listed.
bool verify_item(Checker& ck, const DItem& it, bool strided, int V, int MT, int S, const int (*chunks)[2], int nch) {
  const Problem& p = ck.p;
  const int VK = p.layout == BSL ? 1 : V;
  for (int ci = 0; ci < nch; ++ci) {
    const int l0 = chunks[ci][0], lp = chunks[ci][1];
    const int np = direct_x_pieces(p.layout, strided, lp, V, S);
    const int pe = direct_x_piece_elems(p.layout, strided, lp, V, S);
    if (pe * S != 16 && pe * S != 8) return ck.fail("X piece is not 8 or 16 bytes", pe * S);
    if (np * pe != lp * V) return ck.fail("X pieces do not tile the lane block", np);
    for (int lane = 0; lane < 64; ++lane) {
      const int n = lane & 15, g = lane >> 4;
      const bool valid = direct_lane_valid(p, it, V, n);
      for (int q = 0; q < np; ++q) {
        const int64_t off = direct_x_off(p, it, strided, lp, V, S, l0, n, g, q);
        if ((off * S) % (pe * S)) return ck.fail("X piece not aligned to its size", off);
        ck.read_x(off, pe);
        for (int e = 0; valid && e < pe; ++e)
          if (off + e != expected_x(p, it, V, lp, l0, n, g, q * pe + e))
            return ck.fail("operand element is not the X value the product needs", off + e);
      }
      for (int mt = 0; mt < MT; ++mt)
        for (int e = 0; e < VK; ++e) {
          const int64_t off = direct_k_off(p, it, lp, l0, n, g, mt, e);
          if ((off * S) % (lp * S)) return ck.fail("K operand not aligned to its size", off);
          ck.read_k(off, lp);
        }
    }
  }
  const int ynp = direct_y_pieces(p.layout, strided, V, S);
  const int ype = direct_y_piece_elems(p.layout, strided, V, S);
  if (ype * S != 16 && ype * S != 8) return ck.fail("Y piece is not 8 or 16 bytes", ype * S);
  for (int mt = 0; mt < MT; ++mt)
    for (int lane = 0; lane < 64; ++lane)
      for (int q = 0; q < ynp; ++q) {
        const int64_t off = direct_y_off(p, it, strided, V, S, mt, lane & 15, lane >> 4, q);
        if (off < 0) continue;
        if ((off * S) % (ype * S)) return ck.fail("Y piece not aligned to its size", off);
        ck.write_y(off, ype);
      }
  return ck.err.empty();
}

// Masked kernel with access width V: every X piece is the V elements of
// value l the product needs (or zero padding), K elements inside the block,
// every Y element of the batch written exactly once, vector accesses aligned.
bool verify_masked_v(Checker& ck, int V, int MT) {
  const Problem& p = ck.p;
  const bool fp8 = p.dtype == FP8;
  const int S = p.dtype == F32 ? 4 : 2, LP = masked_lp(S), CH = 4 * LP;
  // bytes of an X piece / Y piece when it is one vector access (0: element
  // accesses): the masked kernel moves V*S >= 8 bytes as vectors, the FP8
  // kernel V >= 2 bytes of X and 2V >= 8 bytes of Y
  const int xvec = fp8 ? (V >= 2 ? V : 0) : (V * S >= 8 ? V * S : 0);
  const int yvec = fp8 ? (2 * V >= 8 ? 2 * V : 0) : (V * S >= 8 ? V * S : 0);
  const int xs = fp8 ? 1 : S, ys = fp8 ? 2 : S;
  const MaskedTile t = masked_tile(p, V, MT);
  if (t.kgroups * 16 * MT < p.b || t.nchunks * CH < p.c) return ck.fail("masked tiles do not cover the block", V);
  if (p.layout == BSL && p.batch % V) return ck.fail("batch not a multiple of the access width", V);
  if (p.layout == BSF && p.d % V) return ck.fail("d not a multiple of the access width", V);
  const int VK = p.layout == BSL ? 1 : V;
  // FP8 batch-size-first with V = d: a lane's X operand is one run of 8V
  // bytes from value l0 and (b a multiple of 4) its outputs one run of 4V
  // bf16; for d = 8 the runs are 64 bytes and lane row g takes piece g of
  // lane row x's run (x = 0..3).
  const bool runs = fp8 && p.layout == BSF && V == p.d && p.c % 8 == 0 && p.align >= 16;
  const bool rows8 = runs && V == 8;
  const bool yruns = runs && V <= 4 && p.b % 4 == 0;
  for (int item = 0; item < t.items && ck.err.empty(); ++item) {
    const MItem it = masked_item(p, t, V, item);
    if (it.i < 0 || it.i >= p.a) return ck.fail("item i out of range", item);
    for (int lane = 0; lane < 64; ++lane) {
      const int n = lane & 15, g = lane >> 4;
      if (rows8 && masked_col_valid(p, it, V, n)) {
        for (int ch = 0; ch < t.nchunks; ++ch)
          for (int x = 0; x < 4; ++x) {
            const int lx = ch * CH + LP * x;
            if (lx >= p.c) continue;
            const int64_t off = (int64_t)(it.beta0 + n) * p.N + ((int64_t)it.i * p.c + lx) * 8 + 16 * g;
            if (off % 16) return ck.fail("row-run X piece not 16-byte aligned", off);
            ck.read_x(off, 16);
            for (int h = 0; h < 2; ++h)
              if (masked_x_off(p, it, V, lx + 2 * g + h, n) != off + 8 * h)
                return ck.fail("row-run X piece is not the values of its lane row", off);
          }
        for (int mt = 0; mt < MT; ++mt)
          for (int x = 0; x < 4; ++x) {
            MItem im = it;
            im.k0 += 16 * mt;
            const int k = im.k0 + 4 * x + g;
            if (k >= p.b) continue;
            const int64_t off = (int64_t)(im.beta0 + n) * p.M + ((int64_t)im.i * p.b + k) * 8;
            if (off != masked_y_off(p, im, V, n, x, g)) return ck.fail("row-run Y piece is not its output", off);
            if ((off * 2) % 16) return ck.fail("row-run Y piece not 16-byte aligned", off);
            ck.write_y(off, 8);
          }
      }
      if (runs && !rows8 && masked_col_valid(p, it, V, n))
        for (int ch = 0; ch < t.nchunks; ++ch) {
          const int l0 = ch * CH + LP * g;
          const int64_t off = masked_x_off(p, it, V, l0, n);
          if (l0 >= p.c) continue;
          if (off < 0) return ck.fail("X run treated as padding", l0);
          const int nb = LP * V < 16 ? LP * V : 16;
          for (int h = 0; h < LP * V / nb; ++h)
            if ((off + h * nb) % nb) return ck.fail("X run piece not aligned to its size", off + h * nb);
          ck.read_x(off, LP * V);
          for (int q = 0; q < LP; ++q)
            if (masked_x_off(p, it, V, l0 + q, n) != off + q * V) return ck.fail("X run is not the values of the lane", l0 + q);
        }
      if (yruns && masked_col_valid(p, it, V, n))
        for (int mt = 0; mt < MT; ++mt) {
          MItem im = it;
          im.k0 += 16 * mt;
          const int64_t off = masked_y_off(p, im, V, n, g, 0);
          if (off >= 0) {
            const int nb = V == 1 ? 8 : 16;  // bytes per store
            if ((off * 2) % nb) return ck.fail("Y run not aligned to its stores", off);
            for (int r = 0; r < 4; ++r)
              if (masked_y_off(p, im, V, n, g, r) != off + r * V) return ck.fail("Y run is not the lane's outputs", off);
            ck.write_y(off, 4 * V);
          }
        }
      for (int ch = 0; ch < t.nchunks; ++ch)
        for (int q = 0; q < LP; ++q) {
          const int l = ch * CH + LP * g + q;
          const int64_t off = runs ? -1 : masked_x_off(p, it, V, l, n);
          if (off >= 0) {
            if (xvec && (off * xs) % xvec) return ck.fail("X vector not aligned to its size", off);
            ck.read_x(off, V);
            for (int e = 0; e < V; ++e) {
              DItem di;
              di.i = it.i; di.j0 = it.j0; di.k0 = it.k0; di.beta0 = it.beta0;
              // the same element the register-direct kernels' definition gives
              // for (l, column e): BSL batch beta0 + V*n + e, BSF j0 + e
              const int64_t want = p.layout == BSL
                  ? ((int64_t)it.i * p.c * p.d + (int64_t)l * p.d + it.j0) * p.batch + it.beta0 + V * n + e
                  : (int64_t)(it.beta0 + n) * p.N + (int64_t)it.i * p.c * p.d + (int64_t)l * p.d + it.j0 + e;
              (void)di;
              if (off + e != want) return ck.fail("masked operand element is not the X value needed", off + e);
            }
          } else if (!runs && l < p.c && masked_col_valid(p, it, V, n)) {
            return ck.fail("needed X piece treated as padding", l);
          }
          for (int mt = 0; mt < MT; ++mt) {
            const int m = 16 * mt + n;  // K row k0 + m
            if (t.kvec && q == 0)
              for (int e = 0; e < VK; ++e) {
                const int64_t ko = masked_k_off(p, it, e, m, l);
                if (ko >= 0) {
                  if ((ko * xs) % (LP * xs)) return ck.fail("K operand vector not aligned to its size", ko);
                  ck.read_k(ko, LP);
                }
              }
            for (int e = 0; e < VK; ++e) {
              const int64_t ko = masked_k_off(p, it, e, m, l);
              if (ko >= 0) {
                ck.read_k(ko, 1);
                if (ko != (((int64_t)it.i * p.d + it.j0 + e) * p.b + it.k0 + m) * p.c + l)
                  return ck.fail("masked K element is not the block value needed", ko);
              } else if (it.k0 + m < p.b && l < p.c) {
                return ck.fail("needed K value treated as padding", l);
              }
            }
          }
        }
      for (int mt = 0; mt < MT && !rows8 && !yruns; ++mt)
        for (int r = 0; r < 4; ++r) {
          MItem im = it;
          im.k0 += 16 * mt;
          const int64_t off = masked_y_off(p, im, V, n, g, r);
          if (off < 0) continue;
          if (yvec && (off * ys) % yvec) return ck.fail("Y vector not aligned to its size", off);
          ck.write_y(off, V);
        }
    }
  }
  return ck.err.empty();
}

// The planned access width, then every narrower one the planner would pick
// for less aligned buffers (each with its own coverage check).
bool verify_masked(Checker& ck, const Plan& pl) {
  // the planned width and M-tiles, then the narrower widths with one M-tile
  if (!verify_masked_v(ck, pl.vec, pl.variant == V_FP8 ? pl.waves_m : 1)) return false;
  for (int V = pl.vec / 2; V >= 1; V /= 2) {
    if (!ck.coverage()) return false;
    std::fill(ck.cover.begin(), ck.cover.end(), 0);
    if (!verify_masked_v(ck, V, 1)) return false;
  }
  return ck.err.empty();
}

bool verify_direct(Checker& ck, const Plan& pl) {
  const Problem& p = ck.p;
  const DirectTile t = direct_tile(p, pl);
  const int V = pl.vec, MT = pl.waves_m, S = p.dtype == F32 ? 4 : 2;
  const bool strided = pl.unroll != 0;
  const int LP = S == 4 ? 4 : 8, CH = 4 * LP;
  if (t.kgroups * 16 * MT != p.b) return ck.fail("M-tiles do not cover b", p.b);
  if (p.c % 16) return ck.fail("c not a multiple of 16", p.c);
  if (t.waves < 1 || t.waves > 4 || (int)pl.block != 64 * t.waves) return ck.fail("bad workgroup size", pl.block);
  if ((int64_t)pl.grid * t.waves < t.items) return ck.fail("grid does not cover the items", pl.grid);
  if (p.layout == BSF && (p.d % V || (!strided && V != p.d))) return ck.fail("bad j-vector", V);
  if (p.layout == BSL && p.batch % V) return ck.fail("batch not a multiple of the vector width", p.batch);
  int chunks[16][2], nch = 0;
  for (int l0 = 0; l0 + CH <= p.c; l0 += CH) { chunks[nch][0] = l0; chunks[nch][1] = LP; ++nch; }
  if (S == 2 && p.c % CH) { chunks[nch][0] = p.c - 16; chunks[nch][1] = 4; ++nch; }
  if (nch == 0) return ck.fail("no chunk covers c", p.c);
  for (int item = 0; item < t.items && ck.err.empty(); ++item) {
    // The kernels decode items with multiply-shift divisions: same item.
    const DItem a1 = direct_item(p, t, V, MT, item), a2 = direct_item_fast(p, t, V, MT, item);
    if (a1.i != a2.i || a1.j0 != a2.j0 || a1.k0 != a2.k0 || a1.beta0 != a2.beta0)
      return ck.fail("fast item decode differs", item);
    if (!verify_item(ck, a1, strided, V, MT, S, chunks, nch)) return false;
  }
  return ck.err.empty();
}

// Structured epilogue of the batch-size-first staged and DMA kernels: every
// cell of the LDS output tile is written once by the lane holding that output,
// then stored by its 16-byte unit.
bool verify_bsf_epilogue(Checker& ck, const StagedTile& t, const STile& st, int V, int MT, int S) {
  const Problem& p = ck.p;
  const int kr = staged_y_kr(t, MT), rows = 16 * t.RS * t.NT;
  std::vector<int64_t> ytile((size_t)rows * t.ypitch / S, -1);
  for (int w = 0; w < t.W; ++w) {
    const SItem si = staged_item(p, t, st, V, MT, w);
    for (int lu = 0; lu < 64 * t.NT; ++lu) {
      const int lane = lu & 63, u = lu >> 6;
      const int n = lane & 15, g = lane >> 4, r = 16 * (t.NT * si.rs + u) + n;
      if (si.beta0 + 16 * u != st.bt * 16 * t.RS * t.NT + 16 * (t.NT * si.rs + u))
        return ck.fail("row group base does not match the tile", si.beta0);
      for (int mt = 0; mt < MT; ++mt)
        for (int r4 = 0; r4 < 4; ++r4)
          for (int e = 0; e < V; ++e) {
            const int k = si.k0 + 16 * mt + 4 * g + r4, j = si.j0 + e;
            const int o = staged_y_lds(p, t, st, MT, S, r, k, j);
            if (e == 0 && o % (V * S)) return ck.fail("output tile write not aligned to its size", o);
            if (o < 0 || o + S > rows * t.ypitch) return ck.fail("output tile write out of range", o);
            int64_t& cell = ytile[(size_t)(o / S)];
            if (cell != -1) return ck.fail("output tile cell written twice", o);
            cell = (int64_t)(st.bt * 16 * t.RS * t.NT + r) * p.M + (int64_t)st.i * p.b * p.d + (int64_t)k * p.d + j;
          }
    }
  }
  const int uy = staged_y_units_per_row(p, t, MT, S);
  if (uy * 16 != kr * p.d * S) return ck.fail("output row is not a whole number of units", kr);
  for (int r = 0; r < rows; ++r)
    for (int v = 0; v < uy; ++v) {
      const int64_t off = staged_y_unit(p, t, st, MT, S, r, v);
      if (off < 0) continue;
      if ((off * S) % 16) return ck.fail("Y unit not 16-byte aligned", off);
      for (int e = 0; e < 16 / S; ++e)
        if (ytile[(size_t)((r * t.ypitch + v * 16) / S + e)] != off + e)
          return ck.fail("Y unit does not hold the outputs it is stored to", off + e);
      ck.write_y(off, 16 / S);
    }
  return true;
}

bool verify_staged(Checker& ck, const Plan& pl) {
  const Problem& p = ck.p;
  const StagedTile t = staged_tile_of(p, pl);
  const int V = pl.vec, MT = pl.waves_m, S = p.dtype == F32 ? 4 : 2;
  const bool strided = pl.unroll != 0;
  const int LP = S == 4 ? 4 : 8, CH = 4 * LP, UE = 16 / S;
  if (t.RS * t.JG * t.KGW != t.W || t.W < 1 || t.W > 8) return ck.fail("waves do not split the tile", t.W);
  if (t.kgt * t.KGW * 16 * MT != p.b) return ck.fail("k-groups do not cover b", p.b);
  if (t.LCH % CH || t.LCH / CH != pl.cps) return ck.fail("stage is not a whole number of chunks", t.LCH);
  if ((int)pl.grid != t.tiles || (int)pl.block != 64 * t.W) return ck.fail("grid does not match the tiles", pl.grid);
  if (pl.lds_bytes != t.lds || t.lds < 2 * t.stage) return ck.fail("LDS allocation does not hold two stages", pl.lds_bytes);
  if (p.layout == BSF && t.lds < 16 * t.RS * t.ypitch) return ck.fail("LDS allocation does not hold the output tile", t.lds);
  if (t.remap && t.tiles % 8) return ck.fail("XCD remap needs a multiple of 8 tiles", t.tiles);
  if (p.layout == BSF && (p.d % V || (!strided && V != p.d) || t.JG != p.d / V)) return ck.fail("bad j-vector", V);
  if (p.layout == BSL && p.batch % UE) return ck.fail("batch not a multiple of the 16-byte unit", p.batch);
  std::vector<uint8_t> seen(t.tiles, 0);
  std::vector<int64_t> shadow((size_t)t.stage / S);
  const int nstages = (p.c + t.LCH - 1) / t.LCH;
  for (int blk = 0; blk < t.tiles && ck.err.empty(); ++blk) {
    const STile st = staged_tile(p, t, blk);
    const int logical = t.remap ? staged_remap(blk, t.tiles) : blk;
    if (logical < 0 || logical >= t.tiles || seen[logical]++) return ck.fail("tile visited twice", logical);
    for (int s = 0; s < nstages; ++s) {
      const int ls = s * t.LCH, nl = p.c - ls < t.LCH ? p.c - ls : t.LCH;
      std::fill(shadow.begin(), shadow.end(), (int64_t)-1);
      const int ur = staged_units_per_row(p, t, V, S, nl);
      const int nunits = staged_rows(p, t, nl) * ur;
      if (nunits > 256 * t.W) return ck.fail("stage has more than 4 units per thread", nunits);
      const int64_t xls = p.layout == BSL ? (int64_t)p.d * p.batch : p.d;
      for (int u = 0; u < nunits; ++u) {
        const int r = u / ur, v = u % ur;
        const int64_t off = staged_x_unit(p, t, st, V, S, ls, r, v);
        // the kernel computes the offset once at ls = 0 and shifts it per stage
        if (off != staged_x_unit(p, t, st, V, S, 0, r, v) + (int64_t)ls * xls)
          return ck.fail("X unit offset is not linear in the stage start", off);
        if ((off * S) % 16) return ck.fail("X unit not 16-byte aligned", off);
        ck.read_x(off, UE);
        const int lo = staged_lds_unit(t, r, v);
        if (lo < 0 || lo + 16 > t.stage) return ck.fail("LDS unit out of the stage buffer", lo);
        for (int e = 0; e < UE; ++e) {
          int64_t& cell = shadow[(size_t)(lo / S + e)];
          if (cell != -1) return ck.fail("LDS cell written twice in a stage", lo);
          cell = off + e;
        }
      }
      for (int w = 0; w < t.W; ++w) {
        const SItem si = staged_item(p, t, st, V, MT, w);
        DItem it;
        it.i = st.i; it.j0 = si.j0; it.k0 = si.k0; it.beta0 = si.beta0;
        // MFMA chunks of this stage: full chunks, then the 16-bit tail
        int chunks[8][2], nch = 0;
        for (int q = 0; (q + 1) * CH <= nl; ++q) { chunks[nch][0] = q * CH; chunks[nch][1] = LP; ++nch; }
        if (nl % CH) {
          if (S != 2 || nl % CH != 16) return ck.fail("stage leaves values of l uncovered", nl);
          chunks[nch][0] = nl - 16; chunks[nch][1] = 4; ++nch;
        }
        for (int ci = 0; ci < nch; ++ci) {
          const int l0 = chunks[ci][0], lp = chunks[ci][1];
          const int pe = direct_x_piece_elems(p.layout, strided, lp, V, S);
          const int np = lp * V / pe, pb = pe * S;
          if (pb != 16 && pb != 8) return ck.fail("operand piece is not 8 or 16 bytes", pb);
          const int olstride = staged_op_lstride(p, t, S), oqstride = staged_op_qstride(p, t, strided, pe, S);
          for (int lane = 0; lane < 64; ++lane) {
            const int n = lane & 15, g = lane >> 4;
            const bool valid = direct_lane_valid(p, it, V, n);
            const int ob = staged_op_base(p, t, si, lp, V, S, n, g);
            for (int q = 0; q < np; ++q) {
              const int o = ob + l0 * olstride + q * oqstride;
              if (o < 0 || o + pb > t.stage || o % pb) return ck.fail("operand read outside the stage or unaligned", o);
              for (int e = 0; e < pe; ++e) {
                const int64_t have = shadow[(size_t)(o / S + e)];
                if (have < 0) return ck.fail("operand read of an LDS cell not written in this stage", o);
                if (valid && have != expected_x(p, it, V, lp, ls + l0, n, g, q * pe + e))
                  return ck.fail("operand element is not the X value the product needs", have);
              }
            }
            for (int mt = 0; mt < MT; ++mt)
              for (int e = 0; e < (p.layout == BSL ? 1 : V); ++e) {
                const int64_t off = direct_k_off(p, it, lp, ls + l0, n, g, mt, e);
                if ((off * S) % (lp * S)) return ck.fail("K operand not aligned to its size", off);
                ck.read_k(off, lp);
              }
          }
        }
      }
    }
    if (p.layout == BSL) {
      for (int w = 0; w < t.W; ++w) {
        const SItem si = staged_item(p, t, st, V, MT, w);
        DItem it;
        it.i = st.i; it.j0 = si.j0; it.k0 = si.k0; it.beta0 = si.beta0;
        const int ynp = direct_y_pieces(p.layout, strided, V, S);
        const int ype = direct_y_piece_elems(p.layout, strided, V, S);
        for (int mt = 0; mt < MT; ++mt)
          for (int lane = 0; lane < 64; ++lane)
            for (int q = 0; q < ynp; ++q) {
              const int64_t off = direct_y_off(p, it, strided, V, S, mt, lane & 15, lane >> 4, q);
              if (off < 0) continue;
              if ((off * S) % (ype * S)) return ck.fail("Y piece not aligned to its size", off);
              ck.write_y(off, ype);
            }
      }
    } else if (!verify_bsf_epilogue(ck, t, st, V, MT, S)) {
      return false;
    }
  }
  return ck.err.empty();
}

// LDS-DMA kernel (ks_dma.h): every lane of every DMA instruction of a stage
// fills one 16-byte unit of the stage buffer (all units exactly once) from an
// in-bounds, 16-byte aligned X address; every operand piece a lane reads from
// the swizzled stage holds the X values its products need; K, the output
// tile and the Y stores as in the staged kernel.
// Batch-size-last DMA kernel (ks_dma_bsl.h): every stage's DMA units land on
// distinct LDS cells inside the buffer, each operand piece a lane reads holds
// the X values its products need, K operands inside the block, the stage
// buffers inside the allocation, and every Y element written once by the
// register-direct store.
bool verify_dma_bsl(Checker& ck, const Plan& pl) {
  const Problem& p = ck.p;
  const StagedTile t = staged_tile_of(p, pl);
  const int S = p.dtype == F32 ? 4 : 2, V = 16 / S, LP = S == 4 ? 4 : 8, CH = 4 * LP, MT = pl.waves_m;
  if (pl.vec != V || pl.unroll != 0 || pl.cps != LP) return ck.fail("bad vector or lane depth", pl.vec);
  if (p.batch % V) return ck.fail("batch not a multiple of the vector width", p.batch);
  if (MT < 1 || MT > (S == 4 ? 4 : 2)) return ck.fail("no instance for this MT", MT);
  if (t.W != 4 || t.RS * t.KGW != t.W || t.JG != 1 || (t.RS != 1 && t.RS != 2 && t.RS != 4))
    return ck.fail("waves do not split the tile", t.W);
  if (t.kgt * t.KGW * 16 * MT != p.b) return ck.fail("k-groups do not cover b", p.b);
  if (t.LCH != CH || p.c % CH) return ck.fail("stages do not cover c", t.LCH);
  if (t.UR != 16 * t.RS || (1 << t.lUR) != t.UR || (1 << t.lRS) != t.RS)
    return ck.fail("stage row is not the tile's units", t.UR);
  if (t.stage != CH * t.UR * 16 || t.UD * 64 * t.W * 16 != t.stage) return ck.fail("stage is not whole DMA instructions", t.stage);
  if ((int)pl.grid != t.tiles || (int)pl.block != 64 * t.W) return ck.fail("grid does not match the tiles", pl.grid);
  const int nst = p.c / CH;
  {
    int top = 0;
    for (int s = 0; s < nst; ++s) top = std::max(top, s % 3);
    if (pl.lds_bytes != t.lds || t.lds < (int64_t)(top + 1) * t.stage || dma_stage_buffers(nst) != top + 1)
      return ck.fail("LDS allocation does not hold the stage buffers the kernel touches", t.lds);
  }
  if (t.remap && t.tiles % 8) return ck.fail("XCD remap needs a multiple of 8 tiles", t.tiles);
  std::vector<uint8_t> seen(t.tiles, 0);
  std::vector<int64_t> shadow((size_t)t.stage / S);
  for (int blk = 0; blk < t.tiles && ck.err.empty(); ++blk) {
    const STile st = staged_tile(p, t, blk);
    const int logical = t.remap ? staged_remap(blk, t.tiles) : blk;
    if (logical < 0 || logical >= t.tiles || seen[logical]++) return ck.fail("tile visited twice", logical);
    const STile sf = dma_bsl_tile(p, t, blk);
    if (sf.i != st.i || sf.bt != st.bt || sf.kt != st.kt || sf.j != st.j) return ck.fail("fast tile decode differs", blk);
    for (int w = 0; w < t.W; ++w) {
      const SItem a1 = staged_item(p, t, st, V, MT, w), a2 = dma_bsl_item(t, st, V, MT, w);
      if (a1.rs != a2.rs || a1.kgw != a2.kgw || a1.j0 != a2.j0 || a1.k0 != a2.k0 || a1.beta0 != a2.beta0)
        return ck.fail("fast work-item decode differs", w);
    }
    for (int s = 0; s < nst; ++s) {
      std::fill(shadow.begin(), shadow.end(), (int64_t)-1);
      for (int w = 0; w < t.W; ++w)
        for (int m = 0; m < t.UD; ++m)
          for (int lane = 0; lane < 64; ++lane) {
            const int P = dma_phys_unit(t, m, w, lane);
            if (P < 0 || (P + 1) * 16 > t.stage) return ck.fail("DMA writes outside the stage buffer", P);
            int r, v;
            dma_bsl_unit_of(t, P, &r, &v);
            if (r < 0 || r >= CH || v < 0 || v >= t.UR) return ck.fail("DMA unit outside the stage rows", P);
            // the kernel's form: X + i*c*d*batch (tile) + s*CH*d*batch (stage) + dma_bsl_src
            const int64_t src = dma_bsl_src(p, t, st, V, r, v);
            const int64_t off = (int64_t)st.i * p.c * p.d * p.batch + (int64_t)s * CH * p.d * p.batch + src;
            if ((off * S) % 16) return ck.fail("DMA source not 16-byte aligned", off);
            ck.read_x(off, V);
            for (int e = 0; e < V; ++e) {
              int64_t& cell = shadow[(size_t)(P * 16 / S + e)];
              if (cell != -1) return ck.fail("LDS cell written twice in a stage", P);
              cell = off + e;
            }
          }
      for (int w = 0; w < t.W; ++w) {
        const SItem si = staged_item(p, t, st, V, MT, w);
        DItem it;
        it.i = st.i; it.j0 = si.j0; it.k0 = si.k0; it.beta0 = si.beta0;
        for (int lane = 0; lane < 64; ++lane) {
          const int n = lane & 15, g = lane >> 4;
          const bool valid = direct_lane_valid(p, it, V, n);
          for (int q = 0; q < LP; ++q) {
            const int o = dma_bsl_op_byte(t, si, LP, n, g, q);
            if (o < 0 || o + 16 > t.stage || o % 16) return ck.fail("operand read outside the stage or unaligned", o);
            for (int e = 0; e < V; ++e) {
              const int64_t have = shadow[(size_t)(o / S + e)];
              if (have < 0) return ck.fail("operand read of an LDS cell not written in this stage", o);
              if (valid && have != expected_x(p, it, V, LP, s * CH, n, g, q * V + e))
                return ck.fail("operand element is not the X value the product needs", have);
            }
          }
          for (int mt = 0; mt < MT; ++mt) {
            const int64_t off = direct_k_off(p, it, LP, s * CH, n, g, mt, 0);
            if ((off * S) % (LP * S)) return ck.fail("K operand not aligned to its size", off);
            ck.read_k(off, LP);
          }
        }
      }
    }
    // Y: the register-direct store of each wavefront's item.
    for (int w = 0; w < t.W; ++w) {
      const SItem si = staged_item(p, t, st, V, MT, w);
      DItem it;
      it.i = st.i; it.j0 = si.j0; it.k0 = si.k0; it.beta0 = si.beta0;
      for (int mt = 0; mt < MT; ++mt)
        for (int lane = 0; lane < 64; ++lane)
          for (int q = 0; q < 4; ++q) {
            const int64_t off = direct_y_off(p, it, false, V, S, mt, lane & 15, lane >> 4, q);
            if (off < 0) continue;
            if ((off * S) % 16) return ck.fail("Y piece not aligned to 16 bytes", off);
            ck.write_y(off, V);
          }
    }
  }
  return ck.err.empty();
}

bool verify_dma(Checker& ck, const Plan& pl) {
  const Problem& p = ck.p;
  if (p.layout == BSL) return verify_dma_bsl(ck, pl);
  const StagedTile t = staged_tile_of(p, pl);
  const int V = pl.vec, MT = pl.waves_m, S = p.dtype == F32 ? 4 : 2, LP = pl.cps, CH = 4 * LP, UE = 16 / S;
  const bool strided = pl.unroll != 0;
  if (p.layout != BSF || V != (p.d < 4 ? p.d : 4) || p.d % V || strided != (p.d > V)) return ck.fail("bad j-vector", V);
  if (LP != 4 && !(S == 2 && LP == 8)) return ck.fail("bad MFMA lane depth", LP);
  if (t.W != 4 || t.RS * t.JG * t.KGW != t.W || t.JG != p.d / V) return ck.fail("waves do not split the tile", t.W);
  if (t.kgt * t.KGW * 16 * MT != p.b) return ck.fail("k-groups do not cover b", p.b);
  if (t.LCH != CH || p.c % CH) return ck.fail("stages do not cover c", t.LCH);
  if (t.UR * 16 != CH * p.d * S || (t.UR & (t.UR - 1))) return ck.fail("stage row is not a power-of-two of units", t.UR);
  if (t.NT != pl.nt || (t.NT != 1 && t.NT != 2 && t.NT != 4) || MT * t.NT > 4) return ck.fail("bad row groups per wavefront", t.NT);
  if (t.stage != 16 * t.RS * t.NT * t.UR * 16 || t.UD * 64 * t.W * 16 != t.stage ||
      (t.UD != 2 && t.UD != 4 && t.UD != 8))
    return ck.fail("stage is not a whole number of DMA instructions per wavefront", t.stage);
  if ((int)pl.grid != t.tiles || (int)pl.block != 64 * t.W) return ck.fail("grid does not match the tiles", pl.grid);
  // The kernel's stage s reads buffer s % 3 and the DMAs of stage s + 2
  // (issued only when s + 2 < nst) write buffer (s + 2) % 3: buffers
  // 0 .. min(nst, 3) - 1 are touched.
  {
    const int nst_v = p.c / CH;
    int top = 0;
    for (int s = 0; s < nst_v; ++s) top = std::max(top, s % 3);
    if (pl.lds_bytes != t.lds || t.lds < (int64_t)(top + 1) * t.stage || dma_stage_buffers(nst_v) != top + 1)
      return ck.fail("LDS allocation does not hold the stage buffers the kernel touches", t.lds);
  }
  if (t.lds < 16 * t.RS * t.NT * t.ypitch) return ck.fail("LDS allocation does not hold the output tile", t.lds);
  if (t.remap && t.tiles % 8) return ck.fail("XCD remap needs a multiple of 8 tiles", t.tiles);
  const int pe = direct_x_piece_elems(BSF, strided, LP, V, S), np = LP * V / pe, pb = pe * S;
  std::vector<uint8_t> seen(t.tiles, 0);
  std::vector<int64_t> shadow((size_t)t.stage / S);
  const int nst = p.c / CH;
  if ((1 << t.lUR) != t.UR || (1 << t.lRS) != t.RS || (1 << t.lJG) != t.JG ||
      (16 << t.lUY) != staged_y_kr(t, MT) * p.d * S)
    return ck.fail("tile sizes are not the powers of two the kernel shifts by", t.UR);
  for (int blk = 0; blk < t.tiles && ck.err.empty(); ++blk) {
    const STile st = staged_tile(p, t, blk);
    const int logical = t.remap ? staged_remap(blk, t.tiles) : blk;
    if (logical < 0 || logical >= t.tiles || seen[logical]++) return ck.fail("tile visited twice", logical);
    // The kernel's decode (multiply-shift divisions, shifts) gives the same tile and items.
    const STile sf = dma_tile(t, blk);
    if (sf.i != st.i || sf.bt != st.bt || sf.kt != st.kt) return ck.fail("fast tile decode differs", blk);
    for (int w = 0; w < t.W; ++w) {
      const SItem a1 = staged_item(p, t, st, V, MT, w), a2 = dma_item(t, st, V, MT, w);
      if (a1.rs != a2.rs || a1.jg != a2.jg || a1.kgw != a2.kgw || a1.j0 != a2.j0 || a1.k0 != a2.k0 ||
          a1.beta0 != a2.beta0)
        return ck.fail("fast work-item decode differs", w);
    }
    for (int s = 0; s < nst; ++s) {
      std::fill(shadow.begin(), shadow.end(), (int64_t)-1);
      for (int w = 0; w < t.W; ++w)
        for (int m = 0; m < t.UD; ++m)
          for (int lane = 0; lane < 64; ++lane) {
            const int P = dma_phys_unit(t, m, w, lane);
            if (P < 0 || (P + 1) * 16 > t.stage) return ck.fail("DMA writes outside the stage buffer", P);
            int r, v, r2, v2;
            dma_unit_of(t, P, &r, &v);
            dma_unit_of_fast(t, P, &r2, &v2);
            if (r2 != r || v2 != v) return ck.fail("fast DMA unit mapping differs", P);
            if (r < 0 || r >= 16 * t.RS * t.NT || v < 0 || v >= t.UR) return ck.fail("DMA unit outside the stage rows", P);
            int beta = st.bt * 16 * t.RS * t.NT + r;
            if (beta >= p.batch) beta = p.batch - 1;
            // the kernel's form: row base i*c*d, stage offset s*CH*d, lane offset beta*N + v*UE
            const int64_t off = (int64_t)st.i * p.c * p.d + (int64_t)s * CH * p.d + ((int64_t)beta * p.N + v * UE);
            if ((off * S) % 16) return ck.fail("DMA source not 16-byte aligned", off);
            if ((int64_t)beta * p.N + v * UE > 0x7fffffff) return ck.fail("DMA lane offset exceeds 32 bits", beta);
            ck.read_x(off, UE);
            for (int e = 0; e < UE; ++e) {
              int64_t& cell = shadow[(size_t)(P * 16 / S + e)];
              if (cell != -1) return ck.fail("LDS cell written twice in a stage", P);
              cell = off + e;
            }
          }
      for (int w = 0; w < t.W; ++w) {
        const SItem si = staged_item(p, t, st, V, MT, w);
        DItem it;
        it.i = st.i; it.j0 = si.j0; it.k0 = si.k0; it.beta0 = si.beta0;
        for (int lu = 0; lu < 64 * t.NT; ++lu) {
          // lane of row group u: the kernel reads group 0's offset + u * (16 rows)
          const int lane = lu & 63, u = lu >> 6;
          const int n = lane & 15, g = lane >> 4, r = 16 * (t.NT * si.rs + u) + n;
          DItem itu = it;
          itu.beta0 = it.beta0 + 16 * u;
          const bool valid = direct_lane_valid(p, itu, V, n);
          for (int q = 0; q < np; ++q) {
            const int b = dma_op_byte(p, si, LP, V, strided, pe, S, 0, g, q);
            if ((b & 15) + pb > 16 || b % pb) return ck.fail("operand piece crosses a 16-byte unit", b);
            const int o = dma_lds_byte(t, r, b);
            if (o != dma_lds_byte(t, 16 * t.NT * si.rs + n, b) + u * 16 * t.UR * 16)
              return ck.fail("row group operand offset is not group 0's plus 16 rows", o);
            if (o < 0 || o + pb > t.stage || o % pb) return ck.fail("operand read outside the stage or unaligned", o);
            for (int e = 0; e < pe; ++e) {
              const int64_t have = shadow[(size_t)(o / S + e)];
              if (have < 0) return ck.fail("operand read of an LDS cell not written in this stage", o);
              if (valid && have != expected_x(p, itu, V, LP, s * CH, n, g, q * pe + e))
                return ck.fail("operand element is not the X value the product needs", have);
            }
          }
          if (u > 0) continue;
          for (int mt = 0; mt < MT; ++mt)
            for (int e = 0; e < V; ++e) {
              const int64_t off = direct_k_off(p, it, LP, s * CH, n, g, mt, e);
              if ((off * S) % (LP * S)) return ck.fail("K operand not aligned to its size", off);
              ck.read_k(off, LP);
            }
        }
      }
    }
    if (!verify_bsf_epilogue(ck, t, st, V, MT, S)) return false;
    // The kernel's own epilogue offsets: per-lane LDS base plus constants, and
    // Y = tile base + row offset for rows inside the batch.
    for (int w = 0; w < t.W; ++w) {
      const SItem si = staged_item(p, t, st, V, MT, w);
      for (int lane = 0; lane < 64; ++lane) {
        const int n = lane & 15, g = lane >> 4;
        for (int u = 0; u < t.NT; ++u)
          for (int mt = 0; mt < MT; ++mt)
            for (int r4 = 0; r4 < 4; ++r4) {
              const int k = si.k0 + 16 * mt + 4 * g + r4, r = 16 * (t.NT * si.rs + u) + n;
              const int o = dma_y_lds_lane(p, t, si, MT, S, n, g) + u * 16 * t.ypitch + (16 * mt + r4) * p.d * S;
              if (o != staged_y_lds(p, t, st, MT, S, r, k, si.j0)) return ck.fail("output tile offset differs", o);
            }
      }
    }
    const int uy = 1 << t.lUY, rows_valid = p.batch - st.bt * 16 * t.RS * t.NT;
    for (int r = 0; r < 16 * t.RS * t.NT; ++r)
      for (int v = 0; v < uy; ++v) {
        const int64_t want = staged_y_unit(p, t, st, MT, S, r, v);
        const int64_t have = r < rows_valid ? dma_y_tile_base(p, t, st, MT) + dma_y_row(p, r, v, S) : -1;
        if (want != have) return ck.fail("output store offset differs", r);
      }
  }
  return ck.err.empty();
}

}  // namespace
}  // namespace ks

using namespace ks;

extern "C" ks_status_t ks_plan_verify(int64_t a, int64_t b, int64_t c, int64_t d, int64_t batch, int layout,
                                      int dtype, char* report, size_t len) {
  Problem p;
  Plan pl;
  ks_status_t st;
  if (report && len) report[0] = 0;
  if (!plan_for_verify(a, b, c, d, batch, layout, dtype, &p, &pl, &st)) {
    if (report && len) snprintf(report, len, "%s", st == KS_OK ? "empty" : "no plan");
    return st;
  }
  Checker ck(p);
  bool ok = false;
  switch (pl.variant) {
    case V_GENERIC: ok = verify_generic(ck, pl); break;
    case V_VALU_BSL: ok = verify_valu_bsl(ck, pl); break;
    case V_VALU_BSF: ok = verify_valu_bsf(ck, pl); break;
    case V_DIRECT: ok = verify_direct(ck, pl); break;
    case V_STAGED: ok = verify_staged(ck, pl); break;
    case V_DMA: ok = verify_dma(ck, pl); break;
    case V_MASKED: ok = verify_masked(ck, pl); break;
    case V_FP8: ok = verify_masked(ck, pl); break;
    default: ck.fail("unknown variant", pl.variant);
  }
  if (ok) ok = ck.coverage();
  if (report && len) snprintf(report, len, "%s", ok ? "ok" : ck.err.c_str());
  return ok ? KS_OK : KS_ERR_UNSUPPORTED;
}

// ---------------------------------------------------------------------------
// Fused chains (ks_chain_fused.hip): replay of every workgroup's tile loads
// and stores and of every factor's work units, with the kernel's own index
// functions (ks_chain_fused.h).
// ---------------------------------------------------------------------------
#include "ks_chain_fused.h"

namespace ks {
bool chain_fused_plan(const ks_factor_t* f, int n, int64_t batch, int layout, int dtype, FusedChain* fc);
namespace {

struct FusedChecker {
  std::string err;
  bool fail(const char* what, int64_t v) {
    if (err.empty()) {
      char buf[200];
      snprintf(buf, sizeof buf, "%s (value %lld)", what, (long long)v);
      err = buf;
    }
    return false;
  }
};

// Global element ranges of one pass over a tile (load of X or store of Y) in
// the 16-byte form (E elements per unit) or the element form (E = 1).
bool verify_fused_io(FusedChecker& ck, const FusedChain& fc, int width, int E, bool store,
                     std::vector<uint8_t>* cover) {
  const int64_t B = fc.batch, total = (int64_t)B * width;
  const int NC = fc.cols;
  const int tiles = (int)((B + NC - 1) / NC);
  const int units = width * NC / E;
  const int rows_lds = fc.buf_rows;
  if (NC != kFusedCols && !(fc.mfma && NC == 2 * kFusedCols)) return ck.fail("tile width", NC);
  if (fc.pitch != NC + 4) return ck.fail("LDS pitch", fc.pitch);
  for (int tile = 0; tile < tiles; ++tile) {
    const int col0 = tile * NC;
    for (int u = 0; u < units; ++u) {
      int row, col;
      if (E > 1) {
        fused_vec_unit(fc.layout, E, u, &row, &col, NC);
      } else if (fc.layout == BSL) {
        row = u / NC;
        col = u % NC;
      } else {
        col = u % NC;
        row = u / NC;
      }
      // The element(s) this unit moves: BSL a run of E columns of one row,
      // BSF a run of E rows (vector elements) of one batch row.
      const int r_hi = fc.layout == BSL ? row : row + E - 1;
      const int c_hi = fc.layout == BSL ? col + E - 1 : col;
      if (row < 0 || r_hi >= width || r_hi >= rows_lds) return ck.fail("tile row out of range", row);
      if (col < 0 || c_hi >= NC) return ck.fail("tile column out of range", col);
      const int bcol = col0 + (fc.layout == BSL ? col : col);
      const bool valid = fc.layout == BSL ? bcol < B : bcol < B;
      if (!valid) continue;  // beyond the batch: loads fill zeros, stores skip
      if (fc.layout == BSL && E > 1 && bcol + E > B) return ck.fail("vector straddles the batch end", bcol);
      const int64_t off = fc.layout == BSL ? (int64_t)row * B + bcol : (int64_t)bcol * width + row;
      if (off < 0 || off + E > total) return ck.fail(store ? "Y access out of bounds" : "X access out of bounds", off);
      if (E > 1 && off % E) return ck.fail("16-byte access not aligned to its vector", off);
      if (cover)
        for (int e = 0; e < E; ++e) (*cover)[(size_t)(off + e)]++;
    }
  }
  return ck.err.empty();
}

// MFMA form (ks_chain_mfma.hip): the kernel applies factor nf-1 .. 0, one per
// pass; wavefront w of W takes blocks w, w + W, ...; lane (n, g) reads the
// 4-value runs K[ij][16kt + n][16ct + 4g ..] and the LDS rows
// in_row(16ct + 4g + t), writes rows out_row(16kt + 4g + r), all at column n
// (the kernel addresses them as in_row(4g) plus multiples of d).  Replays
// every wavefront's blocks and every lane's accesses.
bool verify_fused_mfma(FusedChecker& ck, const FusedChain& fc, int dtype) {
  constexpr int W = kFusedThreads / 64;
  if (!fc.inplace) return ck.fail("MFMA form not in place", 0);
  // Per-wavefront load of the first factor's blocks (d = 1): each X element
  // of the batch read once, by the wavefront whose blocks hold its row, in
  // both access forms.
  if (fc.d[fc.nf - 1] == 1) {
    const int f = fc.nf - 1, B = fc.b[f], NC = fc.cols, nb = fused_mfma_blocks(fc, f), N = fc.width_in;
    const int esize = dtype == F32 ? 4 : 2;
    const int64_t Bt = fc.batch;
    const bool bsl = fc.layout == BSL;
    const bool vec_ok = bsl ? Bt % (16 / esize) == 0 : N % (16 / esize) == 0;
    std::vector<uint8_t> xin((size_t)Bt * N);
    for (int form = 0; form < (vec_ok ? 2 : 1); ++form) {
      const int EP = form ? 16 / esize : 1, PPB = B * NC / EP, PPL = (PPB + 63) / 64;
      std::fill(xin.begin(), xin.end(), 0);
      for (int64_t col0 = 0; col0 < Bt; col0 += NC)
        for (int w = 0; w < W; ++w)
          for (int ij = w; ij < nb; ij += W)
            for (int i = 0; i < PPL; ++i)
              for (int lane = 0; lane < 64; ++lane) {
                const int p = i * 64 + lane;
                if (p >= PPB) continue;
                int r, c;
                fused_block_piece(fc.layout, B, NC, EP, p, &r, &c);
                if (r < 0 || r + (bsl ? 0 : EP - 1) >= B || c < 0 || c + (bsl ? EP - 1 : 0) >= NC)
                  return ck.fail("block piece outside the block", p);
                if (col0 + c >= Bt) continue;
                const int64_t off = bsl ? (int64_t)(ij * B + r) * Bt + col0 + c : (col0 + c) * N + ij * B + r;
                if (EP > 1 && off % EP) return ck.fail("block piece not aligned to its size", off);
                for (int e = 0; e < EP; ++e) xin[(size_t)(off + (bsl ? e : e))]++;
              }
      for (size_t e = 0; e < xin.size(); ++e)
        if (xin[e] != 1) return ck.fail("X element not loaded exactly once by the block loads", (int64_t)e);
    }
  }
  for (int f = fc.nf - 1; f >= 0; --f) {
    const int a = fc.a[f], b = fc.b[f], d = fc.d[f];
    if (b != fc.c[f] || b % 16 || b < 16 || b > kFusedMfmaMaxB) return ck.fail("MFMA form block not square 16..64", f);
    if (b != 16 * fused_mfma_bt(fc)) return ck.fail("MFMA form blocks of different sizes", f);
    const int BT = b / 16, nblk = fused_mfma_blocks(fc, f), width = a * b * d;
    if (nblk != a * d) return ck.fail("MFMA block count", f);
    const int64_t kcount = (int64_t)a * d * b * b;
    const int NC = fc.cols, H = NC / 16;
    if (NC != 16 && NC != 32) return ck.fail("MFMA form tile width", NC);
    if (NC == 32 && BT > 2) return ck.fail("32-column tiles only for blocks up to 32", b);
    std::vector<uint8_t> blk(nblk, 0), cover((size_t)width * NC, 0);
    std::vector<uint8_t> kcov((size_t)kcount, 0);
    for (int w = 0; w < W; ++w) {
      for (int ij = w; ij < nblk; ij += W) {
        blk[ij]++;
        const int i = (int)div_fast((uint32_t)ij, fc.md[f], fc.sd[f]), j = ij - i * d;
        if (i != ij / d || j < 0 || j >= d) return ck.fail("MFMA block decode", ij);
        std::vector<int> rin, rout;
        for (int lane = 0; lane < 64; ++lane) {
          const int n = lane & 15, g = lane >> 4;
          for (int kt = 0; kt < BT; ++kt)
            for (int ct = 0; ct < BT; ++ct) {
              const int64_t off = (int64_t)ij * b * b + (16 * kt + n) * b + 16 * ct + 4 * g;
              if (off % 4) return ck.fail("MFMA K run not aligned to 4 values", off);
              if (off < 0 || off + 4 > kcount) return ck.fail("MFMA K read out of range", off);
              for (int t = 0; t < 4; ++t) kcov[(size_t)(off + t)]++;
            }
          // the kernel's addressing: row in_row(4g) plus (16ct + t) * d
          const int lane_row = i * b * d + j + 4 * g * d;
          for (int ct = 0; ct < BT; ++ct)
            for (int t = 0; t < 4; ++t) {
              const int r = fused_in_row(fc, f, i, j, 16 * ct + 4 * g + t);
              if (r != lane_row + (16 * ct + t) * d) return ck.fail("MFMA lane row is not the input row", r);
              if (r < 0 || r >= width || r >= fc.buf_rows) return ck.fail("MFMA input row out of range", r);
              if (n == 0) rin.push_back(r);
            }
          for (int kt = 0; kt < BT; ++kt)
            for (int r4 = 0; r4 < 4; ++r4) {
              const int r = fused_out_row(fc, f, i, j, 16 * kt + 4 * g + r4);
              if (r != lane_row + (16 * kt + r4) * d) return ck.fail("MFMA lane row is not the output row", r);
              if (r < 0 || r >= width || r >= fc.buf_rows) return ck.fail("MFMA output row out of range", r);
              for (int h = 0; h < H; ++h) cover[(size_t)r * NC + 16 * h + n]++;
              if (n == 0) rout.push_back(r);
            }
        }
        std::sort(rin.begin(), rin.end());
        std::sort(rout.begin(), rout.end());
        if (rin != rout || (int)rin.size() != b) return ck.fail("MFMA block writes rows it does not read", ij);
      }
    }
    for (int q = 0; q < nblk; ++q)
      if (blk[q] != 1) return ck.fail("MFMA block not taken exactly once", q);
    for (size_t e = 0; e < cover.size(); ++e)
      if (cover[e] != 1) return ck.fail("MFMA factor output not written exactly once", (int64_t)e);
    // Each lane reads every K run of its row tiles once per block; over the
    // 64 lanes and BT x BT tiles that is each value exactly once.
    for (size_t e = 0; e < kcov.size(); ++e)
      if (kcov[e] != 1) return ck.fail("MFMA factor value not read exactly once", (int64_t)e);
  }
  return ck.err.empty();
}

// Butterfly form (ks_chain_bfly.hip): the chain's patterns, which lane of a
// row fetches each block, the kernel's block formulas against the index-set
// definition (each block of each factor applied exactly once per column), the
// LDS row map and the per-wavefront tile loads and stores.
bool verify_fused_bfly(FusedChecker& ck, const FusedChain& fc, int dtype) {
  const int L = fc.bfly, LA = bfly_la(L), LB = L - LA, PA = 1 << LA, PB = 1 << LB, N = PA * PB;
  if (fc.nf != L || fc.width_in != N || fc.width_out != N) return ck.fail("butterfly widths", L);
  for (int q = 0; q < L; ++q)
    if (fc.b[q] != 2 || fc.c[q] != 2 || fc.a[q] != (1 << q) || fc.d[q] != (1 << (L - 1 - q)))
      return ck.fail("factor is not the butterfly pattern", q);
  if (16 * PA > kFusedThreads || 16 * PB > kFusedThreads) return ck.fail("butterfly too wide for one unit per thread", N);
  if (bfly_lds_floats(N) * 4 != fused_lds_bytes(fc) || fused_lds_bytes(fc) > kFusedMaxLds)
    return ck.fail("butterfly LDS", fused_lds_bytes(fc));
  // factor blocks fetched by lane i of a unit's row: pass A block u*PA/2 + i,
  // pass B block j + block(PA*r_i) with r_i the i-th r whose bit t is clear;
  // the butterfly of r reads lane block(r) (A) or its rank among those r (B)
  for (int s = 0; s < L; ++s) {
    const int t = s - LA;
    for (int r = 0; r < (s < LA ? PA : PB); ++r) {
      if (s < LA ? (r & (1 << s)) : (r & (1 << t))) continue;
      const int lanei = s < LA ? bfly_block(r, s) : (((r >> (t + 1)) << t) | (r & ((1 << t) - 1)));
      if (lanei < 0 || lanei >= 16 || lanei >= (s < LA ? PA : PB) / 2) return ck.fail("block lane out of range", lanei);
      if (s >= LA) {
        const int ri = ((lanei >> t) << (t + 1)) | (lanei & ((1 << t) - 1));
        if (ri != r) return ck.fail("pass B block lane does not hold the block of r", r);
      }
    }
  }
  // LDS row map: a bijection of [0, N)
  {
    std::vector<uint8_t> seen(N, 0);
    for (int R = 0; R < N; ++R) {
      const int p = bfly_lds_row(R, LA);
      if (p < 0 || p >= N || seen[p]++) return ck.fail("LDS row map not a bijection", R);
    }
  }
  // blocks of every factor: once per column (n is a column; every column
  // runs the same units, so one column is replayed)
  std::vector<std::vector<uint8_t>> used(L, std::vector<uint8_t>(N / 2, 0));
  auto check_pair = [&](int R, int s, int blk) -> bool {
    const int d = 1 << s, i = R / (2 * d), j = R % (2 * d);
    if (j >= d) return ck.fail("first row of a pair has bit s set", R);
    if (blk != i * d + j || blk != bfly_block(R, s)) return ck.fail("block formula differs from the index sets", R);
    if (blk < 0 || blk >= N / 2) return ck.fail("block out of range", blk);
    used[s][blk]++;
    return true;
  };
  for (int g = 0; g < PB; ++g)
    for (int s = 0; s < LA; ++s)
      for (int r = 0; r < PA; ++r)
        if (!(r & (1 << s)) && !check_pair(g * PA + r, s, g * (PA / 2) + bfly_block(r, s))) return false;
  for (int j = 0; j < PA; ++j)
    for (int s = LA; s < L; ++s)
      for (int r = 0; r < PB; ++r)
        if (!(r & (1 << (s - LA))) && !check_pair(j + PA * r, s, j + bfly_block(PA * r, s))) return false;
  for (int s = 0; s < L; ++s)
    for (int b = 0; b < N / 2; ++b)
      if (used[s][b] != 1) return ck.fail("block not applied exactly once", s * N + b);
  // Tile I/O, wavefront by wavefront as the kernel does it, in both access
  // forms the host may pick (pieces of EP elements when VEC): every X element
  // of the batch read once, every Y element written once, pass-A rows loaded
  // by the wavefront whose units use them, pass-B rows stored by the one that
  // wrote them.
  constexpr int W = kFusedThreads / 64;
  const int esize = dtype == F32 ? 4 : 2;
  const int64_t B = fc.batch;
  const int tiles = (int)((B + kFusedCols - 1) / kFusedCols);
  const bool bsl = fc.layout == BSL;
  const bool vec_ok = bsl ? B % (16 / esize) == 0 : N % (16 / esize) == 0;
  std::vector<uint8_t> xin((size_t)B * N), yout((size_t)B * N);
  for (int form = 0; form < (vec_ok ? 2 : 1); ++form) {
    const bool vec = form == 1;
    const int EP = vec ? 16 / esize : 1, PR = kFusedCols / EP;
    std::fill(xin.begin(), xin.end(), 0);
    std::fill(yout.begin(), yout.end(), 0);
    for (int tile = 0; tile < tiles; ++tile) {
      const int64_t col0 = (int64_t)tile * kFusedCols;
      for (int w = 0; w < W; ++w) {
        if (4 * w < PB) {
          if (bsl) {
            const int TOT = 4 * PA * PR, NP = (TOT + 63) / 64;
            for (int i = 0; i < NP; ++i)
              for (int lane = 0; lane < 64; ++lane) {
                const int p = i * 64 + lane, row = 4 * w * PA + p / PR, col = (p % PR) * EP;
                if (p >= TOT || col0 + col >= B) continue;
                if (row < 4 * w * PA || row >= (4 * w + 4) * PA || row >= N) return ck.fail("pass A piece row", row);
                if (vec && col0 + col + EP > B) return ck.fail("X piece straddles the batch end", col0 + col);
                const int64_t off = (int64_t)row * B + col0 + col;
                if (vec && off % EP) return ck.fail("X piece not aligned to its size", off);
                for (int e = 0; e < EP; ++e) xin[(size_t)(off + e)]++;
              }
          } else {
            const int KP = 4 * PA / EP, NI = (KP + 3) / 4;
            for (int i = 0; i < NI; ++i)
              for (int lane = 0; lane < 64; ++lane) {
                const int k = 4 * i + (lane >> 4), t = lane & 15;
                if (k >= KP || col0 + t >= B) continue;
                const int row = 4 * w * PA + k * EP;
                if (row + EP > (4 * w + 4) * PA || row + EP > N) return ck.fail("pass A piece rows", row);
                const int64_t off = (col0 + t) * N + row;
                if (vec && off % EP) return ck.fail("X piece not aligned to its size", off);
                for (int e = 0; e < EP; ++e) xin[(size_t)(off + e)]++;
              }
          }
        }
        if (4 * w < PA) {
          if (bsl) {
            const int TOT = 4 * PB * PR, NP = (TOT + 63) / 64;
            for (int i = 0; i < NP; ++i)
              for (int lane = 0; lane < 64; ++lane) {
                const int p = i * 64 + lane, rho = p / PR, col = (p % PR) * EP;
                const int row = 4 * w + (rho & 3) + PA * (rho >> 2);
                if (p >= TOT || col0 + col >= B) continue;
                // a row of this wavefront's pass-B units j = 4w .. 4w+3
                if ((row % PA) / 4 != w || row >= N) return ck.fail("pass B piece row", row);
                if (vec && col0 + col + EP > B) return ck.fail("Y piece straddles the batch end", col0 + col);
                const int64_t off = (int64_t)row * B + col0 + col;
                if (vec && off % EP) return ck.fail("Y piece not aligned to its size", off);
                for (int e = 0; e < EP; ++e) yout[(size_t)(off + e)]++;
              }
          }
        }
      }
    }
    // batch-size-first: the shared tile store after the second barrier
    if (!bsl && !verify_fused_io(ck, fc, N, EP, true, &yout)) return false;
    for (size_t e = 0; e < xin.size(); ++e)
      if (xin[e] != 1) return ck.fail("X element not read exactly once", (int64_t)e);
    for (size_t e = 0; e < yout.size(); ++e)
      if (yout[e] != 1) return ck.fail("Y element not written exactly once", (int64_t)e);
  }
  return ck.err.empty();
}

bool verify_fused(FusedChecker& ck, const FusedChain& fc, int dtype) {
  const int esize = dtype == F32 ? 4 : 2, E = 16 / esize;
  // Workgroup -> tile order: a bijection of the grid.
  {
    const int tiles = (int)(((int64_t)fc.batch + fc.cols - 1) / fc.cols);
    std::vector<uint8_t> seen(tiles, 0);
    for (int b = 0; b < tiles; ++b) {
      const int t = fused_tile(b, tiles);
      if (t < 0 || t >= tiles) return ck.fail("workgroup tile out of range", b);
      if (seen[t]++) return ck.fail("tile taken by two workgroups", t);
    }
  }
  // Widths along the chain: input of factor nf-1 ... output of factor 0.
  for (int f = 0; f + 1 < fc.nf; ++f)
    if (fc.a[f] * fc.c[f] * fc.d[f] != fc.a[f + 1] * fc.b[f + 1] * fc.d[f + 1]) return ck.fail("widths", f);
  if (fused_lds_bytes(fc) > kFusedMaxLds) return ck.fail("LDS", fused_lds_bytes(fc));
  if (fc.bfly) return verify_fused_bfly(ck, fc, dtype);  // its own tile I/O and passes
  // Vector rows end where the factor-value copies begin.
  if (fused_kbuf_offset(fc) < (fc.inplace ? 1 : 2) * fc.buf_rows * kFusedPitch) return ck.fail("LDS overlap", 0);
  // Tile I/O, both forms the host may choose (vector form only when the
  // batch (BSL) or the widths (BSF) are whole vectors).
  const bool vec_ok = fc.layout == BSL ? fc.batch % E == 0 : (fc.width_in % E == 0 && fc.width_out % E == 0);
  for (int form = 0; form < 2; ++form) {
    const int e = form == 0 ? 1 : E;
    if (form == 1 && !vec_ok) break;
    if (!verify_fused_io(ck, fc, fc.width_in, e, false, nullptr)) return false;
    std::vector<uint8_t> cover((size_t)fc.batch * fc.width_out, 0);
    if (!verify_fused_io(ck, fc, fc.width_out, e, true, &cover)) return false;
    for (size_t q = 0; q < cover.size(); ++q)
      if (cover[q] != 1) return ck.fail(cover[q] ? "Y element stored more than once" : "Y element never stored",
                                        (int64_t)q);
  }
  // Passes cover the factors in application order, each exactly once.
  {
    int next = fc.nf - 1;
    for (int q = 0; q < fc.npass; ++q) {
      if (fc.pf0[q] != next || fc.pm[q] < 1) return ck.fail("passes do not follow the factors", q);
      int kn = 0;
      for (int t = 0; t < fc.pm[q]; ++t) {
        const int f = fc.pf0[q] - t;
        if (fc.a[f] * fc.b[f] * fc.c[f] * fc.d[f] != fc.pcnt[q]) return ck.fail("pass value count", q);
        kn += fc.pcnt[q];
      }
      if (kn != fc.pk[q] || (!fc.mfma && kn > kFusedKValues)) return ck.fail("pass values exceed the LDS copy", q);
      if (fc.mfma && fc.pm[q] != 1) return ck.fail("MFMA form pass with several factors", q);
      next -= fc.pm[q];
    }
    if (next != -1) return ck.fail("passes do not cover the chain", next);
  }
  if (fc.mfma) return verify_fused_mfma(ck, fc, dtype);
  for (int q = 0; q < fc.npass; ++q) {
    if (fused_is_radix(fc, q)) {
      // Radix pass: every unit's P rows in range, the groups partition the
      // vector, and for every factor of the pass each (block, input l) pair
      // is visited exactly once per piece, at the rows the index sets give.
      const int f0 = fc.pf0[q], p = fc.pp[q], P = fc.pP[q], m = fc.pm[q], d0 = fc.d[f0];
      const int N = fc.a[f0] * fc.c[f0] * d0;
      int PP = 1;
      for (int t = 0; t < m; ++t) PP *= p;
      if (PP != P || P > kFusedMaxGroup) return ck.fail("radix group size", q);
      if (!((p == 2 && (P == 2 || P == 4 || P == 8)) || (p == 4 && P == 4) || (p == 8 && P == 8)))
        return ck.fail("no kernel instance for this radix pass", q);
      for (int t = 0; t < m; ++t) {
        const int f = f0 - t;
        int st = 1;
        for (int u = 0; u < t; ++u) st *= p;
        if (fc.b[f] != p || fc.c[f] != p || fc.d[f] != d0 * st || fc.a[f] * p * st != fc.a[f0] * p)
          return ck.fail("radix pass strides do not nest", f);
      }
      if (fused_radix_units(fc, q) != N / P * 4) return ck.fail("radix unit count", q);
      std::vector<uint8_t> rowcover((size_t)N * 4, 0);
      std::vector<std::vector<uint8_t>> blkcover(m, std::vector<uint8_t>((size_t)N * 4, 0));  // a*d blocks x p inputs = N
      for (int u = 0; u < fused_radix_units(fc, q); ++u) {
        const int g = u >> 2, piece = u & 3;
        int i, j0;
        fused_radix_group(fc, q, g, &i, &j0);
        if (i < 0 || j0 < 0 || j0 >= d0 || (int64_t)i * P * d0 + j0 + (int64_t)d0 * (P - 1) >= N)
          return ck.fail("radix group out of range", g);
        if (i != g / d0 || j0 != g % d0) return ck.fail("radix group decode differs from the division", g);
        const int base = i * P * d0 + j0;
        for (int r = 0; r < P; ++r) rowcover[(size_t)(base + d0 * r) * 4 + piece]++;
        for (int t = 0; t < m; ++t) {
          const int f = f0 - t;
          int st = 1;
          for (int uu = 0; uu < t; ++uu) st *= p;
          for (int r = 0; r < P; ++r) {
            if ((r / st) % p != 0) continue;
            int blk = -1;
            switch (P * 16 + p) {
              case 2 * 16 + 2: blk = fused_radix_block<2, 2>(i, j0, d0, t, r); break;
              case 4 * 16 + 2: blk = fused_radix_block<4, 2>(i, j0, d0, t, r); break;
              case 8 * 16 + 2: blk = fused_radix_block<8, 2>(i, j0, d0, t, r); break;
              case 4 * 16 + 4: blk = fused_radix_block<4, 4>(i, j0, d0, t, r); break;
              case 8 * 16 + 8: blk = fused_radix_block<8, 8>(i, j0, d0, t, r); break;
            }
            if (blk < 0 || blk >= fc.a[f] * fc.d[f]) return ck.fail("radix block out of range", blk);
            const int it = blk / fc.d[f], jt = blk % fc.d[f];
            for (int l = 0; l < p; ++l) {
              if (base + d0 * (r + l * st) != fused_in_row(fc, f, it, jt, l))
                return ck.fail("radix register row is not the block's input row", r + l * st);
              if (fused_in_row(fc, f, it, jt, l) != fused_out_row(fc, f, it, jt, l))
                return ck.fail("radix block not square", f);
              blkcover[t][((size_t)blk * p + l) * 4 + piece]++;
            }
          }
        }
      }
      for (size_t e = 0; e < rowcover.size(); ++e)
        if (rowcover[e] != 1) return ck.fail("radix pass row piece not held exactly once", (int64_t)e);
      for (int t = 0; t < m; ++t)
        for (size_t e = 0; e < blkcover[t].size(); ++e)
          if (blkcover[t][e] != 1) return ck.fail("radix factor input not used exactly once", (int64_t)e);
      continue;
    }
    // Single-factor pass: every unit's rows in range, and the units write
    // every (row, column) of the factor's output exactly once; in place, a
    // unit writes exactly the rows it reads (no unit reads rows another unit
    // writes).
    const int f = fc.pf0[q];
    const int a = fc.a[f], b = fc.b[f], c = fc.c[f], d = fc.d[f];
    const int m = b > c ? b : c;
    const int QN = fused_pieces(m), G = 4 / QN;
    const int win = a * c * d, wout = a * b * d;
    if (fused_units(fc, f) != a * d * G) return ck.fail("unit count", f);
    std::vector<uint8_t> cover((size_t)wout * 4, 0);
    for (int u = 0; u < a * d * G; ++u) {
      int i, j, g;
      fused_unit(fc, f, G, u, &i, &j, &g);
      if (i < 0 || i >= a || j < 0 || j >= d || g < 0 || g >= G) return ck.fail("unit decode", u);
      if (i * d + j != u / G) return ck.fail("unit decode differs from the division", u);
      std::vector<int> rin, rout;
      for (int l = 0; l < c; ++l) {
        const int r = fused_in_row(fc, f, i, j, l);
        if (r < 0 || r >= win || r >= fc.buf_rows) return ck.fail("input row out of range", r);
        rin.push_back(r);
      }
      for (int k = 0; k < b; ++k) {
        const int r = fused_out_row(fc, f, i, j, k);
        if (r < 0 || r >= wout || r >= fc.buf_rows) return ck.fail("output row out of range", r);
        rout.push_back(r);
        for (int qn = 0; qn < QN; ++qn) cover[(size_t)r * 4 + g * QN + qn]++;
      }
      if (fc.inplace) {
        std::sort(rin.begin(), rin.end());
        std::sort(rout.begin(), rout.end());
        if (rin != rout) return ck.fail("in-place unit writes rows it does not read", u);
      }
    }
    for (size_t e = 0; e < cover.size(); ++e)
      if (cover[e] != 1) return ck.fail("factor output piece not written exactly once", (int64_t)e);
  }
  return ck.err.empty();
}

}  // namespace
}  // namespace ks

extern "C" ks_status_t ks_chain_verify(const ks_factor_t* factors, int nfactors, int64_t batch, int layout, int dtype,
                                       char* report, size_t len) {
  if (report && len) report[0] = 0;
  char desc[256];
  ks_status_t st = ks_chain_describe(factors, nfactors, batch, layout, dtype, desc, sizeof desc);
  if (st != KS_OK) return st;
  ks::FusedChain fc;
  if (batch == 0 || !ks::chain_fused_plan(factors, nfactors, batch, layout, dtype, &fc)) {
    if (report && len) snprintf(report, len, "%s", batch == 0 ? "empty" : "not fused");
    return KS_OK;
  }
  ks::FusedChecker ck;
  const bool ok = ks::verify_fused(ck, fc, dtype);
  if (report && len) snprintf(report, len, "%s", ok ? "ok" : ck.err.c_str());
  return ok ? KS_OK : KS_ERR_UNSUPPORTED;
}
