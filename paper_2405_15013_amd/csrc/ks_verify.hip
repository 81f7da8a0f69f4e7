// Host-side plan verifier: replays, on the CPU, the address arithmetic every
// thread of the planned launch would perform, and checks that all global reads
// and writes stay inside their tensors, that every LDS cell a tile reads has
// been written, and that every element of Y is written exactly once (the
// partition property of the row/col index sets, paper Section 4.1).  Nothing is
// enqueued on a GPU.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/ks.h"
#include "ks_internal.h"
#include "ks_mfma_index.h"
#include "ks_direct_index.h"

namespace ks {

// Defined in ks_direct_plan.cpp.
DirectTile direct_tile(const Problem& p, const Plan& pl);

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

bool verify_mfma(Checker& ck, const Plan& pl) {
  const Problem& p = ck.p;
  MfmaTile t;
  t.bt = pl.bt;
  t.jg = pl.jg;
  t.njg = p.d / pl.jg;
  t.nbt = (p.batch + pl.bt - 1) / pl.bt;
  t.mode = pl.unroll;
  t.remap = pl.xcd_remap;
  t.vec = pl.vec;
  const int MT = pl.waves_m, NT = pl.waves_n, V = t.vec, s = p.dtype == F32 ? 4 : 2;
  const int KC = s == 4 ? 16 : 32;
  const int P = x_pitch(p, t), PY = y_pitch(p, t);
  const int xs_cells = t.jg * t.bt * P;
  if (t.njg * t.jg != p.d) return ck.fail("j-group does not divide d", t.jg);
  if (t.bt % (16 * MT)) return ck.fail("batch tile not a multiple of 16*MT", t.bt);
  if ((p.b / 16) % NT) return ck.fail("NT does not divide b/16", NT);
  if (x_chunks(p, t) > 256 * kMaxChunks) return ck.fail("too many X chunks per thread", x_chunks(p, t));
  int64_t lds_need = (int64_t)xs_cells * s + (p.layout == BSF ? (int64_t)t.bt * PY * s : 0);
  if (lds_need > pl.lds_bytes) return ck.fail("LDS allocation too small", lds_need);
  if ((int64_t)t.nbt * p.a * t.njg != (int64_t)pl.grid) return ck.fail("grid does not match the tiles", pl.grid);
  if (t.remap && pl.grid % 8) return ck.fail("XCD remap needs a grid multiple of 8", pl.grid);
  std::vector<uint8_t> seen_tile(pl.grid, 0);
  std::vector<uint8_t> xs(xs_cells), ys;
  for (unsigned blk = 0; blk < pl.grid && ck.err.empty(); ++blk) {
    const TileCoord tc = tile_coord(p, t, blk, pl.grid);
    const int logical = t.remap ? xcd_remap(blk, pl.grid) : (int)blk;
    if (seen_tile[logical]++) return ck.fail("tile visited twice", logical);
    std::fill(xs.begin(), xs.end(), 0);
    const int total = x_chunks(p, t);
    for (int q = 0; q < total; ++q) {
      const int64_t src = x_chunk_src(p, t, tc, q);
      if (src >= 0) ck.read_x(src, V);
      if (src >= 0 && (src % V)) ck.fail("X chunk not vector aligned", src);
      for (int e = 0; e < V; ++e) {
        const int li = x_chunk_lds(p, t, q, e);
        if (li < 0 || li >= xs_cells) return ck.fail("Xs write out of bounds", li);
        if (xs[li]++) return ck.fail("Xs cell written twice", li);
      }
    }
    // every cell the MFMA reads must have been written
    for (int jj = 0; jj < t.jg; ++jj)
      for (int r = 0; r < t.bt; ++r)
        for (int l = 0; l < p.c; ++l)
          if (!xs[(jj * t.bt + r) * P + l]) return ck.fail("Xs cell read but never written", (jj * t.bt + r) * P + l);
    if (p.layout == BSF) ys.assign((size_t)t.bt * PY, 0);
    const int items = mfma_items(p, t, MT, NT);
    for (int it = 0; it < items; ++it) {
      const Item itm = mfma_item(p, t, MT, NT, it);
      for (int lane = 0; lane < 64; ++lane) {
        const int n = lane & 15, g = lane >> 4;
        for (int nt = 0; nt < NT; ++nt) {
          const int k = (itm.ngi * NT + nt) * 16 + n;
          const int64_t krow = ((int64_t)(tc.i * p.d + tc.j0 + itm.jj) * p.b + k) * p.c;
          ck.read_k(krow, p.c);
          for (int mt = 0; mt < MT; ++mt) {
            const int bl = (itm.mgi * MT + mt) * 16 + 4 * g;
            const int arow = itm.jj * t.bt + (itm.mgi * MT + mt) * 16 + n;
            if (arow >= t.jg * t.bt) return ck.fail("A operand row out of range", arow);
            if (p.layout == BSL) {
              const int beta = tc.beta0 + bl;
              if (beta < p.batch) {
                if (beta + 4 > p.batch) return ck.fail("BSL store straddles the batch end", beta);
                ck.write_y((int64_t)(tc.i * p.b * p.d + k * p.d + tc.j0 + itm.jj) * p.batch + beta, 4);
              }
            } else {
              for (int r = 0; r < 4; ++r) {
                const int yi = (bl + r) * PY + k * t.jg + itm.jj;
                if (yi >= (int)ys.size()) return ck.fail("Ys write out of bounds", yi);
                if (ys[yi]++) return ck.fail("Ys cell written twice", yi);
              }
            }
          }
        }
      }
    }
    (void)KC;
    if (p.layout == BSF) {
      const int ych = y_chunks(p, t);
      for (int q = 0; q < ych; ++q) {
        int lds;
        const int64_t dst = y_chunk_dst(p, t, tc, q, &lds);
        if (dst < 0) continue;
        for (int e = 0; e < V; ++e)
          if (!ys[lds + e]) return ck.fail("Ys cell stored but never written", lds + e);
        if (dst % V) return ck.fail("Y chunk not vector aligned", dst);
        ck.write_y(dst, V);
      }
    }
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
  // chunks: (l0, values of l per lane group)
  int chunks[16][2], nch = 0;
  for (int l0 = 0; l0 + CH <= p.c; l0 += CH) { chunks[nch][0] = l0; chunks[nch][1] = LP; ++nch; }
  if (S == 2 && p.c % CH) { chunks[nch][0] = p.c - 16; chunks[nch][1] = 4; ++nch; }
  if (nch == 0) return ck.fail("no chunk covers c", p.c);
  const int VK = p.layout == BSL ? 1 : V;
  for (int item = 0; item < t.items && ck.err.empty(); ++item) {
    const DItem it = direct_item(p, t, V, MT, item);
    for (int ci = 0; ci < nch; ++ci) {
      const int l0 = chunks[ci][0], lp = chunks[ci][1];
      const int np = direct_x_pieces(p.layout, strided, lp, V, S);
      const int pe = direct_x_piece_elems(p.layout, strided, lp, V, S);
      if (pe * S != 16 && pe * S != 8) return ck.fail("X piece is not 8 or 16 bytes", pe * S);
      if (np * pe != lp * V) return ck.fail("X pieces do not tile the lane block", np);
      for (int lane = 0; lane < 64; ++lane) {
        const int n = lane & 15, g = lane >> 4;
        for (int q = 0; q < np; ++q) {
          const int64_t off = direct_x_off(p, it, strided, lp, V, S, l0, n, g, q);
          if (off < 0) continue;
          if ((off * S) % (pe * S)) return ck.fail("X piece not aligned to its size", off);
          ck.read_x(off, pe);
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
    case V_MFMA: ok = verify_mfma(ck, pl); break;
    case V_DIRECT: ok = verify_direct(ck, pl); break;
    default: ck.fail("unknown variant", pl.variant);
  }
  if (ok) ok = ck.coverage();
  if (report && len) snprintf(report, len, "%s", ok ? "ok" : ck.err.c_str());
  return ok ? KS_OK : KS_ERR_UNSUPPORTED;
}
