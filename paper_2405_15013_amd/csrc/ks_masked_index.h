// Index arithmetic of the masked register-direct MFMA kernel (ks_masked.h),
// shared by the kernel and by the host-side plan verifier.
//
// The masked kernel runs the patterns and buffers the other MFMA kernels do
// not take: b or c not a multiple of 16, a batch-size-last batch that is not a
// multiple of the 16-byte vector, buffers that are not 16-byte aligned.  Its
// work decomposition is the register-direct one (output-stationary items of
// Section 4.1, Algorithm 2): one wavefront per item = (batch tile, i, j or
// j-group, 16 output rows k), lanes (n, g) = (lane % 16, lane / 16) in the
// MFMA operand layout.  The 16 x 16 tiles are padded with zeros: rows
// k >= b and values l >= c read nothing and contribute zero, outputs of
// padded rows are not stored.  Memory accesses are pieces of V consecutive
// elements (V * sizeof(T) bytes, 2 to 16, aligned to their size): along the
// batch in BSL (the planner picks V dividing the batch and the buffers'
// alignment), along j in BSF (V divides d); K is read element by element.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

#include "ks_internal.h"

#define KS_MHD __host__ __device__ __forceinline__

namespace ks {

struct MaskedTile {
  int mt;        // 16-row output tiles per wavefront (1; the FP8 kernel also 2 or 4)
  int kgroups;   // ceil(b / (16 * mt))
  int jgroups;   // BSL: d; BSF: d / V
  int nbt;       // batch tiles (16*V entries in BSL, 16 rows in BSF)
  int items;     // nbt * a * jgroups * kgroups
  int nchunks;   // ceil(c / CH), CH = 4 * LP values of l per chunk
  int kvec;      // K read as LP-element operands (c a multiple of LP, K_values aligned to them)
};

struct MItem {
  int i, j0, k0, beta0;
};


// LP values of l per lane and chunk: 4 (fp32, 16x16x4 MFMA), 8 (16-bit and
// FP8, 16x16x32 MFMAs).
KS_MHD int masked_lp(int esize) { return esize == 4 ? 4 : 8; }

KS_MHD MaskedTile masked_tile(const Problem& p, int V, int mt = 1) {
  MaskedTile t;
  t.mt = mt;
  t.kgroups = (p.b + 16 * mt - 1) / (16 * mt);
  t.jgroups = p.layout == BSL ? p.d : p.d / V;
  const int span = p.layout == BSL ? 16 * V : 16;
  t.nbt = (p.batch + span - 1) / span;
  t.items = t.nbt * p.a * t.jgroups * t.kgroups;
  const int lp = masked_lp(p.dtype == F32 ? 4 : 2), ch = 4 * lp;
  t.nchunks = (p.c + ch - 1) / ch;
  // A lane's LP values of l (from a multiple of LP) are one vector of its K
  // row when c is a multiple of LP: wholly inside the row or wholly padding.
  const int esize = p.dtype == F32 ? 4 : (p.dtype == FP8 ? 1 : 2);
  t.kvec = (p.c % lp == 0 && (reinterpret_cast<uintptr_t>(p.kv) % (uintptr_t)(lp * esize)) == 0) ? 1 : 0;
  return t;
}

// Item order as in the register-direct kernels: k-group fastest, then batch
// tile, then j-group, then i.
KS_MHD MItem masked_item(const Problem& p, const MaskedTile& t, int V, int item) {
  MItem it;
  int rest = item;
  const int kg = rest % t.kgroups;
  rest /= t.kgroups;
  const int bt = rest % t.nbt;
  rest /= t.nbt;
  const int jg = rest % t.jgroups;
  it.i = rest / t.jgroups;
  it.k0 = 16 * t.mt * kg;
  if (p.layout == BSL) {
    it.j0 = jg;
    it.beta0 = bt * 16 * V;
  } else {
    it.j0 = jg * V;
    it.beta0 = bt * 16;
  }
  return it;
}

// True when lane column n holds real batch entries.
KS_MHD bool masked_col_valid(const Problem& p, const MItem& it, int V, int n) {
  return p.layout == BSL ? it.beta0 + V * n < p.batch : it.beta0 + n < p.batch;
}

// X piece (V elements) of value l for lane column n, or -1 when l >= c or the
// column lies beyond the batch (the piece is zero).
KS_MHD int64_t masked_x_off(const Problem& p, const MItem& it, int V, int l, int n) {
  if (l >= p.c || !masked_col_valid(p, it, V, n)) return -1;
  if (p.layout == BSL)
    return ((int64_t)it.i * p.c * p.d + (int64_t)l * p.d + it.j0) * p.batch + it.beta0 + V * n;
  return (int64_t)(it.beta0 + n) * p.N + (int64_t)it.i * p.c * p.d + (int64_t)l * p.d + it.j0;
}

// K element (k0 + m, l) of block (i, j0 + e), or -1 in the padding.
KS_MHD int64_t masked_k_off(const Problem& p, const MItem& it, int e, int m, int l) {
  const int k = it.k0 + m;
  if (k >= p.b || l >= p.c) return -1;
  return (((int64_t)it.i * p.d + it.j0 + e) * p.b + k) * p.c + l;
}

// Y piece (V elements) of output row k = k0 + 4g + r for lane column n, or -1
// when the row is padding or the column lies beyond the batch.
KS_MHD int64_t masked_y_off(const Problem& p, const MItem& it, int V, int n, int g, int r) {
  const int k = it.k0 + 4 * g + r;
  if (k >= p.b || !masked_col_valid(p, it, V, n)) return -1;
  if (p.layout == BSL)
    return ((int64_t)it.i * p.b * p.d + (int64_t)k * p.d + it.j0) * p.batch + it.beta0 + V * n;
  return (int64_t)(it.beta0 + n) * p.M + (int64_t)it.i * p.b * p.d + (int64_t)k * p.d + it.j0;
}

}  // namespace ks
